// sma_bwd.hip -- backward of the state-memory attention with the gated residual.
//
// Paper: Sec. 3 ("State-Memory Attention", "Gated Residual Integration"),
// App. B.1 (normalised scores) and App. C (the backward recomputes the scores
// from the stored log-sum-exp instead of keeping the attention weights).
//
// For the loss sum_t dy_t . y_t, token t of chunk i, memory j < i, with
// p_j = exp(l_j - LSE_t) (the forward's weights, recovered exactly), gate
// g = SiLU(z_t), s = 1/sqrt(N) and the key side Kh_j = r_j (.) dH_j:
//   dwy_j = dy_t . V_j = C_t . (dH_j dy_t)     Dy = sum_j p_j dwy_j = R_t . dy_t
//   dl_j  = g p_j (dwy_j - Dy)                 (softmax backward, dR = g dy)
//   dC_t  += g p_j dH_j dy_t                   (V_j = C_t dH_j)
//   dQbar += s dl_j Kh_j Ebar_t                (l_j = s Qbar . Kh_j Ebar)
//   dEbar += s dl_j Kh_j^T Qbar_t
//   dz_t   = SiLU'(z_t) Dy                     (summed over heads for one gate)
// and, per memory j, over the later tokens t:
//   M1 = sum_t g p_j[t] C_t^T dy_t,   M2 = sum_t s dl_j[t] Qbar_t^T Ebar_t
//   ddH_j = M1 + r_j (.) M2 - (r_j^3 / P) (.) rowsum(dH_j (.) M2) (.) dH_j
// (the last term through r_j = (mean_p dH_j^2 + eps)^-1/2 of the stored
// values; r = 1 and no such term without normalisation).  q and e gradients
// follow through RMSNorm with the weights held constant.
//
// Kernels, in launch order:
//   k_sma_keys          key side Kh_j (cache layout, bf16 as hi + lo) and 1 / r_j
//   k_bwd_prep          Qbar' = Qbar log2(e)/sqrt(N) (storage dtype, the
//                       forward's operand exactly), q (.) w as hi + lo and its
//                       RMSNorm row scale, Ebar (float, and bf16 for the memory
//                       kernel) per token
//   k_bwd_scores        one workgroup per (64 or 128 tokens of one chunk, block
//                       of heads of one group), 8 waves, a pair per token group
//                       splitting the rows of each product; per (head, memory)
//                       the logit to about 16 bits (W' = Kh^T (q (.) w) from the
//                       hi + lo operands, times the row scale) and
//                       dwy = C . X, X = diag(1/r) Kh dy^T, written per
//                       (b, h, j, t); at the head's end the exact log-sum-exp of
//                       these logits and Dy = sum_j p_j dwy_j per (b, t, h)
//   k_bwd_tokens        same blocks: with p_j and dl_j known at every step,
//                       dQbar += s dl_j Z_j (Z = Kh Ebar^T), dEbar += ln2 dl_j W'_j,
//                       dC += g p_j X_j on MFMA; it writes g p_j[t] over the
//                       logit for the memory kernel and per-head-block partial
//                       sums of dQbar, dEbar, dC
//   k_bwd_mem           one workgroup per (b, h, 4 memories): M1 and M2 over
//                       the later tokens, the token stream copied into LDS by
//                       DMA once for the four memories, dl_j[t] formed from
//                       the stored g p_j, dwy_j and Dy and applied to the
//                       MFMA operand fragments in registers; then the
//                       epilogue above.  Heavy memories (small j) go first.
//   k_bwd_finish        one wave per (b, t, group): sums the partials over the
//                       group's head blocks, RMSNorm backward, dz.
#include <type_traits>

#include "dart_common.hpp"
#include "dart_internal.hpp"

namespace dart {
namespace {

constexpr int kP = 64;
constexpr int kTokWaves = 4;               // 16-token groups (and copying waves) per
                                           // k_bwd_tokens workgroup; two waves a group
constexpr int kTokBlock = 16 * kTokWaves;  // tokens per k_bwd_tokens workgroup
constexpr int kMemJ = 4;                   // memories per k_bwd_mem workgroup
constexpr int kHeadsPerBlock = 8;

// Sum over the 64 lanes in every lane (DPP within rows, then row swaps); call
// from wave-uniform control flow.
__device__ __forceinline__ float wave_sum(float v) { return row4_sum(dpp_group_sum<16>(v)); }

// An empty use of every register of a fragment, so the compiler waits for its
// loads at this point (operands of at most 128 bits each).
__device__ __forceinline__ void keep(const bf16x8& f) { asm volatile("" ::"v"(f)); }
__device__ __forceinline__ void keep(const f32x8& f) {
    const f32x4 a{f[0], f[1], f[2], f[3]}, b{f[4], f[5], f[6], f[7]};
    asm volatile("" ::"v"(a), "v"(b));
}

__device__ __forceinline__ float silu_grad(float z) {
    const float sg = 1.0f / (1.0f + __expf(-z));
    return sg * (1.0f + z * (1.0f - sg));
}

// DMA copy of one XOR-swizzled tile of TILE bytes (rows of RB bytes, chunk c
// of row r stored at chunk c ^ (r & MASK)) from a contiguous global tile,
// with the per-lane offsets fixed at set-up and the tile base passed as a
// scalar, so issuing a copy costs no vector address arithmetic.  Wave w of NW
// copies the 1 KiB pieces w, w + NW, ...; lane i of a piece lands 16 i bytes
// into it.  Invisible to the compiler's wait counting: the caller waits with
// vmcnt (count() copies per call).
template <int RB, int TILE, int NW>
struct TileCopy {
    static constexpr int CPR = RB / 16;
    static constexpr int MASK = (CPR < 8 ? CPR : 8) - 1;
    static constexpr int NI = TILE / 1024;  // pieces per tile
    static constexpr int KPW = NI / NW;     // pieces per wave
    static_assert(NI % NW == 0 && KPW >= 1, "pieces must tile the waves");
    uint32_t goff[KPW];
    int wave;
    __device__ void init(int w, int lane) {
        wave = __builtin_amdgcn_readfirstlane(w);
#pragma unroll
        for (int k = 0; k < KPW; ++k) {
            const int q = (w + k * NW) * 64 + lane;
            const int row = q / CPR, pos = q % CPR;
            goff[k] = (uint32_t)(row * RB + ((pos ^ (row & MASK)) << 4));
            asm volatile("" : "+v"(goff[k]));
        }
    }
    static constexpr int count() { return KPW; }
    __device__ __forceinline__ void issue(const void* gtile, char* ltile) const {
        const uint64_t gb = (uint64_t)(uintptr_t)gtile;
        const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(gb >> 32));
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)gb);
        const uint64_t base = ((uint64_t)hi << 32) | (uint64_t)lo;
        const uint32_t l0 = lds_addr(ltile);
#pragma unroll
        for (int k = 0; k < KPW; ++k) {
            const uint32_t m0 = (uint32_t)__builtin_amdgcn_readfirstlane(
                (int)(l0 + (uint32_t)((wave + k * NW) * 1024)));
            uint32_t save;
            asm volatile(
                "s_mov_b32 %0, m0\n\t"
                "s_mov_b32 m0, %3\n\t"
                "s_nop 0\n\t"
                "global_load_lds_dwordx4 %1, %2\n\t"
                "s_mov_b32 m0, %0"
                : "=&s"(save)
                : "v"(goff[k]), "s"(base), "s"(m0)
                : "memory");
        }
    }
};

// ---- per (b, t, g) row: one wave per row -----------------------------------
// qb = Qbar' = RMSNorm(q) w * log2(e)/sqrt(N) in the storage dtype (the
// operand of the gradient products); the score operand of the logits is kept
// exact instead: qh = q (.) w (the storage value itself when w = NULL), in
// bf16 also its rounding residual ql, and the per-row scale qsc with
// Qbar' = (q (.) w) qsc.  Ebar = RMSNorm(e) w in float, and (ebt != NULL)
// also in the storage dtype.  Without normalisation: raw q and e, qsc =
// log2(e)/sqrt(N).
template <typename T, int N>
__global__ __launch_bounds__(256) void k_bwd_prep(const T* __restrict__ q, const T* __restrict__ e,
                                                  const float* __restrict__ qw,
                                                  const float* __restrict__ ew, T* __restrict__ qb,
                                                  T* __restrict__ qh, bf16* __restrict__ ql,
                                                  float* __restrict__ qsc, float* __restrict__ eb,
                                                  T* __restrict__ ebt, float eps, int normalize,
                                                  int64_t rows) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows) return;
    constexpr int QE = (N + 63) / 64;
    float qv[QE];
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < QE; ++k) {
        const int n = lane + 64 * k;
        qv[k] = n < N ? to_f(q[row * N + n]) : 0.f;
        ss += qv[k] * qv[k];
    }
    ss = wave_sum(ss);
    const float qscale = kLog2e / sqrtf((float)N);
    const float qinv = (normalize ? 1.0f / sqrtf(ss * (1.0f / N) + eps) : 1.0f) * qscale;
#pragma unroll
    for (int k = 0; k < QE; ++k) {
        const int n = lane + 64 * k;
        if (n < N) {
            const float qwv = qw ? qv[k] * qw[n] : qv[k];
            qb[row * N + n] = from_f<T>(qwv * qinv);
            const T hi = from_f<T>(qwv);
            qh[row * N + n] = hi;
            if (ql) ql[row * N + n] = (bf16)(qwv - to_f(hi));
        }
    }
    if (lane == 0) qsc[row] = qinv;
    const float ev = to_f(e[row * kP + lane]);
    const float es = wave_sum(ev * ev);
    const float einv = normalize ? 1.0f / sqrtf(es * (1.0f / kP) + eps) : 1.0f;
    float v = ev * einv;
    if (ew) v *= ew[lane];
    eb[row * kP + lane] = v;
    if (ebt) ebt[row * kP + lane] = from_f<T>(v);
}

// Block order shared by the two token kernels.  Workgroups are dealt to the
// 8 XCDs round-robin by block index and each XCD has its own L2.  When the
// number of (b, head block) pairs is a multiple of 8, XCD x runs only pairs
// x, x+8, ..., so the blocks of one pair share an L2; token blocks go
// heaviest first over all pairs, so that the longest blocks start first and
// the short ones fill in behind them.
__device__ __forceinline__ void tok_block(int64_t bid, int nblk, int64_t BHC, int& blk,
                                          int64_t& bhc) {
    if (BHC % 8 == 0) {
        const int64_t slot = bid >> 3, ng8 = BHC >> 3;
        blk = nblk - 1 - (int)(slot / ng8);
        bhc = (slot % ng8) * 8 + (bid & 7);
    } else {
        blk = nblk - 1 - (int)(bid / BHC);
        bhc = bid % BHC;
    }
}

// LDS ring stages of the token kernels: four when NTILES tiles of a stage fit
// 32 KiB, else two.
template <typename T, int N, int NTILES>
constexpr int tok_stages() {
    return (NTILES * N * kP * (int)sizeof(T) * 4 <= 131072) ? 4 : 2;
}

// The k-permuted fragments of one token's row of N values (a B operand with
// the contraction over n): k step ks holds n = 32 ks + 4 (lane/16) + 0..3 and
// + 16.
template <typename T, typename S, int N>
__device__ __forceinline__ void load_row_frags(const S* row, int grp, Frag<T> (&f)[N / 32]) {
#pragma unroll
    for (int ks = 0; ks < N / 32; ++ks) {
        float a[4], c[4], v[8];
        load4(row + ks * 32 + 4 * grp, a);
        load4(row + ks * 32 + 16 + 4 * grp, c);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[i] = a[i];
            v[4 + i] = c[i];
        }
        f[ks] = make_frag<T>(v);
    }
}

// ---- scores: exact logits and dy . V per (head, memory, token) ---------------
// Workgroup: 64 RT consecutive tokens of chunk i >= 1 and hpb heads of one
// group, 8 waves; waves w and w + 4 share the RT 16-token column tiles of
// tokens 16 RT w .. 16 RT w + 16 RT - 1 and split the rows: rows p of
// W'^T = Kh^T (q (.) w) (this half's part of every logit) and rows n of
// X^T = diag(1/r) Kh dy^T (its part of dy . V = C . X).  Every memory
// fragment read from LDS feeds the RT column tiles.  The two partial sums
// meet in LDS once per step.
//
// The logits are formed to about 16 bits although the operands are stored in
// bf16: the key side streams as hi + lo (the lo tile holds the rounding
// residual of r (.) dH), the query operand is q (.) w, exact when w = NULL
// (then q is the stored bf16 value) and otherwise hi + lo as well, and the
// row scale of RMSNorm multiplies the finished sum.  So W' = Kh_hi^T q_hi +
// Kh_lo^T q_hi (+ Kh_hi^T q_lo).  The softmax backward differences the
// weights (dl_j = g p_j (dy . V_j - Dy)) and its sums over memories cancel,
// so bf16-rounded logits (an absolute error of about 1e-2 at logits of rms
// sqrt(P)) would move the gradients by several per cent; with these logits
// they move by about 1e-5.
//
// Per (head, memory) it writes the logit l2 (log2 units) and dwy; at the
// head's last memory, with d = sum_j exp2(l2_j - lse2) over the forward's
// log-sum-exp lse2 (log2 units), the exact log-sum-exp of these logits
// lse2 + log2(d) and Dy = sum_j p_j dwy_j with p_j = exp2(l2_j - lse2) / d:
// the weights the gradient kernels use are the softmax of the exact logits,
// whatever rounding the forward's log-sum-exp carries.  Tiles stream through
// an NS-stage LDS ring by DMA, NS - 1 steps ahead, copied by waves 0-3.
template <typename T, int N, int RT>
__global__ __launch_bounds__(512) void k_bwd_scores(
    const T* __restrict__ qh, const bf16* __restrict__ ql, const float* __restrict__ qsc,
    const float* __restrict__ eb, const T* __restrict__ Cm, const float* __restrict__ rinv,
    const T* __restrict__ kmem, const T* __restrict__ klo, const float* __restrict__ lse,
    const T* __restrict__ dy, float* __restrict__ lw, float* __restrict__ dwv,
    float* __restrict__ lsep, float* __restrict__ rdy, int use_ql, int64_t L, int64_t Ls, int H,
    int G, int S, int64_t Mp, int hpb, int blk0, int nblk, int64_t BHC) {
    constexpr bool LO = sizeof(T) == 2;
    constexpr int NTL = LO ? 2 : 1;  // tiles per stage: key side (and its residual)
    constexpr int RB = kP * (int)sizeof(T);
    constexpr int TILE = N * RB;
    constexpr int NT = N / 16;
    constexpr int KQ = N / 32;
    constexpr int NTH = NT / 2;
    constexpr int NS = tok_stages<T, N, NTL>();
    constexpr int TB = kTokBlock * RT;  // tokens per workgroup
    using Copy = TileCopy<RB, TILE, kTokWaves>;
    constexpr int RPW = N / 16;
    constexpr int CPS = NTL * Copy::count() + 1;
    __shared__ __attribute__((aligned(16))) char ring[NS][NTL][TILE];
    __shared__ __attribute__((aligned(16))) float rring[NS][N];
    __shared__ float xch[2][2][kTokWaves][16 * RT];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
    const int col = lane & 15, grp = lane >> 4;
    const int tg = wave & 3, nh = wave >> 2;
    const bool copier = wave < kTokWaves;
    int blk;
    int64_t bhc;
    tok_block(blockIdx.x, nblk, BHC, blk, bhc);
    const int nhb = H / hpb;
    const int64_t b = bhc / nhb;
    const int hb = (int)(bhc % nhb);
    const int64_t t0 = (int64_t)(blk0 + blk) * TB;
    const int nj = (int)(t0 / S);
    const int h0 = hb * hpb;
    const int g = h0 / (H / G);
    const int nt0 = nh * NTH;
    const int pt0 = nh * 2;
    bool valid[RT];
    int64_t tc[RT], bt[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const int64_t t = t0 + tg * 16 * RT + rt * 16 + col;
        valid[rt] = t < L;
        tc[rt] = valid[rt] ? t : L - 1;
        bt[rt] = b * L + tc[rt];
    }

    Frag<T> qf[RT][KQ];
    Frag<bf16> qlf[RT][LO ? KQ : 1];
    float qs[RT], ea[RT][2][4];
    typedef T T4 __attribute__((ext_vector_type(4)));
    T4 ca[RT][NTH];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        load_row_frags<T, T, N>(qh + (bt[rt] * G + g) * N, grp, qf[rt]);
        if constexpr (LO) {
            if (use_ql) {
                load_row_frags<bf16, bf16, N>(ql + (bt[rt] * G + g) * N, grp, qlf[rt]);
            } else {
#pragma unroll
                for (int ks = 0; ks < KQ; ++ks) qlf[rt][ks] = bf16x8{};
            }
        }
        qs[rt] = qsc[bt[rt] * G + g];
        const float* erow = eb + (bt[rt] * G + g) * kP;
#pragma unroll
        for (int q = 0; q < 2; ++q) load4(erow + 16 * (pt0 + q) + 4 * grp, ea[rt][q]);
        const T* crow = Cm + (bt[rt] * G + g) * N;
#pragma unroll
        for (int k = 0; k < NTH; ++k)
            ca[rt][k] = *reinterpret_cast<const T4*>(crow + 16 * (nt0 + k) + 4 * grp);
    }
    const f32x4 zero4{0.f, 0.f, 0.f, 0.f};
    const int nsteps = hpb * nj;
    Copy copy;
    copy.init(tg, lane);
    // (head, memory) of the next copy and of the current step, advanced in
    // order (no division in the stream)
    int ih = 0, ij = 0;
    auto issue_tiles = [&](int k) {
        const int hh = ih, j = ij;
        if (++ij == nj) {
            ij = 0;
            ++ih;
        }
        if (!copier) return;
        const int64_t hj = (b * Mp + j) * H + h0 + hh;
        copy.issue(kmem + hj * N * kP, ring[k % NS][0]);
        if constexpr (LO) copy.issue(klo + hj * N * kP, ring[k % NS][NTL - 1]);
        if (lane < RPW)
            lds_dma16_untracked_at(rinv + hj * N + (tg * RPW + lane) * 4,
                                   lds_addr(&rring[k % NS][0]) + tg * RPW * 16);
    };

#pragma unroll
    for (int k = 0; k < NS - 1; ++k)
        if (k < nsteps) issue_tiles(k);

    Frag<T> dyf[RT][2];
    float lse2[RT], dsum[RT], dyacc[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) lse2[rt] = dsum[rt] = dyacc[rt] = 0.f;
    int hh = 0, j = 0;
    for (int k = 0; k < nsteps; ++k) {
        const int h = h0 + hh;
        const int ahead = nsteps - 1 - k < NS - 2 ? nsteps - 1 - k : NS - 2;
        if (ahead >= 2) {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * CPS));
        } else if (ahead == 1) {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(CPS));
        } else {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
        }
        lds_barrier();
        if (j == 0) {
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                const T* dyrow = dy + (bt[rt] * H + h) * kP;
                dyf[rt][0] = load_frag(dyrow + 8 * grp);
                dyf[rt][1] = load_frag(dyrow + 32 + 8 * grp);
                lse2[rt] = lse[bt[rt] * H + h] * kLog2e;
                dsum[rt] = dyacc[rt] = 0.f;
                keep(dyf[rt][0]);
                keep(dyf[rt][1]);
                asm volatile("" ::"v"(lse2[rt]));
            }
        }
        if (k + NS - 1 < nsteps) issue_tiles(k + NS - 1);
        const char* kt = ring[k % NS][0];
        // this half's rows p of W'^T, every column tile per fragment read
        f32x4 w[RT][2];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int q = 0; q < 2; ++q) w[rt][q] = zero4;
#pragma unroll
        for (int ks = 0; ks < KQ; ++ks) {
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                const int r0 = 32 * ks + 4 * grp, r1 = r0 + 16, cb = 16 * (pt0 + q);
                const Frag<T> a = frag_km<T, RB>(kt, r0, r1, cb, lane);
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) w[rt][q] = mma16(w[rt][q], a, qf[rt][ks]);
                if constexpr (LO) {
                    const char* kl = ring[k % NS][NTL - 1];
                    const Frag<T> al = frag_km<T, RB>(kl, r0, r1, cb, lane);
#pragma unroll
                    for (int rt = 0; rt < RT; ++rt) {
                        w[rt][q] = mma16(w[rt][q], al, qf[rt][ks]);
                        if (use_ql) w[rt][q] = mma16(w[rt][q], a, qlf[rt][ks]);
                    }
                }
            }
        }
        float l2[RT], dw[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            l2[rt] = 0.f;
            dw[rt] = 0.f;
#pragma unroll
            for (int q = 0; q < 2; ++q)
#pragma unroll
                for (int i = 0; i < 4; ++i) l2[rt] += ea[rt][q][i] * w[rt][q][i];
        }
        // this half's rows n of X^T = diag(1/r) Kh dy^T, then C . X
#pragma unroll
        for (int q = 0; q < NTH; ++q) {
            const int nt = nt0 + q;
            f32x4 x[RT];
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) x[rt] = zero4;
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const Frag<T> a = frag_rowmajor<T, RB>(kt, 16 * nt + col, 32 * ks + 8 * grp);
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) x[rt] = mma16(x[rt], a, dyf[rt][ks]);
            }
            const f32x4 ri = *reinterpret_cast<const f32x4*>(&rring[k % NS][16 * nt + 4 * grp]);
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int i = 0; i < 4; ++i) dw[rt] += to_f(ca[rt][q][i]) * (x[rt][i] * ri[i]);
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            l2[rt] = row4_sum(l2[rt]);
            dw[rt] = row4_sum(dw[rt]);
            if (lane < 16) {
                xch[0][nh][tg][16 * rt + col] = l2[rt];
                xch[1][nh][tg][16 * rt + col] = dw[rt];
            }
        }
        lds_barrier();
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const float lv = (l2[rt] + xch[0][nh ^ 1][tg][16 * rt + col]) * qs[rt];
            const float dv = dw[rt] + xch[1][nh ^ 1][tg][16 * rt + col];
            const float p = fast_exp2(lv - lse2[rt]);
            dsum[rt] += p;
            dyacc[rt] += p * dv;
            if (nh == 0 && lane < 16 && valid[rt]) {
                const int64_t si = ((b * H + h) * Mp + j) * Ls + tc[rt];
                lw[si] = lv;
                dwv[si] = dv;
                if (j == nj - 1) {
                    lsep[bt[rt] * H + h] = lse2[rt] + __log2f(dsum[rt]);
                    rdy[bt[rt] * H + h] = dyacc[rt] / dsum[rt];
                }
            }
        }
        if (++j == nj) {
            j = 0;
            ++hh;
        }
    }
}

// ---- token-side gradients ------------------------------------------------------
// Same workgroup and block order as k_bwd_scores.  Waves w and w + 4 share
// the RT 16-token column tiles of tokens 16 RT w .. 16 RT w + 16 RT - 1 and
// split the rows of each product: rows p of W' (and dEbar), rows n of X and Z
// (and dQbar, dC).  In every MFMA product the memory tile is the A operand
// (rows n or p) and the tokens are the columns, so lane l works on token
// l % 16 of each column tile and its rows 4 (l / 16) + 0..3 of each 16-row
// tile; every fragment read from LDS feeds the RT column tiles.
//
// The scores kernel has left, per (head, memory, token), the exact logit and
// dwy, and per (token, head) the exact log-sum-exp and Dy; these rows (the
// block's tokens of one head and memory) arrive by DMA with the key tile, so
// each step knows p_j = exp2(l2_j - lse2') and dl_j = g p_j (dwy_j - Dy) at
// once:
//   dQbar += s dl_j Z_j,   Z = Kh Ebar^T;
//   dEbar += s dl_j Kh_j^T Qbar = ln2 dl_j W'_j,   W' = Kh^T Qbar'^T;
//   dC    += g p_j X_j,    X = diag(1/r) Kh dy^T = dH dy^T;
// the three products from the key side alone (bf16 rounding of these
// operands is not amplified: each sum over memories carries the exact
// weights).  g p_j replaces the logit in place for the memory kernel.
template <typename T, int N, int RT>
__global__ __launch_bounds__(512) void k_bwd_tokens(
    const T* __restrict__ qb, const float* __restrict__ eb, const float* __restrict__ rinv,
    const T* __restrict__ kmem, const T* __restrict__ z, const float* __restrict__ lsep,
    const float* __restrict__ rdy, const T* __restrict__ dy, float* __restrict__ gpw,
    const float* __restrict__ gdw, float* __restrict__ part, int z_per_head, int64_t L, int64_t Ls,
    int H, int G, int S, int64_t Mp, int hpb, int blk0, int nblk, int64_t BHC) {
    constexpr int RB = kP * (int)sizeof(T);  // bytes of one tile row (fixed n)
    constexpr int TILE = N * RB;
    constexpr int NT = N / 16;
    constexpr int KQ = N / 32;
    constexpr int NTH = NT / 2;          // n tiles per wave
    // (three stages with two column tiles: room for the lane slots below)
    constexpr int NS = RT > 1 && tok_stages<T, N, 1>() > 3 ? 3 : tok_stages<T, N, 1>();
    constexpr int TB = kTokBlock * RT;   // tokens per workgroup
    using Copy = TileCopy<RB, TILE, kTokWaves>;
    constexpr int RPW = N / 16;              // 16-byte pieces of the 1/r row per copying wave
    constexpr int CPS = Copy::count() + 2;   // DMA copies per copying wave per step
    __shared__ __attribute__((aligned(16))) char ring[NS][TILE];
    __shared__ __attribute__((aligned(16))) float rring[NS][N];
    __shared__ __attribute__((aligned(16))) float lring[NS][kTokWaves][2][16 * RT];  // logit, dwy
    // with two column tiles, each lane's Qbar' and Ebar fragments live in LDS
    // (one 16-byte slot per thread and fragment, conflict-free) rather than
    // in registers
    constexpr int QL = RT > 1 ? RT * (KQ + 2) : 1;
    __shared__ __attribute__((aligned(16))) Frag<T> qslot[QL][512];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
    const int col = lane & 15, grp = lane >> 4;
    const int tg = wave & 3, nh = wave >> 2;  // token group, half of n
    const bool copier = wave < kTokWaves;
    int blk;
    int64_t bhc;
    tok_block(blockIdx.x, nblk, BHC, blk, bhc);
    const int nhb = H / hpb;
    const int64_t b = bhc / nhb;
    const int hb = (int)(bhc % nhb);
    const int64_t t0 = (int64_t)(blk0 + blk) * TB;
    const int nj = (int)(t0 / S);  // memories every token of the block attends
    const int h0 = hb * hpb;
    const int g = h0 / (H / G);
    const float isn = 1.0f / sqrtf((float)N);
    const int nt0 = nh * NTH;  // first n tile of this wave
    const int pt0 = nh * 2;    // first p tile of this wave
    bool valid[RT];
    int64_t tc[RT], bt[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const int64_t t = t0 + tg * 16 * RT + rt * 16 + col;
        valid[rt] = t < L;
        tc[rt] = valid[rt] ? t : L - 1;
        bt[rt] = b * L + tc[rt];
    }

    // group-shared token operands (Qbar' whole; Ebar)
    Frag<T> qf[RT > 1 ? 1 : RT][KQ], ef[RT > 1 ? 1 : RT][2];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        if constexpr (RT > 1) {
            Frag<T> tmp[KQ];
            load_row_frags<T, T, N>(qb + (bt[rt] * G + g) * N, grp, tmp);
#pragma unroll
            for (int ks = 0; ks < KQ; ++ks) qslot[rt * KQ + ks][threadIdx.x] = tmp[ks];
        } else {
            load_row_frags<T, T, N>(qb + (bt[rt] * G + g) * N, grp, qf[rt]);
        }
        const float* erow = eb + (bt[rt] * G + g) * kP;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            float v[8];
            load8(erow + ks * 32 + 8 * grp, v);
            if constexpr (RT > 1) {
                qslot[RT * KQ + rt * 2 + ks][threadIdx.x] = make_frag<T>(v);
            } else {
                ef[rt][ks] = make_frag<T>(v);
            }
        }
    }

    const f32x4 zero4{0.f, 0.f, 0.f, 0.f};
    f32x4 dQ[RT][NTH], dC[RT][NTH], dE[RT][2];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
        for (int k = 0; k < NTH; ++k) dQ[rt][k] = dC[rt][k] = zero4;
#pragma unroll
        for (int q = 0; q < 2; ++q) dE[rt][q] = zero4;
    }

    const int nsteps = hpb * nj;
    Copy copy;
    copy.init(tg, lane);
    // (head, memory) of the next copy and of the current step, advanced in
    // order (no division in the stream)
    int ih = 0, ij = 0;
    auto issue_tiles = [&](int k) {
        const int hh = ih, j = ij;
        if (++ij == nj) {
            ij = 0;
            ++ih;
        }
        if (!copier) return;
        const int64_t hj = (b * Mp + j) * H + h0 + hh;
        copy.issue(kmem + hj * N * kP, ring[k % NS]);
        if (lane < RPW)
            lds_dma16_untracked_at(rinv + hj * N + (tg * RPW + lane) * 4,
                                   lds_addr(&rring[k % NS][0]) + tg * RPW * 16);
        // this token group's 16 RT logits (lanes 0 .. 4 RT - 1) and dwy (the next 4 RT)
        if (lane < 8 * RT) {
            const int64_t srow = ((b * H + h0 + hh) * Mp + j) * Ls + t0 + 16 * RT * tg + 4 * (lane % (4 * RT));
            lds_dma16_untracked_at(lane < 4 * RT ? (const float*)gpw + srow : gdw + srow,
                                   lds_addr(&lring[k % NS][tg][0][0]));
        }
    };

#pragma unroll
    for (int k = 0; k < NS - 1; ++k)
        if (k < nsteps) issue_tiles(k);

    Frag<T> dyf[RT][2];
    float lse2[RT], gate[RT], Dy[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) lse2[rt] = gate[rt] = Dy[rt] = 0.f;
    int hh = 0, j = 0;
    for (int k = 0; k < nsteps; ++k) {
        const int h = h0 + hh;
        // this step's copies (the ones of the later steps in flight may stay)
        const int ahead = nsteps - 1 - k < NS - 2 ? nsteps - 1 - k : NS - 2;
        if (ahead >= 2) {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * CPS));
        } else if (ahead == 1) {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(CPS));
        } else {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
        }
        lds_barrier();
        if (j == 0) {
            // this head's per-token operands, waited for here (copies issued
            // earlier in the stream complete first, so a head's start waits
            // for them too)
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                const T* dyrow = dy + (bt[rt] * H + h) * kP;
                dyf[rt][0] = load_frag(dyrow + 8 * grp);
                dyf[rt][1] = load_frag(dyrow + 32 + 8 * grp);
                lse2[rt] = lsep[bt[rt] * H + h];
                Dy[rt] = rdy[bt[rt] * H + h];
                gate[rt] = silu(to_f(z[z_per_head ? bt[rt] * H + h : bt[rt]]));
                keep(dyf[rt][0]);
                keep(dyf[rt][1]);
                asm volatile("" ::"v"(lse2[rt]), "v"(Dy[rt]), "v"(gate[rt]));
            }
        }
        // the next copies go out at the end of the step when two steps
        // separate them from their use (they then do not hold up the step's
        // first MFMAs: 978 -> 935 us at B4 L8192 H32 N128 S256), else here
        if (NS < 3 && k + NS - 1 < nsteps) issue_tiles(k + NS - 1);
        const char* kt = ring[k % NS];
        // lane coordinates made opaque per step, so that the fragment offsets
        // are recomputed in the loop rather than held live across it
        int ln = lane;
        asm volatile("" : "+v"(ln));
        const int col = ln & 15, grp = ln >> 4;
        // bf16: the step's fragment offsets, once per step: the transposing
        // reads of W' (column tile pt0 + q; k blocks move by 32 rows, an
        // immediate) and the row reads of X and Z (k half ks; n tiles move by
        // 16 rows, an immediate)
        KmOffBf16<RB> kofs[2];
        uint32_t xofs[2];
        if constexpr (sizeof(T) == 2) {
#pragma unroll
            for (int q = 0; q < 2; ++q) kofs[q].init(4 * grp, 16 + 4 * grp, 16 * (pt0 + q), ln);
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) xofs[ks] = (uint32_t)SwzTile<RB>::off(col, (32 * ks + 8 * grp) * 2);
        }
        float gp[RT], dl[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const float p = fast_exp2(lring[k % NS][tg][0][16 * rt + col] - lse2[rt]);
            gp[rt] = gate[rt] * p;
            dl[rt] = gp[rt] * (lring[k % NS][tg][1][16 * rt + col] - Dy[rt]);
        }
        // this half's rows p of W'^T = Kh^T Qbar'^T: dEbar += ln2 dl W'
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            f32x4 w[RT];
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) w[rt] = zero4;
#pragma unroll
            for (int ks = 0; ks < KQ; ++ks) {
                Frag<T> a;
                if constexpr (sizeof(T) == 2) {
                    a = kofs[q].read(kt, ks * 32 * RB);
                } else {
                    a = frag_km<T, RB>(kt, 32 * ks + 4 * grp, 32 * ks + 16 + 4 * grp, 16 * (pt0 + q), ln);
                }
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) {
                    if constexpr (RT > 1) {
                        w[rt] = mma16(w[rt], a, qslot[rt * KQ + ks][threadIdx.x]);
                    } else {
                        w[rt] = mma16(w[rt], a, qf[rt][ks]);
                    }
                }
            }
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) dE[rt][q] += (kLn2 * dl[rt]) * w[rt];
            if constexpr (RT > 1) __builtin_amdgcn_sched_barrier(0);
        }
        // X^T = diag(1/r) Kh dy^T and Z^T = Kh Ebar^T on this half's n tiles
#pragma unroll
        for (int q = 0; q < NTH; ++q) {
            const int nt = nt0 + q;
            f32x4 x[RT], zz[RT];
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) x[rt] = zz[rt] = zero4;
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                Frag<T> a;
                if constexpr (sizeof(T) == 2) {
                    a = *reinterpret_cast<const bf16x8*>(kt + xofs[ks] + 16 * nt * RB);
                } else {
                    a = frag_rowmajor<T, RB>(kt, 16 * nt + col, 32 * ks + 8 * grp);
                }
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) {
                    x[rt] = mma16(x[rt], a, dyf[rt][ks]);
                    if constexpr (RT > 1) {
                        zz[rt] = mma16(zz[rt], a, qslot[RT * KQ + rt * 2 + ks][threadIdx.x]);
                    } else {
                        zz[rt] = mma16(zz[rt], a, ef[rt][ks]);
                    }
                }
            }
            const f32x4 ri = *reinterpret_cast<const f32x4*>(&rring[k % NS][16 * nt + 4 * grp]);
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                dC[rt][q] += gp[rt] * (x[rt] * ri);
                dQ[rt][q] += (isn * dl[rt]) * zz[rt];
            }
            if constexpr (RT > 1) __builtin_amdgcn_sched_barrier(0);  // bounds the live fragments
        }
        if (nh == 0 && lane < 16) {
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
                if (valid[rt]) gpw[((b * H + h) * Mp + j) * Ls + tc[rt]] = gp[rt];
        }
        if (NS >= 3 && k + NS - 1 < nsteps) issue_tiles(k + NS - 1);
        if (++j == nj) {
            j = 0;
            ++hh;
        }
    }

    // per-head-block partial sums: dQbar [N], dEbar [P], dC [N]
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        if (!valid[rt]) continue;
        float* pr = part + (bt[rt] * nhb + hb) * (2 * N + kP);
#pragma unroll
        for (int q = 0; q < NTH; ++q) {
            const int nt = nt0 + q;
            *reinterpret_cast<f32x4*>(pr + 16 * nt + 4 * grp) = dQ[rt][q];
            *reinterpret_cast<f32x4*>(pr + N + kP + 16 * nt + 4 * grp) = dC[rt][q];
        }
#pragma unroll
        for (int q = 0; q < 2; ++q)
            *reinterpret_cast<f32x4*>(pr + N + 16 * (pt0 + q) + 4 * grp) = dE[rt][q];
    }
}

// ---- memory-side gradients -------------------------------------------------------
// Workgroup (b, h, block of kMemJ memories j0 .. j0 + kMemJ - 1), 8 waves:
//   M1_j = sum_t C_t^T (g p_j[t] dy_t),   M2_j = sum_t Qbar'_t^T (ln2 dl_j[t] Ebar_t)
// over the tokens t >= (j + 1) S.  The token stream (C, Qbar', dy, Ebar in the
// storage dtype, unscaled) is read once for all the block's memories: TB
// tokens per step are copied into LDS by DMA one step ahead, and the
// per-(memory, token) factors g p_j and ln2 dl_j (zero where memory j is not
// attended) scale the dy and Ebar fragments in registers.  Wave w owns the
// output columns p = 16 (w % 4) .. + 15; for bf16 it takes two of the four
// memories (2 (w / 4), + 1) over every n tile, so each scaled fragment feeds
// N/16 MFMAs of each product and no two waves scale the same fragment; for
// fp32 (operands twice as wide) it takes every memory over half the n tiles.
// The token
// tiles stream through a 3-stage LDS ring, two steps ahead: waves 0-3 issue
// the DMA copies (and wait for their own with exact counts), waves 4-7 load
// the factors of the step two ahead and write them to LDS at the end of the
// current one, so the ordinary loads never make a copying wave drain its
// copies.  Memories j >= M - 1 (attended by no token) are written as zeros.
template <typename T>
constexpr int mem_tb() { return sizeof(T) == 2 ? 64 : 32; }

template <typename T>
__device__ __forceinline__ Frag<T> scale_frag(Frag<T> f, const f32x4& s0, const f32x4& s1) {
    Frag<T> r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        r[i] = from_f<T>(to_f(f[i]) * s0[i]);
        r[4 + i] = from_f<T>(to_f(f[4 + i]) * s1[i]);
    }
    return r;
}

template <typename T, int N>
__global__ __launch_bounds__(512) void k_bwd_mem(const T* __restrict__ qb,
                                                 const T* __restrict__ ebt,
                                                 const T* __restrict__ Cm, const T* __restrict__ dy,
                                                 const T* __restrict__ mem,
                                                 const float* __restrict__ gpw,
                                                 const float* __restrict__ gdw,
                                                 const float* __restrict__ rdy,
                                                 float* __restrict__ dmem, float eps, int normalize,
                                                 int64_t L, int64_t Ls, int H, int G, int S,
                                                 int64_t Mcap, int64_t Mp, int64_t BH) {
    constexpr int J = kMemJ;
    constexpr int ES = (int)sizeof(T);
    constexpr int TB = mem_tb<T>();
    constexpr int RBN = N * ES, RBP = kP * ES;
    constexpr int CT = TB * RBN, DT = TB * RBP;
    // C and Qbar' tiles: pair-spread swizzle where their rows span 256 bytes
    using SwN = std::conditional_t<(ES == 2 && RBN >= 256), SwzTilePair<RBN>, SwzTile<RBN>>;
    constexpr int STAGE = 2 * CT + 2 * DT;
    constexpr bool MSPLIT = ES == 2;           // waves split the memories (else the n tiles)
    constexpr int NT = MSPLIT ? N / 16 : N / 32;  // n tiles per wave
    constexpr int JW = MSPLIT ? J / 2 : J;        // memories per wave
    static_assert(NT >= 1 && J % 2 == 0, "whole n tiles, memories in two halves");
    constexpr int NS = 3;
    // DMA copies per copying wave per step (every tile is a multiple of 256 pieces)
    constexpr int CPW = (2 * TB * RBN / 16 + 2 * TB * RBP / 16) / 256;
    static_assert((TB * RBP / 16) % 256 == 0, "tiles must split evenly over four waves");
    __shared__ __attribute__((aligned(16))) char buf[NS][STAGE];
    __shared__ __attribute__((aligned(16))) float sc[NS][J][2][TB];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
    const int col = lane & 15, grp = lane >> 4;
    const int pt = wave & 3;                       // p tile of the wave
    const int jh = MSPLIT ? (wave >> 2) * JW : 0;  // its first memory
    const int nt0 = MSPLIT ? 0 : (wave >> 2) * NT; // its first n tile
    const int64_t jb = (int64_t)blockIdx.x / BH;
    const int64_t bh = (int64_t)blockIdx.x - jb * BH;
    const int64_t b = bh / H;
    const int h = (int)(bh - b * H);
    const int g = h / (H / G);
    const int64_t j0 = jb * J;
    const int p = 16 * pt + col;
    auto out_of = [&](int jl) { return dmem + ((b * Mcap + j0 + jl) * H + h) * (int64_t)N * kP; };
    if (j0 >= Mp) {
        // no memory of the block is attended: zeros (slots up to Mcap)
        for (int jl = 0; jl < J; ++jl) {
            if (j0 + jl >= Mcap) break;
            float* out = out_of(jl);
            for (int q = tid; q < N * kP / 4; q += 512)
                reinterpret_cast<f32x4*>(out)[q] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        return;
    }
    const int64_t tbeg = (j0 + 1) * S;
    const int nstep = (int)((L - tbeg + TB - 1) / TB);
    const int64_t grow = (b * L) * G + g;  // row of token 0 in the [B][L][G] layout

    const bool copier = wave < 4;
    // copies of whole steps from per-lane offsets fixed here (C and Qbar' share
    // a row stride and layout); a ragged last step takes the general path
    TilePlan<RBN, TB, 4, SwN> pnc;
    TilePlan<RBP, TB, 4> pdy, pet;
    if (copier) {
        pnc.init(wave, lane, (uint32_t)(G * RBN), TB);
        pdy.init(wave, lane, (uint32_t)(H * RBP), TB);
        pet.init(wave, lane, (uint32_t)(G * RBP), TB);
    }
    const uint32_t buf_lds = lds_addr(&buf[0][0]);
    auto issue = [&](int st) {
        if (!copier || st >= nstep) return;
        const int64_t t0 = tbeg + (int64_t)st * TB;
        const int rv = (int)(L - t0 < TB ? L - t0 : TB);
        if (rv == TB) {
            const uint32_t dl = buf_lds + (uint32_t)((st % NS) * STAGE);
            pnc.issue(Cm + (grow + t0 * G) * N, dl, wave);
            pnc.issue(qb + (grow + t0 * G) * N, dl + CT, wave);
            pdy.issue(dy + ((b * L + t0) * H + h) * kP, dl + 2 * CT, wave);
            pet.issue(ebt + (grow + t0 * G) * kP, dl + 2 * CT + DT, wave);
            return;
        }
        char* d = buf[st % NS];
        dma_tile<RBN, true, SwN>(d, reinterpret_cast<const char*>(Cm + (grow + t0 * G) * N),
                                 (int64_t)G * RBN, TB, rv, wave, 4, lane);
        dma_tile<RBN, true, SwN>(d + CT, reinterpret_cast<const char*>(qb + (grow + t0 * G) * N),
                                 (int64_t)G * RBN, TB, rv, wave, 4, lane);
        dma_tile<RBP, true>(d + 2 * CT,
                            reinterpret_cast<const char*>(dy + ((b * L + t0) * H + h) * kP),
                            (int64_t)H * RBP, TB, rv, wave, 4, lane);
        dma_tile<RBP, true>(d + 2 * CT + DT,
                            reinterpret_cast<const char*>(ebt + (grow + t0 * G) * kP),
                            (int64_t)G * RBP, TB, rv, wave, 4, lane);
    };
    // factors of step st: g p_j[t] and ln2 dl_j[t] = ln2 g p_j (dwy_j - Dy),
    // loaded and stored by waves 4-7 (thread ft = tid - 256 of J * TB = 256)
    static_assert(J * TB <= 256, "one factor per thread of waves 4-7");
    // The loaded values stay raw until the store at the end of the step, so the
    // wait for the loads falls behind the step's MFMA work.
    const int ft = tid - 256;
    float fgp = 0.f, fgw = 0.f, fry = 0.f;
    auto load_factors = [&](int st) {
        fgp = fgw = fry = 0.f;
        if (ft >= 0 && ft < J * TB && st < nstep) {
            const int jl = ft / TB, tk = ft % TB;
            const int64_t j = j0 + jl, t = tbeg + (int64_t)st * TB + tk;
            if (j < Mp && t < L && t >= (j + 1) * S) {
                const int64_t si = ((b * H + h) * Mp + j) * Ls + t;
                fgp = gpw[si];
                fgw = gdw[si];
                fry = rdy[(b * L + t) * H + h];
            }
        }
    };
    auto store_factors = [&](int st) {
        if (ft >= 0 && ft < J * TB && st < nstep) {
            const int jl = ft / TB, tk = ft % TB;
            sc[st % NS][jl][0][tk] = fgp;
            sc[st % NS][jl][1][tk] = kLn2 * fgp * (fgw - fry);
        }
    };

    f32x4 m1[JW][NT], m2[JW][NT];
#pragma unroll
    for (int jw = 0; jw < JW; ++jw)
#pragma unroll
        for (int k = 0; k < NT; ++k) m1[jw][k] = m2[jw][k] = f32x4{0.f, 0.f, 0.f, 0.f};

    issue(0);
    issue(1);
    load_factors(0);
    store_factors(0);
    load_factors(1);
    store_factors(1);
    for (int st = 0; st < nstep; ++st) {
        // this step's copies landed (the next step's may stay in flight)
        if (st + 1 < nstep) {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(CPW));
        } else {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
        }
        lds_barrier();
        load_factors(st + 2);
        const char* cs = buf[st % NS];
        const char* qs = cs + CT;
        const char* dyt = cs + 2 * CT;
        const char* et = dyt + DT;
#pragma unroll
        for (int ks = 0; ks < TB / 32; ++ks) {
            const int r0 = 32 * ks + 4 * grp, r1 = r0 + 16;
            const Frag<T> bd = frag_km<T, RBP>(dyt, r0, r1, 16 * pt, lane);
            const Frag<T> be = frag_km<T, RBP>(et, r0, r1, 16 * pt, lane);
            Frag<T> bdj[JW], bej[JW];
#pragma unroll
            for (int jw = 0; jw < JW; ++jw) {
                const int jl = jh + jw;
                const f32x4 g0 = *reinterpret_cast<const f32x4*>(&sc[st % NS][jl][0][r0]);
                const f32x4 g1 = *reinterpret_cast<const f32x4*>(&sc[st % NS][jl][0][r1]);
                const f32x4 d0 = *reinterpret_cast<const f32x4*>(&sc[st % NS][jl][1][r0]);
                const f32x4 d1 = *reinterpret_cast<const f32x4*>(&sc[st % NS][jl][1][r1]);
                bdj[jw] = scale_frag<T>(bd, g0, g1);
                bej[jw] = scale_frag<T>(be, d0, d1);
            }
#pragma unroll
            for (int k = 0; k < NT; ++k) {
                const Frag<T> ac = frag_km<T, RBN, SwN>(cs, r0, r1, 16 * (nt0 + k), lane);
                const Frag<T> aq = frag_km<T, RBN, SwN>(qs, r0, r1, 16 * (nt0 + k), lane);
#pragma unroll
                for (int jw = 0; jw < JW; ++jw) {
                    m1[jw][k] = mma16(m1[jw][k], ac, bdj[jw]);
                    m2[jw][k] = mma16(m2[jw][k], aq, bej[jw]);
                }
            }
        }
        store_factors(st + 2);
        // the copies of step st + 2 go out after the work (and after the
        // factor loads were waited for by their stores)
        issue(st + 2);
    }
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    lds_barrier();

    // epilogue per memory: r[n] and dr[n] = sum_p dH[n,p] M2[n,p] reduced over
    // the four column waves through LDS (the stage buffers are free now)
    float* red = reinterpret_cast<float*>(&buf[0][0]);  // [J][2][4][N]
#pragma unroll
    for (int jw = 0; jw < JW; ++jw) {
        const int jl = jh + jw;
        const int64_t j = j0 + jl;
        if (j >= Mp) continue;
        const T* hsrc = mem + ((b * Mcap + j) * H + h) * (int64_t)N * kP;
#pragma unroll
        for (int k = 0; k < NT; ++k)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int n = 16 * (nt0 + k) + 4 * grp + i;
                const float hv = to_f(hsrc[n * kP + p]);
                const float s2 = dpp_group_sum<16>(hv * hv);
                const float d2 = dpp_group_sum<16>(hv * m2[jw][k][i]);
                if (col == 0) {
                    red[((jl * 2 + 0) * 4 + pt) * N + n] = s2;
                    red[((jl * 2 + 1) * 4 + pt) * N + n] = d2;
                }
            }
    }
    __syncthreads();
#pragma unroll
    for (int jw = 0; jw < JW; ++jw) {
        const int jl = jh + jw;
        const int64_t j = j0 + jl;
        if (j >= Mcap) break;
        float* out = out_of(jl);
        const T* hsrc = mem + ((b * Mcap + j) * H + h) * (int64_t)N * kP;
#pragma unroll
        for (int k = 0; k < NT; ++k)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int n = 16 * (nt0 + k) + 4 * grp + i;
                float o = 0.f;
                if (j < Mp) {
                    o = m1[jw][k][i];
                    if (normalize) {
                        const float* r0 = red + (jl * 2 + 0) * 4 * N + n;
                        const float* r1 = red + (jl * 2 + 1) * 4 * N + n;
                        const float ss = r0[0] + r0[N] + r0[2 * N] + r0[3 * N];
                        const float dr = r1[0] + r1[N] + r1[2 * N] + r1[3 * N];
                        const float r = __builtin_amdgcn_rsqf(ss * (1.0f / kP) + eps);
                        const float hv = to_f(hsrc[n * kP + p]);
                        o += r * m2[jw][k][i] - (r * r * r * (1.0f / kP)) * dr * hv;
                    } else {
                        o += m2[jw][k][i];
                    }
                }
                out[n * kP + p] = o;
            }
    }
}

// ---- finishing: per (b, t, g) -------------------------------------------------------
template <typename T, int N>
__global__ __launch_bounds__(256) void k_bwd_finish(
    const T* __restrict__ q, const T* __restrict__ e, const T* __restrict__ z,
    const float* __restrict__ qw, const float* __restrict__ ew, const float* __restrict__ part,
    const float* __restrict__ rdy, float* __restrict__ dq, float* __restrict__ de,
    float* __restrict__ dC, float* __restrict__ dz, float eps, int normalize, int z_per_head,
    int64_t L, int H, int G, int S, int hpb, int64_t rows) {
    constexpr int QE = (N + 63) / 64;
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows) return;
    const int g = (int)(row % G);
    const int64_t bt = row / G;
    const int64_t t = bt % L;
    const bool hist = t >= S;  // tokens of the first chunk get no gradient
    const int hpg = H / G;
    const int nhb = H / hpb;
    const int hb0 = g * hpg / hpb, hb1 = (g + 1) * hpg / hpb;
    float sq[QE], sc[QE], se = 0.f;
#pragma unroll
    for (int k = 0; k < QE; ++k) sq[k] = sc[k] = 0.f;
    if (hist) {
        for (int hb = hb0; hb < hb1; ++hb) {
            const float* pr = part + (bt * nhb + hb) * (2 * N + kP);
#pragma unroll
            for (int k = 0; k < QE; ++k) {
                const int n = lane + 64 * k;
                if (n < N) {
                    sq[k] += pr[n];
                    sc[k] += pr[N + kP + n];
                }
            }
            se += pr[N + lane];
        }
    }
    // q: dq = inv u - q inv^3 (u . q) / N with u = dQbar (.) w
    float qv[QE], u[QE];
    float ss = 0.f, uq = 0.f;
#pragma unroll
    for (int k = 0; k < QE; ++k) {
        const int n = lane + 64 * k;
        qv[k] = n < N ? to_f(q[row * N + n]) : 0.f;
        u[k] = n < N ? sq[k] * (normalize && qw ? qw[n] : 1.0f) : 0.f;
        ss += qv[k] * qv[k];
        uq += u[k] * qv[k];
    }
    ss = wave_sum(ss);
    uq = wave_sum(uq);
    const float qi = 1.0f / sqrtf(ss * (1.0f / N) + eps);
#pragma unroll
    for (int k = 0; k < QE; ++k) {
        const int n = lane + 64 * k;
        if (n < N) {
            dq[row * N + n] = normalize ? u[k] * qi - qv[k] * qi * qi * qi * uq * (1.0f / N) : sq[k];
            dC[row * N + n] = sc[k];
        }
    }
    const float ev = to_f(e[row * kP + lane]);
    const float ue = se * (normalize && ew ? ew[lane] : 1.0f);
    const float es = wave_sum(ev * ev);
    const float ueu = wave_sum(ue * ev);
    const float ei = 1.0f / sqrtf(es * (1.0f / kP) + eps);
    de[row * kP + lane] = normalize ? ue * ei - ev * ei * ei * ei * ueu * (1.0f / kP) : se;
    // gate
    if (z_per_head) {
        for (int k = lane; k < hpg; k += 64) {
            const int h = g * hpg + k;
            dz[bt * H + h] = hist ? silu_grad(to_f(z[bt * H + h])) * rdy[bt * H + h] : 0.f;
        }
    } else if (g == 0) {
        float s = 0.f;
        if (hist)
            for (int h = lane; h < H; h += 64) s += rdy[bt * H + h];
        s = wave_sum(s);
        if (lane == 0) dz[bt] = hist ? silu_grad(to_f(z[bt])) * s : 0.f;
    }
}

// Heads per block of the token kernels (and so of the per-token partials the
// finishing kernel sums): the token blocks are 128 tokens for bf16 at S >= 128,
// else kTokBlock, and the first chunk's blocks are not launched.
int bwd_heads_per_block(const Shape& s) {
    const int tpb = (s.dtype == 1 && s.S >= 128) ? 2 * kTokBlock : kTokBlock;
    return sma_block_heads(s.B, s.H, s.G, s.L, s.S, tpb, kHeadsPerBlock, true);
}

struct BwdWs {
    void* kmem;
    void* klo;    // rounding residual of the bf16 key side (bf16 only)
    void* qb;     // Qbar' in the storage dtype
    void* qh;     // q (.) w in the storage dtype
    void* ql;     // its bf16 rounding residual (bf16 only)
    float* qsc;   // per-row scale: Qbar' = (q (.) w) qsc
    float* eb;
    void* ebt;    // Ebar in the storage dtype (eb itself for fp32)
    float* rinv;  // 1 / r of every attended memory row, [B][M-1][H][N]
    float* gp;    // per (b, h, memory, token): the exact logit, then g p
    float* gd;    // per (b, h, memory, token): dwy
    float* part;
    float* rdy;   // Dy per (b, t, h)
    float* lsep;  // exact log-sum-exp (log2 units) per (b, t, h)
    size_t bytes;
};

// Row stride of the per-(b, h, memory) token arrays: a multiple of the 64
// tokens a token-kernel workgroup reads as one row piece.
// Row stride of the per-(head, memory) token arrays: a multiple of the
// largest token block (128), so a block's rows stay inside the array.
inline int64_t bwd_row_stride(const Shape& s) {
    return (s.L + 2 * kTokBlock - 1) / (2 * kTokBlock) * (2 * kTokBlock);
}

BwdWs bwd_layout(const Shape& s, void* base) {
    const int64_t Mp = s.M > 1 ? s.M - 1 : 0;
    const size_t es = elem_bytes(s.dtype);
    const bool lo = s.dtype == 1;
    const int nhb = s.H / bwd_heads_per_block(s);
    const size_t Ls = (size_t)bwd_row_stride(s);
    size_t o = 0;
    BwdWs w;
    char* p = reinterpret_cast<char*>(base);
    auto take = [&](size_t bytes) {
        void* r = p ? p + o : nullptr;
        o += align256(bytes);
        return r;
    };
    w.kmem = take(es * s.B * Mp * s.H * (size_t)s.N * s.P);
    w.klo = lo ? take(es * s.B * Mp * s.H * (size_t)s.N * s.P) : nullptr;
    w.rinv = (float*)take(4 * s.B * Mp * s.H * (size_t)s.N);
    w.qb = take(es * s.B * s.L * s.G * (size_t)s.N);
    w.qh = take(es * s.B * s.L * s.G * (size_t)s.N);
    w.ql = lo ? take(2 * s.B * s.L * s.G * (size_t)s.N) : nullptr;
    w.qsc = (float*)take(4 * s.B * s.L * (size_t)s.G);
    w.eb = (float*)take(4 * s.B * s.L * s.G * (size_t)s.P);
    w.ebt = lo ? take(es * s.B * s.L * s.G * (size_t)s.P) : (void*)w.eb;
    w.gp = (float*)take(4 * s.B * s.H * Mp * Ls);
    w.gd = (float*)take(4 * s.B * s.H * Mp * Ls);
    w.part = (float*)take(4 * s.B * s.L * nhb * (size_t)(2 * s.N + s.P));
    w.rdy = (float*)take(4 * s.B * s.L * (size_t)s.H);
    w.lsep = (float*)take(4 * s.B * s.L * (size_t)s.H);
    w.bytes = o;
    return w;
}

template <typename T, int N>
hipError_t run_bwd(const Shape& s, const SmaArgs& a, const void* q, const void* e, const void* Cm,
                   const void* mem, const void* z, const float* lse, const void* dy, float* dq,
                   float* de, float* dC, float* dmem, float* dz, void* ws, hipStream_t st) {
    const int64_t Mp = s.M > 1 ? s.M - 1 : 0;
    const BwdWs w = bwd_layout(s, ws);
    const int hpb = bwd_heads_per_block(s);
    const int64_t Ls = bwd_row_stride(s);
    constexpr bool LO = sizeof(T) == 2;
    hipError_t err;
    if (Mp > 0) {
        err = launch_sma_keys(s, a, mem, w.kmem, w.klo, w.rinv, st);
        if (err != hipSuccess) return err;
    }
    const int64_t rows = s.B * s.L * s.G;
    const unsigned rblocks = (unsigned)((rows + 3) / 4);
    prof_begin("k_bwd_prep", st);
    k_bwd_prep<T, N><<<rblocks, 256, 0, st>>>((const T*)q, (const T*)e, a.qw, a.ew, (T*)w.qb,
                                              (T*)w.qh, (bf16*)w.ql, w.qsc, w.eb,
                                              LO ? (T*)w.ebt : nullptr, a.eps, a.normalize, rows);
    prof_end(st);
    const int blk0 = s.S / kTokBlock;
    const int64_t nblk = (s.L + kTokBlock - 1) / kTokBlock - blk0;
    if (Mp > 0 && nblk > 0) {
        const int64_t BHC = s.B * (s.H / hpb);
        // the query operand needs its residual only when a norm weight makes
        // q (.) w inexact in bf16
        const int use_ql = LO && a.qw != nullptr;
        prof_begin("k_bwd_scores", st);
        bool two = false;
        if constexpr (sizeof(T) == 2) {
            if (s.S >= 128) {
                // bf16: 128 tokens per workgroup (S is a multiple of 128, so a
                // block never straddles chunks)
                constexpr int TB2 = 2 * kTokBlock;
                const int sb0 = s.S / TB2;
                const int64_t snblk = (s.L + TB2 - 1) / TB2 - sb0;
                k_bwd_scores<T, N, 2><<<(unsigned)(BHC * snblk), 512, 0, st>>>(
                    (const T*)w.qh, (const bf16*)w.ql, w.qsc, w.eb, (const T*)Cm, w.rinv,
                    (const T*)w.kmem, (const T*)w.klo, lse, (const T*)dy, w.gp, w.gd, w.lsep, w.rdy,
                    use_ql, s.L, Ls, s.H, s.G, s.S, Mp, hpb, sb0, (int)snblk, BHC);
                two = true;
            }
        }
        if (!two) {
            k_bwd_scores<T, N, 1><<<(unsigned)(BHC * nblk), 512, 0, st>>>(
                (const T*)w.qh, (const bf16*)w.ql, w.qsc, w.eb, (const T*)Cm, w.rinv,
                (const T*)w.kmem, (const T*)w.klo, lse, (const T*)dy, w.gp, w.gd, w.lsep, w.rdy,
                use_ql, s.L, Ls, s.H, s.G, s.S, Mp, hpb, blk0, (int)nblk, BHC);
        }
        prof_end(st);
        prof_begin("k_bwd_tokens", st);
        two = false;
        if constexpr (sizeof(T) == 2) {
            if (s.S >= 128) {
                constexpr int TB2 = 2 * kTokBlock;
                const int sb0 = s.S / TB2;
                const int64_t snblk = (s.L + TB2 - 1) / TB2 - sb0;
                k_bwd_tokens<T, N, 2><<<(unsigned)(BHC * snblk), 512, 0, st>>>(
                    (const T*)w.qb, w.eb, w.rinv, (const T*)w.kmem, (const T*)z, w.lsep, w.rdy,
                    (const T*)dy, w.gp, w.gd, w.part, a.z_per_head, s.L, Ls, s.H, s.G, s.S, Mp, hpb,
                    sb0, (int)snblk, BHC);
                two = true;
            }
        }
        if (!two) {
            k_bwd_tokens<T, N, 1><<<(unsigned)(BHC * nblk), 512, 0, st>>>(
                (const T*)w.qb, w.eb, w.rinv, (const T*)w.kmem, (const T*)z, w.lsep, w.rdy,
                (const T*)dy, w.gp, w.gd, w.part, a.z_per_head, s.L, Ls, s.H, s.G, s.S, Mp, hpb,
                blk0, (int)nblk, BHC);
        }
        prof_end(st);
    }
    const int64_t BH = s.B * s.H;
    prof_begin("k_bwd_mem", st);
    const int64_t njb = (s.Mcap + kMemJ - 1) / kMemJ;
    k_bwd_mem<T, N><<<(unsigned)(BH * njb), 512, 0, st>>>(
        (const T*)w.qb, (const T*)w.ebt, (const T*)Cm, (const T*)dy, (const T*)mem, w.gp, w.gd, w.rdy, dmem, a.eps,
        a.normalize, s.L, Ls, s.H, s.G, s.S, s.Mcap, Mp, BH);
    prof_end(st);
    prof_begin("k_bwd_finish", st);
    k_bwd_finish<T, N><<<rblocks, 256, 0, st>>>((const T*)q, (const T*)e, (const T*)z, a.qw, a.ew,
                                                w.part, w.rdy, dq, de, dC, dz, a.eps, a.normalize,
                                                a.z_per_head, s.L, s.H, s.G, s.S, hpb, rows);
    prof_end(st);
    return hipGetLastError();
}

// The generic path: token and memory sides from generic.hip, then the same
// finishing kernel with one head per partial.
GenBwdWs gbwd_layout(const Shape& s, void* base) {
    const int64_t Mp = s.M > 1 ? s.M - 1 : 0;
    const size_t Ls = (size_t)bwd_row_stride(s);
    size_t o = 0;
    char* p = reinterpret_cast<char*>(base);
    auto take = [&](size_t bytes) {
        float* r = p ? reinterpret_cast<float*>(p + o) : nullptr;
        o += align256(bytes);
        return r;
    };
    GenBwdWs w;
    w.gp = take(4 * s.B * s.H * (Mp > 0 ? Mp : 1) * Ls);
    w.dl = take(4 * s.B * s.H * (Mp > 0 ? Mp : 1) * Ls);
    w.rdy = take(4 * s.B * s.L * (size_t)s.H);
    w.part = take(4 * s.B * s.L * s.H * (size_t)(2 * s.N + s.P));
    w.Ls = (int64_t)Ls;
    w.bytes = o;
    return w;
}

template <typename T, int N>
hipError_t run_gbwd(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                    const void* Cm, const void* mem, const void* z, const float* lse,
                    const void* dy, float* dq, float* de, float* dC, float* dmem, float* dz,
                    void* ws, hipStream_t st) {
    (void)lse;  // the generic backward forms the exact log-sum-exp itself
    const GenBwdWs w = gbwd_layout(s, ws);
    hipError_t err = launch_gsma_bwd(s, a, q, e, Cm, mem, z, dy, w, dmem, st);
    if (err != hipSuccess) return err;
    const int64_t rows = s.B * s.L * s.G;
    prof_begin("k_bwd_finish", st);
    k_bwd_finish<T, N><<<(unsigned)((rows + 3) / 4), 256, 0, st>>>(
        (const T*)q, (const T*)e, (const T*)z, a.qw, a.ew, w.part, w.rdy, dq, de, dC, dz, a.eps,
        a.normalize, a.z_per_head, s.L, s.H, s.G, s.S, 1, rows);
    prof_end(st);
    return hipGetLastError();
}

template <typename T>
hipError_t run_gbwd_n(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                      const void* Cm, const void* mem, const void* z, const float* lse,
                      const void* dy, float* dq, float* de, float* dC, float* dmem, float* dz,
                      void* ws, hipStream_t st) {
    switch (s.N) {
        case 16: return run_gbwd<T, 16>(s, a, q, e, Cm, mem, z, lse, dy, dq, de, dC, dmem, dz, ws, st);
        case 32: return run_gbwd<T, 32>(s, a, q, e, Cm, mem, z, lse, dy, dq, de, dC, dmem, dz, ws, st);
        case 64: return run_gbwd<T, 64>(s, a, q, e, Cm, mem, z, lse, dy, dq, de, dC, dmem, dz, ws, st);
        case 128: return run_gbwd<T, 128>(s, a, q, e, Cm, mem, z, lse, dy, dq, de, dC, dmem, dz, ws, st);
    }
    return hipErrorInvalidValue;
}

template <typename T>
hipError_t run_bwd_n(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                     const void* Cm, const void* mem, const void* z, const float* lse,
                     const void* dy, float* dq, float* de, float* dC, float* dmem, float* dz,
                     void* ws, hipStream_t st) {
    switch (s.N) {
        case 32: return run_bwd<T, 32>(s, a, q, e, Cm, mem, z, lse, dy, dq, de, dC, dmem, dz, ws, st);
        case 64: return run_bwd<T, 64>(s, a, q, e, Cm, mem, z, lse, dy, dq, de, dC, dmem, dz, ws, st);
        case 128: return run_bwd<T, 128>(s, a, q, e, Cm, mem, z, lse, dy, dq, de, dC, dmem, dz, ws, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace

size_t sma_bwd_workspace_bytes(const Shape& s) {
    if (!tuned_shape(s)) return gbwd_layout(s, nullptr).bytes;
    return bwd_layout(s, nullptr).bytes;
}

hipError_t launch_sma_bwd(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                          const void* Cm, const void* mem, const void* z, const float* lse,
                          const void* dy, float* dq, float* de, float* dC, float* dmem, float* dz,
                          void* ws, hipStream_t st) {
    if (!tuned_shape(s)) {
        if (s.dtype == 1) return run_gbwd_n<bf16>(s, a, q, e, Cm, mem, z, lse, dy, dq, de, dC, dmem, dz, ws, st);
        return run_gbwd_n<float>(s, a, q, e, Cm, mem, z, lse, dy, dq, de, dC, dmem, dz, ws, st);
    }
    if (s.dtype == 1) return run_bwd_n<bf16>(s, a, q, e, Cm, mem, z, lse, dy, dq, de, dC, dmem, dz, ws, st);
    return run_bwd_n<float>(s, a, q, e, Cm, mem, z, lse, dy, dq, de, dC, dmem, dz, ws, st);
}

}  // namespace dart
