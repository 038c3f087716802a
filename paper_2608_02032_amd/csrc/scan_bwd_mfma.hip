// scan_bwd_mfma.hip -- backward of the chunked SSD scan and its chunk
// memories in the chunked matrix form, on MFMA (bf16 storage, the tuned
// shapes: P = 64, N in {32, 64, 128}, S in {64, 128, 256}).
//
// Paper: Sec. 2 (H_t = a_t H_{t-1} + dt_t B_t^T x_t, y_t = C_t H_t,
// a_t = exp(dt_t A_h), and the dual masked form y = (L o C B^T) diag(dt) x),
// Sec. 3 (chunk memory dH_[c]) and App. A (chunk decomposition).  Gradients of
//   loss = sum_t dy_t . y_t + sum_c <dmem_c, dH_[c]> + <dh_last, H_{L-1}>.
//
// Per chunk c (tokens s, t local; cs the inclusive cumulative log decay of
// the chunk, cs_e its last value) with W_c = R_c + dmem_c, R_c the adjoint
// entering the chunk's end from later chunks and the final state:
//   M1[s,t] = e^{cs_s - cs_t} (C_s . B_t),  M2[s,t] = e^{cs_s - cs_t} (dy_s . x_t)
//   (t <= s, zero otherwise);
//   dx_t = dt_t [ sum_s M1[s,t] dy_s + e^{cs_e - cs_t} B_t W_c ]
//   dB_t = sum_h dt_t [ sum_s M2[s,t] C_s + e^{cs_e - cs_t} W_c x_t ]
//   dC_s = sum_h [ sum_t M2[s,t] dt_t B_t + e^{cs_s} H_[c-1] dy_s ]
// The sums over heads of a group are taken inside the quadratic terms:
// Mbar[s,t] = sum_h dt_t M2_h[s,t] is formed over every head of the group and
// the two N-contractions (Mbar^T C and Mbar B) run once per chunk and group.
//
// The decay gradient.  With l_t = dt_t A_h, dL/dl_t is the sum of the pair
// terms e^{cs_s - cs_s'} (...) over every (input s', output s) pair that
// straddles t (s' < t <= s); a global reverse cumulative sum of per-token
// terms would telescope across the whole sequence and amplify rounding.  Here
// every piece is local to the chunk of t:
//   (a) pairs inside the chunk: D[s,t] = M1[s,t] (dy_s . x_t) dt_t,
//       r_s = sum_t D[s,t], c_t = sum_s D[s,t]:  sum_{s>=t} (r_s - c_s);
//   (b) s' in the chunk, s after it (through W_c):  sum_{s'<t} dt_s' v_s',
//       v_s' = e^{cs_e - cs_s'} (B_s' W_c) . x_s';
//   (c) s' before the chunk, s in it (through H_[c-1]):  sum_{s>=t} w_s,
//       w_s = e^{cs_s} C_s . (H_[c-1] dy_s);
//   (d) s' before, s after:  K_c = e^{cs_e} <R_c, H_[c-1]>  (every t of c).
// ddt_t = (B_t Lam_t) . x_t + A_h dL/dl_t and dA_h = sum_{b,t} dt_t dL/dl_t.
// D, r and c use the same rounded M1 that the dx product sees, so that (a)
// cancels its non-straddling pairs exactly.
//
// Kernels, in launch order:
//   k_sbwd_contract<0>  per (b, c, g, head slice): dH_[c] = B^T diag(e^{cs_e - cs} dt) x
//                       (bf16), the chunk's cumulative log decay, and B^T of
//                       the chunk (bf16, [N][S]);
//   k_sbwd_contract<1>  the same for dR_c = C^T diag(e^{cs}) dy and C^T;
//   k_sbwd_pass2        per (b, h, 1024 state elements): forward over chunks
//                       (entry states H_[c-1], bf16), backward (W_c bf16,
//                       partial K_c, dh0);
//   k_sbwd_group        per (b, c, g, set of 64 tokens), every head of the
//                       group: the W_c x and H_[c-1] dy terms of dB and dC
//                       (written to dB, dC), w_s, and Mbar for the set's
//                       token columns;
//   k_sbwd_quad         per (b, c, g, head slice): dx, the (a) (b) pieces and
//                       the chunk scan of dL/dl -> ddt, per-chunk dA partials;
//   k_sbwd_bc           per (b, c, g): + Mbar^T C into dB, + Mbar B into dC;
//   k_sbwd_dA           dA summed over batch and chunks.
// Deterministic (no atomics).
#include "dart_common.hpp"
#include "dart_internal.hpp"

namespace dart {
namespace {

constexpr int kP = 64;

template <int S> constexpr int quad_waves() { return S / 16 >= 8 ? 8 : S / 16; }
// Row tiles of a wave: w, then 2 NW - 1 - w (light and heavy causal rows).
__device__ __forceinline__ int quad_tile(int w, int q, int nw) {
    return q == 0 ? w : 2 * nw - 1 - w;
}
// Row r of the A operand of the 32-row Gram tile u holds token 16 u + r of
// its s block, so that accumulator element 4 u + i of lane l (row
// 4 (l / 16) + i) is token 16 u + 4 (l / 16) + i: the k order of every
// operand that meets these values (s, or n for B_t and W^T) is
// 16 u + 4 (lane / 16) + i, which keeps the transposing reads of
// KmOffSpread free of bank conflicts.
__device__ __forceinline__ int gram_row(int u, int r) { return 16 * u + r; }
// The token (or n) of element e of a lane's 8-value fragment in that order,
// within its 32-block.
__device__ __forceinline__ int korder(int e, int grp) { return 16 * (e >> 2) + 4 * grp + (e & 3); }

__device__ __forceinline__ bf16x8 scale_frag(bf16x8 v, float s) {
    bf16x8 r;
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = (bf16)((float)v[i] * s);
    return r;
}

// k-major fragment reads (as KmOffBf16) whose 16 columns are spread:
// column c = 0..15 of the fragment is tile column cbase + 8 (c / 4) + c % 4.
// With cbase = 32 (pt / 2) + 4 (pt % 2), the accumulator rows 4 g + i of the
// four p tiles pt are the columns 8 g + j and 32 + 8 g + j (j = 4 (pt % 2) + i),
// the k order of the row-major x_t fragments, so x_t . acc needs no exchange.
template <int RB>
struct KmOffSpread {
    uint32_t o0, o1;
    __device__ __forceinline__ void init(int ra, int rb, int cbase, int lane) {
        using Tl = SwzTile<RB>;
        const int j = lane & 15;
        const int col_b = (cbase + 8 * (j & 3)) * 2;
        o0 = (uint32_t)Tl::off(ra + (j >> 2), col_b);
        o1 = (uint32_t)Tl::off(rb + (j >> 2), col_b);
    }
    __device__ __forceinline__ bf16x8 read(const char* tile, int add) const {
        const s16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4*)(tile + add + o0));
        const s16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4*)(tile + add + o1));
        const bf16x4 b0 = __builtin_bit_cast(bf16x4, v0);
        const bf16x4 b1 = __builtin_bit_cast(bf16x4, v1);
        return bf16x8{b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
    }
};
__device__ __forceinline__ int spread_base(int pt) { return 32 * (pt >> 1) + 4 * (pt & 1); }

// block -> (b c g, head slice); the slices of one (b, c, g) share an XCD
__device__ __forceinline__ void block_bcg(int64_t nbcg, int nhs, int64_t& bcg, int& hs) {
    const int64_t bid = blockIdx.x;
    if (nbcg % 8 == 0) {
        const int64_t slot = bid >> 3;
        bcg = (slot / nhs) * 8 + (bid & 7);
        hs = (int)(slot % nhs);
    } else {
        bcg = bid / nhs;
        hs = (int)(bid % nhs);
    }
}

// ---------------------------------------------------------------------------
// Chunk contraction out[n][p] = sum_s w_s Am[s][n] V[s][p] per head (bf16
// out), 512 threads.  MODE 0: Am = B, V = x, w_s = e^{cs_e - cs_s} dt_s (the chunk's own
// state contribution dH); also records cs (log2 units) and the chunk's total
// log decay.  MODE 1: Am = C, V = dy, w_s = e^{cs_s} (the chunk adjoint dR).
// Am^T fragments are read once (k-major from the LDS tile) and kept for every
// head of the slice; each head's V rows arrive by DMA in one of two buffers
// while the previous head computes.  Wave w owns n tiles NTW (w % 2) .. of
// p tile w / 2 of the N x P result (so two waves weight each V fragment);
// the products are formed transposed, a lane holding out[n][p .. p + 3],
// and leave as 8-byte stores.  The slice-0 workgroup also writes Am^T of the
// chunk, [N][S] bf16 (columns past the end repeat the last token; every
// consumer gives them zero weight).
// ---------------------------------------------------------------------------
template <int N, int S, int MODE>
__global__ __launch_bounds__(512) void k_sbwd_contract(
    const bf16* __restrict__ Am, const bf16* __restrict__ V, const float* __restrict__ dt,
    const float* __restrict__ A, bf16* __restrict__ out, float* __restrict__ rec,
    float* __restrict__ lda, bf16* __restrict__ AmT, int64_t L, int H, int G, int64_t M, int hpb,
    int64_t nbcg) {
    constexpr int NW = 8, NT = 512;
    constexpr int VRB = kP * 2;
    constexpr int ARB = N * 2;
    constexpr int VT = S * VRB, ATB = S * ARB;
    constexpr int KST = S / 32;
    constexpr int NTW = N / 32;         // n tiles per wave
    constexpr int NG = 2;               // n-tile groups
    static_assert(NG * NTW * 16 == N && NG * 4 == NW, "tiles cover the waves");
    constexpr int TPL = S / 64;
    constexpr int NST = acc_row_stores<NTW>();  // stores per head and wave

    const int nhs = (H / G) / hpb;
    int64_t bcg;
    int hs;
    block_bcg(nbcg, nhs, bcg, hs);
    const int g = (int)(bcg % G);
    const int64_t bc = bcg / G;
    const int64_t b = bc / M, c = bc % M;
    const int hbase = g * (H / G) + hs * hpb;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = lane >> 4, col = lane & 15;
    const int64_t t0 = c * S;
    const int len = (int)(L - t0 < S ? L - t0 : S);
    const int ng = wave % NG, pg = wave / NG;

    // atile: the Am rows, then the weights of every head [hpb][S] (float)
    __shared__ __attribute__((aligned(16))) char atile[ATB];
    __shared__ __attribute__((aligned(16))) char vbuf[2][VT];
    float* const wall = reinterpret_cast<float*>(atile);

    TilePlan<VRB, S, NW> vplan;
    vplan.init(wave, lane, (uint32_t)(H * VRB), len);
    const uint32_t vbl = lds_addr(vbuf);
    auto issue_v = [&](int hh, int u) __attribute__((always_inline)) {
        vplan.issue(V + ((b * L + t0) * H + hbase + hh) * kP, vbl + (uint32_t)(u * VT), wave);
    };
    {
        TilePlan<ARB, S, NW> aplan;
        aplan.init(wave, lane, (uint32_t)(G * ARB), len);
        aplan.issue(Am + ((b * L + t0) * G + g) * N, lds_addr(atile), wave);
    }
    issue_v(0, 0);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    lds_barrier();
    bf16x8 afr[NTW][KST];
    {
        KmOffBf16<ARB> ao;
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
            ao.init(4 * grp, 16 + 4 * grp, (ng * NTW + j) * 16, lane);
#pragma unroll
            for (int ks = 0; ks < KST; ++ks) afr[j][ks] = ao.read(atile, ks * 32 * ARB);
        }
    }
    if (hs == 0) {
        // Am^T: item (n, 8 tokens) -> one 16-byte store
        bf16* dstT = AmT + bcg * (int64_t)N * S;
        for (int it = tid; it < N * (S / 8); it += NT) {
            const int n = it / (S / 8), s8 = it % (S / 8);
            bf16x8 v;
#pragma unroll
            for (int j = 0; j < 8; ++j)
                v[j] = *reinterpret_cast<const bf16*>(atile + SwzTile<ARB>::off(8 * s8 + j, 2 * n));
            *reinterpret_cast<bf16x8*>(dstT + (int64_t)n * S + 8 * s8) = v;
        }
    }
    lds_barrier();  // every wave holds its Am^T fragments: atile takes the weights
    for (int hd = wave; hd < hpb; hd += NW) {
        const int h = hbase + hd;
        const float a = A[h];
        float dv[TPL], cs[TPL];
        float run = 0.f;
#pragma unroll
        for (int k = 0; k < TPL; ++k) {
            const int tok = TPL * lane + k;
            dv[k] = tok < len ? dt[(b * L + t0 + tok) * H + h] : 0.f;
            run += dv[k] * a;
            cs[k] = run;
        }
        float incl = run;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const float t = __shfl_up(incl, o, 64);
            if (lane >= o) incl += t;
        }
        const float excl = incl - run;
#pragma unroll
        for (int k = 0; k < TPL; ++k) cs[k] += excl;
        const float cse = __shfl(cs[TPL - 1], 63, 64);
#pragma unroll
        for (int k = 0; k < TPL; ++k) {
            const int tok = TPL * lane + k;
            if constexpr (MODE == 0) {
                wall[hd * S + tok] = __expf(cse - cs[k]) * dv[k];
                rec[((b * H + h) * M + c) * S + tok] = cs[k] * kLog2e;
            } else {
                wall[hd * S + tok] = tok < len ? __expf(cs[k]) : 0.f;
            }
        }
        if constexpr (MODE == 0) {
            if (lane == 0) lda[(b * H + h) * M + c] = cse;
        }
    }
    KmOffBf16<VRB> vo;
    vo.init(4 * grp, 16 + 4 * grp, pg * 16, lane);

    for (int hh = 0; hh < hpb; ++hh) {
        const int u = hh & 1;
        // this wave's copies of head hh are in: only its stores of head hh - 1
        // came after them
        if (hh > 0) __builtin_amdgcn_s_waitcnt(vmcnt_imm(NST));
        lds_barrier();
        if (hh + 1 < hpb) issue_v(hh + 1, u ^ 1);
        const float* wv = wall + hh * S;
        f32x4 acc[NTW];
#pragma unroll
        for (int j = 0; j < NTW; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KST; ++ks) {
            const f32x4 w0 = *reinterpret_cast<const f32x4*>(wv + ks * 32 + 4 * grp);
            const f32x4 w1 = *reinterpret_cast<const f32x4*>(wv + ks * 32 + 16 + 4 * grp);
            const bf16x8 vr = vo.read(&vbuf[u][0], ks * 32 * VRB);
            float v[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[i] = (float)vr[i] * w0[i];
                v[4 + i] = (float)vr[4 + i] * w1[i];
            }
            const bf16x8 vf = make_frag<bf16>(v);
#pragma unroll
            for (int j = 0; j < NTW; ++j) acc[j] = mma16(acc[j], vf, afr[j][ks]);
        }
        // acc[j][i] = out[n = 16 (ng NTW + j) + col][p = 16 pg + 4 grp + i]
        store_acc_rows_bf16<NTW>(out + ((b * M + c) * H + hbase + hh) * (int64_t)N * kP + 16 * pg,
                                 kP, 16 * ng * NTW, acc, grp, col);
    }
}

// ---------------------------------------------------------------------------
// Per (b, h, 1024 state elements): forward over the chunks (entry states
// H_[c-1] -> Hb, bf16), then backward: W_c = R_c + dmem_c -> Wb (bf16), the
// partial K_c = e^{lda_c} sum R_c . H_[c-1] of this element block
// (-> Kp[b][h][c][block]) and R_{c-1} = e^{lda_c} R_c + dR_c; dh0 = R_{-1}.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_sbwd_pass2(
    const bf16* __restrict__ dH, const bf16* __restrict__ dR, const float* __restrict__ lda,
    const float* __restrict__ h0, const float* __restrict__ dmem, const float* __restrict__ dhl,
    bf16* __restrict__ Hb, bf16* __restrict__ Wb, float* __restrict__ Kp, float* __restrict__ dh0,
    int H, int NP, int64_t M, int64_t Mcap) {
    __shared__ float red[2][4];
    const int h = blockIdx.y;
    const int64_t b = blockIdx.z;
    const int blk = blockIdx.x, nblk = gridDim.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int e0 = (blk * 256 + tid) * 4;
    const bool ok = e0 < NP;
    const float* ld = lda + (b * H + h) * M;
    float hc[4] = {0.f, 0.f, 0.f, 0.f};
    if (ok && h0) load4(h0 + (b * H + h) * (int64_t)NP + e0, hc);
    for (int64_t c = 0; c < M; ++c) {
        const int64_t o = ((b * M + c) * H + h) * (int64_t)NP + e0;
        if (ok) {
            store4(Hb + o, hc);
            float d[4];
            load4(dH + o, d);
            const float a = __expf(ld[c]);
#pragma unroll
            for (int i = 0; i < 4; ++i) hc[i] = a * hc[i] + d[i];
        }
    }
    float r[4] = {0.f, 0.f, 0.f, 0.f};
    if (ok && dhl) load4(dhl + (b * H + h) * (int64_t)NP + e0, r);
    for (int64_t c = M - 1; c >= 0; --c) {
        const int64_t o = ((b * M + c) * H + h) * (int64_t)NP + e0;
        const float a = __expf(ld[c]);
        float kp = 0.f;
        if (ok) {
            float m[4] = {0.f, 0.f, 0.f, 0.f}, w[4], hb[4], d[4];
            if (dmem) load4(dmem + ((b * Mcap + c) * H + h) * (int64_t)NP + e0, m);
#pragma unroll
            for (int i = 0; i < 4; ++i) w[i] = r[i] + m[i];
            store4(Wb + o, w);
            load4(Hb + o, hb);  // this thread's own entry-state values, stored above
#pragma unroll
            for (int i = 0; i < 4; ++i) kp += r[i] * hb[i];
            load4(dR + o, d);
#pragma unroll
            for (int i = 0; i < 4; ++i) r[i] = a * r[i] + d[i];
        }
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) kp += __shfl_xor(kp, m, 64);
        const int u = (int)(c & 1);
        if (lane == 0) red[u][wave] = kp;
        __syncthreads();
        if (tid == 0) Kp[((b * H + h) * M + c) * nblk + blk] = a * ((red[u][0] + red[u][1]) + (red[u][2] + red[u][3]));
    }
    if (ok && dh0) store4(dh0 + (b * H + h) * (int64_t)NP + e0, r);
}

// ---------------------------------------------------------------------------
// Per (b, c, g, set of four 16-token tiles), every head of the group:
//   the rank-P terms dB_t += dt_t e^{cs_e - cs_t} W_c x_t and
//   dC_s += e^{cs_s} H_[c-1] dy_s ([n][t] tiles: A = W or H rows from LDS,
//   B = the scaled x or dy rows of the token tile), per head
//   w_s = e^{cs_s} C_s . (H_[c-1] dy_s), and
//   Mbar[s][t] = sum_h dt_t e^{cs_s - cs_t} (dy_s . x_t) for the set's token
//   columns (t <= s), in fp32 registers across the heads.
// Set q holds tiles q, NKB - 1 - q, NKB + q and 2 NKB - 1 - q (NKB = S / 32),
// which gives every set the same number of causal (tile, s block) pairs.
// Wave w owns tile w % 4 and half w / 4 of the n tiles and of the tile's
// pairs.  The products take the raw x and dy rows; the per-token factors
// (dt_t e^{cs_e - cs_t}, e^{cs_t}) scale their fp32 results.  dB and dC
// receive the rank-P terms (k_sbwd_bc adds the quadratic ones); Mbar goes out
// as bf16 [S][S] (rows s, columns t, causal blocks).
// ---------------------------------------------------------------------------
template <int N, int S>
__global__ __launch_bounds__(512) void k_sbwd_group(
    const bf16* __restrict__ x, const float* __restrict__ dt, const bf16* __restrict__ Cm,
    const bf16* __restrict__ dy, const float* __restrict__ rec, const bf16* __restrict__ Hb,
    const bf16* __restrict__ Wb, float* __restrict__ dB, float* __restrict__ dC,
    float* __restrict__ wp, bf16* __restrict__ mbar, int64_t L, int H, int G, int64_t M,
    int64_t nbcg) {
    constexpr int NW = 8;
    constexpr int XRB = kP * 2;
    constexpr int DYT = S * XRB, TT = N * XRB, RECB = 3 * S * 4;
    constexpr int UB = DYT + 2 * TT + RECB;
    constexpr int NTH = N / 32;          // n tiles per wave
    constexpr int NSET = S / 64;         // token sets per chunk
    constexpr int NKB = S / 32;
    constexpr int MPW = (NKB + 1) / 2;   // Mbar pairs of a wave (at most)
    int64_t bcg;
    int qs;
    block_bcg(nbcg, NSET, bcg, qs);
    const int g = (int)(bcg % G);
    const int64_t bc = bcg / G;
    const int64_t b = bc / M, c = bc % M;
    const int hpg = H / G;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = lane >> 4, col = lane & 15;
    const int64_t t0 = c * S;
    const int len = (int)(L - t0 < S ? L - t0 : S);
    const int slot = wave & 3, nh = wave >> 2;
    const int T = slot == 0 ? qs : slot == 1 ? NKB - 1 - qs : slot == 2 ? NKB + qs : 2 * NKB - 1 - qs;
    const int t = 16 * T + col;         // token within the chunk
    const bool valid = t < len;
    const int tc = valid ? t : len - 1;
    const int kfirst = (T >> 1) + nh;   // this wave's pairs: s blocks kfirst, kfirst + 2, ...
    const int nk = kfirst < NKB ? (NKB - kfirst + 1) / 2 : 0;

    __shared__ __attribute__((aligned(16))) char ubuf[2][UB];
    __shared__ float wpart[2][2][64];

    TilePlan<XRB, S, NW> dyplan;
    TilePlan<XRB, N, NW> nplan;
    dyplan.init(wave, lane, (uint32_t)(H * XRB), len);
    nplan.init(wave, lane, (uint32_t)XRB, N);
    const uint32_t ubl = lds_addr(ubuf);
    auto issue = [&](int hh, int u) __attribute__((always_inline)) {
        const int h = g * hpg + hh;
        const int64_t o = ((b * M + c) * H + h) * (int64_t)N * kP;
        const uint32_t ub = ubl + (uint32_t)(u * UB);
        dyplan.issue(dy + ((b * L + t0) * H + h) * kP, ub, wave);
        nplan.issue(Wb + o, ub + DYT, wave);
        nplan.issue(Hb + o, ub + DYT + TT, wave);
    };
    // per-token record of head hh (cs, dt, b_s = e^{cs_s - cs at the s block
    // start}): thread tid < S takes token tid; loaded early, stored to LDS
    // before the barrier that opens the head
    float rq[3];
    auto load_rec = [&](int hh) __attribute__((always_inline)) {
        const int h = g * hpg + hh;
        if (tid < S) {
            const float* rc = rec + ((b * H + h) * M + c) * S;
            rq[0] = rc[tid];
            rq[1] = tid < len ? dt[(b * L + t0 + tid) * H + h] : 0.f;
            rq[2] = rc[tid & ~31];
        }
    };
    auto store_rec = [&](int u) __attribute__((always_inline)) {
        if (tid < S) {
            float* r = reinterpret_cast<float*>(&ubuf[u][DYT + 2 * TT]);
            r[tid] = rq[0];
            r[S + tid] = rq[1];
            r[2 * S + tid] = tid < len ? fast_exp2(rq[0] - rq[2]) : 0.f;
        }
    };
    // C_t at the n rows this lane's accumulators hold (16 nt + 4 grp + i)
    float cvf[NTH][4];
#pragma unroll
    for (int j = 0; j < NTH; ++j) {
        const bf16x4 cv = *reinterpret_cast<const bf16x4*>(Cm + ((b * L + t0 + tc) * G + g) * N + (nh * NTH + j) * 16 + 4 * grp);
#pragma unroll
        for (int i = 0; i < 4; ++i) cvf[j][i] = (float)cv[i];
    }
    f32x4 accB[NTH], accC[NTH];
#pragma unroll
    for (int j = 0; j < NTH; ++j) {
        accB[j] = f32x4{0.f, 0.f, 0.f, 0.f};
        accC[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    float mb[MPW][8];
#pragma unroll
    for (int k = 0; k < MPW; ++k)
#pragma unroll
        for (int e = 0; e < 8; ++e) mb[k][e] = 0.f;
    // x_t fragments, one head ahead
    bf16x8 xn0, xn1;
    {
        const bf16* xr = x + ((b * L + t0 + tc) * H + g * hpg) * kP + 8 * grp;
        xn0 = load_frag(xr);
        xn1 = load_frag(xr + 32);
    }
    issue(0, 0);
    load_rec(0);
    store_rec(0);
    for (int hh = 0; hh < hpg; ++hh) {
        const int u = hh & 1;
        const int h = g * hpg + hh;
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
        lds_barrier();  // head hh's inputs are in; buffer u ^ 1 and the exchange slots u ^ 1 are free
        const bf16x8 xf0 = xn0, xf1 = xn1;
        if (hh + 1 < hpg) {
            issue(hh + 1, u ^ 1);
            load_rec(hh + 1);
            const bf16* xr = x + ((b * L + t0 + tc) * H + h + 1) * kP + 8 * grp;
            xn0 = load_frag(xr);
            xn1 = load_frag(xr + 32);
        }
        if (hh > 0 && nh == 0 && grp == 0 && valid) {
            const int tl = slot * 16 + col;
            wp[(b * L + t0 + t) * H + h - 1] = wpart[u ^ 1][0][tl] + wpart[u ^ 1][1][tl];
        }
        const char* dyt = &ubuf[u][0];
        const char* wtl = &ubuf[u][DYT];
        const char* htl = &ubuf[u][DYT + TT];
        const float* rcs = reinterpret_cast<const float*>(&ubuf[u][DYT + 2 * TT]);
        const float* rbs = rcs + 2 * S;
        // the lane's token, opaque per head: the diagonal masks derived from
        // it are formed in the loop rather than held across it
        int tq = t;
        asm volatile("" : "+v"(tq));
        const float cst = rcs[tq], dtt = rcs[S + tq], cse = rcs[S - 1];
        const float sx = valid ? dtt * fast_exp2(cse - cst) : 0.f;
        const float sy = valid ? fast_exp2(cst) : 0.f;
        const bf16x8 y0 = frag_rowmajor<bf16, XRB>(dyt, tc, 8 * grp);
        const bf16x8 y1 = frag_rowmajor<bf16, XRB>(dyt, tc, 32 + 8 * grp);
        // dB_t += dt_t e^{cs_e - cs_t} (W x_t); with dy^ = e^{cs_t} dy_t:
        // dC_t += H dy^, w_t = C_t . H dy^
        float wsum = 0.f;
#pragma unroll
        for (int j = 0; j < NTH; ++j) {
            const int nrow = (nh * NTH + j) * 16 + col;
            const bf16x8 w0 = frag_rowmajor<bf16, XRB>(wtl, nrow, 8 * grp);
            const bf16x8 w1 = frag_rowmajor<bf16, XRB>(wtl, nrow, 32 + 8 * grp);
            const f32x4 pb = mma16(mma16(f32x4{0.f, 0.f, 0.f, 0.f}, w0, xf0), w1, xf1);
            const bf16x8 h0f = frag_rowmajor<bf16, XRB>(htl, nrow, 8 * grp);
            const bf16x8 h1f = frag_rowmajor<bf16, XRB>(htl, nrow, 32 + 8 * grp);
            const f32x4 pc = mma16(mma16(f32x4{0.f, 0.f, 0.f, 0.f}, h0f, y0), h1f, y1);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                accB[j][i] += sx * pb[i];
                wsum += cvf[j][i] * pc[i];
                accC[j][i] += sy * pc[i];
            }
        }
        wsum = row4_sum(wsum * sy);
        if (grp == 0) wpart[u][nh][slot * 16 + col] = wsum;
        // Mbar pairs (tile T, s block K): A = dy rows in gram_row order, B = x_t
#pragma unroll
        for (int k = 0; k < MPW; ++k) {
            if (k < nk) {
                const int K = kfirst + 2 * k;
                f32x4 g2[2];
#pragma unroll
                for (int uu = 0; uu < 2; ++uu) {
                    const int s = 32 * K + gram_row(uu, col);
                    const bf16x8 a0 = frag_rowmajor<bf16, XRB>(dyt, s, 8 * grp);
                    const bf16x8 a1 = frag_rowmajor<bf16, XRB>(dyt, s, 32 + 8 * grp);
                    g2[uu] = mma16(mma16(f32x4{0.f, 0.f, 0.f, 0.f}, a0, xf0), a1, xf1);
                }
                const int s0 = 32 * K + 4 * grp, s1 = s0 + 16;  // tokens of elements 0..3, 4..7
                if (K > (T >> 1)) {
                    const float at = fast_exp2(rcs[32 * K] - cst) * dtt;
                    // (off the diagonal block every s of the block follows t)
                    const f32x4 b0 = *reinterpret_cast<const f32x4*>(rbs + s0);
                    const f32x4 b1 = *reinterpret_cast<const f32x4*>(rbs + s1);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        mb[k][i] += g2[0][i] * (b0[i] * at);
                        mb[k][4 + i] += g2[1][i] * (b1[i] * at);
                    }
                } else {
                    const f32x4 c0 = *reinterpret_cast<const f32x4*>(rcs + s0);
                    const f32x4 c1 = *reinterpret_cast<const f32x4*>(rcs + s1);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        if (s0 + i >= tq && s0 + i < len) mb[k][i] += g2[0][i] * (fast_exp2(c0[i] - cst) * dtt);
                        if (s1 + i >= tq && s1 + i < len) mb[k][4 + i] += g2[1][i] * (fast_exp2(c1[i] - cst) * dtt);
                    }
                }
            }
        }
        if (hh + 1 < hpg) store_rec(u ^ 1);
    }
    lds_barrier();
    if (nh == 0 && grp == 0 && valid) {
        const int u = (hpg - 1) & 1;
        const int tl = slot * 16 + col;
        wp[(b * L + t0 + t) * H + g * hpg + hpg - 1] = wpart[u][0][tl] + wpart[u][1][tl];
    }
    if (valid) {
        const int64_t row = ((b * L + t0 + t) * G + g) * N;
#pragma unroll
        for (int j = 0; j < NTH; ++j) {
            const int n = (nh * NTH + j) * 16 + 4 * grp;
            *reinterpret_cast<f32x4*>(dB + row + n) = accB[j];
            *reinterpret_cast<f32x4*>(dC + row + n) = accC[j];
        }
    }
    bf16* mo = mbar + bcg * (int64_t)S * S;
#pragma unroll
    for (int k = 0; k < MPW; ++k) {
        if (k < nk) {
            const int K = kfirst + 2 * k;
#pragma unroll
            for (int e = 0; e < 8; ++e) mo[(int64_t)(32 * K + korder(e, grp)) * S + t] = (bf16)mb[k][e];
        }
    }
}

// ---------------------------------------------------------------------------
// Quadratic terms per (b, c, g, head slice).  Wave w owns the row tiles
// (16 tokens t) quad_tile(w, q); a pair (tile T, 32-token s block K >= T/2)
// holds, in MFMA accumulator layout with the s order of gram_row, the Gram
// values G1 = C_s . B_t (formed once, kept as bf16 for every head) and per
// head G2 = dy_s . x_t (A = dy rows from LDS, B = x_t).  Per head and pair:
//   decay e^{cs_s - cs_t}: factored at the s block start off the diagonal
//   (b_s = e^{cs_s - cs_K} from LDS, one exp per lane), exact and masked on
//   the diagonal block;
//   M1 = bf16(G1 decay) -> dx^T += dy^T M1 (A = dy^T by transposing reads);
//   D = M1 G2 dt_t -> r_s (lane sums into LDS, per wave).
// The Gram's B operand is x~_t = bf16(dt_t x_t), so D = M1 (dy_s . x~_t) and
// c_t = x~_t . acc (acc = sum_s M1[s,t] dy_s) hold the same products.  Then
// dx^T += W^T (e^{cs_e - cs_t} B_t) (A = W^T from LDS), dx = dt acc,
// v_t = x~_t . (W term), (B Lam) . x = x_t . acc (the accumulator rows are
// spread to the k order of the x_t fragments, see KmOffSpread), and the chunk
// scan of dL/dl (one wave) -> ddt = (B Lam) . x + A_h dL/dl and the chunk's
// dA partial.  Each wave finishes one row tile before the next.
// ---------------------------------------------------------------------------
template <int N, int S>
__global__ __launch_bounds__(64 * quad_waves<S>()) void k_sbwd_quad(
    const bf16* __restrict__ x, const float* __restrict__ dt, const float* __restrict__ A,
    const bf16* __restrict__ Bm, const bf16* __restrict__ Cm, const bf16* __restrict__ dy,
    const float* __restrict__ rec, const bf16* __restrict__ Wb, const float* __restrict__ Kp,
    const float* __restrict__ wp, float* __restrict__ dx, float* __restrict__ ddt,
    float* __restrict__ dAp, int64_t L, int H, int G, int64_t M, int hpb, int64_t nbcg, int nkp) {
    constexpr int NW = quad_waves<S>();
    constexpr int NQ = S / 16 / NW;
    constexpr int NKB = S / 32;
    constexpr int NPW = NQ == 2 ? NKB + 1 : NKB;  // pairs of a wave (at most)
    constexpr int KS = N / 32;
    constexpr int XRB = kP * 2;
    constexpr int DYT = S * XRB, WTB = N * XRB;
    constexpr int REC = 3 * S * 4;                // cs (log2), dt, b_s
    constexpr int UB = DYT + WTB + REC;
    constexpr int TPL = S / 64;
    constexpr int BRB = N * 2;                    // bytes of a B or C row
    constexpr int BCT = S * BRB;
    constexpr int LDSB = 2 * UB > 2 * BCT ? 2 * UB : 2 * BCT;
    static_assert(NQ == 1 || NQ == 2, "one or two row tiles per wave");

    const int nhs = (H / G) / hpb;
    int64_t bcg;
    int hs;
    block_bcg(nbcg, nhs, bcg, hs);
    const int g = (int)(bcg % G);
    const int64_t bc = bcg / G;
    const int64_t b = bc / M, c = bc % M;
    const int hbase = g * (H / G) + hs * hpb;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = lane >> 4, col = lane & 15;
    const int64_t t0 = c * S;
    const int len = (int)(L - t0 < S ? L - t0 : S);

    // the two head buffers; before the head loop the same bytes hold the
    // chunk's B and C rows (swizzled [S][N] tiles) for the G1 pairs
    __shared__ __attribute__((aligned(16))) char lbuf[LDSB];
    char (*const ubuf)[UB] = reinterpret_cast<char (*)[UB]>(lbuf);
    __shared__ float rpart[NW][S];
    __shared__ float tok[3][S];

    TilePlan<XRB, S, NW> dyplan;
    TilePlan<XRB, N, NW> wplan;
    dyplan.init(wave, lane, (uint32_t)(H * XRB), len);
    wplan.init(wave, lane, (uint32_t)XRB, N);
    auto issue = [&](int hh, int u) __attribute__((always_inline)) {
        const int h = hbase + hh;
        const uint32_t ub = lds_addr(lbuf) + (uint32_t)(u * UB);
        dyplan.issue(dy + ((b * L + t0) * H + h) * kP, ub, wave);
        wplan.issue(Wb + ((b * M + c) * H + h) * (int64_t)N * kP, ub + DYT, wave);
    };
    // per-token record of head hh (cs, dt, b_s): thread tid < S takes token
    // tid; loaded early, stored to LDS before the barrier that opens the head
    float rq[3];
    auto load_rec = [&](int hh) __attribute__((always_inline)) {
        const int h = hbase + hh;
        if (tid < S) {
            const float* rc = rec + ((b * H + h) * M + c) * S;
            rq[0] = rc[tid];
            rq[1] = tid < len ? dt[(b * L + t0 + tid) * H + h] : 0.f;
            rq[2] = rc[tid & ~31];
        }
    };
    auto store_rec = [&](int u) __attribute__((always_inline)) {
        if (tid < S) {
            float* r = reinterpret_cast<float*>(&ubuf[u][DYT + WTB]);
            r[tid] = rq[0];
            r[S + tid] = rq[1];
            r[2 * S + tid] = tid < len ? fast_exp2(rq[0] - rq[2]) : 0.f;
        }
    };

    // tiles and pairs of this wave: pair j < nk0 is (tile T0, s block kmin0 + j),
    // pair j >= nk0 is (tile T1, s block kmin1 + j - nk0)
    const int T0 = quad_tile(wave, 0, NW);
    const int T1 = NQ == 2 ? quad_tile(wave, 1, NW) : 0;
    const int kmin0 = T0 >> 1, kmin1 = T1 >> 1;
    const int nk0 = NKB - kmin0;
    const int npw = nk0 + (NQ == 2 ? NKB - kmin1 : 0);

    // the chunk's B and C rows, one copy burst (rows past the end of a
    // partial chunk re-read the last row: finite values, zero weight)
    const uint32_t lb = lds_addr(lbuf);
    {
        TilePlan<BRB, S, NW> bcplan;
        bcplan.init(wave, lane, (uint32_t)(G * BRB), len);
        bcplan.issue(Bm + ((b * L + t0) * G + g) * N, lb, wave);
        bcplan.issue(Cm + ((b * L + t0) * G + g) * N, lb + BCT, wave);
    }
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    lds_barrier();
    // G1 of every pair, kept as bf16
    bf16x8 g1c[NPW];
#pragma unroll
    for (int j = 0; j < NPW; ++j) {
        if (j < npw) {
            const int q = j < nk0 ? 0 : 1;
            const int T = q ? T1 : T0;
            const int K = q ? kmin1 + j - nk0 : kmin0 + j;
            const int t = 16 * T + col;
            f32x4 gg[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
            for (int uu = 0; uu < 2; ++uu) {
                const int s = 32 * K + gram_row(uu, col);
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    gg[uu] = mma16(gg[uu], frag_rowmajor<bf16, BRB>(lbuf + BCT, s, 32 * ks + 8 * grp),
                                   frag_rowmajor<bf16, BRB>(lbuf, t, 32 * ks + 8 * grp));
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                g1c[j][i] = (bf16)gg[0][i];
                g1c[j][4 + i] = (bf16)gg[1][i];
            }
        }
    }
    lds_barrier();  // the B and C tiles are consumed: the head buffers take over
    issue(0, 0);
    load_rec(0);
    store_rec(0);
    KmOffSpread<XRB> ko[4];  // transposing reads of dy^T (k = s) and W^T (k = n), p tile pt
#pragma unroll
    for (int pt = 0; pt < 4; ++pt) ko[pt].init(4 * grp, 16 + 4 * grp, spread_base(pt), lane);

    // x_t fragments of the wave's tiles (each reloaded for the next head once
    // its tile's pairs are done)
    bf16x8 xf[NQ][2];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
        const int t = 16 * (q ? T1 : T0) + col;
        const bf16* xr = x + ((b * L + t0 + (t < len ? t : len - 1)) * H + hbase) * kP + 8 * grp;
        xf[q][0] = load_frag(xr);
        xf[q][1] = load_frag(xr + 32);
    }

    for (int hh = 0; hh < hpb; ++hh) {
        const int u = hh & 1;
        const int h = hbase + hh;
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
        lds_barrier();  // head hh's inputs are in; buffer u ^ 1 is free
        if (hh + 1 < hpb) {
            issue(hh + 1, u ^ 1);
            load_rec(hh + 1);
        }
        // the chunk scan's global inputs, read by wave 0 at the end of the head
        float wq[TPL], kq = 0.f;
        if (wave == 0) {
#pragma unroll
            for (int k = 0; k < TPL; ++k) {
                const int tt = TPL * lane + k;
                wq[k] = tt < len ? wp[(b * L + t0 + tt) * H + h] : 0.f;
            }
            if (lane < nkp) kq = Kp[((b * H + h) * M + c) * nkp + lane];
        }
        const char* dyt = &ubuf[u][0];
        const char* wtl = &ubuf[u][DYT];
        const float* rcs = reinterpret_cast<const float*>(&ubuf[u][DYT + WTB]);
        const float* rdt = rcs + S;
        const float* rbs = rcs + 2 * S;
        for (int i = lane; i < S; i += 64) rpart[wave][i] = 0.f;
        // lane coordinates made opaque per head, so that the per-pair LDS
        // offsets are recomputed in the loop rather than held live across it
        int ln = lane;
        asm volatile("" : "+v"(ln));
        const int grp = ln >> 4, col = ln & 15;
        const float Ah = A[h];
        const float cse = rcs[S - 1];

        // one row tile at a time: its pairs, then its W_c term and outputs
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int T = q ? T1 : T0;
            const int t = 16 * T + col;
            const bool valid = t < len;
            const int tc = valid ? t : len - 1;
            const float cst = rcs[t], dtt = rdt[t];
            bf16x8 bq[KS];  // B_t (k order korder), for the W_c term after the pairs
            const bf16* brow = Bm + ((b * L + t0 + tc) * G + g) * N + 4 * grp;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x4 lo = *reinterpret_cast<const bf16x4*>(brow + 32 * ks);
                const bf16x4 hi = *reinterpret_cast<const bf16x4*>(brow + 32 * ks + 16);
                bq[ks] = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            }
            // x~_t = bf16(dt_t x_t): the Gram B operand, so that r_s (row sums of
            // D = M1 (dy_s . x~_t)) and c_t = x~_t . (sum_s M1[s,t] dy_s) hold the
            // same products
            const bf16x8 xt0 = scale_frag(xf[q][0], dtt), xt1 = scale_frag(xf[q][1], dtt);
            f32x4 acc[4];
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) acc[pt] = f32x4{0.f, 0.f, 0.f, 0.f};
            auto pair = [&](int j, int K) __attribute__((always_inline)) {
                f32x4 g2[2];
#pragma unroll
                for (int uu = 0; uu < 2; ++uu) {
                    const int s = 32 * K + gram_row(uu, col);
                    const bf16x8 a0 = frag_rowmajor<bf16, XRB>(dyt, s, 8 * grp);
                    const bf16x8 a1 = frag_rowmajor<bf16, XRB>(dyt, s, 32 + 8 * grp);
                    g2[uu] = mma16(mma16(f32x4{0.f, 0.f, 0.f, 0.f}, a0, xt0), a1, xt1);
                }
                float f[8];
                const int s0 = 32 * K + 4 * grp, s1 = s0 + 16;  // tokens of elements 0..3, 4..7
                if (K > (T >> 1)) {
                    const float at = fast_exp2(rcs[32 * K] - cst);
                    const f32x4 b0 = *reinterpret_cast<const f32x4*>(rbs + s0);
                    const f32x4 b1 = *reinterpret_cast<const f32x4*>(rbs + s1);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        f[i] = b0[i] * at;
                        f[4 + i] = b1[i] * at;
                    }
                } else {
                    const f32x4 c0 = *reinterpret_cast<const f32x4*>(rcs + s0);
                    const f32x4 c1 = *reinterpret_cast<const f32x4*>(rcs + s1);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        f[i] = (s0 + i >= t && s0 + i < len) ? fast_exp2(c0[i] - cst) : 0.f;
                        f[4 + i] = (s1 + i >= t && s1 + i < len) ? fast_exp2(c1[i] - cst) : 0.f;
                    }
                }
                bf16x8 m1;
                float rv[8];
                // opaque copy: keeps the bf16 -> float conversion of the cached
                // Gram values inside the head loop (hoisted, it would hold 8
                // floats per pair live across heads)
                typedef int i32x4 __attribute__((ext_vector_type(4)));
                i32x4 graw = __builtin_bit_cast(i32x4, g1c[j]);
                asm volatile("" : "+v"(graw));
                const bf16x8 gj = __builtin_bit_cast(bf16x8, graw);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    m1[e] = (bf16)((float)gj[e] * f[e]);
                    rv[e] = (float)m1[e] * (e < 4 ? g2[0][e] : g2[1][e - 4]);
                }
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) acc[pt] = mma16(acc[pt], ko[pt].read(dyt, 32 * K * XRB), m1);
                const float rs = lane_sums8x16_dpp(rv, ln);
                if ((lane & 1) == 0) rpart[wave][32 * K + korder((lane & 15) >> 1, grp)] += rs;
                // keep the scheduler from interleaving pairs (register pressure)
                __builtin_amdgcn_sched_barrier(0);
            };
            if (q == 0) {
#pragma unroll
                for (int j = 0; j < NPW; ++j)
                    if (j < nk0) pair(j, kmin0 + j);
            } else {
#pragma unroll
                for (int j = 0; j < NPW; ++j)
                    if (j >= nk0 && j < npw) pair(j, kmin1 + j - nk0);
            }
            // x . acc for the fragment x (k order 8 g + j, 32 + 8 g + j)
            auto xdot = [&](bf16x8 f0, bf16x8 f1) __attribute__((always_inline)) {
                float d = 0.f;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    d += (float)f0[i] * acc[0][i] + (float)f0[4 + i] * acc[1][i] + (float)f1[i] * acc[2][i] +
                         (float)f1[4 + i] * acc[3][i];
                return row4_sum(d);
            };
            const float cq = xdot(xt0, xt1);  // c_t = dt_t c~_t
            // the W_c term: dx^T += W^T (e^{cs_e - cs_t} B_t)
            const float sB = valid ? fast_exp2(cse - cst) : 0.f;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x8 bfr = scale_frag(bq[ks], sB);
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) acc[pt] = mma16(acc[pt], ko[pt].read(wtl, 32 * ks * XRB), bfr);
            }
            // acc[pt][i] = (B_t Lam_t)[p = spread_base(pt) + 8 grp + i]
            const float cw = xdot(xt0, xt1);
            const float dir = xdot(xf[q][0], xf[q][1]);  // (B_t Lam_t) . x_t
            if (hh + 1 < hpb) {  // this tile's x_t of the next head
                const bf16* xr = x + ((b * L + t0 + tc) * H + h + 1) * kP + 8 * grp;
                xf[q][0] = load_frag(xr);
                xf[q][1] = load_frag(xr + 32);
            }
            if (valid) {
                float* dxr = dx + ((b * L + t0 + t) * H + h) * kP + 8 * grp;
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) {
                    f32x4 v = acc[pt];
#pragma unroll
                    for (int i = 0; i < 4; ++i) v[i] *= dtt;
                    *reinterpret_cast<f32x4*>(dxr + spread_base(pt)) = v;
                }
            }
            if (grp == 0) {
                tok[0][t] = cq;
                tok[1][t] = cw - cq;  // v_t = dt_t v~_t
                tok[2][t] = dir;
            }
        }
        if (hh + 1 < hpb) store_rec(u ^ 1);
        lds_barrier();
        if (wave == 0) {
            // dL/dl_t = sum_{s>=t} (r_s - c_s + w_s) + sum_{s<t} v_s + K_c
            float av[TPL], vv[TPL], asum = 0.f, vsum = 0.f;
#pragma unroll
            for (int k = 0; k < TPL; ++k) {
                const int tt = TPL * lane + k;
                float r = 0.f;
#pragma unroll
                for (int w = 0; w < NW; ++w) r += rpart[w][tt];
                av[k] = r - tok[0][tt] + wq[k];
                vv[k] = tok[1][tt];
                asum += av[k];
                vsum += vv[k];
            }
            float ai = asum, vi = vsum;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const float ta = __shfl_up(ai, o, 64), tv = __shfl_up(vi, o, 64);
                if (lane >= o) {
                    ai += ta;
                    vi += tv;
                }
            }
            const float atot = __shfl(ai, 63, 64);
            float kc = kq;
#pragma unroll
            for (int o = 32; o >= 1; o >>= 1) kc += __shfl_xor(kc, o, 64);
            float suf = atot - (ai - asum);  // sum over s >= first token of this lane
            float pre = vi - vsum;           // sum over s < first token of this lane
            float dA = 0.f;
#pragma unroll
            for (int k = 0; k < TPL; ++k) {
                const int tt = TPL * lane + k;
                const float dl = suf + pre + kc;
                if (tt < len) {
                    ddt[(b * L + t0 + tt) * H + h] = tok[2][tt] + Ah * dl;
                    dA += rdt[tt] * dl;
                }
                suf -= av[k];
                pre += vv[k];
            }
#pragma unroll
            for (int o = 32; o >= 1; o >>= 1) dA += __shfl_xor(dA, o, 64);
            if (lane == 0) dAp[(b * M + c) * H + h] = dA;
        }
    }
}

// ---------------------------------------------------------------------------
// Per (b, c, g, half of the n tiles): Mbar (causal blocks) into LDS, then dB^T[n][t] += C^T Mbar (k = s >= t; A = C^T rows from
// the chunk's C^T, B = Mbar by transposing reads) and dC^T[n][s] += B^T Mbar^T
// (k = t <= s; B = Mbar rows).
// ---------------------------------------------------------------------------
template <int N, int S>
__global__ __launch_bounds__(512) void k_sbwd_bc(const bf16* __restrict__ mbar, const bf16* __restrict__ BT,
                                                 const bf16* __restrict__ CT, float* __restrict__ dB,
                                                 float* __restrict__ dC, int64_t L, int G, int64_t M) {
    constexpr int NW = 8, NT = 512;
    constexpr int RB = 2 * S;
    constexpr int NKB = S / 32;
    constexpr int NTILE = S / 16, NNT = N / 16;
    __shared__ __attribute__((aligned(16))) char mt[S * RB];
    const int64_t bcg = blockIdx.x >> 1;
    const int nhalf = blockIdx.x & 1;  // n tiles [nhalf NNT/2, (nhalf + 1) NNT/2)
    const int g = (int)(bcg % G);
    const int64_t bc = bcg / G;
    const int64_t b = bc / M, c = bc % M;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = tid >> 6;
    const int grp = lane >> 4, col = lane & 15;
    const int64_t t0 = c * S;
    const int len = (int)(L - t0 < S ? L - t0 : S);

    const bf16* mi = mbar + bcg * (int64_t)S * S;
    for (int it = tid; it < S * (S / 8); it += NT) {
        const int s = it / (S / 8), t8 = it % (S / 8);
        if (8 * t8 >= 32 * (s / 32 + 1)) continue;  // above the causal blocks
        *reinterpret_cast<bf16x8*>(mt + SwzTile<RB>::off(s, 16 * t8)) =
            *reinterpret_cast<const bf16x8*>(mi + (int64_t)s * S + 8 * t8);
    }
    __syncthreads();

    const bf16* bt = BT + bcg * (int64_t)N * S;
    const bf16* ct = CT + bcg * (int64_t)N * S;
    KmOffBf16<RB> mo;
    constexpr int NNH = NNT / 2;  // n tiles of this workgroup
    for (int tileid = wave; tileid < NTILE * NNH * 2; tileid += NW) {
        const bool isB = tileid < NTILE * NNH;
        const int id = isB ? tileid : tileid - NTILE * NNH;
        const int T = id / NNH, nt = nhalf * NNH + id % NNH;
        const int tk = 16 * T + col;  // token of this lane's column
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
        // every A fragment of the tile is requested before the first product
        bf16x8 av[NKB];
        if (isB) {
            // dB^T[n][t] = sum_{s >= t} C^T[n][s] Mbar[s][t], k order korder
            // (conflict-free transposing reads of Mbar)
            mo.init(4 * grp, 16 + 4 * grp, 16 * T, lane);
            const bf16* arow = ct + (int64_t)(16 * nt + col) * S + 4 * grp;
#pragma unroll
            for (int K = 0; K < NKB; ++K) {
                if (K >= (T >> 1)) {
                    const bf16x4 lo = *reinterpret_cast<const bf16x4*>(arow + 32 * K);
                    const bf16x4 hi = *reinterpret_cast<const bf16x4*>(arow + 32 * K + 16);
                    av[K] = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                }
            }
#pragma unroll
            for (int K = 0; K < NKB; ++K)
                if (K >= (T >> 1)) acc = mma16(acc, av[K], mo.read(mt, 32 * K * RB));
        } else {
            // dC^T[n][s] = sum_{t <= s} B^T[n][t] Mbar[s][t]
            const bf16* arow = bt + (int64_t)(16 * nt + col) * S + 8 * grp;
#pragma unroll
            for (int K = 0; K < NKB; ++K)
                if (K <= (T >> 1)) av[K] = load_frag(arow + 32 * K);
#pragma unroll
            for (int K = 0; K < NKB; ++K)
                if (K <= (T >> 1))
                    acc = mma16(acc, av[K], frag_rowmajor<bf16, RB>(mt, tk, 32 * K + 8 * grp));
        }
        if (tk < len) {
            float* dst = (isB ? dB : dC) + ((b * L + t0 + tk) * G + g) * N + 16 * nt + 4 * grp;
            f32x4 v = *reinterpret_cast<const f32x4*>(dst);
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] += acc[i];
            *reinterpret_cast<f32x4*>(dst) = v;
        }
    }
}

// one block per head: a fixed-order tree sum over (b, c)
__global__ __launch_bounds__(256) void k_sbwd_dA(const float* __restrict__ dAp, float* __restrict__ dA,
                                                 int64_t BM, int H) {
    __shared__ float red[4];
    const int h = blockIdx.x, tid = threadIdx.x;
    float s = 0.f;
    for (int64_t k = tid; k < BM; k += 256) s += dAp[k * H + h];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
    if ((tid & 63) == 0) red[tid >> 6] = s;
    __syncthreads();
    if (tid == 0) dA[h] = (red[0] + red[1]) + (red[2] + red[3]);
}

// heads per workgroup of the contraction and quadratic kernels
int mfma_hpb(const Shape& s) {
    const int hpg = s.H / s.G;
    for (int c = 8; c > 1; --c)
        if (hpg % c == 0) return c;
    return 1;
}

struct MfmaWs {
    float* rec;   // [B][H][M][S] cs (log2)
    float* lda;   // [B][H][M]
    bf16* dH;     // [B][M][H][N][P]
    bf16* dR;
    bf16* BT;     // [B][M][G][N][S]
    bf16* CT;
    bf16* Hb;     // [B][M][H][N][P]
    bf16* Wb;
    float* Kp;    // [B][H][M][nkp]
    float* wp;    // [B][L][H]
    float* dAp;   // [B][M][H]
    bf16* mbar;   // [B][M][G][S][S]
    int nkp;
    size_t total;
};

MfmaWs mfma_layout(const Shape& s, void* base) {
    const size_t NP = (size_t)s.N * s.P;
    const size_t BHM = (size_t)s.B * s.H * s.M;
    const size_t BMG = (size_t)s.B * s.M * s.G;
    MfmaWs w;
    w.nkp = (int)((NP + 1023) / 1024);
    size_t o = 0;
    char* p = reinterpret_cast<char*>(base);
    auto take = [&](size_t bytes) {
        char* r = p ? p + o : nullptr;
        o += align256(bytes);
        return r;
    };
    w.rec = (float*)take(4 * BHM * s.S);
    w.lda = (float*)take(4 * BHM);
    w.dH = (bf16*)take(2 * BHM * NP);
    w.dR = (bf16*)take(2 * BHM * NP);
    w.BT = (bf16*)take(2 * BMG * s.N * s.S);
    w.CT = (bf16*)take(2 * BMG * s.N * s.S);
    w.Hb = (bf16*)take(2 * BHM * NP);
    w.Wb = (bf16*)take(2 * BHM * NP);
    w.Kp = (float*)take(4 * BHM * w.nkp);
    w.wp = (float*)take(4 * (size_t)s.B * s.L * s.H);
    w.dAp = (float*)take(4 * BHM);
    w.mbar = (bf16*)take(2 * BMG * (size_t)s.S * s.S);
    w.total = o;
    return w;
}

template <int N, int S>
hipError_t run_mfma(const Shape& s, const bf16* x, const float* dt, const float* A, const bf16* Bm,
                    const bf16* Cm, const float* h0, const bf16* dy, const float* dmem, const float* dhl,
                    float* dx, float* ddt, float* dA, float* dB, float* dC, float* dh0, void* ws,
                    hipStream_t st) {
    const MfmaWs w = mfma_layout(s, ws);
    const int hpb = mfma_hpb(s);
    const int64_t nbcg = s.B * s.M * s.G;
    const int nhs = (s.H / s.G) / hpb;
    const unsigned grid = (unsigned)(nbcg * nhs);
    prof_begin("k_sbwd_contract", st);
    k_sbwd_contract<N, S, 0><<<grid, 512, 0, st>>>(Bm, x, dt, A, w.dH, w.rec, w.lda, w.BT, s.L, s.H, s.G, s.M,
                                                   hpb, nbcg);
    k_sbwd_contract<N, S, 1><<<grid, 512, 0, st>>>(Cm, dy, dt, A, w.dR, nullptr, nullptr, w.CT, s.L, s.H, s.G,
                                                   s.M, hpb, nbcg);
    prof_end(st);
    const int NP = s.N * s.P;
    prof_begin("k_sbwd_pass2", st);
    k_sbwd_pass2<<<dim3((unsigned)w.nkp, (unsigned)s.H, (unsigned)s.B), 256, 0, st>>>(
        w.dH, w.dR, w.lda, h0, dmem, dhl, w.Hb, w.Wb, w.Kp, dh0, s.H, NP, s.M, s.Mcap);
    prof_end(st);
    prof_begin("k_sbwd_group", st);
    k_sbwd_group<N, S><<<(unsigned)(nbcg * (S / 64)), 512, 0, st>>>(x, dt, Cm, dy, w.rec, w.Hb, w.Wb, dB, dC,
                                                                    w.wp, w.mbar, s.L, s.H, s.G, s.M, nbcg);
    prof_end(st);
    prof_begin("k_sbwd_quad", st);
    k_sbwd_quad<N, S><<<grid, 64 * quad_waves<S>(), 0, st>>>(x, dt, A, Bm, Cm, dy, w.rec, w.Wb, w.Kp, w.wp, dx,
                                                             ddt, w.dAp, s.L, s.H, s.G, s.M, hpb, nbcg, w.nkp);
    prof_end(st);
    prof_begin("k_sbwd_bc", st);
    k_sbwd_bc<N, S><<<(unsigned)(2 * nbcg), 512, 0, st>>>(w.mbar, w.BT, w.CT, dB, dC, s.L, s.G, s.M);
    prof_end(st);
    prof_begin("k_sbwd_dA", st);
    k_sbwd_dA<<<(unsigned)s.H, 256, 0, st>>>(w.dAp, dA, s.B * s.M, s.H);
    prof_end(st);
    return hipGetLastError();
}

template <int N>
hipError_t run_mfma_s(const Shape& s, const bf16* x, const float* dt, const float* A, const bf16* Bm,
                      const bf16* Cm, const float* h0, const bf16* dy, const float* dmem, const float* dhl,
                      float* dx, float* ddt, float* dA, float* dB, float* dC, float* dh0, void* ws,
                      hipStream_t st) {
    switch (s.S) {
        case 64: return run_mfma<N, 64>(s, x, dt, A, Bm, Cm, h0, dy, dmem, dhl, dx, ddt, dA, dB, dC, dh0, ws, st);
        case 128: return run_mfma<N, 128>(s, x, dt, A, Bm, Cm, h0, dy, dmem, dhl, dx, ddt, dA, dB, dC, dh0, ws, st);
        case 256: return run_mfma<N, 256>(s, x, dt, A, Bm, Cm, h0, dy, dmem, dhl, dx, ddt, dA, dB, dC, dh0, ws, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace

bool sbwd_mfma_shape(const Shape& s) { return s.dtype == 1 && s.P == kP && tuned_shape(s); }

size_t sbwd_mfma_workspace_bytes(const Shape& s) { return mfma_layout(s, nullptr).total; }

hipError_t launch_ssd_bwd_mfma(const Shape& s, const void* x, const float* dt, const float* A,
                               const void* Bm, const void* Cm, const float* h0, const void* dy,
                               const float* dmem, const float* dh_last, float* dx, float* ddt, float* dA,
                               float* dB, float* dC, float* dh0, void* ws, hipStream_t st) {
    const bf16 *xb = (const bf16*)x, *bb = (const bf16*)Bm, *cb = (const bf16*)Cm, *yb = (const bf16*)dy;
    switch (s.N) {
        case 32: return run_mfma_s<32>(s, xb, dt, A, bb, cb, h0, yb, dmem, dh_last, dx, ddt, dA, dB, dC, dh0, ws, st);
        case 64: return run_mfma_s<64>(s, xb, dt, A, bb, cb, h0, yb, dmem, dh_last, dx, ddt, dA, dB, dC, dh0, ws, st);
        case 128: return run_mfma_s<128>(s, xb, dt, A, bb, cb, h0, yb, dmem, dh_last, dx, ddt, dA, dB, dC, dh0, ws, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace dart
