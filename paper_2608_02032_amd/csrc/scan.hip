// scan.hip -- Mamba-2 chunked SSD scan that retains the chunk state memories.
//
// Paper: Sec. 2 (SSD recurrence H_t = a_t H_{t-1} + B_t^T X_t, Y_t = C_t H_t
// and its dual masked-attention form), Sec. 3 (chunk state memory dH_[c]) and
// App. A (chunk decomposition: H_[c] = A_{a_c:b_c} H_[c-1] + dH_[c];
// Y = Y_intra + Y_inter; block form Y_[c] = C<-_[c] H_[c-1] + L_[c] X_[c]).
// Discretisation: a_t = exp(dt_t A_h), input dt_t B_t^T x_t.
//
// Four kernels, one stream:
//   k_chunk_state  per (b, chunk, head): within-chunk cumulative log decay
//                  cs (kept in the workspace, log2 units, for k_chunk_out),
//                  then dH = B^T diag(exp(cs_e - cs_s) dt_s) X on MFMA (B and X
//                  staged through LDS), written to `mem`; the chunk's total log
//                  decay cs_e goes to the workspace.
//   k_chunk_gram   per (b, chunk, group, 4 row tiles): the causal part of the
//                  chunk's Gram matrix G^T = B C^T (it depends on the group,
//                  not the head, so it is formed once for all heads of a
//                  group), stored in the MFMA accumulator layout that
//                  k_chunk_out consumes as its A operand.
//   k_state_pass   per (b, head, element block): sequential over chunks,
//                  H_[c] = exp(cs_e(c)) H_[c-1] + dH_[c]; stores the state
//                  entering every chunk (workspace) and h_last.
//   k_chunk_out    per (b, chunk, head): y = (L o G)(dt X) + (C o e^{cs}) H_[c-1]
//                  on MFMA: the Gram tiles are read straight into registers,
//                  masked and decayed there, and multiplied with X (staged
//                  through LDS).
// Decays are always exponentiated as differences cs_t - cs_s <= 0 (no
// overflow; underflow to 0 is the correct limit).
#include "dart_common.hpp"
#include "dart_internal.hpp"

#include <type_traits>

namespace dart {
namespace {

constexpr int kP = 64;        // head dim
constexpr int kThreads = 256; // 4 waves

// Inclusive prefix sum over the block (thread order).  All threads call it.
__device__ float block_inclusive_scan(float v, float* sred) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const float t = __shfl_up(v, o, 64);
        if (lane >= o) v += t;
    }
    if (lane == 63) sred[wave] = v;
    __syncthreads();
    float add = 0.f;
    for (int w = 0; w < wave; ++w) add += sred[w];
    __syncthreads();
    return v + add;
}

// ---------------------------------------------------------------------------
// Chunk-state contraction: dH_[c] = sum_s exp(cs_e - cs_s) dt_s B_s^T x_s.
// B_c and x_c stream through LDS in 32-token blocks by DMA into a four-stage
// ring, three blocks ahead of the MFMAs that consume them; both MFMA operands
// are read k-major with transpose loads.  Wave w owns p-tile w and all
// n-tiles of the N x P result.  The copies are issued untracked (the compiler
// cannot tell the stage being read from those being filled and would drain
// every copy before each read); each wave waits for its own copies of a stage
// before the barrier that opens it (vector memory operations complete in
// order).
// ---------------------------------------------------------------------------
constexpr int kSB = 32;       // tokens per LDS-staged s block
constexpr int kStages = 4;    // ring stages (kStages - 1 blocks in flight)

// 4-byte global -> LDS copy by DMA (global_load_lds_dword), untracked like
// lds_dma16_untracked: lane i's 4 bytes land at lds_wave_base + 4 i.
__device__ __forceinline__ void lds_dma4_untracked(const void* gsrc, void* lds_wave_base) {
    const uint32_t m0 = (uint32_t)__builtin_amdgcn_readfirstlane(
        (int)(uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)lds_wave_base);
    uint32_t save;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dword %1, off\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(save)
        : "v"(gsrc), "s"(m0)
        : "memory");
}
// s_waitcnt vmcnt(n) for a wave-uniform n in [0, 15].
__device__ __forceinline__ void wait_vm_upto(int n) {
    switch (n) {
#define DART_VMC(k) case k: __builtin_amdgcn_s_waitcnt(vmcnt_imm(k)); break;
        DART_VMC(1) DART_VMC(2) DART_VMC(3) DART_VMC(4) DART_VMC(5) DART_VMC(6) DART_VMC(7)
        DART_VMC(8) DART_VMC(9) DART_VMC(10) DART_VMC(11) DART_VMC(12) DART_VMC(13) DART_VMC(14)
        DART_VMC(15)
#undef DART_VMC
        default: __builtin_amdgcn_s_waitcnt(vmcnt_imm(0)); break;
    }
}
// 1 KiB copies that dma_tile issues from wave w of 4 for a tile of `pieces`
// 16-byte pieces.
__device__ __forceinline__ int dma_copies(int pieces, int w) {
    return pieces > 64 * w ? (pieces - 64 * w + 255) / 256 : 0;
}

template <typename T, int N, int S>
__global__ __launch_bounds__(kThreads) void k_chunk_state(
    const T* __restrict__ x, const float* __restrict__ dt, const float* __restrict__ A,
    const T* __restrict__ Bm, T* __restrict__ mem, float* __restrict__ chunk_lda,
    float* __restrict__ aux, int64_t L, int H, int G, int64_t M, int64_t Mcap) {
    constexpr int XRB = kP * (int)sizeof(T);   // bytes per x row
    constexpr int BRB = N * (int)sizeof(T);    // bytes per B row
    constexpr int XT = kSB * XRB, BT = kSB * BRB;
    constexpr int STB = XT + BT;               // bytes of one ring stage
    constexpr int OUTB = 4 * N * 16 * (int)sizeof(T);  // output strips (reuse the ring)
    constexpr int RINGB = kStages * STB > OUTB ? kStages * STB : OUTB;
    static_assert(S <= kThreads, "one thread per token of the chunk");
    const int c = blockIdx.x, h = blockIdx.y;
    const int64_t b = blockIdx.z;
    const int g = (int)((int64_t)h * G / H);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int grp = lane >> 4;
    const int64_t t0 = (int64_t)c * S;
    const int len = (int)(L - t0 < S ? L - t0 : S);
    const int nsb = (len + kSB - 1) / kSB;

    __shared__ float s_dt[S];
    __shared__ float s_w[S];
    __shared__ float s_red[4];
    __shared__ float s_cse;
    __shared__ __attribute__((aligned(16))) char ring[RINGB];

    // copies: the chunk's dt (with block 0), then the x and B rows of each
    // s block into its ring stage; rows past the end re-read the last row
    // (their weights are zero), blocks past the end are not copied
    if (tid < S) {
        const int tok = tid < len ? tid : len - 1;
        lds_dma4_untracked(dt + (b * L + t0 + tok) * H + h, s_dt + wave * 64);
    }
    const char* xg = reinterpret_cast<const char*>(x + ((b * L + t0) * H + h) * kP);
    const char* bg = reinterpret_cast<const char*>(Bm + ((b * L + t0) * G + g) * N);
    const int64_t xstride = (int64_t)H * XRB, bstride = (int64_t)G * BRB;
    auto stage = [&](int sb) {
        if (sb >= nsb) return;
        char* st = ring + (sb % kStages) * STB;
        const int rv = len - sb * kSB;
        dma_tile<XRB, true>(st, xg + sb * kSB * xstride, xstride, kSB, rv, wave, 4, lane);
        dma_tile<BRB, true>(st + XT, bg + sb * kSB * bstride, bstride, kSB, rv, wave, 4, lane);
    };
    // this wave's copies per s block
    const int cpw = dma_copies(XT / 16, wave) + dma_copies(BT / 16, wave);
    // wait until this wave's copies of block sb are complete: the copies of
    // the (at most kStages - 2) later blocks may still be in flight
    auto wait_block = [&](int sb) {
        const int later = (nsb - 1 - sb) < (kStages - 2) ? (nsb - 1 - sb) : (kStages - 2);
        wait_vm_upto(later * cpw);
    };
#pragma unroll
    for (int sb = 0; sb < kStages - 1; ++sb) stage(sb);

    // block 0 and dt are in: cumulative log decay within the chunk (tokens
    // past L contribute 0) and the weights exp(cs_e - cs_s) dt_s
    wait_block(0);
    __syncthreads();
    const float dts = (tid < len) ? s_dt[tid] : 0.f;
    const float cs = block_inclusive_scan(tid < S ? dts * A[h] : 0.f, s_red);
    if (tid == S - 1) s_cse = cs;
    __syncthreads();
    const float cse = s_cse;
    if (tid < S) s_w[tid] = (tid < len) ? __expf(cse - cs) * dts : 0.f;

    f32x4 acc[N / 16];
#pragma unroll
    for (int nt = 0; nt < N / 16; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    // one s block: x operand (k = s, column p) scaled by w_s, then the B
    // operand of every n tile; bf16 reads use offsets fixed here
    KmOffBf16<XRB> xo;
    KmOffBf16<BRB> bo[N / 16];
    if constexpr (sizeof(T) == 2) {
        xo.init(8 * grp, 8 * grp + 4, wave * 16, lane);
#pragma unroll
        for (int nt = 0; nt < N / 16; ++nt) bo[nt].init(8 * grp, 8 * grp + 4, nt * 16, lane);
    }
    auto consume = [&](int sb, int u) __attribute__((always_inline)) {
        const char* xt = ring + u * STB;
        const char* bt = xt + XT;
        Frag<T> fx;
        if constexpr (sizeof(T) == 2) {
            fx = xo.read(ring, u * STB);
        } else {
            fx = frag_km<T, XRB>(xt, 8 * grp, 8 * grp + 4, wave * 16, lane);
        }
        float xv[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) xv[i] = to_f(fx[i]) * s_w[sb * kSB + 8 * grp + i];
        fx = make_frag<T>(xv);
#pragma unroll
        for (int nt = 0; nt < N / 16; ++nt) {
            Frag<T> fb;
            if constexpr (sizeof(T) == 2) {
                fb = bo[nt].read(ring, u * STB + XT);
            } else {
                fb = frag_km<T, BRB>(bt, 8 * grp, 8 * grp + 4, nt * 16, lane);
            }
            acc[nt] = mma16(acc[nt], fb, fx);
        }
    };
    // the loop is unrolled over the ring so every stage offset is an immediate
    for (int sb0 = 0; sb0 < nsb; sb0 += kStages) {
#pragma unroll
        for (int u = 0; u < kStages; ++u) {
            const int sb = sb0 + u;
            if (sb >= nsb) break;
            if (sb > 0) wait_block(sb);
            lds_barrier();   // block sb (and s_w) are in; every wave is done with block sb - 1
            stage(sb + kStages - 1);
            consume(sb, u);
        }
    }
    // outputs: the chunk's per-token record for the output kernel (cumulative
    // log decay cs in log2 units, dt (0 past the end), and the weight
    // exp2(cs_e - cs_s) dt_s with e the last token of the s's 32-token block),
    // the chunk's total log decay, and dH: acc[nt][i] = dH[n = 16 nt +
    // 4 (lane/16) + i][p = 16 wave + lane%16], each wave's N x 16 strip through
    // LDS (the ring) and out as 16-byte row stores
    {
        const float cs2 = cs * kLog2e;
        const float cse2 = __shfl(cs2, lane | 31);
        if (tid < S) {
            float* rec = aux + ((b * H + h) * M + c) * 3 * S;
            rec[tid] = cs2;
            rec[S + tid] = dts;
            rec[2 * S + tid] = fast_exp2(cse2 - cs2) * dts;
        }
    }
    if (tid == 0) chunk_lda[(b * H + h) * M + c] = cse;
    __syncthreads();
    T* st = reinterpret_cast<T*>(ring) + wave * N * 16;
#pragma unroll
    for (int nt = 0; nt < N / 16; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) st[(nt * 16 + 4 * grp + i) * 16 + (lane & 15)] = from_f<T>(acc[nt][i]);
    T* dst = mem + ((b * Mcap + c) * H + h) * (int64_t)N * kP + wave * 16;
    for (int e8 = lane; e8 < N * 2; e8 += 64) {
        const int n = e8 >> 1, half = e8 & 1;
        float v[8];
        load8(st + n * 16 + half * 8, v);
        store8(dst + n * kP + half * 8, v);
    }
}

// ---------------------------------------------------------------------------
// Chunk-state contraction for bf16, one workgroup per (b, chunk, group, slice
// of hpb heads of the group): the chunk's B rows depend on the group only, so
// each wave reads its B^T operand fragments once (staged through LDS) and
// keeps them in registers for every head of the slice.  The prologue also
// copies the dt of every head of the slice and forms all their within-chunk
// decays at once (wave w takes heads w, w + 8, ...; a wave-level scan of dt A):
// the contraction weights exp(cs_e - cs_s) dt_s stay in LDS (over the B rows,
// no longer needed), the per-token record and the total log decay go to the
// workspace.  Per head, the x rows arrive by DMA in one of two buffers while
// the previous head computes.  Wave w owns n tiles NTW (w % 2) .. of p tile
// w / 2 of the N x P result (so two waves weight each x fragment, by the
// weights of its tokens, before the MFMAs); the products are formed
// transposed, a lane holding dH[n][p .. p + 3], and leave as 8-byte stores.
// ---------------------------------------------------------------------------
template <int N, int S>
__global__ __launch_bounds__(512) void k_chunk_state_heads(
    const bf16* __restrict__ x, const float* __restrict__ dt, const float* __restrict__ A,
    const bf16* __restrict__ Bm, bf16* __restrict__ mem, float* __restrict__ chunk_lda,
    float* __restrict__ aux, int64_t L, int H, int G, int64_t M, int64_t Mcap, int hpb,
    int64_t nbcg) {
    using T = bf16;
    constexpr int NW = 8;
    constexpr int XRB = kP * 2;                 // bytes per x row
    constexpr int BRB = N * 2;                  // bytes per B row
    constexpr int XT = S * XRB, BT = S * BRB;
    constexpr int KST = S / 32;                 // 32-token k steps
    constexpr int NTW = N / 32;                 // n tiles per wave
    constexpr int DHS = acc_row_stores<NTW>();  // dH stores per wave and head
    constexpr int NG = 2;                       // n-tile groups
    static_assert(NG * NTW * 16 == N && NG * 4 == NW, "tiles cover the waves");
    constexpr int TPL = S / 64;                 // tokens per lane in a decay scan
    constexpr int LPB = 32 / TPL;               // lanes per 32-token block

    const int nhs = (H / G) / hpb;
    const int64_t bid = blockIdx.x;
    int64_t bcg;
    int hs;
    if (nbcg % 8 == 0) {
        const int64_t slot = bid >> 3;
        bcg = (slot / nhs) * 8 + (bid & 7);
        hs = (int)(slot % nhs);
    } else {
        bcg = bid / nhs;
        hs = (int)(bid % nhs);
    }
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

    // bt: the B rows, then (after the fragments are read) the weights of
    // every head [hpb][S] fp32; xbuf[1] holds the heads' dt until the first
    // head loop copy
    __shared__ __attribute__((aligned(16))) char bt[BT];
    __shared__ __attribute__((aligned(16))) char xbuf[2][XT];
    float* const wall = reinterpret_cast<float*>(bt);
    const float* const dtall = reinterpret_cast<const float*>(&xbuf[1][0]);
    const uint32_t bt_lds = lds_addr(bt), x_lds = lds_addr(xbuf);

    // copies into swizzled row tiles (rows past the end re-read the last row)
    TilePlan<XRB, S, NW> xplan;
    xplan.init(wave, lane, (uint32_t)(H * XRB), len);
    auto issue_x = [&](int hh, int u) __attribute__((always_inline)) {
        xplan.issue(x + ((b * L + t0) * H + hbase + hh) * kP, x_lds + (uint32_t)(u * XT), wave);
    };

    // prologue copies: B rows, head 0's x rows, every head's dt (one 4-byte
    // copy per token; head hd by wave hd % 8)
    {
        TilePlan<BRB, S, NW> bplan;
        bplan.init(wave, lane, (uint32_t)(G * BRB), len);
        bplan.issue(Bm + ((b * L + t0) * G + g) * N, bt_lds, wave);
    }
    issue_x(0, 0);
    for (int hd = wave; hd < hpb; hd += NW) {
#pragma unroll
        for (int k = 0; k < TPL; ++k) {
            const int tok = k * 64 + lane;
            const int tc = tok < len ? tok : len - 1;
            const uint32_t m0 = x_lds + (uint32_t)(XT + (hd * S + k * 64) * 4);
            const float* src = dt + (b * L + t0 + tc) * H + hbase + hd;
            uint32_t save;
            asm volatile(
                "s_mov_b32 %0, m0\n\t"
                "s_mov_b32 m0, %2\n\t"
                "s_nop 0\n\t"
                "global_load_lds_dword %1, off\n\t"
                "s_mov_b32 m0, %0"
                : "=&s"(save)
                : "v"(src), "s"((uint32_t)__builtin_amdgcn_readfirstlane((int)m0))
                : "memory");
        }
    }
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    lds_barrier();
    bf16x8 bfr[NTW][KST];
    {
        KmOffBf16<BRB> bo;
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
            bo.init(4 * grp, 16 + 4 * grp, (ng * NTW + j) * 16, lane);
#pragma unroll
            for (int ks = 0; ks < KST; ++ks) bfr[j][ks] = bo.read(bt, ks * 32 * BRB);
        }
    }
    lds_barrier();  // every wave holds its B^T fragments: bt takes the weights
    // decays of head hd, lane l holding tokens TPL l .. TPL l + TPL - 1
    for (int hd = wave; hd < hpb; hd += NW) {
        const int h = hbase + hd;
        const float a = A[h];
        float dv[TPL], cs[TPL];
        float run = 0.f;
#pragma unroll
        for (int k = 0; k < TPL; ++k) {
            const int tok = TPL * lane + k;
            dv[k] = tok < len ? dtall[hd * S + tok] : 0.f;
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
        const float cse = __shfl(cs[TPL - 1], 63, 64);                // chunk end
        const float cbe = __shfl(cs[TPL - 1], lane | (LPB - 1), 64);  // 32-token block end
        float* rec = aux + ((b * H + h) * M + c) * 3 * S;
#pragma unroll
        for (int k = 0; k < TPL; ++k) {
            const float cs2 = cs[k] * kLog2e;
            wall[hd * S + TPL * lane + k] = __expf(cse - cs[k]) * dv[k];
            rec[TPL * lane + k] = cs2;
            rec[S + TPL * lane + k] = dv[k];
            rec[2 * S + TPL * lane + k] = fast_exp2(cbe * kLog2e - cs2) * dv[k];
        }
        if (lane == 0) chunk_lda[(b * H + h) * M + c] = cse;
    }
    KmOffBf16<XRB> xo;
    xo.init(4 * grp, 16 + 4 * grp, pg * 16, lane);

    for (int hh = 0; hh < hpb; ++hh) {
        const int u = hh & 1;
        // this wave's copies of head hh are in: only its dH stores of head
        // hh - 1 (DHS) came after them (head 0's were waited for in the prologue)
        if (hh > 0) __builtin_amdgcn_s_waitcnt(vmcnt_imm(DHS));
        lds_barrier();  // copies of head hh and all weights visible; buffer u ^ 1 is free
        if (hh + 1 < hpb) issue_x(hh + 1, u ^ 1);
        const float* wv = wall + hh * S;
        f32x4 acc[NTW];
#pragma unroll
        for (int j = 0; j < NTW; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KST; ++ks) {
            const f32x4 w0 = *reinterpret_cast<const f32x4*>(wv + ks * 32 + 4 * grp);
            const f32x4 w1 = *reinterpret_cast<const f32x4*>(wv + ks * 32 + 16 + 4 * grp);
            const bf16x8 xr = xo.read(&xbuf[u][0], ks * 32 * XRB);
            float v[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[i] = to_f(xr[i]) * w0[i];
                v[4 + i] = to_f(xr[4 + i]) * w1[i];
            }
            const bf16x8 xf = make_frag<T>(v);
#pragma unroll
            for (int j = 0; j < NTW; ++j) acc[j] = mma16(acc[j], xf, bfr[j][ks]);
        }
        // acc[j][i] = dH[n = 16 (ng NTW + j) + col][p = 16 pg + 4 grp + i]
        store_acc_rows_bf16<NTW>(mem + ((b * Mcap + c) * H + hbase + hh) * (int64_t)N * kP + 16 * pg,
                                 kP, 16 * ng * NTW, acc, grp, col);
    }
}

// ---------------------------------------------------------------------------
// Inter-chunk state passing: H_[c] = exp(cs_e(c)) H_[c-1] + dH_[c].
// states[b][c][h] receives the state entering chunk c (H_[c-1]; h0 for c=0).
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kThreads) void k_state_pass(
    const T* __restrict__ mem, const float* __restrict__ chunk_lda, const float* __restrict__ h0,
    T* __restrict__ states, float* __restrict__ h_last, int H, int NP, int64_t M, int64_t Mcap) {
    const int h = blockIdx.y;
    const int64_t b = blockIdx.z;
    const int e0 = (blockIdx.x * kThreads + threadIdx.x) * 4;
    if (e0 >= NP) return;
    float hc[4] = {0.f, 0.f, 0.f, 0.f};
    if (h0) load4(h0 + (b * H + h) * (int64_t)NP + e0, hc);
    const float* lda = chunk_lda + (b * H + h) * M;
#pragma unroll 4
    for (int64_t c = 0; c < M; ++c) {
        store4(states + ((b * M + c) * H + h) * (int64_t)NP + e0, hc);
        float dh[4];
        load4(mem + ((b * Mcap + c) * H + h) * (int64_t)NP + e0, dh);
        const float a = __expf(lda[c]);
#pragma unroll
        for (int i = 0; i < 4; ++i) hc[i] = a * hc[i] + dh[i];
    }
    if (h_last) store4(h_last + (b * H + h) * (int64_t)NP + e0, hc);
}

// ---------------------------------------------------------------------------
// Causal Gram tiles.  Row tile r (tokens t in [16r, 16r+16)) meets the 32-token
// s blocks sk = 0..r/2; pair (r, sk) holds G^T[s][t] = B_s . C_t for
// s = 32 sk + 16u + 4 (lane/16) + i, t = 16 r + lane%16 as 8 floats per lane
// (u, i), which is the accumulator layout of the MFMA below and the A-operand
// layout k_chunk_out wants (any consistent k order is valid).
// ---------------------------------------------------------------------------
__host__ __device__ constexpr int gram_pairs(int S) { return (S / 32) * (S / 32 + 1); }
__device__ __forceinline__ int gram_pair(int r, int sk) {
    const int m = r >> 1;
    return ((r & 1) ? (m + 1) * (m + 1) : m * (m + 1)) + sk;
}

template <typename T, int N, int S>
__global__ __launch_bounds__(kThreads) void k_chunk_gram(const T* __restrict__ Bm,
                                                         const T* __restrict__ Cm,
                                                         float* __restrict__ gram, int64_t L,
                                                         int G, int64_t M) {
    constexpr int KS = N / 32;
    const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int64_t c = blockIdx.y;
    const int64_t bg = blockIdx.z;  // b * G + g
    const int64_t b = bg / G;
    const int g = (int)(bg % G);
    const int lane = threadIdx.x & 63, col = lane & 15, grp = lane >> 4;
    const int64_t t0 = c * S;
    const int len = (int)(L - t0 < S ? L - t0 : S);
    // rows past the end of a partial chunk read the last row (finite values;
    // k_chunk_out gives them zero weight)
    auto row = [&](const T* base, int t) {
        const int tc = t < len ? t : len - 1;
        return base + ((b * L + t0 + tc) * G + g) * N;
    };
    Frag<T> cf[KS];
    const T* crow = row(Cm, r * 16 + col);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) cf[ks] = load_frag(crow + ks * 32 + grp * 8);
    float* out = gram + (bg * M + c) * (int64_t)gram_pairs(S) * 512;
    for (int sk = 0; sk <= (r >> 1); ++sk) {
        f32x4 gacc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const T* brow = row(Bm, sk * 32 + u * 16 + col);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) gacc[u] = mma16(gacc[u], load_frag(brow + ks * 32 + grp * 8), cf[ks]);
        }
        f32x4* dst = reinterpret_cast<f32x4*>(out + ((int64_t)gram_pair(r, sk) * 64 + lane) * 8);
        dst[0] = gacc[0];
        dst[1] = gacc[1];
    }
}

// ---------------------------------------------------------------------------
// Chunk output: y_t = sum_{s<=t} G_ts exp(cs_t - cs_s) dt_s x_s
//                     + exp(cs_t) C_t H_[c-1].
// NW waves (8 for S >= 128); wave w owns the 16-row tiles tile_row(w, q): w,
// then 2 NW - 1 - w, ... (a light and a heavy tile of the causal triangle,
// so every wave has about the same number of causal pairs).  H_[c-1]
// and the chunk's x rows are DMA-staged in natural layout; C rows (for the
// inter-chunk term) and the Gram tiles go straight to registers.
// The intra-chunk term runs over the causal (row tile r, 32-token s block sk)
// pairs only.  For sk < r/2 every s precedes every t, and with e = 32 sk + 31
// the decay factors as exp2(cs_t - cs_e) exp2(cs_e - cs_s), both <= 1: the
// per-token factor b_s = exp2(cs_e - cs_s) dt_s is formed once per block and
// each lane's row factor exp2(cs_t - cs_e) once per pair.  The diagonal pair
// sk = r/2 applies the causal mask and the exact per-element decay.
// ---------------------------------------------------------------------------
template <int S> constexpr int out_waves() { return S / 16 >= 8 ? 8 : S / 16; }
__device__ __forceinline__ int tile_row(int w, int q, int nw) {
    return (q & 1) ? nw * (q + 1) - 1 - w : nw * q + w;
}

template <typename T, int N, int S>
__global__ __launch_bounds__(64 * out_waves<S>()) void k_chunk_out(
    const T* __restrict__ x, const float* __restrict__ dt, const T* __restrict__ Cm,
    const T* __restrict__ states, const float* __restrict__ aux, const float* __restrict__ gram,
    T* __restrict__ y, int64_t L, int H, int G, int64_t M, int64_t BM) {
    constexpr int NW = out_waves<S>();
    constexpr int NT = 64 * NW;
    constexpr int KS = N / 32;     // 32-deep k steps over the state dim
    constexpr int NQ = S / 16 / NW; // row tiles per wave
    constexpr int XRB = kP * (int)sizeof(T);
    constexpr int XT = S * XRB;    // the chunk's x rows
    constexpr int HT = N * XRB;    // H_[c-1] tile, rows n of P values
    // Block order: workgroups are dealt to the 8 XCDs round-robin by block
    // index.  When B*M is a multiple of 8, XCD x runs the heads of chunks
    // (b, c) = x, x+8, ... one after another, so all heads reading one
    // chunk's Gram tiles share one L2.
    const int64_t bid = blockIdx.x;
    int64_t bc;
    int h;
    if (BM % 8 == 0) {
        const int64_t slot = bid >> 3;
        bc = (slot / H) * 8 + (bid & 7);
        h = (int)(slot % H);
    } else {
        bc = bid / H;
        h = (int)(bid % H);
    }
    const int64_t b = bc / M;
    const int64_t c = bc % M;
    const int g = (int)((int64_t)h * G / H);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = lane & 15, grp = lane >> 4;
    const int64_t t0 = c * S;
    const int len = (int)(L - t0 < S ? L - t0 : S);

    __shared__ float s_cs[S];  // within-chunk cumulative log decay, log2 units
    __shared__ float s_dt[S];
    __shared__ __attribute__((aligned(16))) float s_b[S];   // exp2(cs_e - cs_s) dt_s, e = end of the s block
    __shared__ __attribute__((aligned(16))) char ht[HT];
    __shared__ __attribute__((aligned(16))) char xs[XT];

    dma_tile<XRB>(ht, reinterpret_cast<const char*>(states + ((b * M + c) * H + h) * (int64_t)N * kP),
                  XRB, N, N, wave, NW, lane);
    dma_tile<XRB>(xs, reinterpret_cast<const char*>(x + ((b * L + t0) * H + h) * kP),
                  (int64_t)H * XRB, S, len, wave, NW, lane);
    const float* csc = aux + ((b * H + h) * M + c) * 3 * S;
    for (int i = tid; i < S; i += NT) {
        const float csi = csc[i];
        const float cse = csc[i | 31];
        const float dti = (i < len) ? dt[(b * L + t0 + i) * H + h] : 0.f;
        s_cs[i] = csi;
        s_dt[i] = dti;
        s_b[i] = fast_exp2(cse - csi) * dti;
    }
    f32x4 yacc[NQ][4];
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int pt = 0; pt < 4; ++pt) yacc[q][pt] = f32x4{0.f, 0.f, 0.f, 0.f};
    wait_dma();
    __syncthreads();

    // One row tile at a time (few live registers, so several blocks share a
    // CU; the H and x fragments are re-read from LDS per tile).  The C rows of
    // the next tile and the Gram pair of the next s block are requested one
    // step ahead.
    const float* gbase = gram + ((b * G + g) * M + c) * (int64_t)gram_pairs(S) * 512 + lane * 8;
    auto load_c = [&](int q, Frag<T> (&cr)[KS]) {
        const int t = tile_row(wave, q, NW) * 16 + col;
        const int tc = t < len ? t : len - 1;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) cr[ks] = load_frag(Cm + ((b * L + t0 + tc) * G + g) * N + ks * 32 + grp * 8);
    };
    Frag<T> craw[KS];
    load_c(0, craw);
    // bf16 fragment reads at offsets fixed here: H rows 32 ks + 8 grp (+4),
    // x rows 32 sk + 4 grp (+16), column tile pt
    KmOffBf16<XRB> ho[4], xo[4];
    if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int pt = 0; pt < 4; ++pt) {
            ho[pt].init(8 * grp, 8 * grp + 4, pt * 16, lane);
            xo[pt].init(4 * grp, 16 + 4 * grp, pt * 16, lane);
        }
    }
    auto frag_h = [&](int ks, int pt) __attribute__((always_inline)) {
        if constexpr (sizeof(T) == 2) {
            return ho[pt].read(ht, ks * 32 * XRB);
        } else {
            return frag_km<T, XRB>(ht, ks * 32 + 8 * grp, ks * 32 + 8 * grp + 4, pt * 16, lane);
        }
    };
    auto frag_x = [&](int sk, int pt) __attribute__((always_inline)) {
        if constexpr (sizeof(T) == 2) {
            return xo[pt].read(xs, sk * 32 * XRB);
        } else {
            return frag_km<T, XRB>(xs, sk * 32 + 4 * grp, sk * 32 + 16 + 4 * grp, pt * 16, lane);
        }
    };
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
        const int r = tile_row(wave, q, NW);
        const int t = r * 16 + col;
        const float cst = s_cs[t];
        const f32x4* gsrc = reinterpret_cast<const f32x4*>(gbase + (int64_t)gram_pair(r, 0) * 512);
        f32x4 g0 = gsrc[0], g1 = gsrc[1];
        // inter-chunk term: (C_t exp(cs_t)) H_[c-1]; C rows in fragment layout
        // (row t = lane%16), H read k-major (k = n)
        {
            const float sc = fast_exp2(cst);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                float v[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) v[i] = to_f(craw[ks][i]) * sc;
                const Frag<T> fa = make_frag<T>(v);
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) yacc[q][pt] = mma16(yacc[q][pt], fa, frag_h(ks, pt));
            }
        }
        if (q + 1 < NQ) load_c(q + 1, craw);
        // intra-chunk term over the causal s blocks sk <= r/2 (unrolled, so
        // the x fragment offsets are immediates)
#pragma unroll
        for (int sk = 0; sk < S / 32; ++sk) {
            if (sk > (r >> 1)) break;
            const int sbase = sk * 32;
            const f32x4 c0 = g0, c1 = g1;
            if (sk < (r >> 1)) {
                gsrc = reinterpret_cast<const f32x4*>(gbase + (int64_t)gram_pair(r, sk + 1) * 512);
                g0 = gsrc[0];
                g1 = gsrc[1];
            }
            // k order of the A operand: s = sbase + 16 u + 4 grp + i, element 4 u + i
            float mv[8];
            if (sk < (r >> 1)) {
                const float a = fast_exp2(cst - s_cs[sbase + 31]);
                const f32x4 b0 = *reinterpret_cast<const f32x4*>(&s_b[sbase + 4 * grp]);
                const f32x4 b1 = *reinterpret_cast<const f32x4*>(&s_b[sbase + 16 + 4 * grp]);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    mv[i] = c0[i] * (a * b0[i]);
                    mv[4 + i] = c1[i] * (a * b1[i]);
                }
            } else {
#pragma unroll
                for (int u = 0; u < 2; ++u)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int s = sbase + 16 * u + 4 * grp + i;
                        const float gval = u ? c1[i] : c0[i];
                        mv[4 * u + i] = (s <= t) ? gval * fast_exp2(cst - s_cs[s]) * s_dt[s] : 0.f;
                    }
            }
            const Frag<T> fm = make_frag<T>(mv);
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) yacc[q][pt] = mma16(yacc[q][pt], fm, frag_x(sk, pt));
        }
    }

    // yacc[q][pt][i] = y[t = 16 tile_row(wave, q) + 4 grp + i][p = 16 pt + col]:
    // each 16-row tile goes through the wave's LDS scratch (the x rows, no
    // longer read once every wave is done) and leaves as 16-byte stores of
    // whole rows
    __syncthreads();
    T* st = reinterpret_cast<T*>(xs) + wave * 16 * kP;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) st[(4 * grp + i) * kP + pt * 16 + col] = from_f<T>(yacc[q][pt][i]);
        const int tbase = tile_row(wave, q, NW) * 16;
#pragma unroll
        for (int e8 = lane; e8 < 16 * (kP / 8); e8 += 64) {
            const int r = e8 / (kP / 8), k8 = e8 % (kP / 8);
            if (tbase + r < len) {
                float v[8];
                load8(st + r * kP + k8 * 8, v);
                store8(y + ((b * L + t0 + tbase + r) * H + h) * kP + k8 * 8, v);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Chunk output for bf16, one workgroup per (b, chunk, group, slice of hpb
// heads of the group).  The chunk's causal Gram pairs G^T[s][t] = B_s . C_t
// depend on the group only: each wave forms those of its row tiles once (bf16
// registers; the same nine pairs per wave for S = 256, the row tiles being
// paired light with heavy as in k_chunk_out) and keeps them, with its C rows,
// for every head of the slice.  Each head's inputs (x rows, H_[c-1] and the
// chunk's per-token record cs, dt, exp2(cs_e - cs_s) dt_s) arrive by DMA in
// one of two buffers, the next head's copy running under the current head's
// MFMAs.  Per head:
//   y = diag(exp2(cs_t)) (C H_[c-1])            inter-chunk term, the decay
//                                               applied to the accumulator rows
//     + sum over causal s blocks of (G o decay) (x)   intra-chunk term
// with the decay factored over s blocks before the row tile as in k_chunk_out
// and exact on the diagonal block.  A wave's two row tiles share every H and x
// fragment they both use (one LDS read, two MFMAs), and the x fragments of
// the next s block are read while the current one is multiplied.  The k
// order of all operands is s (or n) = 16 u + 4 (lane/16) + i for element
// 4 u + i, which makes the transposing reads of the H and x tiles
// conflict-free.  The products are formed transposed (A = the H or x
// fragment, B = the C or Gram fragment), so that a lane's accumulator holds
// y[t][p .. p + 3] of one token t: the row decay exp2(cs_t) is one factor per
// lane, and each lane stores its outputs as 8-byte pieces straight from
// registers.  The copies use per-lane offsets fixed at set-up.
// ---------------------------------------------------------------------------
// y stores per row tile and head in k_chunk_out_heads (16 bytes per lane)
constexpr int kYStores = 2;

template <int N, int S>
__global__ __launch_bounds__(64 * out_waves<S>()) void k_chunk_out_heads(
    const bf16* __restrict__ x, const bf16* __restrict__ Bm, const bf16* __restrict__ Cm,
    const bf16* __restrict__ states, const float* __restrict__ aux, bf16* __restrict__ y,
    int64_t L, int H, int G, int64_t M, int hpb, int64_t nbcg) {
    using T = bf16;
    constexpr int NW = out_waves<S>();
    constexpr int KS = N / 32;
    constexpr int NQ = S / 16 / NW;
    constexpr int XRB = kP * 2;                   // bytes of an x, H or y row
    constexpr int XT = S * XRB;                   // x rows of the chunk
    constexpr int HT = N * XRB;                   // H_[c-1]
    constexpr int AT = 3 * S * 4;                 // per-token record
    constexpr int UB = XT + HT + AT;              // one head's inputs
    constexpr int MSK0 = ((NW - 1) >> 1) + 1;     // s blocks of row tile q = 0 (at most)
    constexpr int MSK1 = ((2 * NW - 1) >> 1) + 1; // of row tile q = 1
    constexpr int MSKL = NQ == 2 ? MSK1 : MSK0;   // s blocks of the wave (at most)
    static_assert(NQ == 1 || NQ == 2, "one or two row tiles per wave");

    // block -> (b, c, g, head slice); the slices of one (b, c, g) share an XCD
    const int nhs = (H / G) / hpb;
    const int64_t bid = blockIdx.x;
    int64_t bcg;
    int hs;
    if (nbcg % 8 == 0) {
        const int64_t slot = bid >> 3;
        bcg = (slot / nhs) * 8 + (bid & 7);
        hs = (int)(slot % nhs);
    } else {
        bcg = bid / nhs;
        hs = (int)(bid % nhs);
    }
    const int g = (int)(bcg % G);
    const int64_t bc = bcg / G;
    const int64_t b = bc / M, c = bc % M;
    const int hbase = g * (H / G) + hs * hpb;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int col = lane & 15, grp = lane >> 4;
    const int64_t t0 = c * S;
    const int len = (int)(L - t0 < S ? L - t0 : S);

    // the two head buffers; before the head loop the same bytes hold the
    // chunk's B and C rows (swizzled [S][N] tiles) for the Gram pairs
    constexpr int BRB = N * 2;
    constexpr int BCT = S * BRB;
    constexpr int LDSB = 2 * UB > 2 * BCT ? 2 * UB : 2 * BCT;
    __shared__ __attribute__((aligned(16))) char units[LDSB];

    // Copies of one head's inputs into buffer u: x and H_[c-1] into swizzled
    // row tiles (rows past the end of a partial chunk re-read the last row),
    // the record linearly.
    const uint32_t units_lds = lds_addr(units);
    TilePlan<XRB, S, NW> xplan;
    TilePlan<XRB, N, NW> hplan;
    const LinearPlan<AT, NW> rplan;
    xplan.init(wave, lane, (uint32_t)(H * XRB), len);
    hplan.init(wave, lane, (uint32_t)XRB, N);
    auto issue_unit = [&](int hh, int u) __attribute__((always_inline)) {
        const int h = hbase + hh;
        const uint32_t ub = units_lds + (uint32_t)(u * UB);
        xplan.issue(x + ((b * L + t0) * H + h) * kP, ub, wave);
        hplan.issue(states + ((b * M + c) * H + h) * (int64_t)N * kP, ub + XT, wave);
        rplan.issue(aux + ((b * H + h) * M + c) * 3 * S, ub + XT + HT, wave, lane);
    };
    // the chunk's B and C rows, one copy burst (rows past the end of a partial
    // chunk re-read the last row: finite values, zero weight)
    {
        TilePlan<BRB, S, NW> bcplan;
        bcplan.init(wave, lane, (uint32_t)(G * BRB), len);
        bcplan.issue(Bm + ((b * L + t0) * G + g) * N, units_lds, wave);
        bcplan.issue(Cm + ((b * L + t0) * G + g) * N, units_lds + BCT, wave);
    }
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    lds_barrier();
    const char* const btile = units;
    const char* const ctile = units + BCT;

    // the wave's row tiles and their C rows, in the k order above
    int rq[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) rq[q] = tile_row(wave, q, NW);
    auto kfrag = [&](const char* tile, int row, int ks) __attribute__((always_inline)) {
        using Tl = SwzTile<BRB>;
        const bf16x4 lo = *reinterpret_cast<const bf16x4*>(tile + Tl::off(row, (ks * 32 + 4 * grp) * 2));
        const bf16x4 hi = *reinterpret_cast<const bf16x4*>(tile + Tl::off(row, (ks * 32 + 16 + 4 * grp) * 2));
        return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    };
    bf16x8 craw[NQ][KS];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) craw[q][ks] = kfrag(ctile, rq[q] * 16 + col, ks);
    }
    // Gram pairs of the wave's row tiles: element 4 u + i of pair (q, sk) is
    // G^T[s = 32 sk + 16 u + 4 grp + i][t = 16 r_q + col]
    bf16x8 gq0[MSK0], gq1[MSK1];
    auto gram_pair = [&](int q, int sk) __attribute__((always_inline)) {
        f32x4 acc[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            acc[u] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) acc[u] = mma16(acc[u], kfrag(btile, sk * 32 + u * 16 + col, ks), craw[q][ks]);
        }
        const float v[8] = {acc[0][0], acc[0][1], acc[0][2], acc[0][3],
                            acc[1][0], acc[1][1], acc[1][2], acc[1][3]};
        return make_frag<T>(v);
    };
#pragma unroll
    for (int sk = 0; sk < MSK0; ++sk)
        if (sk <= (rq[0] >> 1)) gq0[sk] = gram_pair(0, sk);
    if constexpr (NQ == 2) {
#pragma unroll
        for (int sk = 0; sk < MSK1; ++sk)
            if (sk <= (rq[NQ - 1] >> 1)) gq1[sk] = gram_pair(NQ - 1, sk);
    }
    lds_barrier();  // the B and C tiles are consumed: the head buffers take over
    issue_unit(0, 0);

    // transposing fragment reads at offsets fixed here: rows (k) 4 grp + i and
    // 16 + 4 grp + i of a 32-row block, column tile pt
    KmOffBf16<XRB> ko[4];
#pragma unroll
    for (int pt = 0; pt < 4; ++pt) ko[pt].init(4 * grp, 16 + 4 * grp, pt * 16, lane);

    auto head = [&](int h, const char* ub) __attribute__((always_inline)) {
        // per-lane indices are recomputed for every head (the empty asm keeps
        // the compiler from hoisting the diagonal masks and offsets derived
        // from them out of the head loop, where they would not fit)
        int lc = col, lg = grp;
        asm volatile("" : "+v"(lc), "+v"(lg));
        const char* xt = ub;
        const char* ht = ub + XT;
        const float* rc = reinterpret_cast<const float*>(ub + XT + HT);  // cs | dt | weight
        f32x4 yacc[NQ][4];
#pragma unroll
        for (int q = 0; q < NQ; ++q)
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) yacc[q][pt] = f32x4{0.f, 0.f, 0.f, 0.f};
        // inter-chunk term, each H fragment shared by the row tiles
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) {
                const bf16x8 hf = ko[pt].read(ht, ks * 32 * XRB);
#pragma unroll
                for (int q = 0; q < NQ; ++q) yacc[q][pt] = mma16(yacc[q][pt], hf, craw[q][ks]);
            }
        // the lane's token t = 16 r + col takes exp2(cs_t)
        float cst[NQ];
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            cst[q] = rc[rq[q] * 16 + lc];
            const float e = fast_exp2(cst[q]);
#pragma unroll
            for (int pt = 0; pt < 4; ++pt)
#pragma unroll
                for (int i = 0; i < 4; ++i) yacc[q][pt][i] *= e;
        }
        // intra-chunk term over the s blocks of the heavier row tile
        const int skmax = rq[NQ - 1] >> 1;
        bf16x8 xf[2][4];
#pragma unroll
        for (int pt = 0; pt < 4; ++pt) xf[0][pt] = ko[pt].read(xt, 0);
#pragma unroll
        for (int sk = 0; sk < MSKL; ++sk) {
            if (sk > skmax) break;
            const int cur = sk & 1;
            const int sbase = sk * 32;
            if (sk + 1 <= skmax) {
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) xf[cur ^ 1][pt] = ko[pt].read(xt, (sbase + 32) * XRB);
            }
            const f32x4 b0 = *reinterpret_cast<const f32x4*>(rc + 2 * S + sbase + 4 * lg);
            const f32x4 b1 = *reinterpret_cast<const f32x4*>(rc + 2 * S + sbase + 16 + 4 * lg);
            const float cse = rc[sbase + 31];
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const int rs = rq[q] >> 1;
                if (sk > rs) continue;
                // (q, sk) are constants once the loops are unrolled; q = 0
                // never reaches sk >= MSK0
                bf16x8 gv = q == 0 ? gq0[sk < MSK0 ? sk : MSK0 - 1] : gq1[sk < MSK1 ? sk : MSK1 - 1];
                asm volatile("" : "+v"(gv));  // widened per head, not kept widened
                float mv[8];
                if (sk < rs) {
                    const float a = fast_exp2(cst[q] - cse);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        mv[i] = to_f(gv[i]) * (a * b0[i]);
                        mv[4 + i] = to_f(gv[4 + i]) * (a * b1[i]);
                    }
                } else {
                    const int t = rq[q] * 16 + lc;
#pragma unroll
                    for (int u = 0; u < 2; ++u) {
                        const f32x4 css = *reinterpret_cast<const f32x4*>(rc + sbase + 16 * u + 4 * lg);
                        const f32x4 dts = *reinterpret_cast<const f32x4*>(rc + S + sbase + 16 * u + 4 * lg);
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const int sidx = sbase + 16 * u + 4 * lg + i;
                            mv[4 * u + i] = (sidx <= t) ? to_f(gv[4 * u + i]) * fast_exp2(cst[q] - css[i]) * dts[i]
                                                        : 0.f;
                        }
                    }
                }
                const bf16x8 fm = make_frag<T>(mv);
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) yacc[q][pt] = mma16(yacc[q][pt], xf[cur][pt], fm);
            }
        }
        // yacc[q][pt][i] = y[t = 16 r_q + col][p = 16 pt + 4 grp + i] (the
        // head loop's wait counts on kYStores stores per row tile).  A row
        // swap between the slices pt and pt + 1 (even rows keep slice pt, odd
        // rows slice pt + 1) gives every lane 8 consecutive p of one token:
        // 16-byte stores, half as many as with 4 p per lane.
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int t = rq[q] * 16 + lc;
            uint32_t pk[4][2];
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) {
                const bf16x2 lo = {(bf16)yacc[q][pt][0], (bf16)yacc[q][pt][1]};
                const bf16x2 hi = {(bf16)yacc[q][pt][2], (bf16)yacc[q][pt][3]};
                pk[pt][0] = __builtin_bit_cast(uint32_t, lo);
                pk[pt][1] = __builtin_bit_cast(uint32_t, hi);
            }
            // v_permlane16_swap: odd rows of the first operand trade places
            // with even rows of the second (a row is 16 lanes)
#pragma unroll
            for (int pp = 0; pp < 4; pp += 2) {
#pragma unroll
                for (int k = 0; k < 2; ++k)
                    asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1"
                                 : "+v"(pk[pp][k]), "+v"(pk[pp + 1][k]));
            }
            if (t < len) {
                bf16* yrow = y + ((b * L + t0 + t) * H + h) * kP;
                const int odd = lg & 1;
#pragma unroll
                for (int pp = 0; pp < 4; pp += 2) {
                    const int p0 = 16 * (pp + odd) + 4 * (lg - odd);
                    *reinterpret_cast<uint4*>(yrow + p0) =
                        make_uint4(pk[pp][0], pk[pp][1], pk[pp + 1][0], pk[pp + 1][1]);
                }
            }
        }
    };

    for (int hh = 0; hh < hpb; ++hh) {
        // this wave's copies of head hh are in: only the y stores of head
        // hh - 1 (two per row tile) were issued after them (vector memory
        // operations complete in order); a partial chunk, whose stores are
        // predicated, waits for all
        if (hh == 0 || len < S) {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
        } else {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(kYStores * NQ));
        }
        lds_barrier();  // every wave's copies are in; head hh - 1 is done with its buffer
        if (hh + 1 < hpb) issue_unit(hh + 1, (hh + 1) & 1);
        head(hbase + hh, units + (hh & 1) * UB);
    }
}

// Workspace carve-up of the scan: per-chunk log decay [B][H][M], chunk-entry
// states [B][M][H][N][P] (storage dtype), the per-token record (cs, dt,
// weight) [B][H][M][3][S] and, for fp32 only, the causal Gram tiles
// [B][G][M][pairs][64][8] (float).
struct ScanWs {
    float* lda;
    char* states;
    float* aux;
    float* gram;
    size_t total;
};

}  // namespace

int device_cu_count() {
    static const int cus = [] {
        int dev = 0, n = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
        return n;
    }();
    return cus;
}

namespace {

// Heads per workgroup of the bf16 scan kernels: the largest divisor of the
// heads of a group, at most hmax, that still gives every compute unit a
// workgroup.
int out_heads_per_block(int64_t nbcg, int hg, int hmax) {
    const int cus = device_cu_count();
    for (int hpb = hg < hmax ? hg : hmax; hpb > 1; --hpb)
        if (hg % hpb == 0 && nbcg * (hg / hpb) >= cus) return hpb;
    return 1;
}
ScanWs scan_ws(const Shape& s, void* ws) {
    char* p = reinterpret_cast<char*>(ws);
    ScanWs w;
    size_t off = 0;
    w.lda = reinterpret_cast<float*>(p + off);
    off += align256(sizeof(float) * s.B * s.H * s.M);
    w.states = p + off;
    off += align256(elem_bytes(s.dtype) * s.B * s.M * s.H * (size_t)s.N * s.P);
    if (!tuned_shape(s)) {
        // generic kernels: the chunk contributions and entry states in float
        w.aux = reinterpret_cast<float*>(p + off);
        off += align256(sizeof(float) * s.B * s.M * s.H * (size_t)s.N * s.P);
        w.gram = reinterpret_cast<float*>(p + off);
        off += align256(sizeof(float) * s.B * s.M * s.H * (size_t)s.N * s.P);
        w.total = off;
        return w;
    }
    w.aux = reinterpret_cast<float*>(p + off);
    off += align256(sizeof(float) * s.B * s.H * s.M * 3 * (size_t)s.S);
    w.gram = reinterpret_cast<float*>(p + off);
    if (s.dtype != 1) off += align256(sizeof(float) * s.B * s.G * s.M * (size_t)gram_pairs(s.S) * 512);
    w.total = off;
    return w;
}

template <typename T, int N, int S>
hipError_t run_scan(const Shape& s, const void* x, const float* dt, const float* A, const void* Bm,
                    const void* Cm, const float* h0, void* y_ssd, void* mem, float* h_last,
                    void* ws, hipStream_t st) {
    const ScanWs w = scan_ws(s, ws);
    T* states = reinterpret_cast<T*>(w.states);
    const int64_t nbcg = s.B * s.M * s.G;
    // the chunk-state workgroup keeps every head's dt (S floats) in one x
    // buffer and every head's weights in the B tile: at most 32 and N / 2 heads
    const int hpb = out_heads_per_block(nbcg, s.H / s.G, N / 2 < 32 ? N / 2 : 32);
    prof_begin("k_chunk_state", st);
    if constexpr (sizeof(T) == 2) {
        k_chunk_state_heads<N, S><<<dim3((unsigned)(nbcg * (s.H / s.G / hpb))), 512, 0, st>>>(
            (const bf16*)x, dt, A, (const bf16*)Bm, (bf16*)mem, w.lda, w.aux, s.L, s.H, s.G, s.M,
            s.Mcap, hpb, nbcg);
    } else {
        k_chunk_state<T, N, S><<<dim3((unsigned)s.M, (unsigned)s.H, (unsigned)s.B), kThreads, 0, st>>>(
            (const T*)x, dt, A, (const T*)Bm, (T*)mem, w.lda, w.aux, s.L, s.H, s.G, s.M, s.Mcap);
    }
    prof_end(st);
    if constexpr (sizeof(T) == 4) {
        prof_begin("k_chunk_gram", st);
        k_chunk_gram<T, N, S><<<dim3((unsigned)(S / 64), (unsigned)s.M, (unsigned)(s.B * s.G)),
                                kThreads, 0, st>>>((const T*)Bm, (const T*)Cm, w.gram, s.L, s.G, s.M);
        prof_end(st);
    }
    const int NP = N * kP;
    prof_begin("k_state_pass", st);
    k_state_pass<T><<<dim3((unsigned)(NP / (kThreads * 4)), (unsigned)s.H, (unsigned)s.B), kThreads,
                      0, st>>>((const T*)mem, w.lda, h0, states, h_last, s.H, NP, s.M, s.Mcap);
    prof_end(st);
    prof_begin("k_chunk_out", st);
    if constexpr (sizeof(T) == 2) {
        k_chunk_out_heads<N, S><<<dim3((unsigned)(nbcg * (s.H / s.G / hpb))), 64 * out_waves<S>(), 0,
                                  st>>>((const bf16*)x, (const bf16*)Bm, (const bf16*)Cm, states,
                                        w.aux, (bf16*)y_ssd, s.L, s.H, s.G, s.M, hpb, nbcg);
    } else {
        k_chunk_out<T, N, S><<<dim3((unsigned)(s.B * s.M * s.H)), 64 * out_waves<S>(), 0, st>>>(
            (const T*)x, dt, (const T*)Cm, states, w.aux, w.gram, (T*)y_ssd, s.L, s.H, s.G, s.M,
            s.B * s.M);
    }
    prof_end(st);
    return hipGetLastError();
}

template <typename T, int N>
hipError_t run_scan_s(const Shape& s, const void* x, const float* dt, const float* A,
                      const void* Bm, const void* Cm, const float* h0, void* y, void* mem,
                      float* hl, void* ws, hipStream_t st) {
    switch (s.S) {
        case 64: return run_scan<T, N, 64>(s, x, dt, A, Bm, Cm, h0, y, mem, hl, ws, st);
        case 128: return run_scan<T, N, 128>(s, x, dt, A, Bm, Cm, h0, y, mem, hl, ws, st);
        case 256: return run_scan<T, N, 256>(s, x, dt, A, Bm, Cm, h0, y, mem, hl, ws, st);
    }
    return hipErrorInvalidValue;
}

template <typename T>
hipError_t run_scan_n(const Shape& s, const void* x, const float* dt, const float* A,
                      const void* Bm, const void* Cm, const float* h0, void* y, void* mem,
                      float* hl, void* ws, hipStream_t st) {
    switch (s.N) {
        case 32: return run_scan_s<T, 32>(s, x, dt, A, Bm, Cm, h0, y, mem, hl, ws, st);
        case 64: return run_scan_s<T, 64>(s, x, dt, A, Bm, Cm, h0, y, mem, hl, ws, st);
        case 128: return run_scan_s<T, 128>(s, x, dt, A, Bm, Cm, h0, y, mem, hl, ws, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace

size_t scan_workspace_bytes(const Shape& s) { return scan_ws(s, nullptr).total; }

const void* scan_entry_states(const Shape& s, const void* ws) {
    return scan_ws(s, const_cast<void*>(ws)).states;
}

hipError_t launch_scan(const Shape& s, const void* x, const float* dt, const float* A,
                       const void* Bm, const void* Cm, const float* h0, void* y_ssd, void* mem,
                       float* h_last, void* ws, hipStream_t st) {
    if (!tuned_shape(s)) {
        const ScanWs w = scan_ws(s, ws);
        const GenScanWs g{w.lda, w.states, w.aux, w.gram};
        return launch_gscan(s, x, dt, A, Bm, Cm, h0, y_ssd, mem, h_last, g, st);
    }
    if (s.dtype == 1) return run_scan_n<bf16>(s, x, dt, A, Bm, Cm, h0, y_ssd, mem, h_last, ws, st);
    return run_scan_n<float>(s, x, dt, A, Bm, Cm, h0, y_ssd, mem, h_last, ws, st);
}

}  // namespace dart
