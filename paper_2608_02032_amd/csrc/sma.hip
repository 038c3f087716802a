// sma.hip -- state-memory attention forward with the fused gated residual.
//
// Paper: Sec. 3 "State-Memory Attention" (V_{t,c} = C_t dH_[c],
// K_{t,c} = dH_[c] E_t, l = Q K / sqrt(N), softmax over strictly earlier
// chunks, R_t = 0 without history), "Gated Residual Integration"
// (Y_t = C_t H_t + SiLU(z_t) R_t), App. B.1 (normalised score branch:
// RMSNorm(Q), RMSNorm(E), K = r_c (.) (dH_[c] Ebar)) and Alg. 1 / App. C (a
// query tile fixed, historical memories streamed, online softmax, only R and
// the log-sum-exp leave the chip).
//
// Both precisions run one workgroup per (b, group of heads, token block).
// The block's 8 waves form 4 pairs; each pair owns 16*RT consecutive tokens
// inside one chunk.  In a pair, the score wave holds Qbar and Ebar and the
// value wave holds C and the output accumulator O, so each wave keeps only
// half of the per-token operands and every operand fragment it reads from LDS
// feeds RT independent MFMA chains.  The block streams the memories of its
// heads, head by head; per step:
//   score waves   U^T = (r_s (.) dH_s)^T Qbar^T (P x tokens, MFMA), logits
//                 l_t = sum_p U^T[p,t] Ebar[t,p], online softmax in base 2;
//                 the weights of memory s (and a rescale factor when the
//                 running maximum moved) go to LDS;
//   value waves   V^T = dH^T C^T of an earlier memory (MFMA), O = alpha O + w V;
// with one barrier per step.  Epilogue of each head: the score wave publishes
// its softmax denominators and writes LSE = (m + log2 d) ln 2; the value wave
// writes y = y_ssd + SiLU(z) O/d.
//
// bf16 (k_sma_prep, k_sma): a first kernel writes both sides of every attended
// memory transposed to [P][N] (key side r (.) dH rounded to bf16, value side
// dH), so every MFMA operand fragment is one 16-byte LDS read.  k_sma copies
// the tiles by DMA (global_load_lds, no registers) into XOR-swizzled LDS
// rings, key tiles two steps and value tiles one step ahead; the value waves
// lag the score waves by two memories so neither waits on the other within a
// step, and they copy each head's y_ssd rows and gates into LDS a step before
// the head ends.
//
// fp32 (k_sma_keys, k_sma_regs): a first kernel writes the key side in the
// cache's [N][P] layout; value tiles come straight from the cache, through
// registers one step ahead when four LDS stages do not fit.  Operand fragments
// are read with transposing LDS loads.
#include <algorithm>
#include <cstdlib>

#include "dart_common.hpp"
#include "dart_internal.hpp"

namespace dart {
namespace {

constexpr int kP = 64;
constexpr int kWaves = 8;                  // 4 (score, value) pairs
constexpr int kThreads = kWaves * 64;
constexpr float kRescaleLog2 = 8.0f;       // lazy-rescale threshold (log2 units)
constexpr int kHeadsPerBlock = 8;          // most heads of one group a block can serve (power of 2)
// The forward's chooser stops at four heads per block: measured against
// eight, four take 472 vs 483 us at B 4, L 8192, 32 heads, S 256 and 930 vs
// 965 us at S 128, and tie at the Mamba-2-130M shape (the greedy-order bound
// itself cannot see the difference).
constexpr int kFwdHeadsCap = 4;

// 16-token column tiles per pair: 4 for bf16 (64 tokens), 2 for fp32 (its
// operand fragments take twice the registers).
template <typename T> constexpr int sma_rt() { return sizeof(T) == 2 ? 4 : 2; }
template <typename T> constexpr int sma_tokens_per_block() { return 4 * 16 * sma_rt<T>(); }

// 8 operand values of a token row vector v (length N) in the lane's k order:
// k-group g holds elements 32 ks + 4 g + {0..3} and 32 ks + 16 + 4 g + {0..3},
// the order in which frag_km hands out the rows of a k-major tile.
template <typename T>
__device__ __forceinline__ void load_kperm(const T* row, int ks, int grp, float (&v)[8]) {
    float a[4], b[4];
    load4(row + ks * 32 + 4 * grp, a);
    load4(row + ks * 32 + 16 + 4 * grp, b);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[i] = a[i];
        v[4 + i] = b[i];
    }
}

// Four consecutive elements loaded as one vector (8 B for bf16, 16 B for fp32).
template <typename T>
using Vec4 = T __attribute__((ext_vector_type(4)));
template <typename T>
__device__ __forceinline__ Vec4<T> ld4(const T* p) { return *reinterpret_cast<const Vec4<T>*>(p); }
template <typename T>
__device__ __forceinline__ Frag<T> cat_frag(Vec4<T> a, Vec4<T> b) {
    return Frag<T>{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// Sum of squares of the elements of one 16-byte piece, and the piece scaled.
__device__ __forceinline__ float piece_sumsq(uint4 v, bf16) {
    const bf16x8 h = __builtin_bit_cast(bf16x8, v);
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) s += (float)h[i] * (float)h[i];
    return s;
}
__device__ __forceinline__ float piece_sumsq(uint4 v, float) {
    const f32x4 f = __builtin_bit_cast(f32x4, v);
    return f[0] * f[0] + f[1] * f[1] + f[2] * f[2] + f[3] * f[3];
}
__device__ __forceinline__ uint4 piece_scale(uint4 v, float r, bf16) {
    const bf16x8 h = __builtin_bit_cast(bf16x8, v);
    bf16x8 o;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = (bf16)((float)h[i] * r);
    return __builtin_bit_cast(uint4, o);
}
__device__ __forceinline__ uint4 piece_scale(uint4 v, float r, float) {
    f32x4 f = __builtin_bit_cast(f32x4, v);
#pragma unroll
    for (int i = 0; i < 4; ++i) f[i] *= r;
    return __builtin_bit_cast(uint4, f);
}

// The rounding residual of a scaled bf16 piece: lo = bf16(v r - bf16(v r)), so
// that hi + lo carries v r to about 16 significant bits.
__device__ __forceinline__ uint4 piece_scale_lo(uint4 v, float r) {
    const bf16x8 h = __builtin_bit_cast(bf16x8, v);
    bf16x8 o;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float x = (float)h[i] * r;
        o[i] = (bf16)(x - (float)(bf16)x);
    }
    return __builtin_bit_cast(uint4, o);
}

// Key side of one memory: kmem = r (.) dH, r[n] the inverse RMS of row n of
// the stored values.  The RPC lanes holding one row's 16-byte pieces reduce
// its sum of squares with DPP moves.  rinv (optional, [B][Mp][H][N]) receives
// 1 / r[n]; klo (optional, bf16 only) the rounding residual of the bf16 key
// side, so kmem + klo is r (.) dH to about 16 bits.
template <typename T, int N>
__global__ __launch_bounds__(256) void k_sma_keys(const T* __restrict__ mem, T* __restrict__ kmem,
                                                  T* __restrict__ klo, float* __restrict__ rinv,
                                                  float eps, int normalize, int H, int64_t Mp,
                                                  int64_t Mcap) {
    constexpr int RB = kP * (int)sizeof(T);
    constexpr int PIECES = N * RB / 16;
    constexpr int RPC = RB / 16;
    static_assert(PIECES % 256 == 0, "pieces must tile the block");
    const int64_t j = blockIdx.x;
    const int h = blockIdx.y;
    const int64_t b = blockIdx.z;
    const uint4* src = reinterpret_cast<const uint4*>(mem + ((b * Mcap + j) * H + h) * (int64_t)N * kP);
    const int64_t obase = ((b * Mp + j) * H + h) * (int64_t)N * kP;
    uint4* dst = reinterpret_cast<uint4*>(kmem + obase);
    uint4 v[PIECES / 256];
#pragma unroll
    for (int i = 0; i < PIECES / 256; ++i) v[i] = src[threadIdx.x + i * 256];
#pragma unroll
    for (int i = 0; i < PIECES / 256; ++i) {
        const float ss = dpp_group_sum<RPC>(piece_sumsq(v[i], T()));
        const float rn = normalize ? __builtin_amdgcn_rsqf(ss * (1.0f / kP) + eps) : 1.0f;
        dst[threadIdx.x + i * 256] = piece_scale(v[i], rn, T());
        if constexpr (sizeof(T) == 2) {
            if (klo) reinterpret_cast<uint4*>(klo + obase)[threadIdx.x + i * 256] = piece_scale_lo(v[i], rn);
        }
        const int q = threadIdx.x + i * 256;
        if (rinv && q % RPC == 0) rinv[((b * Mp + j) * H + h) * (int64_t)N + q / RPC] = 1.0f / rn;
    }
}

// The epilogue inputs of one head, for each of a lane's RT tokens: its gate
// pre-activation z and its 4 x 4 y_ssd values (columns 16 pt + 4 (lane/16) ..
// +3).  They are loaded inside one assembly block that also waits for them, so
// the compiler tracks no load of these registers: loads it tracked here, in
// the streaming loop, made it drain the tile copies in flight at later
// register reuses in every step.  Called once per head, where the drain is
// cheap.
template <typename T, int RT>
__device__ __forceinline__ void load_epilogue_inputs(const T* const (&zp)[RT],
                                                     const T* const (&yp)[RT], float (&zz)[RT],
                                                     Vec4<T> (&ys)[RT][4]);
template <>
__device__ __forceinline__ void load_epilogue_inputs<float, 2>(const float* const (&zp)[2],
                                                               const float* const (&yp)[2],
                                                               float (&zz)[2],
                                                               Vec4<float> (&ys)[2][4]) {
    asm volatile(
        "global_load_dword %0, %10, off\n\t"
        "global_load_dword %1, %11, off\n\t"
        "global_load_dwordx4 %2, %12, off\n\t"
        "global_load_dwordx4 %3, %12, off offset:64\n\t"
        "global_load_dwordx4 %4, %12, off offset:128\n\t"
        "global_load_dwordx4 %5, %12, off offset:192\n\t"
        "global_load_dwordx4 %6, %13, off\n\t"
        "global_load_dwordx4 %7, %13, off offset:64\n\t"
        "global_load_dwordx4 %8, %13, off offset:128\n\t"
        "global_load_dwordx4 %9, %13, off offset:192\n\t"
        "s_waitcnt vmcnt(0)"
        : "=&v"(zz[0]), "=&v"(zz[1]), "=&v"(ys[0][0]), "=&v"(ys[0][1]), "=&v"(ys[0][2]),
          "=&v"(ys[0][3]), "=&v"(ys[1][0]), "=&v"(ys[1][1]), "=&v"(ys[1][2]), "=&v"(ys[1][3])
        : "v"(zp[0]), "v"(zp[1]), "v"(yp[0]), "v"(yp[1])
        : "memory");
}

// Copy of one swizzled [N][P] tile (MEMB bytes) from global memory into LDS by
// DMA, issued from inline assembly with a scalar tile base and per-lane byte
// offsets fixed at set-up, so the streaming loop does no vector address work.
// Wave w copies the 1 KiB pieces w, w + 8, ... (or piece w alone when a tile
// has fewer than 8); lane i of a piece lands at piece base + 16 i, which holds
// global chunk (pos ^ (row & 7)) of its row (the tile swizzle is an XOR, its
// own inverse).  Completion is tracked by the wave's vmcnt.
template <int RB, int MEMB>
struct TileDma {
    static constexpr int CPR = RB / 16;
    static constexpr int MASK = (CPR < 8 ? CPR : 8) - 1;
    static constexpr int NI = MEMB / 1024;                      // pieces per tile
    static constexpr int KPW = NI >= kWaves ? NI / kWaves : 1;  // pieces per wave
    static_assert(NI >= kWaves ? NI % kWaves == 0 : true, "pieces must tile the waves");
    uint32_t goff[KPW];
    bool active;
    int wave;
    __device__ void init(int w, int lane) {
        wave = __builtin_amdgcn_readfirstlane(w);
        active = NI >= kWaves || w < NI;
#pragma unroll
        for (int k = 0; k < KPW; ++k) {
            const int q = (w + k * kWaves) * 64 + lane;
            const int row = q / CPR, pos = q % CPR;
            goff[k] = (uint32_t)(row * RB + ((pos ^ (row & MASK)) << 4));
            asm volatile("" : "+v"(goff[k]));
        }
    }
    // copies issued by this wave per tile
    __device__ int count() const { return active ? KPW : 0; }
    __device__ __forceinline__ void issue(const char* gtile, char* ltile) const {
        if (!active) return;
        // readfirstlane returns a signed int: widen through uint32_t so the low
        // half is zero-extended
        const uint64_t gb = (uint64_t)(uintptr_t)gtile;
        const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(gb >> 32));
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)gb);
        const uint64_t base = ((uint64_t)hi << 32) | (uint64_t)lo;
        const uint32_t l0 = (uint32_t)__builtin_amdgcn_readfirstlane(
            (int)(uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)ltile);
#pragma unroll
        for (int k = 0; k < KPW; ++k) {
            const uint32_t m0 =
                (uint32_t)__builtin_amdgcn_readfirstlane((int)(l0 + (uint32_t)((wave + k * kWaves) * 1024)));
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

template <typename T, int N, int S>
__global__ __launch_bounds__(kThreads) void k_sma_regs(
    const T* __restrict__ q, const T* __restrict__ e, const T* __restrict__ Cm,
    const T* __restrict__ mem, const T* __restrict__ kmem, const T* __restrict__ z,
    const T* y_ssd, T* y,
    float* __restrict__ lse, const float* __restrict__ qw, const float* __restrict__ ew, float eps,
    int normalize, int z_per_head, int64_t L, int H, int G, int64_t Mcap, int64_t Mp, int nblk,
    int hpb, int64_t BHC) {
    constexpr int KS = N / 32;
    constexpr int RT = sma_rt<T>();
    constexpr int PT = 16 * RT;                  // tokens per pair
    constexpr int TPB = sma_tokens_per_block<T>();
    constexpr int RB = kP * (int)sizeof(T);      // bytes of one memory row (fixed n)
    constexpr int MEMB = N * RB;                 // bytes of one memory
    constexpr int PIECES = MEMB / 16;            // 16-byte pieces of one memory
    constexpr int PPT = PIECES >= kThreads ? PIECES / kThreads : 1;
    constexpr int RPC = RB / 16;                 // pieces per row
    static_assert(PIECES < kThreads ? kThreads % PIECES == 0 : PIECES % kThreads == 0,
                  "memory pieces must tile the block");
    static_assert(PIECES >= kThreads || PIECES % 64 == 0, "partial copies must be whole waves");
    static_assert(S >= PT, "a pair's tokens must lie in one chunk");
    using Tl = SwzTile<RB>;

    // A block serves `hpb` heads of one projection group (they share q, e and
    // C, loaded once) for one token block, one head after another.
    // Block order.  Workgroups are dealt to the 8 XCDs round-robin by block
    // index, and each XCD has its own L2.  When the number of head groups
    // B*H/hpb is a multiple of 8, XCD x runs only head groups x, x+8, ..., so
    // all blocks reading one head group's memories share one L2.  With one or
    // two groups per XCD they run one group after the other, heaviest first;
    // with more, token blocks go heaviest first over all groups, so that the
    // longest blocks start first and the short ones fill in behind them.
    const int64_t bid = blockIdx.x;
    int blk;
    int64_t bhc;
    if (BHC % 8 == 0) {
        const int64_t slot = bid >> 3, ng8 = BHC >> 3;
        if (ng8 <= 2) {
            // one or two head groups per XCD: one group after the other (its
            // blocks share the L2 while they run; the first group's light
            // blocks meet the second's heavy ones)
            blk = nblk - 1 - (int)(slot % nblk);
            bhc = (slot / nblk) * 8 + (bid & 7);
        } else {
            blk = nblk - 1 - (int)(slot / ng8);
            bhc = (slot % ng8) * 8 + (bid & 7);
        }
    } else {
        blk = nblk - 1 - (int)(bid / BHC);
        bhc = bid % BHC;
    }
    const int hgroups = H / hpb;
    const int64_t b = bhc / hgroups;
    const int h0 = (int)(bhc % hgroups) * hpb;
    const int g = (int)((int64_t)h0 * G / H);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = lane & 15, grp = lane >> 4;
    const bool scorer = wave < 4;
    const int pair = wave & 3;

    const int64_t blk0 = (int64_t)blk * TPB;
    const int64_t pbase = blk0 + pair * PT;                  // first token of the pair
    const int64_t blk_end = (blk0 + TPB < L) ? blk0 + TPB : L;
    const int jmax = (int)((blk_end - 1) / S);              // memories any pair of the block needs
    const bool active = pbase < L;
    const int ip = (int)(pbase / S);                         // the pair's chunk
    const int nj = active ? ip : 0;                          // memories the pair attends

    // LDS: the streamed tiles (see below), the softmax weights (and rescale
    // factors) of the last scored memory per pair, and the final
    // denominators (by head parity).
    constexpr bool kDma = 8 * MEMB + 8192 <= 160 * 1024;  // four (key, value) stages fit
    __shared__ __attribute__((aligned(16))) char st0[2 * MEMB];
    __shared__ __attribute__((aligned(16))) char st1[2 * MEMB];
    __shared__ __attribute__((aligned(16))) char st2[kDma ? 2 * MEMB : 16];
    __shared__ __attribute__((aligned(16))) char st3[kDma ? 2 * MEMB : 16];
    __shared__ float xw[2][4][PT];
    __shared__ float xa[2][4][PT];
    __shared__ int xr[2][4];
    __shared__ float xd[2][4][PT];

    // ---- streaming helpers ---------------------------------------------------
    // The block streams nmem = hpb * jmax memories: index J is memory
    // J % jmax of head h0 + J / jmax.  Indices past the last re-read the last
    // one, so copies are issued on every path and the per-wave count of
    // copies in flight is the same at every wait.  A stage holds the key tile
    // (bytes [0, MEMB)) and the value tile (bytes [MEMB, 2 MEMB)).
    const int nmem = hpb * jmax;
    const char* kbase0 = reinterpret_cast<const char*>(kmem) + (b * Mp * H + h0) * (int64_t)MEMB;
    const char* vbase0 = reinterpret_cast<const char*>(mem) + (b * Mcap * H + h0) * (int64_t)MEMB;
    const int64_t jstride = (int64_t)H * MEMB;
    auto mem_off = [&](int J) {
        const int jj = J < nmem ? J : nmem - 1;
        const int hh = jj / jmax;
        return (int64_t)hh * MEMB + (int64_t)(jj - hh * jmax) * jstride;
    };
    // operand fragments of one 16-column slice (P index pt) of a tile
    auto read_slice = [&](const char* tile, int pt, Frag<T> (&f)[KS]) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            f[ks] = frag_km<T, RB>(tile, ks * 32 + 4 * grp, ks * 32 + 16 + 4 * grp, pt * 16, lane);
    };

    // DMA streaming: step s scores memory s from stage s%4 and accumulates the
    // values of memory s-1 from stage (s-1)%4, while memory s+2 is copied into
    // stage (s+2)%4 (last read in step s-1).  The copies are issued untracked
    // (the compiler would otherwise drain them before every LDS read), and
    // each wave waits for its own copies of memory s+1 before the barrier:
    // vector-memory operations complete in order, so allowing the latest
    // dcnt operations to be outstanding leaves every older copy complete.
    TileDma<RB, MEMB> tdma;
    tdma.init(wave, lane);
    const int dcnt = 2 * tdma.count();  // copies per memory issued by this wave
    auto fetch = [&](int J, char* st) __attribute__((always_inline)) {
        const int64_t off = mem_off(J);
        tdma.issue(kbase0 + off, st);
        tdma.issue(vbase0 + off, st + MEMB);
    };
    auto wait_older = [&]() __attribute__((always_inline)) {
        if (dcnt >= 8) {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(8));
        } else if (dcnt >= 4) {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(4));
        } else if (dcnt >= 2) {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(2));
        }
    };
    static_assert(2 * TileDma<RB, MEMB>::KPW == 2 || 2 * TileDma<RB, MEMB>::KPW == 4 ||
                      2 * TileDma<RB, MEMB>::KPW == 8,
                  "per-wave copy count must be 2, 4 or 8");
    auto stream_dma = [&](auto&& work) {
        wait_older();
        lds_barrier();
        for (int s = 0;; s += 4) {
            fetch(s + 2, st2);
            work(s, st0, st3 + MEMB, 0);
            wait_older();
            lds_barrier();
            if (s + 1 > nmem) break;
            fetch(s + 3, st3);
            work(s + 1, st1, st0 + MEMB, 1);
            wait_older();
            lds_barrier();
            if (s + 2 > nmem) break;
            fetch(s + 4, st0);
            work(s + 2, st2, st1 + MEMB, 0);
            wait_older();
            lds_barrier();
            if (s + 3 > nmem) break;
            fetch(s + 5, st1);
            work(s + 3, st3, st2 + MEMB, 1);
            wait_older();
            lds_barrier();
            if (s + 4 > nmem) break;
        }
    };

    // Register streaming (two stages): memory s+1 is loaded into registers
    // during step s-1 and written to stage (s+1)%2 after step s's work.  Its
    // key tile is needed in step s+1 and its value tile in step s+2, so the
    // value copy of memory s is written one step later than its key copy.
    const bool copier = PIECES >= kThreads || tid < PIECES;
    struct Regs { uint4 k[PPT], v[PPT]; };
    uint32_t loff[PPT];
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
        loff[i] = (uint32_t)(tid + i * kThreads) * 16u;
        // each offset in its own register: every load is a scalar base plus a
        // lane offset
        asm volatile("" : "+v"(loff[i]));
    }
    auto load_regs = [&](int J) {
        Regs r;
        const int64_t off = mem_off(J);
#pragma unroll
        for (int i = 0; i < PPT; ++i) {
            if (copier) {
                r.k[i] = *reinterpret_cast<const uint4*>(kbase0 + off + loff[i]);
                r.v[i] = *reinterpret_cast<const uint4*>(vbase0 + off + loff[i]);
            }
        }
        return r;
    };
    auto put = [&](const uint4 (&src)[PPT], char* tile) {
        if (!copier) return;
#pragma unroll
        for (int i = 0; i < PPT; ++i) {
            const int pc = tid + i * kThreads;
            *reinterpret_cast<uint4*>(tile + Tl::off(pc / RPC, (pc % RPC) * 16)) = src[i];
        }
    };
    Regs r0, r1;
    auto stream_regs = [&](auto&& work) {
        put(r0.k, st0);
        lds_barrier();
        for (int s = 0;; s += 2) {
            work(s, st0, st1 + MEMB, 0);
            put(r0.v, st0 + MEMB);
            put(r1.k, st1);
            r0 = load_regs(s + 2);
            lds_barrier();
            if (s + 1 > nmem) break;
            work(s + 1, st1, st0 + MEMB, 1);
            put(r1.v, st1 + MEMB);
            put(r0.k, st0);
            r1 = load_regs(s + 3);
            lds_barrier();
            if (s + 2 > nmem) break;
        }
    };
    // The first two memories are requested before the token operands, so
    // their latency overlaps the prologue.
    if (nmem > 0) {
        if constexpr (kDma) {
            fetch(0, st0);
            fetch(1, st1);
        } else {
            r0 = load_regs(0);
            r1 = load_regs(1);
        }
    }
    // Both kinds of wave run steps s = 0..nmem and execute the same barriers.
    // The prologue's loads are complete on entry (an explicit wait), so the
    // compiler has no earlier load to wait for inside the loop, where such a
    // wait would also drain the copies in flight.
    auto stream = [&](auto&& work) {
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
        if constexpr (kDma) {
            stream_dma(work);
        } else {
            stream_regs(work);
        }
    };

    // token rows of the pair; rows past the end re-read the last token
    // (their results are zeroed or discarded), so every load is issued up
    // front without branches
    int64_t trow[RT];
    bool tvalid[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const int64_t t = pbase + rt * 16 + col;
        tvalid[rt] = t < L;
        trow[rt] = b * L + (t < L ? t : L - 1);
    }
    const bool hist = ip >= 1;

    if (scorer) {
        // ---- score wave: Qbar and Ebar of the pair's tokens -------------------
        Vec4<T> qraw[RT][KS][2], eraw[RT][4];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const T* qrow = q + (trow[rt] * G + g) * N;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                qraw[rt][ks][0] = ld4(qrow + ks * 32 + 4 * grp);
                qraw[rt][ks][1] = ld4(qrow + ks * 32 + 16 + 4 * grp);
            }
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) eraw[rt][pt] = ld4(e + (trow[rt] * G + g) * kP + pt * 16 + grp * 4);
        }
        Frag<T> qf[RT][KS];
        float ef[RT][4][4];
        const float qscale = kLog2e / sqrtf((float)N);
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const float vmask = tvalid[rt] ? 1.0f : 0.0f;
            float qv[KS][8];
            float ss = 0.f;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    qv[ks][i] = to_f(qraw[rt][ks][0][i]) * vmask;
                    qv[ks][4 + i] = to_f(qraw[rt][ks][1][i]) * vmask;
                }
#pragma unroll
                for (int i = 0; i < 8; ++i) ss += qv[ks][i] * qv[ks][i];
            }
            ss += shfl_xor(ss, 16);
            ss += shfl_xor(ss, 32);
            const float qinv = (normalize ? 1.0f / sqrtf(ss * (1.0f / N) + eps) : 1.0f) * qscale;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
                for (int i = 0; i < 8; ++i) qv[ks][i] *= qinv;
                if (qw) {
                    float w[8];
                    load_kperm(qw, ks, grp, w);
#pragma unroll
                    for (int i = 0; i < 8; ++i) qv[ks][i] *= w[i];
                }
                qf[rt][ks] = make_frag<T>(qv[ks]);
            }
            float es = 0.f;
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    ef[rt][pt][i] = to_f(eraw[rt][pt][i]) * vmask;
                    es += ef[rt][pt][i] * ef[rt][pt][i];
                }
            }
            es += shfl_xor(es, 16);
            es += shfl_xor(es, 32);
            const float einv = normalize ? 1.0f / sqrtf(es * (1.0f / kP) + eps) : 1.0f;
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) {
#pragma unroll
                for (int i = 0; i < 4; ++i) ef[rt][pt][i] *= einv;
                if (ew) {
                    float w[4];
                    load4(ew + pt * 16 + grp * 4, w);
#pragma unroll
                    for (int i = 0; i < 4; ++i) ef[rt][pt][i] *= w[i];
                }
            }
        }
        float m[RT], d[RT];
        // LSE of one head, and its denominators for the value wave
        auto finish_head = [&](int hh) __attribute__((always_inline)) {
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                if (grp == 0) xd[hh & 1][pair][rt * 16 + col] = d[rt];
                if (lse && grp == 0 && tvalid[rt])
                    lse[trow[rt] * H + h0 + hh] = hist ? (m[rt] + log2f(d[rt])) * kLn2 : -INFINITY;
            }
        };
        if (nmem == 0) {
            // no history in this block: LSE = -inf for every head
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) d[rt] = 0.f;
            for (int hh = 0; hh < hpb; ++hh) finish_head(hh);
            return;
        }
        stream([&](int s, const char* kt, const char*, int buf) {
            if (s >= nmem) return;
            const int hh = s / jmax, j = s - hh * jmax;
            if (j == 0) {
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) {
                    m[rt] = -INFINITY;
                    d[rt] = 0.f;
                }
            }
            if (j < nj) {
                // U^T slices: fragments of slice pt+1 are requested before the
                // MFMAs of slice pt
                Frag<T> fb[2][KS];
                read_slice(kt, 0, fb[0]);
                float lp[RT];
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) lp[rt] = 0.f;
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) {
                    if (pt < 3) read_slice(kt, pt + 1, fb[(pt + 1) & 1]);
                        f32x4 u[RT];
#pragma unroll
                    for (int rt = 0; rt < RT; ++rt) u[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
                        for (int rt = 0; rt < RT; ++rt) u[rt] = mma16(u[rt], fb[pt & 1][ks], qf[rt][ks]);
#pragma unroll
                    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                        for (int i = 0; i < 4; ++i) lp[rt] += u[rt][i] * ef[rt][pt][i];
                    }
                // full logit of the lane's token: sum the 4 lanes sharing its
                // column with one fp32 MFMA against a ones matrix
                // (D[i][t] = sum_k B[k][t])
                bool grow = false;
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) {
                    const f32x4 red = __builtin_amdgcn_mfma_f32_16x16x4f32(
                        1.0f, lp[rt], f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                    lp[rt] = red[0];
                    grow |= lp[rt] > m[rt] + kRescaleLog2;
                }
                // lazy rescale: the reference maximum only moves when a logit
                // exceeds it by more than 2^8, so weights stay <= 256 and O is
                // rescaled rarely; R = O/d and LSE = m + log2 d do not depend on
                // the choice of m
                const bool rescale = __builtin_amdgcn_ballot_w64(grow) != 0;
                if (rescale) {
#pragma unroll
                    for (int rt = 0; rt < RT; ++rt) {
                        const float mn = fmaxf(m[rt], lp[rt]);
                        const float al = fast_exp2(m[rt] - mn);
                        d[rt] *= al;
                        m[rt] = mn;
                        if (grp == 0) xa[buf][pair][rt * 16 + col] = al;
                    }
                }
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) {
                    const float pw = fast_exp2(lp[rt] - m[rt]);
                    d[rt] += pw;
                    if (grp == 0) xw[buf][pair][rt * 16 + col] = pw;
                }
                if (lane == 0) xr[buf][pair] = rescale ? 1 : 0;
            }
            if (j == jmax - 1) finish_head(hh);
        });
    } else {
        // ---- value wave: C of the pair's tokens, accumulator O ----------------
        Frag<T> cf[RT][KS];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const T* crow = Cm + (trow[rt] * G + g) * N;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                cf[rt][ks] = cat_frag<T>(ld4(crow + ks * 32 + 4 * grp), ld4(crow + ks * 32 + 16 + 4 * grp));
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            if (!tvalid[rt]) {
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) cf[rt][ks] = Frag<T>{};
            }
        }
        f32x4 o[RT][4];
        // y = y_ssd + SiLU(z) R of one head
        auto finish_head = [&](int hh) __attribute__((always_inline)) {
            const int h = h0 + hh;
            const T* zp[RT];
            const T* yp[RT];
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                zp[rt] = z_per_head ? z + trow[rt] * H + h : z + trow[rt];
                yp[rt] = y_ssd + (trow[rt] * H + h) * kP + grp * 4;
            }
            float zz[RT];
            Vec4<T> ys[RT][4];
            load_epilogue_inputs<T, RT>(zp, yp, zz, ys);
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                if (!tvalid[rt]) continue;
                const float gate = silu(zz[rt]);
                const float invd = hist ? 1.0f / xd[hh & 1][pair][rt * 16 + col] : 0.f;
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) {
                    float yv[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) yv[i] = to_f(ys[rt][pt][i]);
                    if (hist) {
#pragma unroll
                        for (int i = 0; i < 4; ++i) yv[i] += gate * (o[rt][pt][i] * invd);
                    }
                    store4(y + (trow[rt] * H + h) * kP + pt * 16 + grp * 4, yv);
                }
            }
        };
        if (nmem == 0) {
            // no history in this block: y = y_ssd for every head
            for (int hh = 0; hh < hpb; ++hh) finish_head(hh);
            return;
        }
        stream([&](int s, const char*, const char* vt, int buf) {
            // memory s-1, scored in the previous step (weights in slot buf^1)
            if (s < 1) return;
            const int hh = (s - 1) / jmax, j = (s - 1) - hh * jmax;
            if (j == 0) {
#pragma unroll
                for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                    for (int pt = 0; pt < 4; ++pt) o[rt][pt] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
            if (j < nj) {
                const int wb = buf ^ 1;
                // flag and weights first: LDS reads return in order, so the
                // flag test does not wait for the fragment reads
                const int rescale = __builtin_amdgcn_readfirstlane(xr[wb][pair]);
                float pw[RT];
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) pw[rt] = xw[wb][pair][rt * 16 + col];
                Frag<T> fb[2][KS];
                read_slice(vt, 0, fb[0]);
                if (rescale) {
#pragma unroll
                    for (int rt = 0; rt < RT; ++rt) {
                        const float al = xa[wb][pair][rt * 16 + col];
#pragma unroll
                        for (int pt = 0; pt < 4; ++pt) o[rt][pt] *= al;
                    }
                }
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) {
                    if (pt < 3) read_slice(vt, pt + 1, fb[(pt + 1) & 1]);
                        f32x4 v[RT];
#pragma unroll
                    for (int rt = 0; rt < RT; ++rt) v[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
                        for (int rt = 0; rt < RT; ++rt) v[rt] = mma16(v[rt], fb[pt & 1][ks], cf[rt][ks]);
#pragma unroll
                    for (int rt = 0; rt < RT; ++rt) o[rt][pt] += pw[rt] * v[rt];
                    }
            }
            // the head's last memory is in: its denominators were published
            // in the previous step
            if (j == jmax - 1) finish_head(hh);
        });
    }
}

// ---------------------------------------------------------------------------
// bf16 streaming kernel.
//
// Same work split as above (8 waves = 4 (score, value) pairs of 64 tokens, four
// heads of one group per block, one continuous stream of memories), with the
// value wave two steps behind the score wave:
//   step s  score waves  MFMAs of memory s (key tile), and before them the
//                        softmax tail of memory s-1: the last P-slice of its
//                        logit sums, the reduction over the four lanes of a
//                        column (gfx950 row-swap moves), the online-softmax
//                        update and the weights of s-1 written to LDS;
//           value waves  memory s-2: V^T = dH^T C^T on MFMA, O = alpha O + w V;
//                        before the barrier they already read the first
//                        operand fragments of memory s-1;
//           all waves    DMA of memory s+2 (key tile into a 3-stage ring,
//                        value tile into a 5-stage ring).
// So the softmax tail runs while the score wave's first fragment reads are in
// flight and the value waves have MFMA work ready when the barrier opens.
// Operand fragments are read PD fragments ahead of their MFMAs; scheduling
// barriers keep the compiler from sinking the reads next to their use.
// ---------------------------------------------------------------------------

// Reduce-scatter over the four lanes l, l^16, l^32, l^48 that hold one column
// of a 16x16 MFMA accumulator: v0..v3 are the lane's partial sums for column
// tiles 0..3, and the result in 16-lane row g of the wave is the full sum for
// tile g.  v_permlane32_swap exchanges lanes 32..63 of its first operand with
// lanes 0..31 of its second, so after swapping (v0, v2) the sum v0 + v2 holds
// tile 0 over lanes {l, l^32} in the lower half and tile 2 in the upper half
// (likewise v1 + v3 for tiles 1 and 3); v_permlane16_swap then exchanges the
// odd 16-lane rows of its first operand with the even rows of its second, and
// one more sum completes each row's tile.  Issued from assembly: the builtins
// return the second operand unchanged in this compiler.
__device__ __forceinline__ float col_reduce_scatter4(float v0, float v1, float v2, float v3) {
    asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(v0), "+v"(v2));
    asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(v1), "+v"(v3));
    float sa = v0 + v2, sb = v1 + v3;
    asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(sa), "+v"(sb));
    return sa + sb;
}

// s_waitcnt vmcnt(k) for the per-wave copy counts that occur (0, 2, 4 or 8).
__device__ __forceinline__ void wait_vm(int k) {
    if (k >= 8) {
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(8));
    } else if (k >= 4) {
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(4));
    } else if (k >= 2) {
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(2));
    } else {
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    }
}

// Key and value sides of every attended memory for the bf16 kernel, both
// transposed to [P][N]: kT[p][n] = r[n] dH[n][p] (rounded to bf16) and
// vT[p][n] = dH[n][p], with r[n] = (mean_p dH[n,p]^2 + eps)^-1/2 reduced from
// the stored values.  Rows of N consecutive n put the contraction index of
// both SMA products in consecutive bytes, so k_sma reads every MFMA operand
// fragment with one 16-byte LDS load.  The tile is staged in LDS in the
// swizzled row layout; two transposing reads then hand each lane 8
// consecutive n of one p (one 16-byte piece of an output row).  The RPC lanes
// holding one source row reduce its sum of squares with DPP moves.
template <int N>
__global__ __launch_bounds__(256) void k_sma_prep(const bf16* __restrict__ mem,
                                                  bf16* __restrict__ kT, bf16* __restrict__ vT,
                                                  float eps, int normalize, int H, int64_t Mp,
                                                  int64_t Mcap) {
    constexpr int RB = kP * 2;            // bytes of one source row (fixed n)
    constexpr int RPC = RB / 16;          // 16-byte pieces per source row
    constexpr int PIECES = N * RPC;       // 16-byte pieces of one memory
    constexpr int NG = N / 32;            // 32-row bands of the output pieces
    static_assert(PIECES % 256 == 0 || 256 % PIECES == 0, "pieces must tile the block");
    using Tl = SwzTile<RB>;
    const int64_t j = blockIdx.x;
    const int h = blockIdx.y;
    const int64_t b = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    __shared__ __attribute__((aligned(16))) char t[N * RB];
    __shared__ float rs[N];
    // the memories are read once here (streaming loads); the transposed
    // sides are written with ordinary stores so the attention kernel that
    // follows finds them in the caches
    const u32x4_nt* src = reinterpret_cast<const u32x4_nt*>(mem + ((b * Mcap + j) * H + h) * (int64_t)N * kP);
    for (int q = tid; q < PIECES; q += 256) {
        const u32x4_nt vn = __builtin_nontemporal_load(src + q);
        const uint4 v = make_uint4(vn[0], vn[1], vn[2], vn[3]);
        const int n = q / RPC, pc = q % RPC;
        const float ss = dpp_group_sum<RPC>(piece_sumsq(v, bf16()));
        if (pc == 0) rs[n] = normalize ? __builtin_amdgcn_rsqf(ss * (1.0f / kP) + eps) : 1.0f;
        *reinterpret_cast<uint4*>(t + Tl::off(n, pc * 16)) = v;
    }
    __syncthreads();
    // piece w of the 4 NG pieces per wave: columns p = 16 (w % 4) + (lane % 16),
    // rows n = 32 (w / 4) + 8 (lane / 16) .. +7
    const int64_t obase = ((b * Mp + j) * H + h) * (int64_t)N * kP;
    const int g = lane >> 4, c = lane & 15;
    for (int w = wave; w < 4 * NG; w += 4) {
        const int pbase = 16 * (w & 3), nb = 32 * (w >> 2) + 8 * g;
        const bf16x8 v = frag_kmajor_bf16<RB>(t, nb, nb + 4, pbase, lane);
        bf16x8 k;
#pragma unroll
        for (int i = 0; i < 8; ++i) k[i] = (bf16)((float)v[i] * rs[nb + i]);
        const int64_t o = obase + (int64_t)(pbase + c) * N + nb;
        *reinterpret_cast<bf16x8*>(vT + o) = v;
        *reinterpret_cast<bf16x8*>(kT + o) = k;
    }
}

// DMA of one [P][N] bf16 tile (P = 64 rows of RB = 2N bytes) into an LDS tile
// whose 16-byte chunks are XOR-swizzled by row: chunk c of row p sits at
// c ^ key(p), key(p) = (p RB / 256) mod (RB / 16).  The 16 lanes of one
// 16-byte fragment read (rows 16 pt + 0..15, one logical chunk) then cover
// all 64 banks.  Issued from inline assembly with a scalar tile base and
// per-lane offsets fixed at set-up, as TileDma.
template <int N, int NW>
struct TileDmaPN {
    static constexpr int RB = 2 * N;
    static constexpr int CPR = RB / 16;
    static constexpr int MEMB = kP * RB;
    static constexpr int NI = MEMB / 1024;                      // 1 KiB pieces per tile
    static constexpr int KPW = NI >= NW ? NI / NW : 1;  // pieces per issuing wave
    static_assert(NI >= NW ? NI % NW == 0 : true, "pieces must tile the waves");
    __host__ __device__ static constexpr int key(int row) { return (row * RB / 256) & (CPR - 1); }
    uint32_t goff[KPW];
    bool active;
    int wave;
    __device__ void init(int w, int lane) {
        wave = __builtin_amdgcn_readfirstlane(w);
        active = w < NW && (NI >= NW || w < NI);
#pragma unroll
        for (int k = 0; k < KPW; ++k) {
            const int q = (w + k * NW) * 64 + lane;
            const int row = q / CPR, pos = q % CPR;
            goff[k] = (uint32_t)(row * RB + ((pos ^ key(row)) << 4));
            asm volatile("" : "+v"(goff[k]));
        }
    }
    __device__ int count() const { return active ? KPW : 0; }
    __device__ __forceinline__ void issue(const char* gtile, char* ltile) const {
        if (!active) return;
        const uint64_t gb = (uint64_t)(uintptr_t)gtile;
        const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(gb >> 32));
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)gb);
        const uint64_t base = ((uint64_t)hi << 32) | (uint64_t)lo;
        const uint32_t l0 = (uint32_t)__builtin_amdgcn_readfirstlane(
            (int)(uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)ltile);
#pragma unroll
        for (int k = 0; k < KPW; ++k) {
            const uint32_t m0 =
                (uint32_t)__builtin_amdgcn_readfirstlane((int)(l0 + (uint32_t)((wave + k * NW) * 1024)));
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

template <int N, int S>
__global__ __launch_bounds__(kThreads) void k_sma(
    const bf16* __restrict__ q, const bf16* __restrict__ e, const bf16* __restrict__ Cm,
    const bf16* __restrict__ vT, const bf16* __restrict__ kT, const bf16* __restrict__ z,
    const bf16* y_ssd, bf16* y, float* __restrict__ lse, const float* __restrict__ qw,
    const float* __restrict__ ew, float eps, int normalize, int z_per_head, int64_t L, int H, int G,
    int64_t Mp, int nblk, int hpb, int64_t BHC) {
    using T = bf16;
    constexpr int KS = N / 32;
    constexpr int RT = 4;                    // 16-token column tiles per pair
    constexpr int PT = 16 * RT;              // tokens per pair
    constexpr int TPB = 4 * PT;              // tokens per block
    constexpr int RB = 2 * N;                // bytes of one [P][N] tile row (fixed p)
    constexpr int MEMB = kP * RB;            // bytes of one memory
    constexpr int NF = 4 * KS;               // operand fragments per tile (4 P-slices)
    constexpr int PD = 3;                    // fragments read ahead
    constexpr int KST = 3, VST = 4;          // key and value ring stages
    constexpr int YB = PT * kP * 2;          // bytes of a pair's y_ssd tile (bf16)
    static_assert(S >= PT, "a pair's tokens must lie in one chunk");
    static_assert(NF >= 4, "at least one fragment per slice");
    using Dma = TileDmaPN<N, 4>;  // the score waves issue all copies

    // block order: as in k_sma_regs (XCD-aware, heaviest token block first)
    const int64_t bid = blockIdx.x;
    int blk;
    int64_t bhc;
    if (BHC % 8 == 0) {
        const int64_t slot = bid >> 3, ng8 = BHC >> 3;
        if (ng8 <= 2) {
            // one or two head groups per XCD: one group after the other (its
            // blocks share the L2 while they run; the first group's light
            // blocks meet the second's heavy ones)
            blk = nblk - 1 - (int)(slot % nblk);
            bhc = (slot / nblk) * 8 + (bid & 7);
        } else {
            blk = nblk - 1 - (int)(slot / ng8);
            bhc = (slot % ng8) * 8 + (bid & 7);
        }
    } else {
        blk = nblk - 1 - (int)(bid / BHC);
        bhc = bid % BHC;
    }
    const int hgroups = H / hpb;
    const int64_t b = bhc / hgroups;
    const int h0 = (int)(bhc % hgroups) * hpb;
    const int g = (int)((int64_t)h0 * G / H);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: role branches are scalar
    const int col = lane & 15, grp = lane >> 4;
    const bool scorer = wave < 4;
    const int pair = wave & 3;

    const int64_t blk0 = (int64_t)blk * TPB;
    const int64_t pbase = blk0 + pair * PT;
    const int64_t blk_end = (blk0 + TPB < L) ? blk0 + TPB : L;
    const int jmax = (int)((blk_end - 1) / S);
    const bool active = pbase < L;
    const int ip = (int)(pbase / S);
    const int nj = active ? ip : 0;
    const bool hist = ip >= 1;
    const int nmem = hpb * jmax;

    __shared__ __attribute__((aligned(16))) char kring[KST * MEMB];
    __shared__ __attribute__((aligned(16))) char vring[VST * MEMB];
    __shared__ float xw[2][4][PT];
    __shared__ float xa[2][4][PT];
    __shared__ int xr[2][4];
    __shared__ float xd[2][4][PT];
    __shared__ __attribute__((aligned(16))) char ybuf[4 * YB];  // epilogue y_ssd, per pair
    __shared__ uint32_t zbuf[4][PT];                            // epilogue z, per pair

    // ---- memory stream: DMA of whole tiles, each wave its fixed pieces -------
    const char* kbase0 = reinterpret_cast<const char*>(kT) + (b * Mp * H + h0) * (int64_t)MEMB;
    const char* vbase0 = reinterpret_cast<const char*>(vT) + (b * Mp * H + h0) * (int64_t)MEMB;
    const int64_t jstride = (int64_t)H * MEMB;
    Dma tdma;
    tdma.init(wave, lane);
    const int tcnt = tdma.count();      // copies per tile issued by this wave
    // next key and value tiles to copy (memory order: index within a head,
    // then head), as tile addresses advanced by a stride or, at a head's last
    // memory, back to the next head's first one
    const char* kp = kbase0;
    const char* vp = vbase0;
    int kj = 0, vj = 0;
    const int64_t hstep = (int64_t)MEMB - (int64_t)(jmax - 1) * jstride;
    auto advance = [&](const char*& p, int& j) __attribute__((always_inline)) {
        if (++j == jmax) {
            j = 0;
            p += hstep;
        } else {
            p += jstride;
        }
    };
    auto fetch_k = [&](int st) __attribute__((always_inline)) {
        tdma.issue(kp, kring + st * MEMB);
        advance(kp, kj);
    };
    auto fetch_v = [&](int st) __attribute__((always_inline)) {
        tdma.issue(vp, vring + st * MEMB);
        advance(vp, vj);
    };
    if (nmem > 0) {
        fetch_k(0);
        fetch_v(0);
    }
    if (nmem > 1) fetch_k(1);

    // Operand fragment (slice pt, k step ks) of a [P][N] tile: lane (grp, col)
    // takes row p = 16 pt + col, n = 32 ks + 8 grp .. +7, one 16-byte read.
    // Its byte offset is 16 pt RB + koff[ks], koff[ks] = col RB + (chunk ^ key) 16
    // with chunk 4 ks + grp (key(16 pt + col) does not depend on pt).
    uint32_t koff[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
        koff[ks] = (uint32_t)(col * RB + (((4 * ks + grp) ^ Dma::key(col)) << 4));
    auto frag = [&](const char* tile, int f) __attribute__((always_inline)) {
        return *reinterpret_cast<const bf16x8*>(tile + (f / KS) * 16 * RB + koff[f % KS]);
    };

    // token rows of the pair; rows past the end re-read the last token
    int64_t trow[RT];
    bool tvalid[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const int64_t t = pbase + rt * 16 + col;
        tvalid[rt] = t < L;
        trow[rt] = b * L + (t < L ? t : L - 1);
    }

    // One P-slice pt of a tile product: for each k step, the operand fragment
    // PD ahead is requested, then four MFMAs (one per 16-token column tile)
    // accumulate into acc; fma(rt) (four VALU ops on the previous slice's
    // results) is applied for the column tiles assigned to the k step.  The
    // scheduling groups interleave the MFMAs with that VALU work.  The VALU
    // work starts at the second k step, so the MFMAs that produced its inputs
    // were issued at least seven MFMAs earlier and have completed.
    auto fma_lo = [](int ks) { return KS == 1 ? 0 : KS == 2 ? (ks == 1 ? 0 : RT) : ks == 1 ? 0 : ks == 2 ? RT / 2 : RT; };
    auto fma_hi = [](int ks) { return KS == 1 ? RT : KS == 2 ? (ks == 1 ? RT : 0) : ks == 1 ? RT / 2 : ks == 2 ? RT : 0; };
    auto slice_region = [&](Frag<T> (&fr)[4], const char* tile, int pt, f32x4 (&acc)[RT],
                            const Frag<T> (&bop)[RT][KS], auto&& fma) __attribute__((always_inline)) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (KS > 1 && ks == 1) __builtin_amdgcn_sched_barrier(0);
            const int f = pt * KS + ks;
            if (f + PD < NF) fr[(f + PD) & 3] = frag(tile, f + PD);
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
                acc[rt] = mma16(ks == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : acc[rt], fr[f & 3], bop[rt][ks]);
#pragma unroll
            for (int r = fma_lo(ks); r < fma_hi(ks); ++r) fma(r);
        }
        // interleave pattern of the region that holds the VALU work
        if constexpr (KS == 1) {
#pragma unroll
            for (int m = 0; m < RT; ++m) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
            }
        } else {
#pragma unroll
            for (int ks = 1; ks < KS; ++ks) {
                if (pt * KS + ks + PD < NF) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
                for (int m = 0; m < RT; ++m) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    if (KS == 2) {
                        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
                    } else if (ks <= 2) {
                        __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
                    }
                }
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    };

    // One step of the stream for every wave: the wave's work, then the copies
    // of the key tile of memory s+2 and the value tile of memory s+1 (the
    // score waves issue all copies; issued after the work rather than before
    // it, they do not hold up the step's first MFMAs, and one step still
    // covers their latency: 3-5 % faster at every measured shape), barrier.
    // Memory s is scored at step s and its value tile
    // consumed at step s+2 (first fragments read at the end of step s+1), so
    // three key stages and four value stages suffice.  Score waves wait for
    // every copy but this step's and make their LDS writes (the softmax
    // weights) complete before the barrier; value waves write LDS only
    // through their own epilogue copies, which they wait for themselves, and
    // cross the barrier with their reads of the next step's first fragments
    // still in flight (a compiler-level barrier keeps every LDS access on its
    // side of it).
    auto run_stream = [&](auto&& work) __attribute__((always_inline)) {
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));  // prologue loads and first tiles
        lds_barrier();
        int kc = 0, vc = 0;                        // s % KST, s % VST
        for (int s = 0; s < nmem + 2; ++s) {
            const bool kcopy = s + 2 < nmem, vcopy = s + 1 < nmem;
            work(s, kc, vc);
            if (kcopy) fetch_k(kc == 0 ? 2 : kc - 1);
            if (vcopy) fetch_v(vc == VST - 1 ? 0 : vc + 1);
            if (scorer) {
                if (kcopy) {
                    wait_vm(2 * tcnt);
                } else if (vcopy) {
                    wait_vm(tcnt);
                } else {
                    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
                }
                lds_barrier();
            } else {
                asm volatile("s_barrier" ::: "memory");
            }
            kc = kc == KST - 1 ? 0 : kc + 1;
            vc = vc == VST - 1 ? 0 : vc + 1;
        }
    };

    if (scorer) {
        // ---- score wave: Qbar and Ebar of the pair's tokens -------------------
        Frag<T> qraw[RT][KS];
        Vec4<T> eraw[RT][4];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const T* qrow = q + (trow[rt] * G + g) * N;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) qraw[rt][ks] = load_frag(qrow + ks * 32 + 8 * grp);
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) eraw[rt][pt] = ld4(e + (trow[rt] * G + g) * kP + pt * 16 + grp * 4);
        }
        Frag<T> qf[RT][KS];
        float ef[RT][4][4];
        const float qscale = kLog2e / sqrtf((float)N);
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const float vmask = tvalid[rt] ? 1.0f : 0.0f;
            float qv[KS][8];
            float ss = 0.f;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
                for (int i = 0; i < 8; ++i) qv[ks][i] = to_f(qraw[rt][ks][i]) * vmask;
#pragma unroll
                for (int i = 0; i < 8; ++i) ss += qv[ks][i] * qv[ks][i];
            }
            ss += shfl_xor(ss, 16);
            ss += shfl_xor(ss, 32);
            const float qinv = (normalize ? 1.0f / sqrtf(ss * (1.0f / N) + eps) : 1.0f) * qscale;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
                for (int i = 0; i < 8; ++i) qv[ks][i] *= qinv;
                if (qw) {
                    float w[8];
                    load8(qw + ks * 32 + 8 * grp, w);
#pragma unroll
                    for (int i = 0; i < 8; ++i) qv[ks][i] *= w[i];
                }
                qf[rt][ks] = make_frag<T>(qv[ks]);
            }
            float es = 0.f;
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    ef[rt][pt][i] = to_f(eraw[rt][pt][i]) * vmask;
                    es += ef[rt][pt][i] * ef[rt][pt][i];
                }
            }
            es += shfl_xor(es, 16);
            es += shfl_xor(es, 32);
            const float einv = normalize ? 1.0f / sqrtf(es * (1.0f / kP) + eps) : 1.0f;
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) {
#pragma unroll
                for (int i = 0; i < 4; ++i) ef[rt][pt][i] *= einv;
                if (ew) {
                    float w[4];
                    load4(ew + pt * 16 + grp * 4, w);
#pragma unroll
                    for (int i = 0; i < 4; ++i) ef[rt][pt][i] *= w[i];
                }
            }
        }
        // After the reduction, lane (grp, col) owns token 16 grp + col of the
        // pair (column tile grp): its running maximum and denominator.
        const int64_t t_own = pbase + grp * 16 + col;
        const bool own_valid = t_own < L;
        const int64_t own_row = b * L + (own_valid ? t_own : L - 1);
        float m_own = -INFINITY, d_own = 0.f;
        // LSE of one head, and its denominators for the value wave
        auto finish_head = [&](int hh) __attribute__((always_inline)) {
            xd[hh & 1][pair][lane] = d_own;
            if (lse && own_valid)
                lse[own_row * H + h0 + hh] = hist ? (m_own + log2f(d_own)) * kLn2 : -INFINITY;
        };
        if (nmem == 0) {
            for (int hh = 0; hh < hpb; ++hh) finish_head(hh);
            return;
        }
        f32x4 u[2][RT];           // U^T slice accumulators (slice parity)
        float lp[RT];             // logit partial sums of the memory being scored
        Frag<T> fr[4];            // fragment ring
        int jm = 0;               // index within its head of memory s
        int hm = 0;               // head of memory s
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) u[1][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
        // partial logit sums of slice pt (in u[pt & 1]) for column tile rt
        auto lp_fma = [&](int pt, int rt) __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < 4; ++i) lp[rt] += u[pt & 1][rt][i] * ef[rt][pt][i];
        };
        run_stream([&](int s, int kc, int) __attribute__((always_inline)) {
            // memory s is scored by this wave iff mmi < 0 (a scalar integer, so
            // the flag never takes a lane-mask round trip between its uses)
            int mmi = (s - nmem) & (jm - nj);
            asm("" : "+s"(mmi));
            const bool mm = mmi < 0;
            // memory s-1 was scored by this wave
            const bool tail_pending = s >= 1 && s <= nmem && (jm == 0 ? jmax - 1 : jm - 1) < nj;
            const char* kt = kring + kc * MEMB;
            // slice 0 of memory s, with the last slice's logit sums of memory s-1
            if (mm) {
#pragma unroll
                for (int f = 0; f < PD; ++f) fr[f] = frag(kt, f);
                slice_region(fr, kt, 0, u[0], qf, [&](int rt) { lp_fma(3, rt); });
            } else if (tail_pending) {
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) lp_fma(3, rt);
            }
            // ---- softmax tail of memory s-1 --------------------------------------
            if (tail_pending) {
                const float l = col_reduce_scatter4(lp[0], lp[1], lp[2], lp[3]);
                // lazy rescale: the reference maximum moves only when a logit
                // exceeds it by more than 2^8; R = O/d and LSE = m + log2 d do
                // not depend on that choice
                const bool rescale = __builtin_amdgcn_ballot_w64(l > m_own + kRescaleLog2) != 0;
                const int slot = (s - 1) & 1;
                // the factor for O is needed (and written) only when the
                // maximum moves; otherwise it is exactly 1
                float al = 1.0f;
                if (rescale) {
                    const float mn = fmaxf(m_own, l);
                    al = fast_exp2(m_own - mn);
                    m_own = mn;
                    xa[slot][pair][lane] = al;
                }
                const float pw = fast_exp2(l - m_own);
                d_own = d_own * al + pw;
                xw[slot][pair][lane] = pw;
                if (lane == 0) xr[slot][pair] = rescale ? 1 : 0;
            }
            // the head of memory s-1 is complete
            if (s >= 1 && s <= nmem && jm == 0) {
                finish_head(hm - 1);
                m_own = -INFINITY;
                d_own = 0.f;
            }
            // (the sums restart every step, so no step carries them into a
            // step that does not score)
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) lp[rt] = 0.f;
            asm("" : "+s"(mmi));
            if (mmi < 0) {
                // ---- U^T = (r (.) dH_s)^T Qbar^T, slices 1..3; each slice's
                // MFMAs are interleaved with the logit sums of the slice before
#pragma unroll
                for (int pt = 1; pt < 4; ++pt)
                    slice_region(fr, kt, pt, u[pt & 1], qf, [&](int rt) { lp_fma(pt - 1, rt); });
            }
            // (jm, hm) advance in scalar registers
            asm("s_add_i32 %0, %0, 1\n\t"
                "s_cmp_eq_u32 %0, %2\n\t"
                "s_cselect_b32 %0, 0, %0\n\t"
                "s_addc_u32 %1, %1, 0"
                : "+s"(jm), "+s"(hm)
                : "s"(jmax)
                : "scc");
        });
    } else {
        // ---- value wave: C of the pair's tokens, accumulator O ----------------
        Frag<T> cf[RT][KS];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const T* crow = Cm + (trow[rt] * G + g) * N;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                cf[rt][ks] = load_frag(crow + ks * 32 + 8 * grp);
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            if (!tvalid[rt]) {
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) cf[rt][ks] = Frag<T>{};
            }
        }
        f32x4 o[RT][4];
        // Epilogue inputs of head hh (the pair's y_ssd rows and gates) are
        // copied into the pair's LDS buffers a step before the head's last
        // memory is consumed, so their latency hides behind that step.  y_ssd
        // row r (64 bf16, eight 16-byte chunks) goes to ybuf row r with chunk c
        // in slot c ^ (r & 7): copy k moves rows 8k .. 8k+7, lane l taking row
        // 8k + l/8 and slot l % 8.  The gate of token r is one 16-bit copy into
        // the 4-byte slot r of zbuf.  Rows past the end re-read the last token.
        char* const yb = ybuf + pair * YB;
        const int lastr = (int)((L - 1 - pbase < PT - 1) ? L - 1 - pbase : PT - 1);
        const int64_t zstride = z_per_head ? H : 1;
        auto prefetch_epilogue = [&](int hh) __attribute__((always_inline)) {
            if (!active) return;  // no token of the pair exists
            const int h = h0 + hh;
            const uint64_t yg = (uint64_t)(uintptr_t)(y_ssd + ((b * L + pbase) * H + h) * kP);
            const uint64_t zg = (uint64_t)(uintptr_t)(z + (b * L + pbase) * zstride + (z_per_head ? h : 0));
            const uint64_t ybase = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(yg >> 32)) << 32) |
                                   (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)yg);
            const uint64_t zbase = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(zg >> 32)) << 32) |
                                   (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)zg);
            const uint32_t lb = (uint32_t)__builtin_amdgcn_readfirstlane(
                (int)(uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)yb);
            const uint32_t lz = (uint32_t)__builtin_amdgcn_readfirstlane(
                (int)(uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)&zbuf[pair][0]);
            // per-lane offsets are recomputed at each use (the empty asm keeps
            // the compiler from hoisting them out of the stream)
            int ln = lane;
            asm volatile("" : "+v"(ln));
            const uint32_t rowb = (uint32_t)(H * kP * 2);
            const uint32_t slot = (uint32_t)(((ln & 7) ^ (ln >> 3)) << 4);
#pragma unroll
            for (int k = 0; k < PT / 8; ++k) {
                const int r = 8 * k + (ln >> 3);
                const uint32_t off = (uint32_t)(r < lastr ? r : lastr) * rowb + slot;
                const uint32_t m0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)(lb + (uint32_t)(k * 1024)));
                uint32_t save;
                asm volatile(
                    "s_mov_b32 %0, m0\n\t"
                    "s_mov_b32 m0, %3\n\t"
                    "s_nop 0\n\t"
                    "global_load_lds_dwordx4 %1, %2\n\t"
                    "s_mov_b32 m0, %0"
                    : "=&s"(save)
                    : "v"(off), "s"(ybase), "s"(m0)
                    : "memory");
            }
            {
                const uint32_t off = (uint32_t)((ln < lastr ? ln : lastr) * zstride * 2);
                uint32_t save;
                asm volatile(
                    "s_mov_b32 %0, m0\n\t"
                    "s_mov_b32 m0, %3\n\t"
                    "s_nop 0\n\t"
                    "global_load_lds_ushort %1, %2\n\t"
                    "s_mov_b32 m0, %0"
                    : "=&s"(save)
                    : "v"(off), "s"(zbase), "s"(lz)
                    : "memory");
            }
        };
        // y = y_ssd + silu(z) R for head hh, R = O / d, once its copies landed
        auto finish_head = [&](int hh) __attribute__((always_inline)) {
            const int h = h0 + hh;
            int c = col, gq = grp;
            asm volatile("" : "+v"(c), "+v"(gq));
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                const int r = rt * 16 + c;
                const int64_t t = pbase + r;
                if (t >= L) continue;
                // SiLU(z) / d folded into one factor per token, both
                // reciprocals by the hardware rcp (the epilogue's IEEE divides
                // and separate products had made it cost about one stream step
                // per head)
                const float zv = __builtin_bit_cast(float, zbuf[pair][r] << 16);
                const float gd = hist ? zv * __builtin_amdgcn_rcpf(1.0f + __expf(-zv)) *
                                            __builtin_amdgcn_rcpf(xd[hh & 1][pair][r])
                                      : 0.f;
                bf16* yrow = y + ((b * L + t) * H + h) * kP + gq * 4;
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) {
                    const Vec4<T> ys = *reinterpret_cast<const Vec4<T>*>(
                        yb + r * (kP * 2) + ((((2 * pt + (gq >> 1)) ^ (c & 7))) << 4) + (gq & 1) * 8);
                    float yv[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) yv[i] = to_f(ys[i]);
                    if (hist) {
#pragma unroll
                        for (int i = 0; i < 4; ++i) yv[i] = fmaf(gd, o[rt][pt][i], yv[i]);
                    }
                    store4(yrow + pt * 16, yv);
                }
            }
        };
        if (nmem == 0) {
            for (int hh = 0; hh < hpb; ++hh) {
                prefetch_epilogue(hh);
                finish_head(hh);
            }
            return;
        }
        // index of the memory at whose step a head's epilogue copies start
        const int jpf = jmax >= 2 ? jmax - 2 : 0;
        Frag<T> fr[4];             // fragment ring; the first PD of the next step's
                                   // memory are read before the barrier
        int jv = 0, hv = 0;        // (index, head) of memory s-2
        f32x4 v[2][RT];            // V^T slice accumulators (slice parity)
        float pwp[RT];             // weights of the memory whose last slice is pending
        bool pend = false;         // o[.][3] += pwp v[1] is still to be applied
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            v[1][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
            pwp[rt] = 0.f;
        }
        // memory J's value tile sits in stage J % VST; at step s, J = s-2 is in
        // stage (vc + 2) % 4 and the next step's memory s-1 in (vc + 3) % 4
        run_stream([&](int s, int, int vc) __attribute__((always_inline)) {
            const int J = s - 2;
            if (J >= 0) {
                const bool act = jv < nj;
                const char* vt = vring + (vc >= 2 ? vc - 2 : vc + 2) * MEMB;
                if (jv == jpf) prefetch_epilogue(hv);
                if (act) {
                    const int slot = J & 1;
                    float pw[RT];
#pragma unroll
                    for (int rt = 0; rt < RT; ++rt) pw[rt] = xw[slot][pair][rt * 16 + col];
                    const int rescale_v = xr[slot][pair];
                    // slice 0, with the previous memory's last slice (weight 0
                    // when nothing is pending; v[1] is always finite)
                    if (!pend) {
#pragma unroll
                        for (int rt = 0; rt < RT; ++rt) pwp[rt] = 0.f;
                    }
                    slice_region(fr, vt, 0, v[0], cf, [&](int rt) { o[rt][3] += pwp[rt] * v[1][rt]; });
#pragma unroll
                    for (int rt = 0; rt < RT; ++rt) asm volatile("" : "+v"(o[rt][3]));
                    // start of a head, or the running maximum moved: O (which
                    // already holds every earlier memory) is reset or rescaled
                    if (jv == 0) {
#pragma unroll
                        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                            for (int pt = 0; pt < 4; ++pt) o[rt][pt] = f32x4{0.f, 0.f, 0.f, 0.f};
                    } else if (__builtin_amdgcn_readfirstlane(rescale_v)) {
#pragma unroll
                        for (int rt = 0; rt < RT; ++rt) {
                            const float al = xa[slot][pair][rt * 16 + col];
#pragma unroll
                            for (int pt = 0; pt < 4; ++pt) o[rt][pt] *= al;
                        }
                    }
                    // (each slice's O updates are pinned behind its region, so
                    // they stay interleaved with its MFMAs instead of being
                    // sunk to the end of the step)
#pragma unroll
                    for (int pt = 1; pt < 4; ++pt) {
                        slice_region(fr, vt, pt, v[pt & 1], cf,
                                     [&](int rt) { o[rt][pt - 1] += pw[rt] * v[(pt - 1) & 1][rt]; });
#pragma unroll
                        for (int rt = 0; rt < RT; ++rt) asm volatile("" : "+v"(o[rt][pt - 1]));
                    }
                    // the last slice waits for the next memory of the head, if it
                    // is attended; otherwise it completes O now
                    pend = jv + 1 < nj;
                    if (pend) {
#pragma unroll
                        for (int rt = 0; rt < RT; ++rt) pwp[rt] = pw[rt];
                    } else {
#pragma unroll
                        for (int rt = 0; rt < RT; ++rt) o[rt][3] += pw[rt] * v[1][rt];
                    }
                }
                if (jv == jmax - 1) finish_head(hv);
                if (++jv == jmax) {
                    jv = 0;
                    ++hv;
                }
            }
            // first fragments of the next step's memory (s-1), if attended
            if (s >= 1 && s - 1 < nmem && jv < nj) {
                const char* vn = vring + (vc >= 1 ? vc - 1 : vc + 3) * MEMB;
#pragma unroll
                for (int f = 0; f < PD; ++f) fr[f] = frag(vn, f);
            }
        });
    }
}

}  // namespace

// Heads per block of the SMA kernels: the power-of-2 divisor of the group's
// heads, at most hmax, with the least estimated makespan.  A block of hpb
// heads on token block k (tpb tokens) streams hpb * jmax(k) memories (plus two
// pipeline steps) after a set-up of about kSmaSetupSteps steps, jmax(k) being
// the chunk index of its last token; blocks of the first chunk attend no
// memory and, with no_first_chunk, are not launched at all.  Blocks are
// launched heaviest first and each CU takes the next one when it frees, so the
// makespan is about the larger of the longest block and the total work over
// the CUs (the bound of that greedy order).  More heads per block share the
// per-token operands and their set-up; fewer split the longest blocks, so that
// short sequences and small batches still fill every CU evenly.  A split whose
// head-group count B H / hpb is not a multiple of 8 loses the XCD-local block
// order (each head group's memory tiles in one L2) and counts kSmaUnaligned
// times slower (measured at B 1, L 65536, 32 heads: 8 heads per block, 4
// groups, 7.3 ms; 4 heads, 8 groups, 6.7 ms).
constexpr int kSmaSetupSteps = 3;
constexpr double kSmaUnaligned = 1.08;
int sma_block_heads(int64_t B, int H, int G, int64_t L, int S, int tpb, int hmax,
                    bool no_first_chunk) {
    const int per_group = H / G;
    // DART_SMA_HEADS_PER_BLOCK in {1, 2, 4, 8} forces the split when it divides
    // the group's heads, above hmax too (testing and tuning); read at every call
    if (const char* ev = getenv("DART_SMA_HEADS_PER_BLOCK")) {
        const int x = atoi(ev);
        if ((x == 1 || x == 2 || x == 4 || x == 8) && x <= kHeadsPerBlock && per_group % x == 0) return x;
    }
    const int64_t nblk = (L + tpb - 1) / tpb;
    const double cus = (double)device_cu_count();
    int best = 1;
    double best_t = -1.0;
    for (int hpb = hmax; hpb >= 1; hpb >>= 1) {
        if (per_group % hpb != 0) continue;
        const double bhc = (double)(B * (H / hpb));
        double longest = 0.0, total = 0.0;
        for (int64_t k = 0; k < nblk; ++k) {
            const int64_t end = (k + 1) * tpb < L ? (k + 1) * tpb : L;
            const int64_t jmax = (end - 1) / S;
            if (no_first_chunk && jmax == 0) continue;
            const double cost = kSmaSetupSteps + (double)(hpb * jmax) + (jmax > 0 ? 2 : 0);
            longest = std::max(longest, cost);
            total += bhc * cost;
        }
        const double t = std::max(longest, total / cus) *
                         ((B * (H / hpb)) % 8 == 0 ? 1.0 : kSmaUnaligned);
        if (best_t < 0 || t < best_t * 0.97) {  // fewer heads only for a clear gain
            best = hpb;
            best_t = t;
        }
    }
    return best;
}

namespace {

template <typename T, int N, int S>
hipError_t run_sma(const Shape& s, const SmaArgs& a, const void* q, const void* e, const void* Cm,
                   const void* mem, const void* z, const void* y_ssd, void* y, float* lse,
                   void* ws, hipStream_t st) {
    constexpr int TPB = sma_tokens_per_block<T>();
    const int nblk = (int)((s.L + TPB - 1) / TPB);
    const int hpb = sma_block_heads(s.B, s.H, s.G, s.L, s.S, TPB, kFwdHeadsCap, false);
    const int64_t BHC = s.B * (s.H / hpb);
    const int64_t Mp = s.M > 1 ? s.M - 1 : 0;  // memories any token attends to
    T* kmem = reinterpret_cast<T*>(ws);
    if constexpr (sizeof(T) == 2) {
        // bf16: transposed key and value sides ([P][N]) of memories 0..M-2
        T* vT = kmem + (size_t)s.B * Mp * s.H * N * kP;
        if (Mp > 0) {
            prof_begin("k_sma_prep", st);
            k_sma_prep<N><<<dim3((unsigned)Mp, (unsigned)s.H, (unsigned)s.B), 256, 0, st>>>(
                (const T*)mem, kmem, vT, a.eps, a.normalize, s.H, Mp, s.Mcap);
            prof_end(st);
        }
        prof_begin("k_sma", st);
        k_sma<N, S><<<dim3((unsigned)(BHC * nblk)), kThreads, 0, st>>>(
            (const T*)q, (const T*)e, (const T*)Cm, vT, kmem, (const T*)z, (const T*)y_ssd,
            (T*)y, lse, a.qw, a.ew, a.eps, a.normalize, a.z_per_head, s.L, s.H, s.G, Mp, nblk,
            hpb, BHC);
        prof_end(st);
        return hipGetLastError();
    } else {
        if (Mp > 0) {
            prof_begin("k_sma_keys", st);
            k_sma_keys<T, N><<<dim3((unsigned)Mp, (unsigned)s.H, (unsigned)s.B), 256, 0, st>>>(
                (const T*)mem, kmem, nullptr, nullptr, a.eps, a.normalize, s.H, Mp, s.Mcap);
            prof_end(st);
        }
        prof_begin("k_sma", st);
        k_sma_regs<T, N, S><<<dim3((unsigned)(BHC * nblk)), kThreads, 0, st>>>(
            (const T*)q, (const T*)e, (const T*)Cm, (const T*)mem, kmem, (const T*)z,
            (const T*)y_ssd, (T*)y, lse, a.qw, a.ew, a.eps, a.normalize, a.z_per_head, s.L, s.H,
            s.G, s.Mcap, Mp, nblk, hpb, BHC);
        prof_end(st);
        return hipGetLastError();
    }
}

template <typename T, int N>
hipError_t run_sma_s(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                     const void* Cm, const void* mem, const void* z, const void* ys, void* y,
                     float* lse, void* ws, hipStream_t st) {
    switch (s.S) {
        case 64: return run_sma<T, N, 64>(s, a, q, e, Cm, mem, z, ys, y, lse, ws, st);
        case 128: return run_sma<T, N, 128>(s, a, q, e, Cm, mem, z, ys, y, lse, ws, st);
        case 256: return run_sma<T, N, 256>(s, a, q, e, Cm, mem, z, ys, y, lse, ws, st);
    }
    return hipErrorInvalidValue;
}

template <typename T>
hipError_t run_sma_n(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                     const void* Cm, const void* mem, const void* z, const void* ys, void* y,
                     float* lse, void* ws, hipStream_t st) {
    switch (s.N) {
        case 32: return run_sma_s<T, 32>(s, a, q, e, Cm, mem, z, ys, y, lse, ws, st);
        case 64: return run_sma_s<T, 64>(s, a, q, e, Cm, mem, z, ys, y, lse, ws, st);
        case 128: return run_sma_s<T, 128>(s, a, q, e, Cm, mem, z, ys, y, lse, ws, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_sma_keys(const Shape& s, const SmaArgs& a, const void* mem, void* kmem,
                           void* klo, float* rinv, hipStream_t st) {
    const int64_t Mp = s.M > 1 ? s.M - 1 : 0;
    if (Mp == 0) return hipSuccess;
    const dim3 grid((unsigned)Mp, (unsigned)s.H, (unsigned)s.B);
    prof_begin("k_sma_keys", st);
#define DART_KEYS(T, NN)                                                                      \
    k_sma_keys<T, NN><<<grid, 256, 0, st>>>((const T*)mem, (T*)kmem, (T*)klo, rinv, a.eps, \
                                            a.normalize, s.H, Mp, s.Mcap)
    if (s.dtype == 1) {
        switch (s.N) {
            case 32: DART_KEYS(bf16, 32); break;
            case 64: DART_KEYS(bf16, 64); break;
            case 128: DART_KEYS(bf16, 128); break;
        }
    } else {
        switch (s.N) {
            case 32: DART_KEYS(float, 32); break;
            case 64: DART_KEYS(float, 64); break;
            case 128: DART_KEYS(float, 128); break;
        }
    }
#undef DART_KEYS
    prof_end(st);
    return hipGetLastError();
}

size_t sma_workspace_bytes(const Shape& s) {
    if (!tuned_shape(s)) return 0;  // the generic kernel stages memories itself
    const int64_t Mp = s.M > 1 ? s.M - 1 : 0;
    // bf16: key and value sides; fp32: key side only
    return (s.dtype == 1 ? 2 : 1) * elem_bytes(s.dtype) * s.B * Mp * s.H * (size_t)s.N * s.P;
}

hipError_t launch_sma(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                      const void* Cm, const void* mem, const void* z, const void* y_ssd, void* y,
                      float* lse, void* ws, hipStream_t st) {
    if (!tuned_shape(s)) return launch_gsma(s, a, q, e, Cm, mem, z, y_ssd, y, lse, st);
    if (s.dtype == 1) return run_sma_n<bf16>(s, a, q, e, Cm, mem, z, y_ssd, y, lse, ws, st);
    return run_sma_n<float>(s, a, q, e, Cm, mem, z, y_ssd, y, lse, ws, st);
}

}  // namespace dart
