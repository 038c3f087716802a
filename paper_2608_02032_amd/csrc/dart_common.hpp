// dart_common.hpp -- device helpers shared by the DART HIP kernels (gfx950).
//
// Storage types: float (fp32 mode) and __bf16 (bf16 mode).  All arithmetic
// accumulates in float.  Matrix products use the CDNA4 16x16 MFMA tiles:
//   bf16: v_mfma_f32_16x16x32_bf16 (one instruction per 32-deep k step)
//   fp32: v_mfma_f32_16x16x4_f32   (eight instructions per 32-deep k step)
// Operand convention (a "fragment"): lane l of the wave holds 8 consecutive
// k-elements of row (A) or column (B) index l%16; k-group l/16 selects which
// 8 of the 32.  Because A and B use the same per-lane k assignment, any
// consistent permutation of k inside a 32-deep step gives the same product.
// Accumulator layout (f32x4): lane l holds column l%16, rows 4*(l/16)+i.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dart {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

template <typename T> struct FragT;
template <> struct FragT<bf16> { using type = bf16x8; };
template <> struct FragT<float> { using type = f32x8; };
template <typename T> using Frag = typename FragT<T>::type;

__device__ __forceinline__ f32x4 mma16(f32x4 acc, bf16x8 a, bf16x8 b) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma16(f32x4 acc, f32x8 a, f32x8 b) {
#pragma unroll
    for (int i = 0; i < 8; ++i) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[i], acc, 0, 0, 0);
    return acc;
}

// ---- conversions --------------------------------------------------------
__device__ __forceinline__ float to_f(float v) { return v; }
__device__ __forceinline__ float to_f(bf16 v) { return (float)v; }
template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f<bf16>(float v) { return (bf16)v; }

template <typename T> __device__ __forceinline__ Frag<T> make_frag(const float (&v)[8]);
template <> __device__ __forceinline__ bf16x8 make_frag<bf16>(const float (&v)[8]) {
    bf16x8 r;
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = (bf16)v[i];
    return r;
}
template <> __device__ __forceinline__ f32x8 make_frag<float>(const float (&v)[8]) {
    f32x8 r;
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = v[i];
    return r;
}

// ---- 8-element vector loads/stores (16 B for bf16, 32 B for float) -------
// `p` must be aligned to 8 elements.
__device__ __forceinline__ void load8(const bf16* p, float (&v)[8]) {
    const bf16x8 r = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = (float)r[i];
}
__device__ __forceinline__ void load8(const float* p, float (&v)[8]) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(p);
    const f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[i] = a[i];
        v[4 + i] = b[i];
    }
}
__device__ __forceinline__ void store8(bf16* p, const float (&v)[8]) {
    bf16x8 r;
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = (bf16)v[i];
    *reinterpret_cast<bf16x8*>(p) = r;
}
__device__ __forceinline__ void store8(float* p, const float (&v)[8]) {
    f32x4 a, b;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        a[i] = v[i];
        b[i] = v[4 + i];
    }
    *reinterpret_cast<f32x4*>(p) = a;
    *reinterpret_cast<f32x4*>(p + 4) = b;
}
// Streaming variants for data a kernel touches once: nontemporal loads and
// stores (the cache lines are not kept for reuse).
typedef unsigned int u32x4_nt __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void load8_nt(const bf16* p, float (&v)[8]) {
    const bf16x8 r = __builtin_bit_cast(bf16x8, __builtin_nontemporal_load(reinterpret_cast<const u32x4_nt*>(p)));
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = (float)r[i];
}
__device__ __forceinline__ void load8_nt(const float* p, float (&v)[8]) {
    const f32x4 a = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
    const f32x4 b = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + 4));
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[i] = a[i];
        v[4 + i] = b[i];
    }
}
__device__ __forceinline__ void store8_nt(bf16* p, const float (&v)[8]) {
    bf16x8 r;
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = (bf16)v[i];
    __builtin_nontemporal_store(__builtin_bit_cast(u32x4_nt, r), reinterpret_cast<u32x4_nt*>(p));
}
__device__ __forceinline__ void store8_nt(float* p, const float (&v)[8]) {
    f32x4 a, b;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        a[i] = v[i];
        b[i] = v[4 + i];
    }
    __builtin_nontemporal_store(a, reinterpret_cast<f32x4*>(p));
    __builtin_nontemporal_store(b, reinterpret_cast<f32x4*>(p + 4));
}
// Raw fragment load (no conversion) from 8 consecutive elements.
__device__ __forceinline__ bf16x8 load_frag(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }
__device__ __forceinline__ f32x8 load_frag(const float* p) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(p);
    const f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
    f32x8 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        r[i] = a[i];
        r[4 + i] = b[i];
    }
    return r;
}
// 4-element loads/stores (8 B bf16, 16 B float).
__device__ __forceinline__ void load4(const bf16* p, float (&v)[4]) {
    const bf16x4 r = *reinterpret_cast<const bf16x4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = (float)r[i];
}
__device__ __forceinline__ void load4(const float* p, float (&v)[4]) {
    const f32x4 r = *reinterpret_cast<const f32x4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = r[i];
}
__device__ __forceinline__ void store4(bf16* p, const float (&v)[4]) {
    bf16x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = (bf16)v[i];
    *reinterpret_cast<bf16x4*>(p) = r;
}
__device__ __forceinline__ void store4(float* p, const float (&v)[4]) {
    f32x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = v[i];
    *reinterpret_cast<f32x4*>(p) = r;
}

// Stores of NT MFMA accumulator tiles as bf16: lane (grp, col) of tile j holds
// out[row0 + 16 j + col][4 grp + i], i < 4, in rows of `pitch` elements from
// `base`.  With NT even, a row swap between tiles j and j + 1 (even rows keep
// tile j, odd rows take tile j + 1; v_permlane16_swap trades odd rows of its
// first operand with even rows of its second) gives every lane 8 consecutive
// columns of one row: one 16-byte store per tile pair.  Every lane of the
// wave must take part.  acc_row_stores<NT>() is the number of stores each
// lane issues (for wait counts).
template <int NT>
constexpr int acc_row_stores() { return NT % 2 == 0 ? NT / 2 : NT; }
template <int NT>
__device__ __forceinline__ void store_acc_rows_bf16(bf16* base, int64_t pitch, int row0,
                                                    const f32x4 (&acc)[NT], int grp, int col) {
    if constexpr (NT % 2 == 0) {
        uint32_t pk[NT][2];
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            const bf16x2 lo = {(bf16)acc[j][0], (bf16)acc[j][1]};
            const bf16x2 hi = {(bf16)acc[j][2], (bf16)acc[j][3]};
            pk[j][0] = __builtin_bit_cast(uint32_t, lo);
            pk[j][1] = __builtin_bit_cast(uint32_t, hi);
        }
#pragma unroll
        for (int j = 0; j < NT; j += 2) {
#pragma unroll
            for (int k = 0; k < 2; ++k)
                asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(pk[j][k]), "+v"(pk[j + 1][k]));
        }
        const int odd = grp & 1;
#pragma unroll
        for (int j = 0; j < NT; j += 2) {
            const int64_t r = row0 + 16 * (j + odd) + col;
            *reinterpret_cast<uint4*>(base + r * pitch + 4 * (grp - odd)) =
                make_uint4(pk[j][0], pk[j][1], pk[j + 1][0], pk[j + 1][1]);
        }
    } else {
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            const bf16x4 v4 = {(bf16)acc[j][0], (bf16)acc[j][1], (bf16)acc[j][2], (bf16)acc[j][3]};
            *reinterpret_cast<bf16x4*>(base + (int64_t)(row0 + 16 * j + col) * pitch + 4 * grp) = v4;
        }
    }
}

// ---- wave-level helpers ---------------------------------------------------
__device__ __forceinline__ float shfl_xor(float v, int mask) { return __shfl_xor(v, mask, 64); }

// Sum over aligned groups of G = 8 or 16 consecutive lanes with DPP lane moves
// (no LDS round trip): swap within pairs, then within quads, then mirror
// within 8 (and 16) lanes; every lane of a group ends with the group sum.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
template <int G>
__device__ __forceinline__ float dpp_group_sum(float v) {
    static_assert(G == 8 || G == 16, "group of 8 or 16 lanes");
    v += dpp_mov<0xB1>(v);   // quad_perm [1,0,3,2]
    v += dpp_mov<0x4E>(v);   // quad_perm [2,3,0,1]
    v += dpp_mov<0x141>(v);  // row_half_mirror (lane i <-> 7-i within 8)
    if constexpr (G == 16) v += dpp_mov<0x140>(v);  // row_mirror (lane i <-> 15-i within 16)
    return v;
}

// Reduce-scatter over the 64 lanes of the W values of every lane: at step
// MASK a lane keeps one half of its values (the upper half where bit MASK of
// its lane id is set) and adds its partner's copy of that half, so after
// log2(W) steps lane l holds a partial sum of value l / (64 / W); the
// remaining bits are summed by plain butterflies.  W - 1 + log2(64 / W)
// exchanges instead of W full reductions.
template <int R, int W, int MASK>
__device__ __forceinline__ void rs_step(float (&cur)[R], int lane) {
    if constexpr (W > 1) {
        constexpr int half = W / 2;
        const bool hi = (lane & MASK) != 0;
#pragma unroll
        for (int j = 0; j < half; ++j) {
            const float keep = hi ? cur[j + half] : cur[j];
            const float give = hi ? cur[j] : cur[j + half];
            cur[j] = keep + __shfl_xor(give, MASK, 64);
        }
        rs_step<R, half, MASK / 2>(cur, lane);
    }
}

// Sum of each of the R values of every lane over the groups of LANES lanes that
// differ in their low log2(LANES) bits; afterwards lane l holds the group sum of
// value (l % LANES) / (LANES / R).
template <int R, int LANES>
__device__ __forceinline__ float lane_sums(float (&v)[R], int lane) {
    rs_step<R, R, LANES / 2>(v, lane);
    float s = v[0];
#pragma unroll
    for (int m = (LANES / R) / 2; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
    return s;
}

// Sum over the lanes l, l^16, l^32, l^48 (the four 16-lane rows of the wave),
// in every lane, without an LDS round trip: v_permlane32_swap exchanges lanes
// 32..63 of its first operand with lanes 0..31 of its second, so with both
// operands a copy of x their sum is x[l] + x[l^32]; v_permlane16_swap exchanges
// the odd rows of its first operand with the even rows of its second, and the
// same step adds the lane l^16.  Issued from assembly (the builtins return the
// second operand unchanged in this compiler); call from uniform control flow.
__device__ __forceinline__ float row4_sum(float x) {
    float a = x, b = x;
    asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
    float c = a + b, d = c;
    asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(c), "+v"(d));
    return c + d;
}

// lane_sums<8, 16> with DPP moves instead of LDS permutes.  Each step pairs a
// lane with a partner that differs in the step's mask bit (row rotate by 8,
// mirror within 8 lanes, then the two quad swaps); the partner keeps the same
// half of the values at that point, so the keep / give selection by lane bit is
// the one of rs_step and lane l again ends with the 16-lane sum of value
// (l % 16) / 2.
__device__ __forceinline__ float lane_sums8x16_dpp(float (&v)[8], int lane) {
    {
        const bool hi = (lane & 8) != 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float keep = hi ? v[j + 4] : v[j];
            const float give = hi ? v[j] : v[j + 4];
            v[j] = keep + dpp_mov<0x128>(give);  // row_ror:8 (partner lane ^ 8)
        }
    }
    {
        const bool hi = (lane & 4) != 0;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const float keep = hi ? v[j + 2] : v[j];
            const float give = hi ? v[j] : v[j + 2];
            v[j] = keep + dpp_mov<0x141>(give);  // row_half_mirror (partner lane ^ 7)
        }
    }
    {
        const bool hi = (lane & 2) != 0;
        const float keep = hi ? v[1] : v[0];
        const float give = hi ? v[0] : v[1];
        v[0] = keep + dpp_mov<0x4E>(give);  // quad_perm [2,3,0,1] (partner lane ^ 2)
    }
    return v[0] + dpp_mov<0xB1>(v[0]);  // quad_perm [1,0,3,2] (partner lane ^ 1)
}

__device__ __forceinline__ float fast_exp2(float v) { return __builtin_amdgcn_exp2f(v); }

__device__ __forceinline__ float silu(float v) { return v / (1.0f + __expf(-v)); }

// ---- LDS tiles staged by DMA ------------------------------------------------
// 16-byte global -> LDS copy by DMA (global_load_lds_dwordx4).  `lds_wave_base`
// must be the same for the whole wave; lane i's 16 bytes land at
// lds_wave_base + 16 i.  Completion is tracked by the wave's vmcnt.
__device__ __forceinline__ void lds_dma16(const void* gsrc, void* lds_wave_base) {
    __builtin_amdgcn_global_load_lds(gsrc, (__attribute__((address_space(3))) void*)lds_wave_base,
                                     16, 0, 0);
}
__device__ __forceinline__ void wait_dma() { __builtin_amdgcn_s_waitcnt(0); }
// The same copy issued from inline assembly, invisible to the compiler's
// wait-count tracking: the caller must wait for it (s_waitcnt vmcnt) before
// the LDS bytes are read.  Used where the compiler cannot tell a copy in
// flight from the tiles being read and would otherwise drain every copy
// before each LDS read.  M0 (the LDS base) is saved and restored.
__device__ __forceinline__ void lds_dma16_untracked(const void* gsrc, void* lds_wave_base) {
    const uint32_t m0 = (uint32_t)__builtin_amdgcn_readfirstlane(
        (int)(uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)lds_wave_base);
    uint32_t save;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(save)
        : "v"(gsrc), "s"(m0)
        : "memory");
}
// The same copy with the LDS destination given as an LDS byte address (the
// wave's base; lane i lands 16 i bytes further).
__device__ __forceinline__ void lds_dma16_untracked_at(const void* gsrc, uint32_t lds_wave_base) {
    const uint32_t m0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)lds_wave_base);
    uint32_t save;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(save)
        : "v"(gsrc), "s"(m0)
        : "memory");
}
// LDS byte address of a __shared__ object.
template <typename V>
__device__ __forceinline__ uint32_t lds_addr(V* p) {
    return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)p;
}
// s_waitcnt immediate that waits until at most k vector-memory operations of
// the wave are outstanding (expcnt and lgkmcnt left unconstrained; gfx9
// encoding: vmcnt bits [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]).
// Workgroup execution barrier without the memory fence of __syncthreads():
// used in streaming loops where each wave first waits for its own LDS copies
// (vmcnt) and every LDS read of a stage is consumed before the barrier.
__device__ __forceinline__ void block_barrier() { __builtin_amdgcn_s_barrier(); }
// Workgroup barrier that orders LDS only: this wave's LDS writes complete
// before it and no LDS access moves across it, while global loads issued
// earlier stay in flight (a fence on the local address space alone).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}
constexpr int vmcnt_imm(int k) { return (k & 15) | (7 << 4) | (15 << 8) | ((k >> 4) << 14); }

// A natural-layout tile of rows of RB bytes in LDS whose 16-byte chunks are
// XOR-swizzled by row (chunk c of row r is stored at chunk c ^ (r & MASK)), so
// that column reads across consecutive rows spread over the banks.
template <int RB>
struct SwzTile {
    static constexpr int CPR = RB / 16;                  // chunks per row
    static constexpr int MASK = (CPR < 8 ? CPR : 8) - 1;
    __device__ static __forceinline__ int key(int r) { return r & MASK; }
    __device__ static __forceinline__ int off(int r, int byte_in_row) {
        return r * RB + ((((byte_in_row >> 4) ^ key(r)) << 4) | (byte_in_row & 15));
    }
};

// The same with chunk c of row r at chunk c ^ 2 (r & 7), for rows of at least
// 256 bytes: a k-major fragment read takes 32 bytes (an even-aligned chunk
// pair) from each of eight consecutive rows, and with this key the eight rows
// put their pairs on sixteen distinct chunk slots of a 256-byte bank window
// (with c ^ (r & 7) rows r and r ^ 1 share a pair of slots).
template <int RB>
struct SwzTilePair {
    static constexpr int CPR = RB / 16;
    static_assert(CPR >= 16, "rows of at least 256 bytes");
    __device__ static __forceinline__ int key(int r) { return 2 * (r & 7); }
    __device__ static __forceinline__ int off(int r, int byte_in_row) {
        return r * RB + ((((byte_in_row >> 4) ^ key(r)) << 4) | (byte_in_row & 15));
    }
};

// Copy `rows` rows of RB bytes (global row stride gstride bytes) into a
// swizzled LDS tile.  Rows >= rows_valid read the last valid row instead
// (never out of bounds); callers mask their contribution.  rows_valid >= 1.
// Wave w issues copies q0 = 64 w, 64 (w + nwaves), ... of the rows * RB / 1024
// one-KiB pieces.  UNTRACKED selects lds_dma16_untracked.
template <int RB, bool UNTRACKED = false, class Tl = SwzTile<RB>>
__device__ __forceinline__ void dma_tile(char* lds, const char* g, int64_t gstride, int rows,
                                         int rows_valid, int wave, int nwaves, int lane) {
    const int total = rows * Tl::CPR;
    for (int q0 = wave * 64; q0 < total; q0 += nwaves * 64) {
        const int q = q0 + lane;
        if (q < total) {
            const int r = q / Tl::CPR, cs = q % Tl::CPR;
            const int c = cs ^ Tl::key(r);
            const int rr = r < rows_valid ? r : rows_valid - 1;
            if constexpr (UNTRACKED) {
                lds_dma16_untracked(g + rr * gstride + c * 16, lds + q0 * 16);
            } else {
                lds_dma16(g + rr * gstride + c * 16, lds + q0 * 16);
            }
        }
    }
}

// One 16-byte global -> LDS copy per lane: global address = sbase (scalar) +
// voff (per lane, 32-bit), LDS destination = m0 + 16 lane.  Completion is
// tracked by the wave's vmcnt only (the compiler does not see the write).
__device__ __forceinline__ void lds_dma16_sbase(uint32_t voff, uint64_t sbase, uint32_t m0) {
    uint32_t save;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %3\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, %2\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(save)
        : "v"(voff), "s"(sbase), "s"(m0)
        : "memory");
}
// A pointer made wave-uniform (scalar registers).
__device__ __forceinline__ uint64_t uniform_ptr(const void* p) {
    const uint64_t a = (uint64_t)(uintptr_t)p;
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    return ((uint64_t)hi << 32) | (uint64_t)lo;
}

// Copies of one swizzled LDS tile (the Tl layout, SwzTile<RB> by default, ROWS
// rows of RB bytes; rows >= rows_valid re-read the last valid row) issued by NW waves,
// with the per-lane global byte offsets (row * gstride + chunk * 16, 32-bit)
// fixed at set-up, so that issuing a copy costs no vector address work.  Wave
// w copies the 1 KiB pieces w, w + NW, ...; lane l of piece k lands at byte
// 1024 k + 16 l of the tile.
template <int RB, int ROWS, int NW, class Tl = SwzTile<RB>>
struct TilePlan {
    static constexpr int CPR = RB / 16;
    static_assert(ROWS * CPR % 64 == 0, "the tile is whole 1 KiB pieces");
    static constexpr int PIECES = ROWS * CPR / 64;
    static constexpr int KPW = (PIECES + NW - 1) / NW;  // pieces per wave (at most)
    uint32_t goff[KPW];
    __device__ __forceinline__ void init(int wave, int lane, uint32_t gstride, int rows_valid) {
#pragma unroll
        for (int k = 0; k < KPW; ++k) {
            const int q = (wave + k * NW) * 64 + lane;
            const int r = q / CPR, ch = (q % CPR) ^ Tl::key(r);
            const int rr = r < rows_valid ? r : rows_valid - 1;
            goff[k] = (uint32_t)rr * gstride + (uint32_t)(ch * 16);
            asm volatile("" : "+v"(goff[k]));
        }
    }
    // wave: this wave's index (wave-uniform); lds_tile: LDS byte address
    __device__ __forceinline__ void issue(const void* gtile, uint32_t lds_tile, int wave) const {
        const uint64_t sb = uniform_ptr(gtile);
#pragma unroll
        for (int k = 0; k < KPW; ++k) {
            const int piece = wave + k * NW;
            if (PIECES % NW != 0 && piece >= PIECES) break;
            lds_dma16_sbase(goff[k], sb,
                            (uint32_t)__builtin_amdgcn_readfirstlane((int)(lds_tile + (uint32_t)(piece * 1024))));
        }
    }
    // copies this wave issues per tile
    __device__ __forceinline__ int count(int wave) const {
        return PIECES / NW + (wave < PIECES % NW ? 1 : 0);
    }
};
// Copies of BYTES contiguous bytes (a multiple of 16) into LDS at the same
// offsets, NW waves: wave w copies the 1 KiB pieces w, w + NW, ...; lanes past
// the end of a partial last piece copy nothing.
template <int BYTES, int NW>
struct LinearPlan {
    static_assert(BYTES % 16 == 0, "whole 16-byte pieces");
    static constexpr int PIECES = (BYTES + 1023) / 1024;
    static constexpr int KPW = (PIECES + NW - 1) / NW;
    __device__ __forceinline__ void issue(const void* g, uint32_t lds, int wave, int lane) const {
        const uint64_t sb = uniform_ptr(g);
#pragma unroll
        for (int k = 0; k < KPW; ++k) {
            const int piece = wave + k * NW;
            if (PIECES % NW != 0 && piece >= PIECES) break;
            const uint32_t off = (uint32_t)(piece * 1024 + lane * 16);
            const uint32_t m0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)(lds + (uint32_t)(piece * 1024)));
            if (BYTES % 1024 == 0 || off < (uint32_t)BYTES) lds_dma16_sbase(off, sb, m0);
        }
    }
    __device__ __forceinline__ int count(int wave) const {
        return PIECES / NW + (wave < PIECES % NW ? 1 : 0);
    }
};

// MFMA operand fragment from a k-major swizzled tile (rows = k, columns = the
// operand's m or n index): lane l = 16 g + j receives, for its column
// cbase + j, the 8 values of rows krow0(g) + 0..3 and krow1(g) + 0..3.
// bf16 uses two ds_read_b64_tr_b16 (within each 16-lane group, lane j points at
// row r0 + j/4, columns c0 + 4 (j%4); lane i then holds column c0 + i of rows
// r0..r0+3); fp32 falls back to eight scalar reads.
typedef short s16x4 __attribute__((ext_vector_type(4)));
template <int RB, class Tl = SwzTile<RB>>
__device__ __forceinline__ bf16x8 frag_kmajor_bf16(const char* tile, int krow0, int krow1,
                                                   int cbase, int lane) {
    const int j = lane & 15;
    const int col_b = (cbase + 4 * (j & 3)) * 2;
    const char* a0 = tile + Tl::off(krow0 + (j >> 2), col_b);
    const char* a1 = tile + Tl::off(krow1 + (j >> 2), col_b);
    const s16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4*)(a0));
    const s16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4*)(a1));
    const bf16x4 b0 = __builtin_bit_cast(bf16x4, v0);
    const bf16x4 b1 = __builtin_bit_cast(bf16x4, v1);
    return bf16x8{b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
}
template <int RB, class Tl = SwzTile<RB>>
__device__ __forceinline__ f32x8 frag_kmajor_f32(const char* tile, int krow0, int krow1,
                                                 int cbase, int lane) {
    const int col_b = (cbase + (lane & 15)) * 4;
    f32x8 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        r[i] = *reinterpret_cast<const float*>(tile + Tl::off(krow0 + i, col_b));
        r[4 + i] = *reinterpret_cast<const float*>(tile + Tl::off(krow1 + i, col_b));
    }
    return r;
}
template <typename T, int RB, class Tl = SwzTile<RB>>
__device__ __forceinline__ Frag<T> frag_km(const char* tile, int krow0, int krow1, int cbase,
                                           int lane) {
    if constexpr (sizeof(T) == 2) {
        return frag_kmajor_bf16<RB, Tl>(tile, krow0, krow1, cbase, lane);
    } else {
        return frag_kmajor_f32<RB, Tl>(tile, krow0, krow1, cbase, lane);
    }
}

// The two transposing reads of frag_kmajor_bf16 with their per-lane byte
// offsets computed once: rows ra and rb (per lane, + lane/4 within each
// 16-lane group), columns cbase + 4 (lane % 4).  The row swizzle of SwzTile
// depends on the row only modulo 8, so the fragment of rows shifted by a
// multiple of 8 is read at the same offsets plus `add` = rows * RB bytes
// (an immediate when known at compile time), with no address arithmetic.
template <int RB>
struct KmOffBf16 {
    uint32_t o0, o1;
    __device__ __forceinline__ void init(int ra, int rb, int cbase, int lane) {
        using Tl = SwzTile<RB>;
        const int j = lane & 15;
        const int col_b = (cbase + 4 * (j & 3)) * 2;
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

// Fragment from a row-major swizzled tile (rows = the operand's m or n index,
// 8 consecutive k per lane): one 16-byte read (two for fp32).
template <typename T, int RB>
__device__ __forceinline__ Frag<T> frag_rowmajor(const char* tile, int row, int kcol) {
    using Tl = SwzTile<RB>;
    if constexpr (sizeof(T) == 2) {
        return *reinterpret_cast<const bf16x8*>(tile + Tl::off(row, kcol * 2));
    } else {
        const f32x4 a = *reinterpret_cast<const f32x4*>(tile + Tl::off(row, kcol * 4));
        const f32x4 b = *reinterpret_cast<const f32x4*>(tile + Tl::off(row, kcol * 4 + 16));
        return f32x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    }
}

}  // namespace dart
