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

// ---- wave-level helpers ---------------------------------------------------
__device__ __forceinline__ float shfl_xor(float v, int mask) { return __shfl_xor(v, mask, 64); }

__device__ __forceinline__ float fast_exp2(float v) { return __builtin_amdgcn_exp2f(v); }

__device__ __forceinline__ float silu(float v) { return v / (1.0f + __expf(-v)); }

}  // namespace dart
