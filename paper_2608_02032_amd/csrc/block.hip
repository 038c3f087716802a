// block.hip -- the steps either side of the path in a DART (Mamba-2) block:
// the causal width-4 convolution with SiLU over the x, B, C channels of the
// input projection (and its carried state, the decode cache of the
// convolution), the step sizes dt = softplus(raw + bias), and the gated
// RMSNorm ahead of the output projection.  The paper fixes the convolution
// width (4) and RMSNorm (App. D.2, the text after Table 8); the rest follows
// the Mamba-2 block it builds on.  All three are elementwise or row-local and
// bound by HBM: every input element is read once, every output written once.
#include "dart_common.hpp"
#include "dart_internal.hpp"

namespace dart {
namespace {

constexpr int kConvTok = 64;  // tokens per thread of the scalar convolution
constexpr int kConvTok8 = 32; // tokens per thread of the 8-channel convolution

// SiLU through the hardware reciprocal (about 1 ulp) instead of an IEEE
// division: these kernels evaluate it once per element they stream.
__device__ __forceinline__ float silu_rcp(float v) {
    return v * __builtin_amdgcn_rcpf(1.0f + __expf(-v));
}

// One thread per (channel, run of kConvTok tokens): the last three inputs
// live in registers, so each input element is loaded once; consecutive
// threads take consecutive channels (coalesced rows).
template <typename T>
__global__ __launch_bounds__(256) void k_conv1d_silu(const T* __restrict__ in, int64_t stride,
                                                     const float* __restrict__ w,
                                                     const float* __restrict__ bias,
                                                     const float* __restrict__ st_in,
                                                     float* __restrict__ st_out,
                                                     T* __restrict__ out, int64_t L, int C) {
    const int c = blockIdx.x * 256 + threadIdx.x;
    const int64_t t0 = (int64_t)blockIdx.y * kConvTok;
    const int64_t b = blockIdx.z;
    if (c >= C) return;
    const float w0 = w[c * 4 + 0], w1 = w[c * 4 + 1], w2 = w[c * 4 + 2], w3 = w[c * 4 + 3];
    const float bc = bias ? bias[c] : 0.f;
    const T* src = in + (b * L) * stride + c;
    // inputs t0 - 3 .. t0 - 1 (carried state before token 0)
    float win[3];
#pragma unroll
    for (int i = 0; i < 3; ++i) {
        const int64_t s = t0 - 3 + i;
        win[i] = s >= 0 ? to_f(src[s * stride]) : (st_in ? st_in[(b * C + c) * 3 + (3 + s)] : 0.f);
    }
    const int64_t t1 = t0 + kConvTok < L ? t0 + kConvTok : L;
    T* dst = out + (b * L) * C + c;
    for (int64_t t = t0; t < t1; ++t) {
        const float v = to_f(src[t * stride]);
        const float a = bc + w0 * win[0] + w1 * win[1] + w2 * win[2] + w3 * v;
        dst[t * C] = from_f<T>(silu_rcp(a));
        win[0] = win[1];
        win[1] = win[2];
        win[2] = v;
    }
    if (st_out && t1 == L) {
        // the last three inputs, oldest first
#pragma unroll
        for (int i = 0; i < 3; ++i) st_out[(b * C + c) * 3 + i] = win[i];
    }
}

// The same convolution with 8 consecutive channels per thread (16-byte rows
// of bf16, 32 of fp32): used when C, the row stride and the pointers are
// multiples of 8 elements.
template <typename T>
__global__ __launch_bounds__(64) void k_conv1d_silu_v8(const T* __restrict__ in, int64_t stride,
                                                        const float* __restrict__ w,
                                                        const float* __restrict__ bias,
                                                        const float* __restrict__ st_in,
                                                        float* __restrict__ st_out,
                                                        T* __restrict__ out, int64_t L, int C) {
    const int c0 = (blockIdx.x * 64 + threadIdx.x) * 8;
    const int64_t t0 = (int64_t)blockIdx.y * kConvTok8;
    const int64_t b = blockIdx.z;
    if (c0 >= C) return;
    float wk[8][4], bc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const f32x4 wv = *reinterpret_cast<const f32x4*>(w + (c0 + i) * 4);
#pragma unroll
        for (int k = 0; k < 4; ++k) wk[i][k] = wv[k];
        bc[i] = bias ? bias[c0 + i] : 0.f;
    }
    const T* src = in + (b * L) * stride + c0;
    float win[3][8];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        const int64_t s = t0 - 3 + k;
        if (s >= 0) {
            load8(src + s * stride, win[k]);
        } else {
#pragma unroll
            for (int i = 0; i < 8; ++i)
                win[k][i] = st_in ? st_in[(b * C + c0 + i) * 3 + (3 + s)] : 0.f;
        }
    }
    const int64_t t1 = t0 + kConvTok8 < L ? t0 + kConvTok8 : L;
    T* dst = out + (b * L) * C + c0;
#pragma unroll 4
    for (int64_t t = t0; t < t1; ++t) {
        float v[8], o[8];
        load8(src + t * stride, v);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float a = bc[i] + wk[i][0] * win[0][i] + wk[i][1] * win[1][i] +
                            wk[i][2] * win[2][i] + wk[i][3] * v[i];
            o[i] = silu_rcp(a);
            win[0][i] = win[1][i];
            win[1][i] = win[2][i];
            win[2][i] = v[i];
        }
        store8(dst + t * C, o);
    }
    if (st_out && t1 == L) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int k = 0; k < 3; ++k) st_out[(b * C + c0 + i) * 3 + k] = win[k][i];
    }
}

template <typename T>
__global__ __launch_bounds__(256) void k_dt_softplus(const T* __restrict__ raw, int64_t stride,
                                                     const float* __restrict__ bias,
                                                     float* __restrict__ dt, int64_t rows, int H) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= rows * H) return;
    const int64_t r = i / H;
    const int h = (int)(i - r * H);
    const float v = to_f(raw[r * stride + h]) + (bias ? bias[h] : 0.f);
    // softplus, log1p(exp(v)) without overflow
    dt[i] = v > 20.f ? v + log1pf(__expf(-v)) : log1pf(__expf(v));
}

// One wave per (row, group): u = y SiLU(z), out = u rsqrt(mean(u^2) + eps) w.
// Lanes take 8 consecutive channels at a time (group and the row strides are
// multiples of 8); the group sum is a wave reduction in a fixed order.
template <typename T>
__global__ __launch_bounds__(256) void k_gated_rmsnorm(const T* __restrict__ y,
                                                       const T* __restrict__ z, int64_t zstride,
                                                       const float* __restrict__ w, float eps,
                                                       T* __restrict__ out, int64_t rows, int D,
                                                       int group) {
    const int lane = threadIdx.x & 63;
    const int64_t item = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int ngr = D / group;
    if (item >= rows * ngr) return;
    const int64_t r = item / ngr;
    const int g0 = (int)(item - r * ngr) * group;
    const T* yr = y + r * D + g0;
    const T* zr = z + r * zstride + g0;
    T* orow = out + r * D + g0;
    // groups of up to 2048 channels stay in registers between the two
    // passes (four pieces of 8 per lane); longer groups read y and z again
    constexpr int KEEP = 4;
    float u[KEEP][8], wv[KEEP][8];
    float ss = 0.f;
#pragma unroll
    for (int q = 0; q < KEEP; ++q) {
        const int k = lane * 8 + q * 512;
        if (k < group) {
            float yv[8], zv[8];
            load8(yr + k, yv);
            load8(zr + k, zv);
            // the weights of these channels, loaded with the data (vector
            // loads; 8 consecutive floats at a multiple of 8)
            if (w) {
                load8(w + g0 + k, wv[q]);
            } else {
#pragma unroll
                for (int i = 0; i < 8; ++i) wv[q][i] = 1.f;
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                u[q][i] = yv[i] * silu_rcp(zv[i]);
                ss += u[q][i] * u[q][i];
            }
        }
    }
    for (int k = lane * 8 + KEEP * 512; k < group; k += 512) {
        float yv[8], zv[8];
        load8(yr + k, yv);
        load8(zr + k, zv);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float uu = yv[i] * silu_rcp(zv[i]);
            ss += uu * uu;
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o, 64);
    const float inv = 1.0f / sqrtf(ss / group + eps);
#pragma unroll
    for (int q = 0; q < KEEP; ++q) {
        const int k = lane * 8 + q * 512;
        if (k < group) {
            float o[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) o[i] = u[q][i] * inv * wv[q][i];
            store8(orow + k, o);
        }
    }
    for (int k = lane * 8 + KEEP * 512; k < group; k += 512) {
        float yv[8], zv[8], o[8];
        load8(yr + k, yv);
        load8(zr + k, zv);
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] = yv[i] * silu_rcp(zv[i]) * inv * (w ? w[g0 + k + i] : 1.f);
        store8(orow + k, o);
    }
}

}  // namespace

hipError_t launch_conv1d_silu(int dtype, int64_t B, int64_t L, int C, int64_t stride,
                              const void* in, const float* w, const float* bias,
                              const float* st_in, float* st_out, void* out, hipStream_t st) {
    const dim3 grid((unsigned)((C + 255) / 256), (unsigned)((L + kConvTok - 1) / kConvTok),
                    (unsigned)B);
    const size_t es = dtype == 1 ? 2 : 4;
    if (C % 8 == 0 && stride % 8 == 0 && (uintptr_t)in % (8 * es) == 0 &&
        (uintptr_t)out % (8 * es) == 0 && (uintptr_t)w % 16 == 0) {
        const dim3 g8((unsigned)((C / 8 + 63) / 64), (unsigned)((L + kConvTok8 - 1) / kConvTok8),
                      (unsigned)B);
        prof_begin("k_conv1d_silu", st);
        if (dtype == 1) {
            k_conv1d_silu_v8<bf16><<<g8, 64, 0, st>>>((const bf16*)in, stride, w, bias, st_in,
                                                      st_out, (bf16*)out, L, C);
        } else {
            k_conv1d_silu_v8<float><<<g8, 64, 0, st>>>((const float*)in, stride, w, bias, st_in,
                                                       st_out, (float*)out, L, C);
        }
        prof_end(st);
        return hipGetLastError();
    }
    prof_begin("k_conv1d_silu", st);
    if (dtype == 1) {
        k_conv1d_silu<bf16><<<grid, 256, 0, st>>>((const bf16*)in, stride, w, bias, st_in, st_out,
                                                  (bf16*)out, L, C);
    } else {
        k_conv1d_silu<float><<<grid, 256, 0, st>>>((const float*)in, stride, w, bias, st_in,
                                                   st_out, (float*)out, L, C);
    }
    prof_end(st);
    return hipGetLastError();
}

hipError_t launch_dt_softplus(int dtype, int64_t rows, int H, const void* raw, int64_t stride,
                              const float* bias, float* dt, hipStream_t st) {
    const unsigned blocks = (unsigned)((rows * H + 255) / 256);
    prof_begin("k_dt_softplus", st);
    if (dtype == 1) {
        k_dt_softplus<bf16><<<blocks, 256, 0, st>>>((const bf16*)raw, stride, bias, dt, rows, H);
    } else {
        k_dt_softplus<float><<<blocks, 256, 0, st>>>((const float*)raw, stride, bias, dt, rows, H);
    }
    prof_end(st);
    return hipGetLastError();
}

hipError_t launch_gated_rmsnorm(int dtype, int64_t rows, int D, int group, const void* y,
                                const void* z, int64_t zstride, const float* w, float eps,
                                void* out, hipStream_t st) {
    const int64_t items = rows * (D / group);
    const unsigned blocks = (unsigned)((items + 3) / 4);
    prof_begin("k_gated_rmsnorm", st);
    if (dtype == 1) {
        k_gated_rmsnorm<bf16><<<blocks, 256, 0, st>>>((const bf16*)y, (const bf16*)z, zstride, w,
                                                      eps, (bf16*)out, rows, D, group);
    } else {
        k_gated_rmsnorm<float><<<blocks, 256, 0, st>>>((const float*)y, (const float*)z, zstride,
                                                       w, eps, (float*)out, rows, D, group);
    }
    prof_end(st);
    return hipGetLastError();
}

}  // namespace dart
