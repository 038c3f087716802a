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
            load8_nt(yr + k, yv);
            load8_nt(zr + k, zv);
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
            store8_nt(orow + k, o);
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

// ---- backward of the block kernels ------------------------------------------------
// Gradients for a loss whose gradient with respect to each kernel's output is
// `dout` (float).  Sums over tokens or rows (weights, biases) go to per-block
// partials in the workspace and a second kernel adds them in a fixed order.

__device__ __forceinline__ float silu_grad_f(float u) {
    const float sg = 1.0f / (1.0f + __expf(-u));
    return sg * (1.0f + u * (1.0f - sg));
}

constexpr int kConvBwdTok = 32;  // tokens per thread of the convolution backward

// One thread per (channel, run of kConvBwdTok tokens, batch row).  With
// u_t = bias + sum_k w_k in[t-3+k] and du_t = dout_t SiLU'(u_t):
//   din[s] = w3 du_s + w2 du_{s+1} + w1 du_{s+2} + w0 du_{s+3},
//   dw_k = sum_t du_t in[t-3+k],  dbias = sum_t du_t,
//   dstate[j] (input -3+j) = sum_{t <= j} du_t w_{j-t}.
// A run computes du for its own tokens and the three after it, so din of its
// tokens is complete; the weight sums cover its own tokens only.
template <typename T>
__global__ __launch_bounds__(256) void k_conv1d_silu_bwd(
    const T* __restrict__ in, int64_t stride, const float* __restrict__ w,
    const float* __restrict__ bias, const float* __restrict__ st_in,
    const float* __restrict__ dout, float* __restrict__ din, int64_t dstride,
    float* __restrict__ dst_in, float* __restrict__ part, int64_t L, int C, int nruns) {
    const int c = blockIdx.x * 256 + threadIdx.x;
    const int run = blockIdx.y;
    const int64_t b = blockIdx.z;
    if (c >= C) return;
    const int64_t t0 = (int64_t)run * kConvBwdTok;
    const int64_t t1 = t0 + kConvBwdTok < L ? t0 + kConvBwdTok : L;
    const int64_t tend = t1 + 3 < L ? t1 + 3 : L;
    const float w0 = w[c * 4 + 0], w1 = w[c * 4 + 1], w2 = w[c * 4 + 2], w3 = w[c * 4 + 3];
    const float bc = bias ? bias[c] : 0.f;
    const T* src = in + (b * L) * stride + c;
    const float* dsrc = dout + (b * L) * C + c;
    float* dd = din + (b * L) * dstride + c;
    float win[3];
#pragma unroll
    for (int i = 0; i < 3; ++i) {
        const int64_t s = t0 - 3 + i;
        win[i] = s >= 0 ? to_f(src[s * stride]) : (st_in ? st_in[(b * C + c) * 3 + (3 + s)] : 0.f);
    }
    float q0 = 0.f, q1 = 0.f, q2 = 0.f, q3 = 0.f;  // du at t-3 .. t
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f, ab = 0.f;
    float d0 = 0.f, d1 = 0.f, d2 = 0.f;  // du at t0, t0+1, t0+2
    for (int64_t t = t0; t < tend; ++t) {
        const float v = to_f(src[t * stride]);
        const float u = bc + w0 * win[0] + w1 * win[1] + w2 * win[2] + w3 * v;
        const float du = dsrc[t * C] * silu_grad_f(u);
        if (t < t1) {
            a0 += du * win[0];
            a1 += du * win[1];
            a2 += du * win[2];
            a3 += du * v;
            ab += du;
        }
        if (t == t0) d0 = du;
        if (t == t0 + 1) d1 = du;
        if (t == t0 + 2) d2 = du;
        q0 = q1;
        q1 = q2;
        q2 = q3;
        q3 = du;
        if (t - 3 >= t0) dd[(t - 3) * dstride] = w3 * q0 + w2 * q1 + w1 * q2 + w0 * q3;
        win[0] = win[1];
        win[1] = win[2];
        win[2] = v;
    }
    // tokens whose later inputs end at L (du beyond L is zero); q3 = du at
    // tend - 1 and so on
    for (int64_t s = (tend - 3 > t0 ? tend - 3 : t0); s < t1; ++s) {
        const int64_t k = tend - s;  // 3, 2 or 1 tokens from s to the end
        float v = 0.f;
        if (k == 3) v = w3 * q1 + w2 * q2 + w1 * q3;
        if (k == 2) v = w3 * q2 + w2 * q3;
        if (k == 1) v = w3 * q3;
        dd[s * dstride] = v;
    }
    if (dst_in && t0 == 0) {
        dst_in[(b * C + c) * 3 + 0] = d0 * w0;
        dst_in[(b * C + c) * 3 + 1] = d0 * w1 + d1 * w0;
        dst_in[(b * C + c) * 3 + 2] = d0 * w2 + d1 * w1 + d2 * w0;
    }
    float* pr = part + ((b * nruns + run) * (int64_t)C + c) * 5;
    pr[0] = a0;
    pr[1] = a1;
    pr[2] = a2;
    pr[3] = a3;
    pr[4] = ab;
}

// Sum of nparts partial rows of K floats per item: out[i][k] = sum_p part[p][i][k].
__global__ __launch_bounds__(256) void k_sum_parts(const float* __restrict__ part,
                                                   int64_t nparts, int64_t width,
                                                   float* __restrict__ out, int K, int keep,
                                                   float* __restrict__ out2) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= width) return;
    float s = 0.f;
    for (int64_t p = 0; p < nparts; ++p) s += part[p * width + i];
    // items of K values: the first `keep` go to out ([item][keep]), the rest
    // (at most one) to out2 ([item])
    const int64_t item = i / K;
    const int k = (int)(i - item * K);
    if (k < keep) {
        if (out) out[item * keep + k] = s;
    } else if (out2) {
        out2[item] = s;
    }
}

// dt = softplus(raw + bias): draw = ddt sigmoid(raw + bias), dbias = sum over
// rows.  One thread per (head, block of 256 rows).
constexpr int kDtRows = 256;
template <typename T>
__global__ __launch_bounds__(256) void k_dt_softplus_bwd(const T* __restrict__ raw, int64_t stride,
                                                         const float* __restrict__ bias,
                                                         const float* __restrict__ ddt,
                                                         float* __restrict__ draw,
                                                         int64_t dstride, float* __restrict__ part,
                                                         int64_t rows, int H) {
    const int h = blockIdx.x * 256 + threadIdx.x;
    const int64_t rb = blockIdx.y;
    if (h >= H) return;
    const int64_t r0 = rb * kDtRows;
    const int64_t r1 = r0 + kDtRows < rows ? r0 + kDtRows : rows;
    const float bh = bias ? bias[h] : 0.f;
    float acc = 0.f;
    for (int64_t r = r0; r < r1; ++r) {
        const float v = to_f(raw[r * stride + h]) + bh;
        const float g = ddt[r * H + h] / (1.0f + __expf(-v));
        draw[r * dstride + h] = g;
        acc += g;
    }
    part[rb * H + h] = acc;
}

// Gated RMSNorm backward, one wave per (block of kNormRows rows, group); the
// group's channels (at most 2048) stay in registers, 8 per lane per piece.
// With u = y SiLU(z), inv = (mean u^2 + eps)^-1/2, g = dout (.) w:
//   du = inv g - u inv^3 (g . u) / group,  dy = du SiLU(z),
//   dz = du y SiLU'(z),  dw += dout u inv (summed over the block's rows).
constexpr int kNormRows = 16;
template <typename T>
__global__ __launch_bounds__(256) void k_gated_rmsnorm_bwd(
    const T* __restrict__ y, const T* __restrict__ z, int64_t zstride, const float* __restrict__ w,
    float eps, const float* __restrict__ dout, float* __restrict__ dy, float* __restrict__ dz,
    int64_t dzstride, float* __restrict__ part, int64_t rows, int D, int group) {
    const int lane = threadIdx.x & 63;
    const int64_t item = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int ngr = D / group;
    const int64_t nrb = (rows + kNormRows - 1) / kNormRows;
    if (item >= nrb * ngr) return;
    const int64_t rb = item / ngr;
    const int g0 = (int)(item - rb * ngr) * group;
    constexpr int KEEP = 4;
    float wacc[KEEP][8];
#pragma unroll
    for (int q = 0; q < KEEP; ++q)
#pragma unroll
        for (int i = 0; i < 8; ++i) wacc[q][i] = 0.f;
    const int64_t r1 = (rb + 1) * kNormRows < rows ? (rb + 1) * kNormRows : rows;
    for (int64_t r = rb * kNormRows; r < r1; ++r) {
        float u[KEEP][8], g[KEEP][8], ss = 0.f, gu = 0.f;
#pragma unroll
        for (int q = 0; q < KEEP; ++q) {
            const int k = lane * 8 + q * 512;
            if (k < group) {
                float yv[8], zv[8], dv[8];
                load8(y + r * D + g0 + k, yv);
                load8(z + r * zstride + g0 + k, zv);
                load8(dout + r * D + g0 + k, dv);
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    u[q][i] = yv[i] * silu_rcp(zv[i]);
                    g[q][i] = dv[i] * (w ? w[g0 + k + i] : 1.f);
                    ss += u[q][i] * u[q][i];
                    gu += g[q][i] * u[q][i];
                }
            }
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            ss += __shfl_xor(ss, o, 64);
            gu += __shfl_xor(gu, o, 64);
        }
        const float inv = 1.0f / sqrtf(ss / group + eps);
        const float c3 = inv * inv * inv * gu / group;
#pragma unroll
        for (int q = 0; q < KEEP; ++q) {
            const int k = lane * 8 + q * 512;
            if (k < group) {
                float yv[8], zv[8], dv[8], oy[8], oz[8];
                load8(y + r * D + g0 + k, yv);
                load8(z + r * zstride + g0 + k, zv);
                load8(dout + r * D + g0 + k, dv);
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const float du = inv * g[q][i] - u[q][i] * c3;
                    const float sz = silu_rcp(zv[i]);
                    oy[i] = du * sz;
                    oz[i] = du * yv[i] * silu_grad_f(zv[i]);
                    wacc[q][i] += dv[i] * u[q][i] * inv;
                }
                store8(dy + r * D + g0 + k, oy);
                store8(dz + r * dzstride + g0 + k, oz);
            }
        }
    }
#pragma unroll
    for (int q = 0; q < KEEP; ++q) {
        const int k = lane * 8 + q * 512;
        if (k < group) store8(part + rb * D + g0 + k, wacc[q]);
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

size_t conv1d_silu_bwd_workspace_bytes(int64_t B, int64_t L, int C) {
    const int64_t nruns = (L + kConvBwdTok - 1) / kConvBwdTok;
    return align256(sizeof(float) * (size_t)B * nruns * C * 5);
}

hipError_t launch_conv1d_silu_bwd(int dtype, int64_t B, int64_t L, int C, int64_t stride,
                                  const void* in, const float* w, const float* bias,
                                  const float* st_in, const float* dout, float* din,
                                  int64_t dstride, float* dw, float* db, float* dst_in, void* ws,
                                  hipStream_t st) {
    const int nruns = (int)((L + kConvBwdTok - 1) / kConvBwdTok);
    float* part = reinterpret_cast<float*>(ws);
    const dim3 grid((unsigned)((C + 255) / 256), (unsigned)nruns, (unsigned)B);
    prof_begin("k_conv1d_silu_bwd", st);
    if (dtype == 1) {
        k_conv1d_silu_bwd<bf16><<<grid, 256, 0, st>>>((const bf16*)in, stride, w, bias, st_in, dout,
                                                      din, dstride, dst_in, part, L, C, nruns);
    } else {
        k_conv1d_silu_bwd<float><<<grid, 256, 0, st>>>((const float*)in, stride, w, bias, st_in,
                                                       dout, din, dstride, dst_in, part, L, C, nruns);
    }
    prof_end(st);
    const int64_t width = (int64_t)C * 5;
    prof_begin("k_sum_parts", st);
    k_sum_parts<<<(unsigned)((width + 255) / 256), 256, 0, st>>>(part, B * nruns, width, dw, 5, 4, db);
    prof_end(st);
    return hipGetLastError();
}

size_t dt_softplus_bwd_workspace_bytes(int64_t rows, int H) {
    return align256(sizeof(float) * (size_t)((rows + kDtRows - 1) / kDtRows) * H);
}

hipError_t launch_dt_softplus_bwd(int dtype, int64_t rows, int H, const void* raw, int64_t stride,
                                  const float* bias, const float* ddt, float* draw,
                                  int64_t dstride, float* dbias, void* ws, hipStream_t st) {
    const int64_t nrb = (rows + kDtRows - 1) / kDtRows;
    float* part = reinterpret_cast<float*>(ws);
    const dim3 grid((unsigned)((H + 255) / 256), (unsigned)nrb);
    prof_begin("k_dt_softplus_bwd", st);
    if (dtype == 1) {
        k_dt_softplus_bwd<bf16><<<grid, 256, 0, st>>>((const bf16*)raw, stride, bias, ddt, draw,
                                                      dstride, part, rows, H);
    } else {
        k_dt_softplus_bwd<float><<<grid, 256, 0, st>>>((const float*)raw, stride, bias, ddt, draw,
                                                       dstride, part, rows, H);
    }
    prof_end(st);
    if (dbias) {
        prof_begin("k_sum_parts", st);
        k_sum_parts<<<(unsigned)((H + 255) / 256), 256, 0, st>>>(part, nrb, H, dbias, 1, 1, nullptr);
        prof_end(st);
    }
    return hipGetLastError();
}

size_t gated_rmsnorm_bwd_workspace_bytes(int64_t rows, int D) {
    return align256(sizeof(float) * (size_t)((rows + kNormRows - 1) / kNormRows) * D);
}

hipError_t launch_gated_rmsnorm_bwd(int dtype, int64_t rows, int D, int group, const void* y,
                                    const void* z, int64_t zstride, const float* w, float eps,
                                    const float* dout, float* dy, float* dz, int64_t dzstride,
                                    float* dw, void* ws, hipStream_t st) {
    const int64_t nrb = (rows + kNormRows - 1) / kNormRows;
    float* part = reinterpret_cast<float*>(ws);
    const int64_t items = nrb * (D / group);
    prof_begin("k_gated_rmsnorm_bwd", st);
    if (dtype == 1) {
        k_gated_rmsnorm_bwd<bf16><<<(unsigned)((items + 3) / 4), 256, 0, st>>>(
            (const bf16*)y, (const bf16*)z, zstride, w, eps, dout, dy, dz, dzstride, part, rows, D,
            group);
    } else {
        k_gated_rmsnorm_bwd<float><<<(unsigned)((items + 3) / 4), 256, 0, st>>>(
            (const float*)y, (const float*)z, zstride, w, eps, dout, dy, dz, dzstride, part, rows,
            D, group);
    }
    prof_end(st);
    if (dw) {
        prof_begin("k_sum_parts", st);
        k_sum_parts<<<(unsigned)((D + 255) / 256), 256, 0, st>>>(part, nrb, D, dw, 1, 1, nullptr);
        prof_end(st);
    }
    return hipGetLastError();
}

}  // namespace dart
