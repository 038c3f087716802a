// decode.hip -- single-token decode step over the cached chunk memories.
//
// Paper: Sec. 4 "Inference Cache" (the decode cache is one N x P memory per
// completed chunk plus the recurrent state), Sec. 3 (SMA over strictly earlier
// chunks, gated residual) and App. B.1 (normalised score branch).  Keys depend
// on the current token (K = r (.) (dH E_t)), so every step re-reads every
// cached memory: the step is a stream over B*H*m*N*P storage elements and is
// bound by HBM bandwidth.
//
//   k_decode_partial      grid (split, head, batch): each block streams up to
//                         decode_mps() memories, one wave per memory at a time;
//                         lanes own 8 consecutive p of N/8 rows.  Each wave
//                         keeps the next memory's rows in flight while it
//                         reduces the current one (r, the logit and C dH on
//                         the fly; online softmax (m, d, O[P])).  Waves merge
//                         in LDS; one partial per split goes to the workspace.
//   k_decode_state_merge  grid (head, batch): recurrent update of h_state and
//                         of the running chunk contribution, y_ssd = C h_state,
//                         the append of the running contribution when the
//                         token closes its chunk (slot m, never read by this
//                         step), the deterministic LSE merge of the split
//                         partials and y = y_ssd + SiLU(z) R.
// Keeping the state traffic out of the streaming kernel measured faster than
// giving it to one split per head (that split then lags the others).
#include "dart_common.hpp"
#include "dart_internal.hpp"

#include <cstdlib>
#include <mutex>

#include "dart.h"

namespace dart {
namespace {

constexpr int kP = 64;
constexpr int kThreads = 256;
// Memories per split.  Long splits amortise each block's set-up (measured:
// at 64 x 32 heads and 256 memories, 128-memory splits beat 32-memory ones by
// 4 % on a uniform batch and 18 % on a ragged one); the split size is halved
// (down to 8) while that leaves fewer than 4096 blocks (16 per CU).
// DART_DECODE_MPS in {8, 16, 32, 64, 128} forces a size (tuning); the workspace is
// sized for the smallest.
int decode_mps(int64_t bh, int64_t m) {
    static const int forced = [] {
        const char* e = getenv("DART_DECODE_MPS");
        const int x = e ? atoi(e) : 0;
        return (x == 8 || x == 16 || x == 32 || x == 64 || x == 128) ? x : 0;
    }();
    if (forced) return forced;
    int mps = 128;
    while (mps > 8 && bh * ((m + mps - 1) / mps) < 4096) mps >>= 1;
    return mps;
}
constexpr int kMinMPS = kDecodeMinMemPerSplit;

__device__ __forceinline__ bf16x2 as_bf2(uint32_t u) { return __builtin_bit_cast(bf16x2, u); }
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(as_bf2(a), as_bf2(b), c, false);
}
__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
    const bf16x2 v{(bf16)lo, (bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}

// One memory row chunk held by a lane: 8 consecutive p of one row n.
template <typename T> struct RowChunk;
template <> struct RowChunk<bf16> { uint4 v; };
template <> struct RowChunk<float> { f32x4 a, b; };

// The cache is read once per step: nontemporal loads keep it from displacing
// anything in the caches (and stream faster than ordinary loads).
__device__ __forceinline__ void load_row(const bf16* p, RowChunk<bf16>& r) {
    const u32x4_nt w = __builtin_nontemporal_load(reinterpret_cast<const u32x4_nt*>(p));
    r.v = make_uint4(w.x, w.y, w.z, w.w);
}
__device__ __forceinline__ void load_row(const float* p, RowChunk<float>& r) {
    r.a = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
    r.b = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + 4));
}

// Workspace layout: partials [B][H][nsplit][P+2] (O[P], m, d), then y_ssd
// [B][H][P] (float).
inline size_t decode_part_floats(int64_t B, int H, int nsplit) {
    return (size_t)B * H * nsplit * (kP + 2);
}

template <typename T, int N>
__device__ __forceinline__ void state_update(const T* __restrict__ x, const float* __restrict__ dt,
                                             const float* __restrict__ A, const T* __restrict__ Bm,
                                             const T* __restrict__ Cm, float* __restrict__ h_state,
                                             float* __restrict__ chunk_acc, T* __restrict__ mem,
                                             float* __restrict__ yssd, int H, int G, int S,
                                             int64_t Mcap, int64_t pos, int64_t m, int64_t b, int h,
                                             int g, float* s_x, float* s_B, float* s_C,
                                             float (*s_y)[kP]) {
    const int tid = threadIdx.x;
    const int pq = tid & 15, rg = tid >> 4;  // p quad, row group
    const bool reset = (pos % S) == 0;
    const bool append = (pos % S) == S - 1;
    if (tid < kP) s_x[tid] = to_f(x[(b * H + h) * kP + tid]);
    if (tid < N) {
        s_B[tid] = to_f(Bm[(b * G + g) * N + tid]);
        s_C[tid] = to_f(Cm[(b * G + g) * N + tid]);
    }
    __syncthreads();
    const float dtv = dt[b * H + h];
    const float a = __expf(dtv * A[h]);
    float yp[4] = {0.f, 0.f, 0.f, 0.f};
    const int64_t sbase = (b * H + h) * (int64_t)N * kP;
    T* mdst = mem + ((b * Mcap + m) * H + h) * (int64_t)N * kP;
#pragma unroll 4
    for (int k = 0; k < N / 16; ++k) {
        const int n = rg + 16 * k;
        const int64_t off = sbase + n * kP + 4 * pq;
        float hs[4], ca[4];
        load4(h_state + off, hs);
        if (reset) {
#pragma unroll
            for (int i = 0; i < 4; ++i) ca[i] = 0.f;
        } else {
            load4(chunk_acc + off, ca);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float u = dtv * s_B[n] * s_x[4 * pq + i];
            hs[i] = a * hs[i] + u;
            ca[i] = a * ca[i] + u;
            yp[i] += s_C[n] * hs[i];
        }
        store4(h_state + off, hs);
        store4(chunk_acc + off, ca);
        if (append) store4(mdst + n * kP + 4 * pq, ca);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) s_y[rg][4 * pq + i] = yp[i];
    __syncthreads();
    if (tid < kP) {
        float ys = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) ys += s_y[r][tid];
        yssd[(b * H + h) * kP + tid] = ys;
    }
}

template <typename T, int N>
__global__ __launch_bounds__(kThreads) void k_decode_partial(
    const T* __restrict__ mem_rd, const T* __restrict__ q, const T* __restrict__ e,
    const T* __restrict__ Cm, const float* __restrict__ qw, const float* __restrict__ ew,
    float* __restrict__ part, float eps, int normalize, int H, int G, int S, int64_t Mcap,
    int64_t m, const int64_t* __restrict__ pos_rows, int64_t pos_lim, int nsplit, int mps) {
    constexpr int R = N / 8;  // rows per lane (row n = rg + 8 k)
    const int s = blockIdx.x, h = blockIdx.y;
    const int64_t b = blockIdx.z;
    const int g = (int)((int64_t)h * G / H);
    if (pos_rows) {
        // ragged batch: this row's own position; rows outside [0, pos_lim]
        // take no part in the step
        const int64_t pb = pos_rows[b];
        if (pb < 0 || pb > pos_lim) return;
        m = pb / S;
    }
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int po = lane & 7, rg = lane >> 3;

    __shared__ float s_q[N];
    __shared__ float s_e[kP];
    __shared__ float s_part[4][kP + 2];

    const int64_t j0 = (int64_t)s * mps;
    const int64_t j1 = (j0 + mps < m) ? j0 + mps : m;
    if (j0 >= j1) return;  // block-uniform: no cached memory in this split

    if (wave == 0) {
        const float v0 = lane < N ? to_f(q[(b * G + g) * N + lane]) : 0.f;
        const float v1 = lane + 64 < N ? to_f(q[(b * G + g) * N + lane + 64]) : 0.f;
        float ss = v0 * v0 + v1 * v1;
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) ss += shfl_xor(ss, o);
        const float inv = (normalize ? 1.0f / sqrtf(ss * (1.0f / N) + eps) : 1.0f) *
                          (kLog2e / sqrtf((float)N));
        if (lane < N) s_q[lane] = v0 * inv * (qw ? qw[lane] : 1.0f);
        if (lane + 64 < N) s_q[lane + 64] = v1 * inv * (qw ? qw[lane + 64] : 1.0f);
    } else if (wave == 1) {
        const float v = to_f(e[(b * G + g) * kP + lane]);
        float ss = v * v;
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) ss += shfl_xor(ss, o);
        const float inv = normalize ? 1.0f / sqrtf(ss * (1.0f / kP) + eps) : 1.0f;
        s_e[lane] = v * inv * (ew ? ew[lane] : 1.0f);
    }
    __syncthreads();

    float eb[8], qb[R], cb[R];
#pragma unroll
    for (int i = 0; i < 8; ++i) eb[i] = s_e[po * 8 + i];
#pragma unroll
    for (int k = 0; k < R; ++k) {
        qb[k] = s_q[rg + 8 * k];
        cb[k] = to_f(Cm[(b * G + g) * N + rg + 8 * k]);
    }
    // packed bf16 copies for the dot2 path
    uint32_t ebp[4], cbp[R / 2];
#pragma unroll
    for (int i = 0; i < 4; ++i) ebp[i] = pack_bf2(eb[2 * i], eb[2 * i + 1]);
#pragma unroll
    for (int k = 0; k < R / 2; ++k) cbp[k] = pack_bf2(cb[2 * k], cb[2 * k + 1]);

    float mx = -INFINITY, den = 0.f, o[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = 0.f;

    auto load_mem = [&](int64_t j, RowChunk<T>(&xr)[R]) {
        const T* src = mem_rd + ((b * Mcap + j) * H + h) * (int64_t)N * kP;
#pragma unroll
        for (int k = 0; k < R; ++k) load_row(src + (rg + 8 * k) * kP + po * 8, xr[k]);
    };
    auto reduce_mem = [&](const RowChunk<T>(&xr)[R]) {
        float lsum = 0.f, v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = 0.f;
#pragma unroll
        for (int k = 0; k < R; ++k) {
            float ss, kv;
            if constexpr (sizeof(T) == 2) {
                const uint32_t w[4] = {xr[k].v.x, xr[k].v.y, xr[k].v.z, xr[k].v.w};
                ss = dot2(w[0], w[0], 0.f);
                kv = dot2(w[0], ebp[0], 0.f);
#pragma unroll
                for (int i = 1; i < 4; ++i) {
                    ss = dot2(w[i], w[i], ss);
                    kv = dot2(w[i], ebp[i], kv);
                }
                if (k & 1) {
                    // value side: pair rows k-1 and k so one dot2 covers both
                    // (v_perm: the low halves of rows k-1, k, then the high halves)
                    const uint32_t u[4] = {xr[k - 1].v.x, xr[k - 1].v.y, xr[k - 1].v.z,
                                           xr[k - 1].v.w};
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const uint32_t lo = __builtin_amdgcn_perm(w[i], u[i], 0x05040100u);
                        const uint32_t hi = __builtin_amdgcn_perm(w[i], u[i], 0x07060302u);
                        v[2 * i] = dot2(lo, cbp[k >> 1], v[2 * i]);
                        v[2 * i + 1] = dot2(hi, cbp[k >> 1], v[2 * i + 1]);
                    }
                }
            } else {
                const float xv[8] = {xr[k].a[0], xr[k].a[1], xr[k].a[2], xr[k].a[3],
                                     xr[k].b[0], xr[k].b[1], xr[k].b[2], xr[k].b[3]};
                ss = 0.f;
                kv = 0.f;
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    ss += xv[i] * xv[i];
                    kv += xv[i] * eb[i];
                    v[i] += cb[k] * xv[i];
                }
            }
            // the row's sum of squares over its 8 lanes (DPP), then its inverse
            // RMS; the logit partial kv is summed over the lanes once per memory
            ss = dpp_group_sum<8>(ss);
            const float r = normalize ? __builtin_amdgcn_rsqf(ss * (1.0f / kP) + eps) : 1.0f;
            lsum += qb[k] * r * kv;
        }
        lsum = dpp_group_sum<16>(lsum);
        lsum = row4_sum(lsum);
        const float mn = fmaxf(mx, lsum);
        const float al = fast_exp2(mx - mn), pw = fast_exp2(lsum - mn);
        den = den * al + pw;
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] = o[i] * al + pw * v[i];
        mx = mn;
    };
    // wave w takes memories j0 + w, j0 + w + 4, ...; the next one's rows are
    // loaded before the current one is reduced (two register buffers)
    RowChunk<T> xa[R], xb[R];
    int64_t j = j0 + wave;
    if (j < j1) load_mem(j, xa);
    while (j < j1) {
        if (j + 4 < j1) load_mem(j + 4, xb);
        reduce_mem(xa);
        j += 4;
        if (j >= j1) break;
        if (j + 4 < j1) load_mem(j + 4, xa);
        reduce_mem(xb);
        j += 4;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        o[i] += shfl_xor(o[i], 8);
        o[i] += shfl_xor(o[i], 16);
        o[i] += shfl_xor(o[i], 32);
    }
    if (rg == 0) {
#pragma unroll
        for (int i = 0; i < 8; ++i) s_part[wave][po * 8 + i] = o[i];
    }
    if (lane == 0) {
        s_part[wave][kP] = mx;
        s_part[wave][kP + 1] = den;
    }
    __syncthreads();
    if (tid < kP) {
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < 4; ++w) M = fmaxf(M, s_part[w][kP]);
        float D = 0.f, O = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const float mw = s_part[w][kP];
            if (mw == -INFINITY) continue;
            const float sc = fast_exp2(mw - M);
            D += s_part[w][kP + 1] * sc;
            O += s_part[w][tid] * sc;
        }
        float* out = part + (((b * H + h) * nsplit) + s) * (kP + 2);
        out[tid] = O;
        if (tid == 0) {
            out[kP] = M;
            out[kP + 1] = D;
        }
    }
}

// Recurrent update (h_state, running chunk contribution, y_ssd, append), then
// the deterministic LSE merge of the split partials and the gate.
template <typename T, int N>
__global__ __launch_bounds__(kThreads) void k_decode_state_merge(
    const T* __restrict__ x, const float* __restrict__ dt, const float* __restrict__ A,
    const T* __restrict__ Bm, const T* __restrict__ Cm, const T* __restrict__ z,
    float* __restrict__ h_state, float* __restrict__ chunk_acc, T* __restrict__ mem,
    T* __restrict__ y, const float* __restrict__ part, float* __restrict__ yssd, int H, int G,
    int S, int64_t Mcap, int64_t pos, int64_t m, const int64_t* __restrict__ pos_rows,
    int64_t pos_lim, int nsplit, int z_per_head, int mps) {
    const int h = blockIdx.x;
    const int64_t b = blockIdx.y;
    const int g = (int)((int64_t)h * G / H);
    if (pos_rows) {
        pos = pos_rows[b];
        if (pos < 0 || pos > pos_lim) return;  // the row takes no part in the step
        m = pos / S;
    }
    __shared__ float s_x[kP], s_B[N], s_C[N];
    __shared__ float s_y[16][kP];
    state_update<T, N>(x, dt, A, Bm, Cm, h_state, chunk_acc, mem, yssd, H, G, S, Mcap, pos, m, b,
                       h, g, s_x, s_B, s_C, s_y);
    const int p = threadIdx.x;
    if (p >= kP) return;
    float R = 0.f;
    if (m > 0) {
        const int ns = (int)((m + mps - 1) / mps);
        const float* pb = part + (b * H + h) * nsplit * (int64_t)(kP + 2);
        float M = -INFINITY;
        for (int s = 0; s < ns; ++s) M = fmaxf(M, pb[s * (kP + 2) + kP]);
        float D = 0.f, O = 0.f;
        for (int s = 0; s < ns; ++s) {
            const float sc = fast_exp2(pb[s * (kP + 2) + kP] - M);
            D += pb[s * (kP + 2) + kP + 1] * sc;
            O += pb[s * (kP + 2) + p] * sc;
        }
        R = O / D;
    }
    const float zz = to_f(z_per_head ? z[b * H + h] : z[b]);
    y[(b * H + h) * kP + p] = from_f<T>(yssd[(b * H + h) * kP + p] + silu(zz) * R);
}

// Number of splits of a step that attends m memories.
inline int decode_splits(const Shape& s, int64_t m) {
    if (m <= 0) return 0;
    const int mps = decode_mps(s.B * s.H, m);
    return (int)((m + mps - 1) / mps);
}

// nsplit_stride: the partials' split stride in the workspace (0: the
// workspace's worst case over positions that fit the cache).
template <typename T, int N>
hipError_t run_decode(const Shape& s, const SmaArgs& a, int64_t pos, const int64_t* pos_rows,
                      const void* x, const float* dt, const float* A, const void* Bm,
                      const void* Cm, const void* q, const void* e, const void* z, float* h_state,
                      float* chunk_acc, void* mem, void* y, void* ws, int nsplit_stride,
                      hipStream_t st) {
    // ragged batches size the grid for the largest position (pos = pos_lim)
    const int64_t m = pos / s.S;
    const int mps = decode_mps(s.B * s.H, m);
    const int nsplit_cap =
        nsplit_stride > 0 ? nsplit_stride : (int)((s.Mcap + kMinMPS - 1) / kMinMPS);
    float* part = reinterpret_cast<float*>(ws);
    float* yssd = part + decode_part_floats(s.B, s.H, nsplit_cap);
    if (m > 0) {
        const int ns = (int)((m + mps - 1) / mps);
        prof_begin("k_decode_partial", st);
        k_decode_partial<T, N><<<dim3((unsigned)ns, (unsigned)s.H, (unsigned)s.B), kThreads, 0, st>>>(
            (const T*)mem, (const T*)q, (const T*)e, (const T*)Cm, a.qw, a.ew, part, a.eps,
            a.normalize, s.H, s.G, s.S, s.Mcap, m, pos_rows, pos, nsplit_cap, mps);
        prof_end(st);
    }
    prof_begin("k_decode_state_merge", st);
    k_decode_state_merge<T, N><<<dim3((unsigned)s.H, (unsigned)s.B), kThreads, 0, st>>>(
        (const T*)x, dt, A, (const T*)Bm, (const T*)Cm, (const T*)z, h_state, chunk_acc, (T*)mem,
        (T*)y, part, yssd, s.H, s.G, s.S, s.Mcap, pos, m, pos_rows, pos, nsplit_cap, a.z_per_head,
        mps);
    prof_end(st);
    return hipGetLastError();
}

template <typename T>
hipError_t run_decode_n(const Shape& s, const SmaArgs& a, int64_t pos, const int64_t* pr,
                        const void* x, const float* dt, const float* A, const void* Bm,
                        const void* Cm, const void* q, const void* e, const void* z, float* hs,
                        float* ca, void* mem, void* y, void* ws, int nss, hipStream_t st) {
    switch (s.N) {
        case 16: return run_decode<T, 16>(s, a, pos, pr, x, dt, A, Bm, Cm, q, e, z, hs, ca, mem, y, ws, nss, st);
        case 32: return run_decode<T, 32>(s, a, pos, pr, x, dt, A, Bm, Cm, q, e, z, hs, ca, mem, y, ws, nss, st);
        case 64: return run_decode<T, 64>(s, a, pos, pr, x, dt, A, Bm, Cm, q, e, z, hs, ca, mem, y, ws, nss, st);
        case 128: return run_decode<T, 128>(s, a, pos, pr, x, dt, A, Bm, Cm, q, e, z, hs, ca, mem, y, ws, nss, st);
    }
    return hipErrorInvalidValue;
}

// Fixed device scratch of the allocation-free decode step: the partials
// [B][H][nsplit][P+2] of that step's own split count and y_ssd [B][H][P]
// (float).  Each device holds its own copy; host code reaches it only through
// the address hipGetSymbolAddress returns on that device.
static __device__ __align__(256) char scratch[DART_DECODE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's scratch address, looked up once per device (with that
// device current) and kept.
hipError_t scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

// Prefill -> decode handoff for row b of length L_b (lengths[b]; rows with
// L_b < 0 are left untouched): h_state = h_last and chunk_acc = the running
// contribution of the partial chunk floor(L_b/S), which the forward scan left
// in mem slot floor(L_b/S) (0 when L_b is a multiple of S: the next token
// opens a chunk).
template <typename T, int N>
__global__ __launch_bounds__(kThreads) void k_decode_handoff(const T* __restrict__ mem,
                                                             const float* __restrict__ h_last,
                                                             const int64_t* __restrict__ lengths,
                                                             float* __restrict__ h_state,
                                                             float* __restrict__ chunk_acc, int H,
                                                             int S, int64_t Mcap) {
    const int h = blockIdx.x;
    const int64_t b = blockIdx.y;
    const int64_t len = lengths[b];
    if (len < 0) return;
    const int64_t mi = len / S;
    const bool partial = (len % S) != 0 && mi < Mcap;
    const int64_t base = (b * H + h) * (int64_t)N * kP;
    const T* src = mem + ((b * Mcap + (partial ? mi : 0)) * H + h) * (int64_t)N * kP;
    for (int e0 = threadIdx.x * 4; e0 < N * kP; e0 += kThreads * 4) {
        float v[4];
        load4(h_last + base + e0, v);
        store4(h_state + base + e0, v);
        if (partial) {
            load4(src + e0, v);
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = 0.f;
        }
        store4(chunk_acc + base + e0, v);
    }
}

template <typename T>
hipError_t run_handoff_n(const Shape& s, const void* mem, const float* h_last,
                         const int64_t* lengths, float* h_state, float* chunk_acc, hipStream_t st) {
    const dim3 grid((unsigned)s.H, (unsigned)s.B);
    prof_begin("k_decode_handoff", st);
    switch (s.N) {
        case 16: k_decode_handoff<T, 16><<<grid, kThreads, 0, st>>>((const T*)mem, h_last, lengths, h_state, chunk_acc, s.H, s.S, s.Mcap); break;
        case 32: k_decode_handoff<T, 32><<<grid, kThreads, 0, st>>>((const T*)mem, h_last, lengths, h_state, chunk_acc, s.H, s.S, s.Mcap); break;
        case 64: k_decode_handoff<T, 64><<<grid, kThreads, 0, st>>>((const T*)mem, h_last, lengths, h_state, chunk_acc, s.H, s.S, s.Mcap); break;
        case 128: k_decode_handoff<T, 128><<<grid, kThreads, 0, st>>>((const T*)mem, h_last, lengths, h_state, chunk_acc, s.H, s.S, s.Mcap); break;
        default: prof_end(st); return hipErrorInvalidValue;
    }
    prof_end(st);
    return hipGetLastError();
}

}  // namespace

size_t decode_workspace_bytes(const Shape& s) {
    const int64_t nsplit = (s.Mcap + kMinMPS - 1) / kMinMPS;
    return align256(sizeof(float) * (decode_part_floats(s.B, s.H, (int)(nsplit > 0 ? nsplit : 1)) +
                                     (size_t)s.B * s.H * s.P));
}

hipError_t launch_decode(const Shape& s, const SmaArgs& a, int64_t pos, const int64_t* pos_rows,
                         const void* x, const float* dt, const float* A, const void* Bm,
                         const void* Cm, const void* q, const void* e, const void* z,
                         float* h_state, float* chunk_acc, void* mem, void* y, void* ws,
                         hipStream_t st) {
    if (s.dtype == 1)
        return run_decode_n<bf16>(s, a, pos, pos_rows, x, dt, A, Bm, Cm, q, e, z, h_state, chunk_acc,
                                  mem, y, ws, 0, st);
    return run_decode_n<float>(s, a, pos, pos_rows, x, dt, A, Bm, Cm, q, e, z, h_state, chunk_acc, mem,
                               y, ws, 0, st);
}

size_t decode_noalloc_scratch_bytes(const Shape& s, int64_t pos) {
    const int ns = decode_splits(s, pos / s.S);
    return sizeof(float) * (decode_part_floats(s.B, s.H, ns > 0 ? ns : 1) + (size_t)s.B * s.H * s.P);
}

hipError_t launch_decode_noalloc(const Shape& s, const SmaArgs& a, int64_t pos, const void* x,
                                 const float* dt, const float* A, const void* Bm, const void* Cm,
                                 const void* q, const void* e, const void* z, float* h_state,
                                 float* chunk_acc, void* mem, void* y, hipStream_t st) {
    void* ws = nullptr;
    const hipError_t err = scratch_address(&ws);
    if (err != hipSuccess) return err;
    const int ns = decode_splits(s, pos / s.S);
    const int nss = ns > 0 ? ns : 1;
    if (s.dtype == 1)
        return run_decode_n<bf16>(s, a, pos, nullptr, x, dt, A, Bm, Cm, q, e, z, h_state, chunk_acc,
                                  mem, y, ws, nss, st);
    return run_decode_n<float>(s, a, pos, nullptr, x, dt, A, Bm, Cm, q, e, z, h_state, chunk_acc, mem,
                               y, ws, nss, st);
}

hipError_t launch_decode_handoff(const Shape& s, const void* mem, const float* h_last,
                                 const int64_t* lengths, float* h_state, float* chunk_acc,
                                 hipStream_t st) {
    if (s.dtype == 1) return run_handoff_n<bf16>(s, mem, h_last, lengths, h_state, chunk_acc, st);
    return run_handoff_n<float>(s, mem, h_last, lengths, h_state, chunk_acc, st);
}

}  // namespace dart
