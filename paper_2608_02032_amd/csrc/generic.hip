// generic.hip -- the untuned path: every shape outside the tuned set
// (N in {32, 64, 128} with S in {64, 128, 256}), i.e. any chunk size S >= 1
// and N in {16, 32, 64, 128}, P = 64, both storage dtypes.  Plain fp32 VALU
// kernels, correct before fast; the tuned MFMA kernels serve the benchmark
// shapes.  The paper trains at S = 16, N in {16, 64} (MQAR, App. D.1) and
// evaluates one checkpoint at S = 64 and 32 (Sec. 5.2).
//
// Scan (Sec. 2 recurrence, Sec. 3 / App. A chunk memories), chunk-parallel
// with the recurrence itself inside each chunk:
//   k_gscan_chunk  per (b, c, h): run the chunk's tokens from a zero state;
//                  the state at the chunk's end is dH_[c] (App. A), kept in
//                  float and written to the memories in the storage dtype;
//                  the chunk's log decay sum_t dt_t A_h;
//   k_gscan_pass   per (b, h, 1024 state elements): H_[c] = e^{lda_c} H_[c-1]
//                  + dH_[c] over the chunks, in float; every chunk's entry
//                  state (float, and in the storage dtype for the backward)
//                  and h_last;
//   k_gscan_out    per (b, c, h): run the chunk's tokens again from its entry
//                  state, y_t = C_t H_t.
// SMA forward (Sec. 3, App. B.1, Alg. 1's online softmax):
//   k_gsma         per (b, h, chunk i, up to 32 tokens of it): memory j < i
//                  staged in LDS with its row inverse-RMS r_j, then every
//                  token's logit and value on the lanes (lane = p), the
//                  online softmax, and the gated residual with the LSE.
// SMA backward (App. C: scores recomputed; exact softmax of the recomputed
// logits):
//   k_gsma_bwd_tok per (b, h, chunk i, up to 32 tokens): pass 1 over the
//                  memories for the logits, dy . V_j, the LSE and
//                  Dy = R . dy; pass 2 for dl_j = g p_j (dy . V_j - Dy) and
//                  the token-side gradients dQbar, dEbar, dC (per head; the
//                  finishing kernel sums a group's heads);
//   k_gsma_bwd_mem per (b, h, memory): M1 = sum_t g p_j C_t^T dy_t and
//                  M2 = sum_t dl_j Qbar_t^T Ebar_t / sqrt(N), then the memory
//                  gradient through r_j.
#include "dart_common.hpp"
#include "dart_internal.hpp"

namespace dart {
namespace {

constexpr int kP = 64;
constexpr int kGT = 256;  // threads per block
constexpr int kTileTok = 32;  // tokens per SMA block at most

// Thread layout over an N x P state: row group rg = tid / 16 holds rows
// rg + 16 k (k < N / 16, so N >= 16), column quad pq = tid % 16 holds
// columns 4 pq .. 4 pq + 3.
template <int N>
struct StateLayout {
    static constexpr int RK = N / 16;
    static_assert(N % 16 == 0, "N must be a multiple of 16");
};

// ---- scan --------------------------------------------------------------------------
constexpr int kScanTok = 32;  // tokens staged per barrier in k_gscan_chunk

template <typename T, int N>
__global__ __launch_bounds__(kGT) void k_gscan_chunk(const T* __restrict__ x,
                                                     const float* __restrict__ dt,
                                                     const float* __restrict__ A,
                                                     const T* __restrict__ Bm, T* __restrict__ mem,
                                                     float* __restrict__ dh32,
                                                     float* __restrict__ lda, int64_t L, int H,
                                                     int G, int S, int64_t M, int64_t Mcap) {
    constexpr int RK = StateLayout<N>::RK;
    const int64_t c = blockIdx.x;
    const int h = blockIdx.y;
    const int64_t b = blockIdx.z;
    const int g = (int)((int64_t)h * G / H);
    const int tid = threadIdx.x, rg = tid >> 4, pq = tid & 15;
    const int64_t t0 = c * S;
    const int64_t t1 = t0 + S < L ? t0 + S : L;
    const float Ah = A[h];
    __shared__ float s_x[kScanTok][kP], s_B[kScanTok][N], s_d[kScanTok];
    float st[RK][4];
#pragma unroll
    for (int k = 0; k < RK; ++k)
#pragma unroll
        for (int i = 0; i < 4; ++i) st[k][i] = 0.f;
    float la = 0.f;
    for (int64_t tb = t0; tb < t1; tb += kScanTok) {
        const int nt = (int)(t1 - tb < kScanTok ? t1 - tb : kScanTok);
        __syncthreads();
        for (int e = tid; e < nt * kP; e += kGT) {
            const int k = e / kP, p = e % kP;
            s_x[k][p] = to_f(x[((b * L + tb + k) * H + h) * kP + p]);
        }
        for (int e = tid; e < nt * N; e += kGT) {
            const int k = e / N, n = e % N;
            s_B[k][n] = to_f(Bm[((b * L + tb + k) * G + g) * N + n]);
        }
        if (tid < nt) s_d[tid] = dt[(b * L + tb + tid) * H + h];
        __syncthreads();
        for (int k = 0; k < nt; ++k) {
            const float d = s_d[k];
            const float a = __expf(d * Ah);
            la += d * Ah;
#pragma unroll
            for (int kk = 0; kk < RK; ++kk) {
                const float bn = d * s_B[k][rg + 16 * kk];
#pragma unroll
                for (int i = 0; i < 4; ++i) st[kk][i] = a * st[kk][i] + bn * s_x[k][4 * pq + i];
            }
        }
    }
    const int64_t ch = (b * M + c) * H + h;
#pragma unroll
    for (int k = 0; k < RK; ++k) {
        const int o = (rg + 16 * k) * kP + 4 * pq;
        store4(dh32 + ch * (int64_t)N * kP + o, st[k]);
        if (mem) store4(mem + ((b * Mcap + c) * H + h) * (int64_t)N * kP + o, st[k]);
    }
    if (tid == 0) lda[(b * H + h) * M + c] = la;
}

template <typename T>
__global__ __launch_bounds__(kGT) void k_gscan_pass(const float* __restrict__ dh32,
                                                    const float* __restrict__ lda,
                                                    const float* __restrict__ h0,
                                                    float* __restrict__ st32, T* __restrict__ states,
                                                    float* __restrict__ h_last, int H, int NP,
                                                    int64_t M) {
    const int h = blockIdx.y;
    const int64_t b = blockIdx.z;
    const int e0 = (blockIdx.x * kGT + threadIdx.x) * 4;
    if (e0 >= NP) return;
    float hc[4] = {0.f, 0.f, 0.f, 0.f};
    if (h0) load4(h0 + (b * H + h) * (int64_t)NP + e0, hc);
    for (int64_t c = 0; c < M; ++c) {
        const int64_t o = ((b * M + c) * H + h) * (int64_t)NP + e0;
        store4(st32 + o, hc);
        if (states) store4(states + o, hc);
        float d4[4];
        load4(dh32 + o, d4);
        const float a = __expf(lda[(b * H + h) * M + c]);
#pragma unroll
        for (int i = 0; i < 4; ++i) hc[i] = a * hc[i] + d4[i];
    }
    if (h_last) store4(h_last + (b * H + h) * (int64_t)NP + e0, hc);
}

template <typename T, int N>
__global__ __launch_bounds__(kGT) void k_gscan_out(const T* __restrict__ x,
                                                   const float* __restrict__ dt,
                                                   const float* __restrict__ A,
                                                   const T* __restrict__ Bm, const T* __restrict__ Cm,
                                                   const float* __restrict__ st32,
                                                   T* __restrict__ y, int64_t L, int H, int G, int S,
                                                   int64_t M) {
    constexpr int RK = StateLayout<N>::RK;
    const int64_t c = blockIdx.x;
    const int h = blockIdx.y;
    const int64_t b = blockIdx.z;
    const int g = (int)((int64_t)h * G / H);
    const int tid = threadIdx.x, rg = tid >> 4, pq = tid & 15;
    const int64_t t0 = c * S;
    const int64_t t1 = t0 + S < L ? t0 + S : L;
    const float Ah = A[h];
    __shared__ float s_x[2][kP], s_B[2][N], s_C[2][N];
    __shared__ float s_d[2];
    __shared__ float s_y[2][16][kP];
    float st[RK][4];
    const float* src = st32 + ((b * M + c) * H + h) * (int64_t)N * kP;
#pragma unroll
    for (int k = 0; k < RK; ++k) load4(src + (rg + 16 * k) * kP + 4 * pq, st[k]);
    // token t uses buffer (t - t0) & 1; one barrier per token orders both the
    // staged inputs and the partial sums of the previous token
    for (int64_t t = t0; t < t1; ++t) {
        const int bf = (int)((t - t0) & 1);
        if (tid < kP) s_x[bf][tid] = to_f(x[((b * L + t) * H + h) * kP + tid]);
        if (tid < N) {
            s_B[bf][tid] = to_f(Bm[((b * L + t) * G + g) * N + tid]);
            s_C[bf][tid] = to_f(Cm[((b * L + t) * G + g) * N + tid]);
        }
        if (tid == 0) s_d[bf] = dt[(b * L + t) * H + h];
        __syncthreads();
        if (t > t0 && tid < kP) {
            float ys = 0.f;
#pragma unroll
            for (int r = 0; r < 16; ++r) ys += s_y[bf ^ 1][r][tid];
            y[((b * L + (t - 1)) * H + h) * kP + tid] = from_f<T>(ys);
        }
        const float d = s_d[bf];
        const float a = __expf(d * Ah);
        float yp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < RK; ++k) {
            const int n = rg + 16 * k;
            const float bn = d * s_B[bf][n], cn = s_C[bf][n];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                st[k][i] = a * st[k][i] + bn * s_x[bf][4 * pq + i];
                yp[i] += cn * st[k][i];
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) s_y[bf][rg][4 * pq + i] = yp[i];
        // the next token's barrier (or the one below) orders these writes
        // before their sum; the buffer is rewritten two tokens later, after
        // the reads of the next token's barrier interval
    }
    __syncthreads();
    if (t1 > t0 && tid < kP) {
        const int bf = (int)((t1 - 1 - t0) & 1);
        float ys = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) ys += s_y[bf][r][tid];
        y[((b * L + (t1 - 1)) * H + h) * kP + tid] = from_f<T>(ys);
    }
}

// ---- SMA: shared staging -----------------------------------------------------------
// Memory j of head h in LDS as float with rows padded to kP + 1 (row reads by
// lane n and column reads by lane p are both conflict-free), and its row
// inverse-RMS r[n] (1 without normalisation).
template <typename T, int N>
__device__ __forceinline__ void stage_memory(const T* __restrict__ src, float (*hm)[kP + 1],
                                             float* r, float eps, int normalize) {
    const int tid = threadIdx.x;
    for (int e = tid; e < N * kP; e += kGT) hm[e / kP][e % kP] = to_f(src[e]);
    __syncthreads();
    if (tid < N) {
        float ss = 0.f;
        for (int p = 0; p < kP; ++p) ss += hm[tid][p] * hm[tid][p];
        r[tid] = normalize ? 1.0f / sqrtf(ss * (1.0f / kP) + eps) : 1.0f;
    }
    __syncthreads();
}

// Qbar = RMSNorm(q) w and Ebar = RMSNorm(e) w of one token, by one wave
// (without normalisation the raw vectors).
template <typename T, int N>
__device__ __forceinline__ void norm_rows(const T* __restrict__ qrow, const T* __restrict__ erow,
                                          const float* __restrict__ qw, const float* __restrict__ ew,
                                          float eps, int normalize, float* qb, float* eb) {
    const int lane = threadIdx.x & 63;
    float qv[(N + 63) / 64];
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < (N + 63) / 64; ++k) {
        const int n = lane + 64 * k;
        qv[k] = n < N ? to_f(qrow[n]) : 0.f;
        ss += qv[k] * qv[k];
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o, 64);
    const float qi = normalize ? 1.0f / sqrtf(ss * (1.0f / N) + eps) : 1.0f;
#pragma unroll
    for (int k = 0; k < (N + 63) / 64; ++k) {
        const int n = lane + 64 * k;
        if (n < N) qb[n] = qv[k] * qi * (qw ? qw[n] : 1.0f);
    }
    const float ev = to_f(erow[lane]);
    float es = ev * ev;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) es += __shfl_xor(es, o, 64);
    const float ei = normalize ? 1.0f / sqrtf(es * (1.0f / kP) + eps) : 1.0f;
    eb[lane] = ev * ei * (ew ? ew[lane] : 1.0f);
}

__device__ __forceinline__ float wave_sum64(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// ---- SMA forward -------------------------------------------------------------------
// Block (tile of up to 32 tokens of chunk i, head h, batch b), 4 waves; wave w
// serves tokens w, w + 4, ... of the tile, lane = p.  Each token's online
// softmax state (m, d, O[P]) lives in LDS.
template <typename T, int N>
__global__ __launch_bounds__(kGT) void k_gsma(
    const T* __restrict__ q, const T* __restrict__ e, const T* __restrict__ Cm,
    const T* __restrict__ mem, const T* __restrict__ z, const T* __restrict__ y_ssd,
    T* __restrict__ y, float* __restrict__ lse, const float* __restrict__ qw,
    const float* __restrict__ ew, float eps, int normalize, int z_per_head, int64_t L, int H,
    int G, int S, int64_t Mcap, int tiles) {
    const int64_t i = blockIdx.x / tiles;
    const int tile = (int)(blockIdx.x % tiles);
    const int h = blockIdx.y;
    const int64_t b = blockIdx.z;
    const int g = (int)((int64_t)h * G / H);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t tb = i * S + (int64_t)tile * kTileTok;
    const int64_t cend = (i + 1) * S < L ? (i + 1) * S : L;
    if (tb >= cend) return;
    const int ntok = (int)(cend - tb < kTileTok ? cend - tb : kTileTok);
    __shared__ float s_q[kTileTok][N], s_e[kTileTok][kP], s_c[kTileTok][N];
    __shared__ float s_h[N][kP + 1];
    __shared__ float s_r[N];
    __shared__ float s_o[kTileTok][kP], s_m[kTileTok], s_d[kTileTok];
    const float isn = 1.0f / sqrtf((float)N);
    for (int k = wave; k < ntok; k += 4) {
        const int64_t bt = b * L + tb + k;
        norm_rows<T, N>(q + (bt * G + g) * N, e + (bt * G + g) * kP, qw, ew, eps, normalize,
                        s_q[k], s_e[k]);
        for (int n = lane; n < N; n += 64) s_c[k][n] = to_f(Cm[(bt * G + g) * N + n]);
        s_o[k][lane] = 0.f;
        if (lane == 0) {
            s_m[k] = -INFINITY;
            s_d[k] = 0.f;
        }
    }
    for (int64_t j = 0; j < i; ++j) {
        __syncthreads();
        stage_memory<T, N>(mem + ((b * Mcap + j) * H + h) * (int64_t)N * kP, s_h, s_r, eps, normalize);
        for (int k = wave; k < ntok; k += 4) {
            float up = 0.f, vp = 0.f;
#pragma unroll 8
            for (int n = 0; n < N; ++n) {
                const float hv = s_h[n][lane];
                up += s_q[k][n] * s_r[n] * hv;
                vp += s_c[k][n] * hv;
            }
            const float l = wave_sum64(s_e[k][lane] * up) * isn;
            const float mo = s_m[k];
            const float mn = fmaxf(mo, l);
            const float al = __expf(mo - mn), pw = __expf(l - mn);
            s_o[k][lane] = s_o[k][lane] * al + pw * vp;
            // every lane has read m and d before lane 0 rewrites them
            const float dn = s_d[k] * al + pw;
            __builtin_amdgcn_wave_barrier();
            if (lane == 0) {
                s_m[k] = mn;
                s_d[k] = dn;
            }
            __builtin_amdgcn_wave_barrier();
        }
    }
    for (int k = wave; k < ntok; k += 4) {
        const int64_t bt = b * L + tb + k;
        const int64_t yi = (bt * H + h) * kP + lane;
        if (i == 0) {
            y[yi] = y_ssd[yi];
            if (lse && lane == 0) lse[bt * H + h] = -INFINITY;
        } else {
            const float R = s_o[k][lane] / s_d[k];
            const float gz = silu(to_f(z[z_per_head ? bt * H + h : bt]));
            y[yi] = from_f<T>(to_f(y_ssd[yi]) + gz * R);
            if (lse && lane == 0) lse[bt * H + h] = s_m[k] + logf(s_d[k]);
        }
    }
}

// ---- SMA backward ------------------------------------------------------------------
// Per-(b, h, memory, token) arrays: the logit (then g p_j) and dy . V_j (then
// dl_j), row stride Ls; per (b, t, h): Dy.  part [B][L][H][2N+P]: per head
// dQbar, dEbar, dC of the token (the finishing kernel sums a group's heads).
// Per-token state in LDS as in the forward.
template <typename T, int N>
__global__ __launch_bounds__(kGT) void k_gsma_bwd_tok(
    const T* __restrict__ q, const T* __restrict__ e, const T* __restrict__ Cm,
    const T* __restrict__ mem, const T* __restrict__ z, const T* __restrict__ dy,
    const float* __restrict__ qw, const float* __restrict__ ew, float eps, int normalize,
    int z_per_head, float* __restrict__ gpw, float* __restrict__ dlw, float* __restrict__ rdy,
    float* __restrict__ part, int64_t L, int64_t Ls, int H, int G, int S, int64_t Mcap,
    int64_t Mp, int tiles) {
    const int64_t i = blockIdx.x / tiles + 1;  // chunks 1 .. M-1
    const int tile = (int)(blockIdx.x % tiles);
    const int h = blockIdx.y;
    const int64_t b = blockIdx.z;
    const int g = (int)((int64_t)h * G / H);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t tb = i * S + (int64_t)tile * kTileTok;
    const int64_t cend = (i + 1) * S < L ? (i + 1) * S : L;
    if (tb >= cend) return;
    const int ntok = (int)(cend - tb < kTileTok ? cend - tb : kTileTok);
    __shared__ float s_q[kTileTok][N], s_e[kTileTok][kP], s_c[kTileTok][N], s_dy[kTileTok][kP];
    __shared__ float s_h[N][kP + 1];
    __shared__ float s_r[N];
    __shared__ float s_dq[kTileTok][N], s_dc[kTileTok][N], s_de[kTileTok][kP];
    __shared__ float s_st[kTileTok][4];  // m, d, sum p dwy (then gate, Dy, lse)
    const float isn = 1.0f / sqrtf((float)N);
    for (int k = wave; k < ntok; k += 4) {
        const int64_t bt = b * L + tb + k;
        norm_rows<T, N>(q + (bt * G + g) * N, e + (bt * G + g) * kP, qw, ew, eps, normalize,
                        s_q[k], s_e[k]);
        for (int n = lane; n < N; n += 64) {
            s_c[k][n] = to_f(Cm[(bt * G + g) * N + n]);
            s_dq[k][n] = s_dc[k][n] = 0.f;
        }
        s_dy[k][lane] = to_f(dy[(bt * H + h) * kP + lane]);
        s_de[k][lane] = 0.f;
        if (lane == 0) {
            s_st[k][0] = -INFINITY;
            s_st[k][1] = s_st[k][2] = 0.f;
        }
    }
    auto sidx = [&](int64_t j, int k) { return ((b * H + h) * Mp + j) * Ls + tb + k; };
    // pass 1: logits, dy . V, online LSE and Dy
    for (int64_t j = 0; j < i; ++j) {
        __syncthreads();
        stage_memory<T, N>(mem + ((b * Mcap + j) * H + h) * (int64_t)N * kP, s_h, s_r, eps, normalize);
        for (int k = wave; k < ntok; k += 4) {
            float up = 0.f, vp = 0.f;
#pragma unroll 8
            for (int n = 0; n < N; ++n) {
                const float hv = s_h[n][lane];
                up += s_q[k][n] * s_r[n] * hv;
                vp += s_c[k][n] * hv;
            }
            const float l = wave_sum64(s_e[k][lane] * up) * isn;
            const float dw = wave_sum64(s_dy[k][lane] * vp);
            const float mo = s_st[k][0];
            const float mn = fmaxf(mo, l);
            const float al = __expf(mo - mn), pw = __expf(l - mn);
            const float dn = s_st[k][1] * al + pw, an = s_st[k][2] * al + pw * dw;
            __builtin_amdgcn_wave_barrier();
            if (lane == 0) {
                gpw[sidx(j, k)] = l;
                dlw[sidx(j, k)] = dw;
                s_st[k][0] = mn;
                s_st[k][1] = dn;
                s_st[k][2] = an;
            }
            __builtin_amdgcn_wave_barrier();
        }
    }
    __syncthreads();
    for (int k = wave; k < ntok; k += 4) {
        if (lane == 0) {
            const int64_t bt = b * L + tb + k;
            const float lsev = s_st[k][0] + logf(s_st[k][1]);
            const float Dy = s_st[k][2] / s_st[k][1];
            s_st[k][0] = silu(to_f(z[z_per_head ? bt * H + h : bt]));
            s_st[k][1] = Dy;
            s_st[k][2] = lsev;
            rdy[bt * H + h] = Dy;
        }
    }
    // pass 2: the gradients
    for (int64_t j = 0; j < i; ++j) {
        __syncthreads();
        stage_memory<T, N>(mem + ((b * Mcap + j) * H + h) * (int64_t)N * kP, s_h, s_r, eps, normalize);
        for (int k = wave; k < ntok; k += 4) {
            // every lane reads the logit and dy . V that lane 0 wrote in pass 1
            // (the barriers since then order the writes before these reads)
            const float l = gpw[sidx(j, k)];
            const float dw = dlw[sidx(j, k)];
            const float p = __expf(l - s_st[k][2]);
            const float gp = s_st[k][0] * p;
            const float dl = gp * (dw - s_st[k][1]);
            // lane = p: dEbar_p += dl s sum_n dH[n][p] r_n Qbar_n
            float up = 0.f;
#pragma unroll 8
            for (int n = 0; n < N; ++n) up += s_q[k][n] * s_r[n] * s_h[n][lane];
            s_de[k][lane] += dl * isn * up;
            // lane = n: dQbar_n += dl s r_n K_n, dC_n += g p_j (dH dy)_n
            for (int n = lane; n < N; n += 64) {
                float kn = 0.f, xn = 0.f;
#pragma unroll 8
                for (int pp = 0; pp < kP; ++pp) {
                    const float hv = s_h[n][pp];
                    kn += hv * s_e[k][pp];
                    xn += hv * s_dy[k][pp];
                }
                s_dq[k][n] += dl * isn * s_r[n] * kn;
                s_dc[k][n] += gp * xn;
            }
            __builtin_amdgcn_wave_barrier();
            if (lane == 0) {
                gpw[sidx(j, k)] = gp;
                dlw[sidx(j, k)] = dl;
            }
        }
    }
    for (int k = wave; k < ntok; k += 4) {
        const int64_t bt = b * L + tb + k;
        float* pr = part + (bt * H + h) * (int64_t)(2 * N + kP);
        for (int n = lane; n < N; n += 64) {
            pr[n] = s_dq[k][n];
            pr[N + kP + n] = s_dc[k][n];
        }
        pr[N + lane] = s_de[k][lane];
    }
}

// Tokens of chunk 0 (no history): zero partials and Dy.
__global__ __launch_bounds__(kGT) void k_gsma_bwd_zero(float* __restrict__ part,
                                                      float* __restrict__ rdy, int64_t L, int H,
                                                      int S, int NP2, int64_t B) {
    const int64_t idx = (int64_t)blockIdx.x * kGT + threadIdx.x;
    const int64_t t0n = L < S ? L : S;
    const int64_t rows = B * t0n * H;
    if (idx >= rows) return;
    const int h = (int)(idx % H);
    const int64_t t = (idx / H) % t0n;
    const int64_t b = idx / (H * t0n);
    const int64_t bt = b * L + t;
    rdy[bt * H + h] = 0.f;
    float* pr = part + (bt * H + h) * (int64_t)NP2;
    for (int k = 0; k < NP2; ++k) pr[k] = 0.f;
}

// Memory side: per (b, h, memory j), thread elements as StateLayout, tokens
// staged 32 at a time.
template <typename T, int N>
__global__ __launch_bounds__(kGT) void k_gsma_bwd_mem(
    const T* __restrict__ q, const T* __restrict__ e, const T* __restrict__ Cm,
    const T* __restrict__ dy, const T* __restrict__ mem, const float* __restrict__ qw,
    const float* __restrict__ ew, const float* __restrict__ gpw, const float* __restrict__ dlw,
    float* __restrict__ dmem, float eps, int normalize, int64_t L, int64_t Ls, int H, int G,
    int S, int64_t Mcap, int64_t Mp) {
    constexpr int RK = StateLayout<N>::RK;
    constexpr int TT = 32;
    const int64_t j = blockIdx.x;
    const int h = blockIdx.y;
    const int64_t b = blockIdx.z;
    const int g = (int)((int64_t)h * G / H);
    const int tid = threadIdx.x, rg = tid >> 4, pq = tid & 15, lane = tid & 63, wave = tid >> 6;
    float* out = dmem + ((b * Mcap + j) * H + h) * (int64_t)N * kP;
    if (j >= Mp) {
        for (int e0 = tid * 4; e0 < N * kP; e0 += kGT * 4) {
            float zz[4] = {0.f, 0.f, 0.f, 0.f};
            store4(out + e0, zz);
        }
        return;
    }
    __shared__ float s_q[TT][N], s_c[TT][N], s_e[TT][kP], s_dy[TT][kP], s_gp[TT], s_dl[TT];
    __shared__ float s_red[16][kP];
    __shared__ float s_rs[N];
    const float isn = 1.0f / sqrtf((float)N);
    float m1[RK][4], m2[RK][4];
#pragma unroll
    for (int k = 0; k < RK; ++k)
#pragma unroll
        for (int i2 = 0; i2 < 4; ++i2) m1[k][i2] = m2[k][i2] = 0.f;
    const int64_t tbeg = (j + 1) * S;
    for (int64_t t0 = tbeg; t0 < L; t0 += TT) {
        const int nt = (int)(L - t0 < TT ? L - t0 : TT);
        __syncthreads();
        for (int k = wave; k < nt; k += 4) {
            const int64_t bt = b * L + t0 + k;
            norm_rows<T, N>(q + (bt * G + g) * N, e + (bt * G + g) * kP, qw, ew, eps, normalize,
                            s_q[k], s_e[k]);
            for (int n = lane; n < N; n += 64) s_c[k][n] = to_f(Cm[(bt * G + g) * N + n]);
            s_dy[k][lane] = to_f(dy[(bt * H + h) * kP + lane]);
            if (lane == 0) {
                const int64_t si = ((b * H + h) * Mp + j) * Ls + t0 + k;
                s_gp[k] = gpw[si];
                s_dl[k] = dlw[si] * isn;
            }
        }
        __syncthreads();
        for (int k = 0; k < nt; ++k) {
#pragma unroll
            for (int kk = 0; kk < RK; ++kk) {
                const int n = rg + 16 * kk;
                const float cg = s_gp[k] * s_c[k][n], qd = s_dl[k] * s_q[k][n];
#pragma unroll
                for (int i2 = 0; i2 < 4; ++i2) {
                    m1[kk][i2] += cg * s_dy[k][4 * pq + i2];
                    m2[kk][i2] += qd * s_e[k][4 * pq + i2];
                }
            }
        }
    }
    // through r_j: ddH = M1 + r M2 - (r^3 / P) rowsum(dH M2) dH
    const T* hsrc = mem + ((b * Mcap + j) * H + h) * (int64_t)N * kP;
    float hv[RK][4];
#pragma unroll
    for (int kk = 0; kk < RK; ++kk) load4(hsrc + (rg + 16 * kk) * kP + 4 * pq, hv[kk]);
    // row sums over p: the 16 column-quad threads of a row, through LDS
    for (int kk = 0; kk < RK; ++kk) {
        float s1 = 0.f, s2 = 0.f;
#pragma unroll
        for (int i2 = 0; i2 < 4; ++i2) {
            s1 += hv[kk][i2] * hv[kk][i2];
            s2 += hv[kk][i2] * m2[kk][i2];
        }
        __syncthreads();
        s_red[rg][pq] = s1;
        s_red[rg][16 + pq] = s2;
        __syncthreads();
        if (tid < 16) {
            float a1 = 0.f, a2 = 0.f;
            for (int c2 = 0; c2 < 16; ++c2) {
                a1 += s_red[tid][c2];
                a2 += s_red[tid][16 + c2];
            }
            s_rs[tid + 16 * kk] = a1;
            s_red[tid][32] = a2;
        }
        __syncthreads();
        const int n = rg + 16 * kk;
        float o4[4];
        if (normalize) {
            const float r = 1.0f / sqrtf(s_rs[n] * (1.0f / kP) + eps);
            const float dr = s_red[rg][32];
#pragma unroll
            for (int i2 = 0; i2 < 4; ++i2)
                o4[i2] = m1[kk][i2] + r * m2[kk][i2] - (r * r * r * (1.0f / kP)) * dr * hv[kk][i2];
        } else {
#pragma unroll
            for (int i2 = 0; i2 < 4; ++i2) o4[i2] = m1[kk][i2] + m2[kk][i2];
        }
        store4(out + n * kP + 4 * pq, o4);
    }
}

// ---- launchers -----------------------------------------------------------------------
template <typename T, int N>
hipError_t run_gscan(const Shape& s, const void* x, const float* dt, const float* A,
                     const void* Bm, const void* Cm, const float* h0, void* y, void* mem,
                     float* hl, const GenScanWs& w, hipStream_t st) {
    const dim3 grid((unsigned)s.M, (unsigned)s.H, (unsigned)s.B);
    prof_begin("k_gscan_chunk", st);
    k_gscan_chunk<T, N><<<grid, kGT, 0, st>>>((const T*)x, dt, A, (const T*)Bm, (T*)mem, w.dh32,
                                              w.lda, s.L, s.H, s.G, s.S, s.M, s.Mcap);
    prof_end(st);
    const int NP = N * kP;
    prof_begin("k_gscan_pass", st);
    k_gscan_pass<T><<<dim3((unsigned)((NP / 4 + kGT - 1) / kGT), (unsigned)s.H, (unsigned)s.B), kGT,
                      0, st>>>(w.dh32, w.lda, h0, w.st32, (T*)w.states, hl, s.H, NP, s.M);
    prof_end(st);
    prof_begin("k_gscan_out", st);
    k_gscan_out<T, N><<<grid, kGT, 0, st>>>((const T*)x, dt, A, (const T*)Bm, (const T*)Cm, w.st32,
                                            (T*)y, s.L, s.H, s.G, s.S, s.M);
    prof_end(st);
    return hipGetLastError();
}

template <typename T, int N>
hipError_t run_gsma(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                    const void* Cm, const void* mem, const void* z, const void* ys, void* y,
                    float* lse, hipStream_t st) {
    const int tiles = (s.S + kTileTok - 1) / kTileTok;
    prof_begin("k_gsma", st);
    k_gsma<T, N><<<dim3((unsigned)(s.M * tiles), (unsigned)s.H, (unsigned)s.B), kGT, 0, st>>>(
        (const T*)q, (const T*)e, (const T*)Cm, (const T*)mem, (const T*)z, (const T*)ys, (T*)y,
        lse, a.qw, a.ew, a.eps, a.normalize, a.z_per_head, s.L, s.H, s.G, s.S, s.Mcap, tiles);
    prof_end(st);
    return hipGetLastError();
}

template <typename T, int N>
hipError_t run_gsma_bwd(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                        const void* Cm, const void* mem, const void* z, const void* dy,
                        const GenBwdWs& w, float* dmem, hipStream_t st) {
    const int64_t Mp = s.M > 1 ? s.M - 1 : 0;
    const int tiles = (s.S + kTileTok - 1) / kTileTok;
    const int NP2 = 2 * s.N + kP;
    const int64_t zrows = s.B * (s.L < s.S ? s.L : s.S) * s.H;
    prof_begin("k_gsma_bwd_zero", st);
    k_gsma_bwd_zero<<<(unsigned)((zrows + kGT - 1) / kGT), kGT, 0, st>>>(w.part, w.rdy, s.L, s.H,
                                                                        s.S, NP2, s.B);
    prof_end(st);
    if (Mp > 0) {
        prof_begin("k_gsma_bwd_tok", st);
        k_gsma_bwd_tok<T, N><<<dim3((unsigned)(Mp * tiles), (unsigned)s.H, (unsigned)s.B), kGT, 0,
                               st>>>(
            (const T*)q, (const T*)e, (const T*)Cm, (const T*)mem, (const T*)z, (const T*)dy, a.qw,
            a.ew, a.eps, a.normalize, a.z_per_head, w.gp, w.dl, w.rdy, w.part, s.L, w.Ls, s.H, s.G,
            s.S, s.Mcap, Mp, tiles);
        prof_end(st);
    }
    prof_begin("k_gsma_bwd_mem", st);
    k_gsma_bwd_mem<T, N><<<dim3((unsigned)s.Mcap, (unsigned)s.H, (unsigned)s.B), kGT, 0, st>>>(
        (const T*)q, (const T*)e, (const T*)Cm, (const T*)dy, (const T*)mem, a.qw, a.ew, w.gp, w.dl,
        dmem, a.eps, a.normalize, s.L, w.Ls, s.H, s.G, s.S, s.Mcap, Mp);
    prof_end(st);
    return hipGetLastError();
}

template <typename T, int N>
hipError_t run_scan_states(const Shape& s, const void* x, const float* dt, const float* A,
                           const void* Bm, const float* h0, float* lda, float* dh32, float* st32,
                           hipStream_t st) {
    prof_begin("k_gscan_chunk", st);
    k_gscan_chunk<T, N><<<dim3((unsigned)s.M, (unsigned)s.H, (unsigned)s.B), kGT, 0, st>>>(
        (const T*)x, dt, A, (const T*)Bm, nullptr, dh32, lda, s.L, s.H, s.G, s.S, s.M, s.M);
    prof_end(st);
    const int NP = N * kP;
    prof_begin("k_gscan_pass", st);
    k_gscan_pass<T><<<dim3((unsigned)((NP / 4 + kGT - 1) / kGT), (unsigned)s.H, (unsigned)s.B), kGT,
                      0, st>>>(dh32, lda, h0, st32, nullptr, nullptr, s.H, NP, s.M);
    prof_end(st);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_scan_states_f32(const Shape& s, const void* x, const float* dt, const float* A,
                                  const void* Bm, const float* h0, float* lda, float* dh32,
                                  float* st32, hipStream_t st) {
#define DART_SS(T, NN) run_scan_states<T, NN>(s, x, dt, A, Bm, h0, lda, dh32, st32, st)
    if (s.dtype == 1) {
        switch (s.N) {
            case 16: return DART_SS(bf16, 16);
            case 32: return DART_SS(bf16, 32);
            case 64: return DART_SS(bf16, 64);
            case 128: return DART_SS(bf16, 128);
        }
    } else {
        switch (s.N) {
            case 16: return DART_SS(float, 16);
            case 32: return DART_SS(float, 32);
            case 64: return DART_SS(float, 64);
            case 128: return DART_SS(float, 128);
        }
    }
#undef DART_SS
    return hipErrorInvalidValue;
}

bool tuned_shape(const Shape& s) {
    return (s.N == 32 || s.N == 64 || s.N == 128) && (s.S == 64 || s.S == 128 || s.S == 256);
}

hipError_t launch_gscan(const Shape& s, const void* x, const float* dt, const float* A,
                        const void* Bm, const void* Cm, const float* h0, void* y_ssd, void* mem,
                        float* h_last, const GenScanWs& w, hipStream_t st) {
#define DART_GS(T, NN) run_gscan<T, NN>(s, x, dt, A, Bm, Cm, h0, y_ssd, mem, h_last, w, st)
    if (s.dtype == 1) {
        switch (s.N) {
            case 16: return DART_GS(bf16, 16);
            case 32: return DART_GS(bf16, 32);
            case 64: return DART_GS(bf16, 64);
            case 128: return DART_GS(bf16, 128);
        }
    } else {
        switch (s.N) {
            case 16: return DART_GS(float, 16);
            case 32: return DART_GS(float, 32);
            case 64: return DART_GS(float, 64);
            case 128: return DART_GS(float, 128);
        }
    }
#undef DART_GS
    return hipErrorInvalidValue;
}

hipError_t launch_gsma(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                       const void* Cm, const void* mem, const void* z, const void* y_ssd, void* y,
                       float* lse, hipStream_t st) {
#define DART_GM(T, NN) run_gsma<T, NN>(s, a, q, e, Cm, mem, z, y_ssd, y, lse, st)
    if (s.dtype == 1) {
        switch (s.N) {
            case 16: return DART_GM(bf16, 16);
            case 32: return DART_GM(bf16, 32);
            case 64: return DART_GM(bf16, 64);
            case 128: return DART_GM(bf16, 128);
        }
    } else {
        switch (s.N) {
            case 16: return DART_GM(float, 16);
            case 32: return DART_GM(float, 32);
            case 64: return DART_GM(float, 64);
            case 128: return DART_GM(float, 128);
        }
    }
#undef DART_GM
    return hipErrorInvalidValue;
}

hipError_t launch_gsma_bwd(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                           const void* Cm, const void* mem, const void* z, const void* dy,
                           const GenBwdWs& w, float* dmem, hipStream_t st) {
#define DART_GB(T, NN) run_gsma_bwd<T, NN>(s, a, q, e, Cm, mem, z, dy, w, dmem, st)
    if (s.dtype == 1) {
        switch (s.N) {
            case 16: return DART_GB(bf16, 16);
            case 32: return DART_GB(bf16, 32);
            case 64: return DART_GB(bf16, 64);
            case 128: return DART_GB(bf16, 128);
        }
    } else {
        switch (s.N) {
            case 16: return DART_GB(float, 16);
            case 32: return DART_GB(float, 32);
            case 64: return DART_GB(float, 64);
            case 128: return DART_GB(float, 128);
        }
    }
#undef DART_GB
    return hipErrorInvalidValue;
}

}  // namespace dart
