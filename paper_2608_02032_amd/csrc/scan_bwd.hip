// scan_bwd.hip -- backward of the chunked SSD scan and of its chunk memories.
//
// Paper: Sec. 2 (the recurrence H_t = a_t H_{t-1} + dt_t B_t^T x_t,
// y_t = C_t H_t, a_t = exp(dt_t A_h)) and Sec. 3 / App. A (the chunk memory
// dH_[c], the chunk's own contribution).  Gradients of
//   loss = sum_t dy_t . y_t + sum_c <dmem_c, dH_[c]> + <dh_last, H_{L-1}>
// with respect to x, dt, A, B, C and h0.  With Lam_t the adjoint of the
// token's input term u_t = dt_t B_t^T x_t (through later outputs, through
// H_{L-1} and through its own chunk's memory):
//   Lam_t = C_t^T dy_t + a_{t+1} Lam_{t+1} inside chunk c, starting at the
//           chunk's last token from W_c = R_c + dmem_c, where R_c is the
//           adjoint entering chunk c's end from the later chunks:
//           R_{M-1} = dh_last, R_{c-1} = e^{cs_e(c)} R_c + dR_c,
//           dR_c = sum_{s in c} e^{cs_s} C_s^T dy_s (cs inclusive within c),
//           dh0 = R_{-1};
//   dx_t = dt_t B_t Lam_t,  dB_t = dt_t Lam_t x_t,  dC_t = H_t dy_t;
//   the decay gradient, per (b, h) a reverse cumulative sum of scalars
//   (a_t <G_t, H_{t-1}> = <G_t, H_t> - <G_t, u_t> telescopes):
//     g_t = sum_{s >= t} (y_s . dy_s - dx_s . x_s) + <dh_last, H_{L-1}>
//           + sum_{c' >= c(t)} <dmem_c', dH_[c']>,
//   ddt_t = dx_t . x_t / dt_t + A_h g_t,  dA_h = sum_{b,t} dt_t g_t.
//
// Kernels, in launch order (after a forward scan into the workspace, which
// gives y_ssd, the memories, H_{L-1} and every chunk's entry state):
//   k_sbwd_chunk   per (b, c, h): dR_c and the chunk's total decay;
//   k_sbwd_pass    per (b, h, 1024 elements): the reverse chunk pass -> R_c,
//                  dh0;
//   k_sbwd_tokens  per (b, c, block of heads of one group): for each head a
//                  forward sweep over the chunk's tokens (H_t from the entry
//                  state, dC) and a reverse one (Lam_t, dx, dB).  Each of the
//                  4 waves holds N/4 rows of the N x P state, each lane N/16
//                  rows by 4 columns, so the sums over p are short in-lane
//                  sums plus a reduce-scatter over 16 lanes, and the sum over
//                  n of dx meets in LDS once per 16 tokens.  The same sweeps give
//                  the pieces of the decay gradient (y.dy, (B Lam).x and the
//                  memory terms) on one consistent trajectory;
//   k_sbwd_decay   per (b, h): the reverse cumulative sum -> ddt, dA partials;
//   k_sbwd_finish  per (b, t, g): dB, dC summed over the group's head blocks;
//                  dA summed over the batch.
#include "dart_common.hpp"
#include "dart_internal.hpp"

namespace dart {
namespace {

constexpr int kP = 64;
constexpr int kHpb = 4;  // heads per k_sbwd_tokens workgroup (at most)

__device__ __forceinline__ float block_sum(float v, float* red) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    __syncthreads();
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float s = 0.f;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) s += red[w];
    return s;
}

// ---- per (b, c, h): chunk adjoint and total decay -------------------------------
// Thread (n, slice of P/TPR columns); the running product e^{cs_s} advances
// token by token.
template <typename T, int N>
__global__ __launch_bounds__(256) void k_sbwd_chunk(const T* __restrict__ Cm,
                                                    const T* __restrict__ dy,
                                                    const float* __restrict__ dt,
                                                    const float* __restrict__ A,
                                                    float* __restrict__ dR,
                                                    float* __restrict__ dec, int64_t L, int H,
                                                    int G, int S, int64_t M) {
    constexpr int TPR = 256 / N;
    constexpr int PPT = kP / TPR;
    const int64_t c = blockIdx.x;
    const int h = blockIdx.y;
    const int64_t b = blockIdx.z;
    const int g = h / (H / G);
    const int tid = threadIdx.x;
    const int n = tid / TPR, p0 = (tid % TPR) * PPT;
    const int64_t a0 = c * S;
    const int64_t e = (c + 1) * S < L ? (c + 1) * S - 1 : L - 1;
    const float Ah = A[h];
    float acc[PPT];
#pragma unroll
    for (int i = 0; i < PPT; ++i) acc[i] = 0.f;
    float w = 1.f;
    for (int64_t s = a0; s <= e; ++s) {
        w *= __expf(dt[(b * L + s) * H + h] * Ah);
        const float cw = w * to_f(Cm[((b * L + s) * G + g) * N + n]);
        const T* dyr = dy + ((b * L + s) * H + h) * kP + p0;
#pragma unroll
        for (int i = 0; i < PPT; i += 4) {
            float d4[4];
            load4(dyr + i, d4);
#pragma unroll
            for (int k = 0; k < 4; ++k) acc[i + k] += cw * d4[k];
        }
    }
    float* out = dR + ((b * M + c) * H + h) * (int64_t)N * kP + n * kP + p0;
#pragma unroll
    for (int i = 0; i < PPT; i += 4) {
        float v4[4] = {acc[i], acc[i + 1], acc[i + 2], acc[i + 3]};
        store4(out + i, v4);
    }
    if (tid == 0) dec[(b * H + h) * M + c] = w;
}

// ---- per (b, h, element block): reverse chunk pass ----------------------------
__global__ __launch_bounds__(256) void k_sbwd_pass(const float* __restrict__ dR,
                                                   const float* __restrict__ dec,
                                                   const float* __restrict__ dhl,
                                                   float* __restrict__ Rs, float* __restrict__ dh0,
                                                   int H, int NP, int64_t M) {
    const int h = blockIdx.y;
    const int64_t b = blockIdx.z;
    const int e0 = (blockIdx.x * 256 + threadIdx.x) * 4;
    if (e0 >= NP) return;
    float r[4] = {0.f, 0.f, 0.f, 0.f};
    if (dhl) load4(dhl + (b * H + h) * (int64_t)NP + e0, r);
    for (int64_t c = M - 1; c >= 0; --c) {
        const int64_t ch = (b * M + c) * H + h;
        store4(Rs + ch * NP + e0, r);
        float d[4];
        load4(dR + ch * NP + e0, d);
        const float dc = dec[(b * H + h) * M + c];
#pragma unroll
        for (int i = 0; i < 4; ++i) r[i] = dc * r[i] + d[i];
    }
    if (dh0) store4(dh0 + (b * H + h) * (int64_t)NP + e0, r);
}

template <int K>
__device__ __forceinline__ void load_k(const bf16* p, float (&v)[K]) {
    if constexpr (K % 8 == 0) {
#pragma unroll
        for (int i = 0; i < K; i += 8) {
            float t[8];
            load8(p + i, t);
#pragma unroll
            for (int k = 0; k < 8; ++k) v[i + k] = t[k];
        }
    } else if constexpr (K == 4) {
        load4(p, v);
    } else {
#pragma unroll
        for (int i = 0; i < K; ++i) v[i] = (float)p[i];
    }
}
template <int K>
__device__ __forceinline__ void load_k(const float* p, float (&v)[K]) {
    if constexpr (K % 4 == 0) {
#pragma unroll
        for (int i = 0; i < K; i += 4) {
            float t[4];
            load4(p + i, t);
#pragma unroll
            for (int k = 0; k < 4; ++k) v[i + k] = t[k];
        }
    } else {
#pragma unroll
        for (int i = 0; i < K; ++i) v[i] = p[i];
    }
}

// K storage elements kept raw in registers (converted where used), so that a
// load issued one token ahead is not waited for at once.
template <typename T, int K>
struct alignas(sizeof(T) * K >= 16 ? 16 : sizeof(T) * K) RawVec {
    T v[K];
};
template <typename T, int K>
__device__ __forceinline__ RawVec<T, K> raw_load(const T* p) {
    return *reinterpret_cast<const RawVec<T, K>*>(p);
}

// ---- per (b, c, head block): the two sweeps ----------------------------------------
// Wave w holds state rows n0 = w N/4 .. n0 + N/4 - 1; inside the wave lane
// (ng, pg) = (lane / 16, lane % 16) holds the RL = N/16 rows n0 + ng RL + i and
// the 4 columns 4 pg + c.  Sums over p (dC, dB) are then 4-term in-lane sums
// followed by a reduce-scatter over the 16 pg lanes; the sum over n of dx is an
// in-lane sum over RL rows, a reduce-scatter over the 4 ng lanes and an LDS
// exchange between the waves once per 16 tokens.
// Besides dx, dB and dC this records, per wave, the pieces of the decay
// gradient that the same recomputed trajectory gives: y_t . dy_t
// (= C_t . dC_t), (B_t Lam_t) . x_t, and <dmem_c, dH_[c]> (+ <dh_last, H_{L-1}>
// in the last chunk), so that the reverse cumulative sum telescopes exactly.
template <typename T, int N>
__global__ __launch_bounds__(256) void k_sbwd_tokens(
    const T* __restrict__ x, const float* __restrict__ dt, const float* __restrict__ A,
    const T* __restrict__ Bm, const T* __restrict__ Cm, const T* __restrict__ dy,
    const float* __restrict__ states, const float* __restrict__ Rs, const float* __restrict__ dmem,
    const float* __restrict__ dhl, float* __restrict__ dx, float* __restrict__ bxl,
    float* __restrict__ ydyp, float* __restrict__ mdp, float* __restrict__ dBp,
    float* __restrict__ dCp, int64_t L, int H, int G, int S, int64_t M, int64_t Mcap, int hpb) {
    constexpr int RL = N / 16;       // rows per lane
    constexpr int GRP = 16 / RL;     // pg lanes that share one row sum
    constexpr int TB = 16;           // tokens per dx exchange
    __shared__ float xpart[2][TB][4][kP];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int ng = lane >> 4, pg = lane & 15;
    const int64_t c = blockIdx.x;
    const int hb = blockIdx.y;
    const int64_t b = blockIdx.z;
    const int nhb = H / hpb;
    const int h0 = hb * hpb;
    const int g = h0 / (H / G);
    const int nl = wave * (N / 4) + ng * RL;  // first row of this lane
    const int pl = pg * 4;                    // first column of this lane
    const int64_t a0 = c * S;
    const int64_t e = (c + 1) * S < L ? (c + 1) * S - 1 : L - 1;
    const int nsum = wave * (N / 4) + ng * RL + pg / GRP;  // row of this lane's sum
    const bool writer = pg % GRP == 0;

    for (int hh = 0; hh < hpb; ++hh) {
        const int h = h0 + hh;
        const float Ah = A[h];
        const int64_t ch = (b * M + c) * H + h;
        const int64_t sm = ((b * Mcap + c) * H + h) * (int64_t)N * kP;
        // forward sweep: H_t from the entry state; dC_t = H_t dy_t; the
        // chunk's own contribution dH accumulates beside it
        float st[RL][4], dh[RL][4];
#pragma unroll
        for (int i = 0; i < RL; ++i) {
            float t4[4];
            load4(states + ch * (int64_t)N * kP + (nl + i) * kP + pl, t4);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                st[i][k] = t4[k];
                dh[i][k] = 0.f;
            }
        }
        // the next token's rows are loaded while this one is swept
        RawVec<T, 4> xr, yr;
        RawVec<T, RL> br;
        float dn, on = 0.f;  // on: the previous heads' partial of the row sum
        const bool rmw = hh > 0 && writer;
        auto fetch_f = [&](int64_t t) {
            const int64_t th = (b * L + t) * H + h;
            dn = dt[th];
            if (rmw) on = dCp[((b * L + t) * nhb + hb) * (int64_t)N + nsum];
            xr = raw_load<T, 4>(x + th * kP + pl);
            yr = raw_load<T, 4>(dy + th * kP + pl);
            br = raw_load<T, RL>(Bm + ((b * L + t) * G + g) * N + nl);
        };
        fetch_f(a0);
        for (int64_t t = a0; t <= e; ++t) {
            const int64_t th = (b * L + t) * H + h;
            const float d = dn, oc = on;
            const RawVec<T, 4> xc = xr, yc = yr;
            const RawVec<T, RL> bc = br;
            if (t < e) fetch_f(t + 1);
            const float a = __expf(d * Ah);
            float xv[4], dyv[4], bv[RL];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                xv[k] = to_f(xc.v[k]);
                dyv[k] = to_f(yc.v[k]);
            }
#pragma unroll
            for (int i = 0; i < RL; ++i) bv[i] = to_f(bc.v[i]);
#pragma unroll
            for (int k = 0; k < 4; ++k) xv[k] *= d;
            float v[RL];
#pragma unroll
            for (int i = 0; i < RL; ++i) {
                float acc = 0.f;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const float u = bv[i] * xv[k];
                    st[i][k] = a * st[i][k] + u;
                    dh[i][k] = a * dh[i][k] + u;
                    acc += st[i][k] * dyv[k];
                }
                v[i] = acc;
            }
            const float sc = lane_sums<RL, 16>(v, lane);
            if (writer) dCp[((b * L + t) * nhb + hb) * (int64_t)N + nsum] = oc + sc;
            // y_t . dy_t over this wave's rows: C_n dC_n summed over the rows
            float yd = writer ? to_f(Cm[((b * L + t) * G + g) * N + nsum]) * sc : 0.f;
#pragma unroll
            for (int m = 32; m >= 1; m >>= 1) yd += __shfl_xor(yd, m, 64);
            if (lane == 0) ydyp[th * 4 + wave] = yd;
        }
        float md = 0.f;
        if (dmem) {
#pragma unroll
            for (int i = 0; i < RL; ++i) {
                float t4[4];
                load4(dmem + sm + (nl + i) * kP + pl, t4);
#pragma unroll
                for (int k = 0; k < 4; ++k) md += t4[k] * dh[i][k];
            }
        }
        if (dhl && c == M - 1) {
            const float* hr = dhl + (b * H + h) * (int64_t)N * kP;
#pragma unroll
            for (int i = 0; i < RL; ++i) {
                float t4[4];
                load4(hr + (nl + i) * kP + pl, t4);
#pragma unroll
                for (int k = 0; k < 4; ++k) md += t4[k] * st[i][k];
            }
        }
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) md += __shfl_xor(md, m, 64);
        if (lane == 0) mdp[((b * H + h) * M + c) * 4 + wave] = md;

        // reverse sweep: Lam from W_c = R_c + dmem_c; dx, dB
        float lam[RL][4];
#pragma unroll
        for (int i = 0; i < RL; ++i) {
            const int64_t o = (nl + i) * kP + pl;
            float r4[4], m4[4] = {0.f, 0.f, 0.f, 0.f};
            load4(Rs + ch * (int64_t)N * kP + o, r4);
            if (dmem) load4(dmem + sm + o, m4);
#pragma unroll
            for (int k = 0; k < 4; ++k) lam[i][k] = r4[k] + m4[k];
        }
        const int ntok = (int)(e - a0 + 1);
        RawVec<T, RL> cr;
        auto fetch_r = [&](int64_t t) {
            const int64_t th = (b * L + t) * H + h;
            dn = dt[th];
            if (rmw) on = dBp[((b * L + t) * nhb + hb) * (int64_t)N + nsum];
            xr = raw_load<T, 4>(x + th * kP + pl);
            yr = raw_load<T, 4>(dy + th * kP + pl);
            br = raw_load<T, RL>(Bm + ((b * L + t) * G + g) * N + nl);
            cr = raw_load<T, RL>(Cm + ((b * L + t) * G + g) * N + nl);
        };
        fetch_r(e);
        for (int k = 0; k < ntok; ++k) {
            const int64_t t = e - k;
            const float d = dn, ob = on;
            const RawVec<T, 4> xc = xr, yc = yr;
            const RawVec<T, RL> bc = br, cc = cr;
            if (k + 1 < ntok) fetch_r(t - 1);
            float xv[4], dyv[4], bv[RL], cv[RL];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                xv[q] = to_f(xc.v[q]);
                dyv[q] = to_f(yc.v[q]);
            }
#pragma unroll
            for (int i = 0; i < RL; ++i) {
                bv[i] = to_f(bc.v[i]);
                cv[i] = to_f(cc.v[i]);
            }
            float px[4] = {0.f, 0.f, 0.f, 0.f}, v[RL];
#pragma unroll
            for (int i = 0; i < RL; ++i) {
                float acc = 0.f;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    lam[i][q] += cv[i] * dyv[q];
                    px[q] += bv[i] * lam[i][q];
                    acc += lam[i][q] * xv[q];
                }
                v[i] = acc;
            }
            const float sb = lane_sums<RL, 16>(v, lane);
            if (writer) dBp[((b * L + t) * nhb + hb) * (int64_t)N + nsum] = ob + d * sb;
            // sum of px over the 4 ng lanes: lane (ng, pg) keeps column 4 pg + ng
            rs_step<4, 4, 32>(px, lane);
            const int slot = k % TB, buf = (k / TB) & 1;
            xpart[buf][slot][wave][pl + ng] = px[0];
            // carry to t - 1: Lam_{t-1} = C_{t-1}^T dy_{t-1} + a_t Lam_t
            const float a = __expf(d * Ah);
#pragma unroll
            for (int i = 0; i < RL; ++i)
#pragma unroll
                for (int q = 0; q < 4; ++q) lam[i][q] *= a;
            if (slot == TB - 1 || k == ntok - 1) {
                __syncthreads();
                // wave w finishes tokens w, w + 4, ... of this batch
                const int kb = k - slot;
                for (int q = wave; q <= slot; q += 4) {
                    const int64_t tq = (b * L + (e - (kb + q))) * H + h;
                    const float s4 = xpart[buf][q][0][lane] + xpart[buf][q][1][lane] +
                                     xpart[buf][q][2][lane] + xpart[buf][q][3][lane];
                    dx[tq * kP + lane] = dt[tq] * s4;
                    float pr = s4 * to_f(x[tq * kP + lane]);
#pragma unroll
                    for (int o = 32; o >= 1; o >>= 1) pr += __shfl_xor(pr, o, 64);
                    if (lane == 0) bxl[tq] = pr;
                }
            }
        }
        __syncthreads();
    }
}

// ---- per (b, h): the decay gradient by a reverse cumulative sum -------------------
// g_t = sum_{s >= t} (y_s . dy_s - dt_s (B_s Lam_s) . x_s) + sum_{c' >= c(t)} md_c',
// ddt_t = (B_t Lam_t) . x_t + A_h g_t, dA partial = sum_t dt_t g_t.
__global__ __launch_bounds__(256) void k_sbwd_decay(
    const float* __restrict__ dt, const float* __restrict__ A, const float* __restrict__ bxl,
    const float* __restrict__ ydyp, const float* __restrict__ mdp, float* __restrict__ ddt,
    float* __restrict__ dAp, float* __restrict__ mdsuf, int64_t L, int H, int S, int64_t M) {
    __shared__ float red[4];
    __shared__ float carry_s;
    const int h = blockIdx.x;
    const int64_t b = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const float Ah = A[h];
    // suffix sums over chunks of the memory (and final-state) terms
    float* suf = mdsuf + (b * H + h) * M;
    if (tid == 0) {
        float s = 0.f;
        for (int64_t c = M - 1; c >= 0; --c) {
            const float* m4 = mdp + ((b * H + h) * M + c) * 4;
            s += (m4[0] + m4[1]) + (m4[2] + m4[3]);
            suf[c] = s;
        }
        carry_s = 0.f;
    }
    __syncthreads();
    float dA = 0.f;
    const int64_t nblk = (L + 255) / 256;
    for (int64_t blk = 0; blk < nblk; ++blk) {
        // thread i takes token t = L - 1 - (256 blk + i): a suffix in token order
        const int64_t t = L - 1 - (blk * 256 + tid);
        float v = 0.f, d = 0.f, bx = 0.f;
        if (t >= 0) {
            const int64_t th = (b * L + t) * H + h;
            const float* y4 = ydyp + th * 4;
            d = dt[th];
            bx = bxl[th];
            v = (y4[0] + y4[1]) + (y4[2] + y4[3]) - d * bx;
        }
        float sc = v;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const float u = __shfl_up(sc, o, 64);
            if (lane >= o) sc += u;
        }
        if (lane == 63) red[wave] = sc;
        __syncthreads();
        float add = carry_s;
        for (int w2 = 0; w2 < wave; ++w2) add += red[w2];
        const float total = carry_s + red[0] + red[1] + red[2] + red[3];
        sc += add;
        if (t >= 0) {
            const float gsum = sc + suf[t / S];
            ddt[(b * L + t) * H + h] = bx + Ah * gsum;
            dA += d * gsum;
        }
        __syncthreads();
        if (tid == 0) carry_s = total;
        __syncthreads();
    }
    dA = block_sum(dA, red);
    if (tid == 0) dAp[b * H + h] = dA;
}

// ---- per (b, t, g): group sums of dB, dC; dA over the batch -----------------------
template <int N>
__global__ __launch_bounds__(256) void k_sbwd_finish(const float* __restrict__ dBp,
                                                     const float* __restrict__ dCp,
                                                     const float* __restrict__ dAp,
                                                     float* __restrict__ dB, float* __restrict__ dC,
                                                     float* __restrict__ dA, int64_t rows, int H,
                                                     int G, int hpb, int64_t B) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int nhb = H / hpb, per = (H / G) / hpb;
    if (i < rows * N) {
        const int64_t row = i / N;  // (b, t, g)
        const int n = (int)(i - row * N);
        const int g = (int)(row % G);
        const int64_t bt = row / G;
        float sb = 0.f, sc = 0.f;
        for (int k = 0; k < per; ++k) {
            const int hb = g * per + k;
            sb += dBp[(bt * nhb + hb) * (int64_t)N + n];
            sc += dCp[(bt * nhb + hb) * (int64_t)N + n];
        }
        dB[i] = sb;
        dC[i] = sc;
    }
    if (blockIdx.x == 0) {
        for (int h = threadIdx.x; h < H; h += 256) {
            float s = 0.f;
            for (int64_t b = 0; b < B; ++b) s += dAp[b * H + h];
            dA[h] = s;
        }
    }
}

int sbwd_heads_per_block(const Shape& s) {
    const int per = s.H / s.G;
    for (int c = kHpb; c > 1; --c)
        if (per % c == 0) return c;
    return 1;
}

struct SbwdWs {
    float* lda;
    float* dh32;
    float* st32;
    float* dR;
    float* Rs;
    float* dec;
    float* mdp;
    float* mdsuf;
    float* bxl;
    float* ydyp;
    float* dBp;
    float* dCp;
    float* dAp;
    size_t total;
};

// Workspace: the chunk log decays, chunk contributions and entry states of
// the forward recomputed in float, then the backward's: chunk adjoints dR
// and R, chunk decays, per-wave memory terms [B][H][M][4] and their suffix
// sums, per-token (B Lam) . x [B][L][H] and per-wave y . dy [B][L][H][4],
// per-head-block dB / dC partials [B][L][H/hpb][N], per-batch dA partials.
SbwdWs sbwd_layout(const Shape& s, void* base) {
    const size_t NP = (size_t)s.N * s.P;
    const size_t BLH = (size_t)s.B * s.L * s.H;
    const size_t BHM = (size_t)s.B * s.H * s.M;
    const int nhb = s.H / sbwd_heads_per_block(s);
    SbwdWs w;
    size_t o = 0;
    char* p = reinterpret_cast<char*>(base);
    auto take = [&](size_t bytes) {
        char* r = p ? p + o : nullptr;
        o += align256(bytes);
        return r;
    };
    w.lda = (float*)take(4 * BHM);
    w.dh32 = (float*)take(4 * BHM * NP);
    w.st32 = (float*)take(4 * BHM * NP);
    w.dR = (float*)take(4 * BHM * NP);
    w.Rs = (float*)take(4 * BHM * NP);
    w.dec = (float*)take(4 * BHM);
    w.mdp = (float*)take(16 * BHM);
    w.mdsuf = (float*)take(4 * BHM);
    w.bxl = (float*)take(4 * BLH);
    w.ydyp = (float*)take(16 * BLH);
    w.dBp = (float*)take(4 * (size_t)s.B * s.L * nhb * s.N);
    w.dCp = (float*)take(4 * (size_t)s.B * s.L * nhb * s.N);
    w.dAp = (float*)take(4 * (size_t)s.B * s.H);
    w.total = o;
    return w;
}

template <typename T, int N>
hipError_t run_sbwd(const Shape& s, const void* x, const float* dt, const float* A,
                    const void* Bm, const void* Cm, const float* h0, const void* dy,
                    const float* dmem, const float* dhl, float* dx, float* ddt, float* dA,
                    float* dB, float* dC, float* dh0, void* ws, hipStream_t st) {
    const SbwdWs w = sbwd_layout(s, ws);
    // the forward again, in float, for every chunk's entry state
    hipError_t err = launch_scan_states_f32(s, x, dt, A, Bm, h0, w.lda, w.dh32, w.st32, st);
    if (err != hipSuccess) return err;
    const int hpb = sbwd_heads_per_block(s);
    const int NP = s.N * s.P;
    prof_begin("k_sbwd_chunk", st);
    k_sbwd_chunk<T, N><<<dim3((unsigned)s.M, (unsigned)s.H, (unsigned)s.B), 256, 0, st>>>(
        (const T*)Cm, (const T*)dy, dt, A, w.dR, w.dec, s.L, s.H, s.G, s.S, s.M);
    prof_end(st);
    prof_begin("k_sbwd_pass", st);
    k_sbwd_pass<<<dim3((unsigned)((NP / 4 + 255) / 256), (unsigned)s.H, (unsigned)s.B), 256, 0, st>>>(
        w.dR, w.dec, dhl, w.Rs, dh0, s.H, NP, s.M);
    prof_end(st);
    prof_begin("k_sbwd_tokens", st);
    k_sbwd_tokens<T, N><<<dim3((unsigned)s.M, (unsigned)(s.H / hpb), (unsigned)s.B), 256, 0, st>>>(
        (const T*)x, dt, A, (const T*)Bm, (const T*)Cm, (const T*)dy, w.st32, w.Rs, dmem, dhl, dx,
        w.bxl, w.ydyp, w.mdp, w.dBp, w.dCp, s.L, s.H, s.G, s.S, s.M, s.Mcap, hpb);
    prof_end(st);
    prof_begin("k_sbwd_decay", st);
    k_sbwd_decay<<<dim3((unsigned)s.H, (unsigned)s.B), 256, 0, st>>>(
        dt, A, w.bxl, w.ydyp, w.mdp, ddt, w.dAp, w.mdsuf, s.L, s.H, s.S, s.M);
    prof_end(st);
    const int64_t rows = s.B * s.L * s.G;
    prof_begin("k_sbwd_finish", st);
    k_sbwd_finish<N><<<(unsigned)((rows * N + 255) / 256), 256, 0, st>>>(
        w.dBp, w.dCp, w.dAp, dB, dC, dA, rows, s.H, s.G, hpb, s.B);
    prof_end(st);
    return hipGetLastError();
}

template <typename T>
hipError_t run_sbwd_n(const Shape& s, const void* x, const float* dt, const float* A,
                      const void* Bm, const void* Cm, const float* h0, const void* dy,
                      const float* dmem, const float* dhl, float* dx, float* ddt, float* dA,
                      float* dB, float* dC, float* dh0, void* ws, hipStream_t st) {
    switch (s.N) {
        case 16: return run_sbwd<T, 16>(s, x, dt, A, Bm, Cm, h0, dy, dmem, dhl, dx, ddt, dA, dB, dC, dh0, ws, st);
        case 32: return run_sbwd<T, 32>(s, x, dt, A, Bm, Cm, h0, dy, dmem, dhl, dx, ddt, dA, dB, dC, dh0, ws, st);
        case 64: return run_sbwd<T, 64>(s, x, dt, A, Bm, Cm, h0, dy, dmem, dhl, dx, ddt, dA, dB, dC, dh0, ws, st);
        case 128: return run_sbwd<T, 128>(s, x, dt, A, Bm, Cm, h0, dy, dmem, dhl, dx, ddt, dA, dB, dC, dh0, ws, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace

size_t ssd_bwd_workspace_bytes(const Shape& s) {
    return sbwd_mfma_shape(s) ? sbwd_mfma_workspace_bytes(s) : sbwd_layout(s, nullptr).total;
}

hipError_t launch_ssd_bwd(const Shape& s, const void* x, const float* dt, const float* A,
                          const void* Bm, const void* Cm, const float* h0, const void* dy,
                          const float* dmem, const float* dh_last, float* dx, float* ddt, float* dA,
                          float* dB, float* dC, float* dh0, void* ws, hipStream_t st) {
    if (sbwd_mfma_shape(s))
        return launch_ssd_bwd_mfma(s, x, dt, A, Bm, Cm, h0, dy, dmem, dh_last, dx, ddt, dA, dB, dC, dh0, ws, st);
    if (s.dtype == 1)
        return run_sbwd_n<bf16>(s, x, dt, A, Bm, Cm, h0, dy, dmem, dh_last, dx, ddt, dA, dB, dC, dh0, ws, st);
    return run_sbwd_n<float>(s, x, dt, A, Bm, Cm, h0, dy, dmem, dh_last, dx, ddt, dA, dB, dC, dh0, ws, st);
}

}  // namespace dart
