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
// Two kernels:
//   k_sma_prep  per (b, memory j, head): r_j[n] = (mean_p dH_j[n,p]^2 + eps)^-1/2
//               from the stored values; writes two copies of the memory in the
//               MFMA A-operand order (key side scaled by r_j, value side as
//               stored) so the main loop streams them with plain 16-byte loads.
//   k_sma_main  per (b, head, 256-token block; 4 waves x 64 tokens, each wave
//               inside one chunk): for every earlier memory j, on MFMA
//                 U^T = (r_j (.) dH_j)^T Qbar^T   (P x tokens)
//                 V^T = dH_j^T C^T                (P x tokens)
//               then l_t = sum_p U^T[p,t] Ebar[t,p] (the P axis lives in the
//               lane's own registers plus 2 cross-lane steps), an online
//               softmax in base 2, O = alpha O + g V.  Epilogue:
//               y = y_ssd + SiLU(z) O/d and LSE = (m + log2 d) ln 2.
// The transposed products put one token per lane column, so each lane owns its
// tokens' softmax statistics and no per-row broadcast is needed.
#include "dart_common.hpp"
#include "dart_internal.hpp"

namespace dart {
namespace {

constexpr int kP = 64;
constexpr int kThreads = 256;
constexpr int kPad = 8;
constexpr int kTokPerBlock = 256;

template <typename T, int N>
__global__ __launch_bounds__(kThreads) void k_sma_prep(const T* __restrict__ mem,
                                                        T* __restrict__ kfrag,
                                                        T* __restrict__ vfrag, float eps,
                                                        int normalize, int H, int64_t Mp,
                                                        int64_t Mcap) {
    const int64_t j = blockIdx.x;
    const int h = blockIdx.y;
    const int64_t b = blockIdx.z;
    const int tid = threadIdx.x;
    __shared__ __attribute__((aligned(16))) T sm[N][kP + kPad];
    __shared__ float sr[N];
    const T* src = mem + ((b * Mcap + j) * H + h) * (int64_t)N * kP;
    for (int ci = tid; ci < N * (kP / 8); ci += kThreads) {
        const int r = ci >> 3, k8 = ci & 7;
        float v[8];
        load8(src + r * kP + k8 * 8, v);
        store8(&sm[r][k8 * 8], v);
    }
    __syncthreads();
    if (tid < N) {
        float ss = 0.f;
#pragma unroll 8
        for (int p = 0; p < kP; ++p) {
            const float v = to_f(sm[tid][p]);
            ss += v * v;
        }
        sr[tid] = normalize ? 1.0f / sqrtf(ss * (1.0f / kP) + eps) : 1.0f;
    }
    __syncthreads();
    constexpr int kFrag = (N / 32) * 4;  // fragments (k step, p tile) per memory
    const int64_t base = ((b * Mp + j) * H + h) * (int64_t)N * kP;
    for (int pi = tid; pi < kFrag * 64; pi += kThreads) {
        const int f = pi >> 6, l = pi & 63;
        const int ks = f >> 2, pt = f & 3;
        const int p = pt * 16 + (l & 15);
        const int n0 = ks * 32 + (l >> 4) * 8;
        float v[8], kv[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            v[i] = to_f(sm[n0 + i][p]);
            kv[i] = v[i] * sr[n0 + i];
        }
        store8(vfrag + base + (int64_t)pi * 8, v);
        store8(kfrag + base + (int64_t)pi * 8, kv);
    }
}

template <typename T, int N, int S, int RT>
__global__ __launch_bounds__(16 / RT * 64) void k_sma_main(
    const T* __restrict__ q, const T* __restrict__ e, const T* __restrict__ Cm,
    const T* __restrict__ kfrag, const T* __restrict__ vfrag, const T* __restrict__ z,
    const T* y_ssd, T* y, float* __restrict__ lse, const float* __restrict__ qw,
    const float* __restrict__ ew, float eps, int normalize, int z_per_head, int64_t L, int H, int G,
    int64_t Mp, int nblk, int64_t BH) {
    constexpr int KS = N / 32;
    constexpr int NW = 16 / RT;                            // waves; 16*RT tokens each
    constexpr int WT = 16 * RT;                            // tokens per wave
    constexpr int MEMEL = N * kP;                          // elements per memory
    constexpr int PIECES = MEMEL * (int)sizeof(T) / 1024;  // 1 KiB operand fragments per copy
    static_assert(PIECES * 1024 == MEMEL * (int)sizeof(T), "memory must be whole fragments");
    static_assert(S >= WT, "a wave's tokens must lie in one chunk");

    // Block order.  Workgroups are dealt to the 8 XCDs round-robin by block
    // index, and each XCD has its own L2.  When B*H is a multiple of 8, XCD x
    // runs whole heads (b, h) = x, x+8, ... one after another, heaviest token
    // block first, so all blocks reading one head's memories share one L2.
    const int64_t bid = blockIdx.x;
    int blk;
    int64_t bh;
    if (BH % 8 == 0) {
        const int64_t slot = bid >> 3;
        blk = nblk - 1 - (int)(slot % nblk);
        bh = (slot / nblk) * 8 + (bid & 7);
    } else {
        blk = nblk - 1 - (int)(bid / BH);
        bh = bid % BH;
    }
    const int64_t b = bh / H;
    const int h = (int)(bh % H);
    const int g = (int)((int64_t)h * G / H);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = lane & 15, grp = lane >> 4;

    const int64_t blk0 = (int64_t)blk * kTokPerBlock;
    const int64_t wbase = blk0 + wave * WT;
    const int64_t blk_end = (blk0 + kTokPerBlock < L) ? blk0 + kTokPerBlock : L;
    const int jmax = (int)((blk_end - 1) / S);             // memories any wave of the block needs
    const bool active = wbase < L;
    const int iw = (int)(wbase / S);                        // this wave's chunk
    const int nj = active ? iw : 0;

    // Three stages (key copy then value copy of one memory each) as distinct
    // LDS objects: the compiler can see that a DMA into one stage does not
    // alias reads of another, so prefetches two memories ahead overlap the
    // MFMAs instead of being waited for.
    constexpr bool kThree = 3 * 2 * MEMEL * (int)sizeof(T) <= 160 * 1024;
    __shared__ __attribute__((aligned(16))) T st0[2 * MEMEL];
    __shared__ __attribute__((aligned(16))) T st1[2 * MEMEL];
    __shared__ __attribute__((aligned(16))) T st2[kThree ? 2 * MEMEL : 8];

    // ---- prologue: Qbar, C and Ebar of this wave's 64 tokens -------------
    Frag<T> qf[RT][KS], cf[RT][KS];
    float ef[RT][4][4];
    const float qscale = kLog2e / sqrtf((float)N);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const int64_t t = wbase + rt * 16 + col;
        const bool valid = active && t < L;
        float qv[KS][8];
        float ss = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (valid) {
                load8(q + ((b * L + t) * G + g) * N + ks * 32 + grp * 8, qv[ks]);
            } else {
#pragma unroll
                for (int i = 0; i < 8; ++i) qv[ks][i] = 0.f;
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
                load8(qw + ks * 32 + grp * 8, w);
#pragma unroll
                for (int i = 0; i < 8; ++i) qv[ks][i] *= w[i];
            }
            qf[rt][ks] = make_frag<T>(qv[ks]);
            float cv[8];
            if (valid) {
                load8(Cm + ((b * L + t) * G + g) * N + ks * 32 + grp * 8, cv);
            } else {
#pragma unroll
                for (int i = 0; i < 8; ++i) cv[i] = 0.f;
            }
            cf[rt][ks] = make_frag<T>(cv);
        }
        float es = 0.f;
#pragma unroll
        for (int pt = 0; pt < 4; ++pt) {
            if (valid) {
                load4(e + ((b * L + t) * G + g) * kP + pt * 16 + grp * 4, ef[rt][pt]);
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) ef[rt][pt][i] = 0.f;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) es += ef[rt][pt][i] * ef[rt][pt][i];
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
    f32x4 o[RT][4];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        m[rt] = -INFINITY;
        d[rt] = 0.f;
#pragma unroll
        for (int pt = 0; pt < 4; ++pt) o[rt][pt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // ---- stream the earlier memories through LDS (double buffered) -------
    // Each wave copies whole 1 KiB operand fragments straight from global
    // memory into LDS (global_load_lds_dwordx4: lane i writes 16 B at the
    // wave-uniform LDS base + 16 i), so no registers hold the prefetch.
    const int64_t mstride = (int64_t)H * MEMEL;
    const char* kbase = reinterpret_cast<const char*>(kfrag + (b * Mp * H + h) * (int64_t)MEMEL);
    const char* vbase = reinterpret_cast<const char*>(vfrag + (b * Mp * H + h) * (int64_t)MEMEL);
    static_assert(PIECES % NW == 0, "every wave copies the same number of fragments");
    constexpr int kDmaPerMem = 2 * PIECES / NW;  // DMA instructions per memory per wave
    auto fetch = [&](int j, T* dstage) {
        const char* kj = kbase + (int64_t)j * mstride * (int64_t)sizeof(T);
        const char* vj = vbase + (int64_t)j * mstride * (int64_t)sizeof(T);
        char* kd = reinterpret_cast<char*>(dstage);
        char* vd = kd + MEMEL * (int)sizeof(T);
#pragma unroll
        for (int pc = wave; pc < PIECES; pc += NW) {
            lds_dma16(kj + pc * 1024 + lane * 16, kd + pc * 1024);
            lds_dma16(vj + pc * 1024 + lane * 16, vd + pc * 1024);
        }
    };
    auto consume = [&](const T* kc, const T* vc) {
        float lp[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) lp[rt] = 0.f;
#pragma unroll
        for (int pt = 0; pt < 4; ++pt) {
            f32x4 u[RT];
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) u[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const Frag<T> fa = load_frag(&kc[((ks * 4 + pt) * 64 + lane) * 8]);
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) u[rt] = mma16(u[rt], fa, qf[rt][ks]);
            }
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int i = 0; i < 4; ++i) lp[rt] += u[rt][i] * ef[rt][pt][i];
        }
        float al[RT], pw[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            float l = lp[rt];
            l += shfl_xor(l, 16);
            l += shfl_xor(l, 32);
            const float mn = fmaxf(m[rt], l);
            al[rt] = fast_exp2(m[rt] - mn);
            pw[rt] = fast_exp2(l - mn);
            d[rt] = d[rt] * al[rt] + pw[rt];
            m[rt] = mn;
        }
#pragma unroll
        for (int pt = 0; pt < 4; ++pt) {
            f32x4 v[RT];
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) v[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const Frag<T> fa = load_frag(&vc[((ks * 4 + pt) * 64 + lane) * 8]);
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) v[rt] = mma16(v[rt], fa, cf[rt][ks]);
            }
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) o[rt][pt] = o[rt][pt] * al[rt] + pw[rt] * v[rt];
        }
    };
    // wait until at most `pending` memories' copies of this wave are in flight
    auto wait_copies = [&](bool one_pending) {
        if (one_pending) {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(kDmaPerMem));
        } else {
            wait_dma();
        }
    };
    if constexpr (kThree) {
        if (jmax > 0) fetch(0, st0);
        if (jmax > 1) fetch(1, st1);
        wait_copies(jmax > 1);
        block_barrier();
        // memory j is consumed from stage j % 3 while j+1 (already issued) and j+2
        // stream into the other two; one barrier per memory
        for (int j = 0; j < jmax; j += 3) {
            if (j + 2 < jmax) fetch(j + 2, st2);
            if (j < nj) consume(st0, st0 + MEMEL);
            wait_copies(j + 2 < jmax);
            block_barrier();
            if (j + 1 >= jmax) break;
            if (j + 3 < jmax) fetch(j + 3, st0);
            if (j + 1 < nj) consume(st1, st1 + MEMEL);
            wait_copies(j + 3 < jmax);
            block_barrier();
            if (j + 2 >= jmax) break;
            if (j + 4 < jmax) fetch(j + 4, st1);
            if (j + 2 < nj) consume(st2, st2 + MEMEL);
            wait_copies(j + 4 < jmax);
            block_barrier();
        }
    } else {
        // two stages (when three do not fit in LDS): j+1 streams while j is consumed
        if (jmax > 0) fetch(0, st0);
        wait_dma();
        __syncthreads();
        for (int j = 0; j < jmax; j += 2) {
            if (j + 1 < jmax) fetch(j + 1, st1);
            if (j < nj) consume(st0, st0 + MEMEL);
            wait_dma();
            __syncthreads();
            if (j + 1 >= jmax) break;
            if (j + 2 < jmax) fetch(j + 2, st0);
            if (j + 1 < nj) consume(st1, st1 + MEMEL);
            wait_dma();
            __syncthreads();
        }
    }

    // ---- epilogue: y = y_ssd + SiLU(z) R, LSE ------------------------------
    const bool hist = iw >= 1;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const int64_t t = wbase + rt * 16 + col;
        if (!active || t >= L) continue;
        const float zz = to_f(z_per_head ? z[(b * L + t) * H + h] : z[b * L + t]);
        const float gate = silu(zz);
        const float invd = hist ? 1.0f / d[rt] : 0.f;
#pragma unroll
        for (int pt = 0; pt < 4; ++pt) {
            const int64_t off = ((b * L + t) * H + h) * kP + pt * 16 + grp * 4;
            float ys[4];
            load4(y_ssd + off, ys);
            if (hist) {
#pragma unroll
                for (int i = 0; i < 4; ++i) ys[i] += gate * (o[rt][pt][i] * invd);
            }
            store4(y + off, ys);
        }
        if (lse && grp == 0) lse[(b * L + t) * H + h] = hist ? (m[rt] + log2f(d[rt])) * kLn2 : -INFINITY;
    }
}

template <typename T, int N, int S>
hipError_t run_sma(const Shape& s, const SmaArgs& a, const void* q, const void* e, const void* Cm,
                   const void* mem, const void* z, const void* y_ssd, void* y, float* lse,
                   void* ws, hipStream_t st) {
    const int64_t Mp = s.M > 1 ? s.M - 1 : 0;  // memories any token attends to
    T* kfrag = reinterpret_cast<T*>(ws);
    T* vfrag = reinterpret_cast<T*>(reinterpret_cast<char*>(ws) +
                                    align256(sizeof(T) * s.B * Mp * s.H * (size_t)N * kP));
    if (Mp > 0) {
        prof_begin("k_sma_prep", st);
        k_sma_prep<T, N><<<dim3((unsigned)Mp, (unsigned)s.H, (unsigned)s.B), kThreads, 0, st>>>(
            (const T*)mem, kfrag, vfrag, a.eps, a.normalize, s.H, Mp, s.Mcap);
        prof_end(st);
    }
    const int nblk = (int)((s.L + kTokPerBlock - 1) / kTokPerBlock);
    const int64_t BH = s.B * s.H;
    // 64 tokens per wave while the per-token operands fit the register file,
    // 32 tokens per wave (8 waves) for the largest state size
    constexpr int RT = (N * (int)sizeof(T) > 128) ? 2 : 4;
    prof_begin("k_sma_main", st);
    k_sma_main<T, N, S, RT><<<dim3((unsigned)(BH * nblk)), 16 / RT * 64, 0, st>>>(
        (const T*)q, (const T*)e, (const T*)Cm, kfrag, vfrag, (const T*)z, (const T*)y_ssd, (T*)y,
        lse, a.qw, a.ew, a.eps, a.normalize, a.z_per_head, s.L, s.H, s.G, Mp, nblk, BH);
    prof_end(st);
    return hipGetLastError();
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

size_t sma_workspace_bytes(const Shape& s) {
    const int64_t Mp = s.M > 1 ? s.M - 1 : 0;
    return 2 * align256(elem_bytes(s.dtype) * s.B * Mp * s.H * (size_t)s.N * s.P);
}

hipError_t launch_sma(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                      const void* Cm, const void* mem, const void* z, const void* y_ssd, void* y,
                      float* lse, void* ws, hipStream_t st) {
    if (s.dtype == 1) return run_sma_n<bf16>(s, a, q, e, Cm, mem, z, y_ssd, y, lse, ws, st);
    return run_sma_n<float>(s, a, q, e, Cm, mem, z, y_ssd, y, lse, ws, st);
}

}  // namespace dart
