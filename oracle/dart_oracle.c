/*
 * dart_oracle.c -- plain, slow, fp64 CPU oracle for the hot path of DART
 * ("Decoded Attention over Recurrent sTates", arXiv 2608.02032).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product (the HIP library and its
 * Python binding) may include, link, load or call this file.  Only the tests,
 * the smoke check and the CPU-baseline leg of the benchmark use it.  It shares
 * no code, header, table or helper with the GPU path.
 *
 * Every routine is the plain definition from the paper, written as literal
 * loops in double precision, with no chunking, blocking, fusion or reordering
 * beyond what the definition states:
 *
 *   dart_oracle_ssd_recurrence   Sec. 2 "State Space Duality": the token-level
 *                                recurrence H_t = A_t H_{t-1} + B_t^T X_t,
 *                                Y_t = C_t H_t, with the scalar transition
 *                                A_t = a_t I_N and the discretisation
 *                                a_t = exp(dt_t * A_h), input term
 *                                dt_t * B_t^T X_t (the paper writes the
 *                                recurrence without dt, while its kernel
 *                                benchmark feeds precomputed X, dt, A, B, C;
 *                                dt arrives already positive, no softplus).
 *   dart_oracle_chunk_memories   Sec. 3 "Chunk State Memories" and App. A
 *                                Eq. (mamba2_delta_h_chunk):
 *                                dH_[c] = sum_{s in [c]} A_{s+1:e(c)} B_s^T X_s,
 *                                the decay product taken literally, the empty
 *                                product being 1.
 *   dart_oracle_sma              Sec. 3 "State-Memory Attention" and
 *                                "Gated Residual Integration", with the
 *                                normalised score branch of App. B.1: for each
 *                                token an explicit two-pass softmax over the
 *                                strictly earlier chunks, then
 *                                Y_t = C_t H_t + SiLU(z_t) R_t.
 *   dart_oracle_ssd_bwd          gradients of the recurrence and the memories
 *                                (loss sum dy . y_ssd + <dmem, dH> + <dh, H_{L-1}>)
 *                                by running the recurrence backwards.
 *   dart_oracle_sma_bwd          gradients of dart_oracle_sma (loss sum dy . y)
 *                                by recomputing every row (App. C) and the chain
 *                                rule through Sec. 3 and App. B.1, written out.
 *   dart_oracle_conv1d_silu,     the block around the path: causal width-4
 *   dart_oracle_dt_softplus,     convolution + SiLU with its carried state,
 *   dart_oracle_gated_rmsnorm    softplus step sizes, gated RMSNorm (the
 *                                conventions of the Mamba-2 block; "parity
 *                                unpinned" beyond the definitions).
 *   dart_oracle_decode_step      one autoregressive token (the paper gives no
 *                                algorithm; the order used is: update the
 *                                recurrent state and the running chunk
 *                                contribution, read the cached memories of
 *                                completed chunks, gate, and append the running
 *                                contribution when the token closes a chunk).
 *
 * Precision: all arithmetic in double.  Callers pass the inputs already
 * rounded to the storage precision the GPU sees, then widened to double.
 *
 * Layouts (row-major, App. B.2 Table 7 order; b = batch, t = token,
 * h = head, g = group = h*G/H, c = chunk, n = state index, p = head-dim index):
 *   x      [B][L][H][P]       dt  [B][L][H]       A  [H]
 *   Bm, Cm [B][L][G][N]       q   [B][L][G][N]    e  [B][L][G][P]
 *   z      [B][L][H] (z_per_head = 1) or [B][L] (z_per_head = 0)
 *   y_ssd, y [B][L][H][P]     lse [B][L][H]
 *   mem    [B][Mcap][H][N][P] with M = ceil(L/S) <= Mcap
 *   h0, h_last, h_state, chunk_acc [B][H][N][P]
 *
 * parity: pinned by the oracle self-tests (SSD duality, boundary-state
 * identity, S = L and S = 1 degenerate cases, closed-form softmax cases,
 * normalisation invariances, decode == forward).  The conventions for the RMS
 * epsilon, the optional norm weights and the gate granularity are readings of
 * the paper, not fixed by it.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>

#define X_AT(b, t, h, p) x[(((size_t)(b) * L + (t)) * H + (h)) * P + (p)]
#define DT_AT(b, t, h) dt[((size_t)(b) * L + (t)) * H + (h)]
#define BM_AT(b, t, g, n) Bm[(((size_t)(b) * L + (t)) * G + (g)) * N + (n)]
#define CM_AT(b, t, g, n) Cm[(((size_t)(b) * L + (t)) * G + (g)) * N + (n)]
#define Y_AT(arr, b, t, h, p) arr[(((size_t)(b) * L + (t)) * H + (h)) * P + (p)]
#define ST_AT(arr, b, h, n, p) arr[(((size_t)(b) * H + (h)) * N + (n)) * P + (p)]
#define MEM_AT(b, c, h, n, p) \
    mem[((((size_t)(b) * Mcap + (c)) * H + (h)) * N + (n)) * P + (p)]

static int group_of(int h, int H, int G) { return (int)(((long)h * G) / H); }

/* ------------------------------------------------------------------------ */
/* Sec. 2 SSD recurrence (and App. A, token-level form).                     */
/* ------------------------------------------------------------------------ */
void dart_oracle_ssd_recurrence(int64_t B, int64_t L, int H, int G, int P, int N,
                                const double* x, const double* dt, const double* A,
                                const double* Bm, const double* Cm,
                                const double* h0, /* may be NULL: zero state */
                                double* y_ssd, double* h_last /* may be NULL */) {
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b) {
        for (int h = 0; h < H; ++h) {
            const int g = group_of(h, H, G);
            double* Hs = (double*)malloc(sizeof(double) * (size_t)N * P);
            for (int n = 0; n < N; ++n)
                for (int p = 0; p < P; ++p)
                    Hs[(size_t)n * P + p] = h0 ? ST_AT(h0, b, h, n, p) : 0.0;
            for (int64_t t = 0; t < L; ++t) {
                const double d = DT_AT(b, t, h);
                const double a = exp(d * A[h]); /* scalar transition a_t */
                /* H_t = a_t H_{t-1} + dt_t B_t^T X_t */
                for (int n = 0; n < N; ++n)
                    for (int p = 0; p < P; ++p)
                        Hs[(size_t)n * P + p] =
                            a * Hs[(size_t)n * P + p] + d * BM_AT(b, t, g, n) * X_AT(b, t, h, p);
                /* Y_t = C_t H_t */
                for (int p = 0; p < P; ++p) {
                    double acc = 0.0;
                    for (int n = 0; n < N; ++n) acc += CM_AT(b, t, g, n) * Hs[(size_t)n * P + p];
                    Y_AT(y_ssd, b, t, h, p) = acc;
                }
            }
            if (h_last)
                for (int n = 0; n < N; ++n)
                    for (int p = 0; p < P; ++p) ST_AT(h_last, b, h, n, p) = Hs[(size_t)n * P + p];
            free(Hs);
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Sec. 3 chunk state memory, App. A Eq. (mamba2_delta_h_chunk).            */
/* Chunk c (0-based) holds tokens [c*S, min((c+1)*S, L)); e(c) is its last   */
/* token.  A partial last chunk is emitted like any other.                   */
/* ------------------------------------------------------------------------ */
void dart_oracle_chunk_memories(int64_t B, int64_t L, int H, int G, int P, int N, int S,
                                int64_t Mcap, const double* x, const double* dt,
                                const double* A, const double* Bm, double* mem) {
    const int64_t M = (L + S - 1) / S;
#pragma omp parallel for collapse(3) schedule(static)
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t c = 0; c < M; ++c) {
            for (int h = 0; h < H; ++h) {
                const int g = group_of(h, H, G);
                const int64_t a0 = c * S;
                const int64_t e = (c + 1) * S < L ? (c + 1) * S - 1 : L - 1;
                for (int n = 0; n < N; ++n)
                    for (int p = 0; p < P; ++p) MEM_AT(b, c, h, n, p) = 0.0;
                for (int64_t s = a0; s <= e; ++s) {
                    /* A_{s+1:e(c)} = prod_{k=s+1}^{e(c)} a_k, empty product = 1 */
                    double decay = 1.0;
                    for (int64_t k = s + 1; k <= e; ++k) decay *= exp(DT_AT(b, k, h) * A[h]);
                    const double w = decay * DT_AT(b, s, h);
                    for (int n = 0; n < N; ++n)
                        for (int p = 0; p < P; ++p)
                            MEM_AT(b, c, h, n, p) += w * BM_AT(b, s, g, n) * X_AT(b, s, h, p);
                }
            }
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Backward of the scan and its memories: gradients of                       */
/*   loss = sum_t dy_t . y_t + sum_c <dmem_c, dH_[c]> + <dh_last, H_{L-1}>    */
/* with respect to x, dt, A, B, C and h0, by running the recurrence of Sec. 2 */
/* backwards.  With u_t = dt_t B_t^T x_t and a_t = exp(dt_t A_h):            */
/*   G_t = C_t^T dy_t + a_{t+1} G_{t+1},  G_{L-1} includes dh_last            */
/*     (the adjoint of H_t through y and h_last);                             */
/*   F_t = a_{t+1} F_{t+1} inside chunk c, F_{e(c)} = dmem_c                  */
/*     (the adjoint of the chunk's running contribution D_t, D reset to 0 at  */
/*     the chunk's first token, dH_[c] = D_{e(c)});                           */
/*   dx_t = dt_t B_t (G_t + F_t),  dB_t = dt_t (G_t + F_t) x_t,               */
/*   dC_t = H_t dy_t,  da_t = <G_t, H_{t-1}> + <F_t, D_{t-1}>,                */
/*   ddt_t = B_t (G_t + F_t) x_t + da_t a_t A_h,  dA_h = sum_t da_t a_t dt_t, */
/*   dh0 = a_0 G_0.                                                          */
/* B and C gradients sum over the heads of their group.  dmem, dh_last and   */
/* h0 may be NULL (zero).  Memory: the states of one (b, h) are kept for the */
/* whole sequence (L N P doubles), fine at the sizes the oracle serves.      */
/* ------------------------------------------------------------------------ */
void dart_oracle_ssd_bwd(int64_t B, int64_t L, int H, int G, int P, int N, int S, int64_t Mcap,
                         const double* x, const double* dt, const double* A, const double* Bm,
                         const double* Cm, const double* h0, const double* dy,
                         const double* dmem, const double* dhl, double* dx, double* ddt,
                         double* dA, double* dB, double* dC, double* dh0) {
    const size_t NP = (size_t)N * P;
    for (size_t k = 0; k < (size_t)B * L * H * P; ++k) dx[k] = 0.0;
    for (size_t k = 0; k < (size_t)B * L * H; ++k) ddt[k] = 0.0;
    for (size_t k = 0; k < (size_t)B * L * G * N; ++k) dB[k] = 0.0, dC[k] = 0.0;
    double* dAb = (double*)calloc((size_t)B * H, sizeof(double));
    /* rows of one batch entry touch only that entry's outputs */
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        double* Hs = (double*)malloc(sizeof(double) * (size_t)(L + 1) * NP); /* H_{-1..L-1} */
        double* Ds = (double*)malloc(sizeof(double) * (size_t)(L + 1) * NP); /* D_{-1..L-1} */
        double* Gt = (double*)malloc(sizeof(double) * NP);
        double* Ft = (double*)malloc(sizeof(double) * NP);
        for (int h = 0; h < H; ++h) {
            const int g = group_of(h, H, G);
            /* forward: every state, and every chunk's running contribution */
            for (size_t k = 0; k < NP; ++k) {
                Hs[k] = h0 ? h0[((size_t)b * H + h) * NP + k] : 0.0;
                Ds[k] = 0.0;
            }
            for (int64_t t = 0; t < L; ++t) {
                const double d = DT_AT(b, t, h);
                const double a = exp(d * A[h]);
                const int first = (t % S) == 0;
                const double* Hp = Hs + (size_t)t * NP;
                const double* Dp = Ds + (size_t)t * NP;
                double* Hn = Hs + (size_t)(t + 1) * NP;
                double* Dn = Ds + (size_t)(t + 1) * NP;
                for (int n = 0; n < N; ++n)
                    for (int p = 0; p < P; ++p) {
                        const size_t k = (size_t)n * P + p;
                        const double u = d * BM_AT(b, t, g, n) * X_AT(b, t, h, p);
                        Hn[k] = a * Hp[k] + u;
                        Dn[k] = (first ? 0.0 : a * Dp[k]) + u;
                    }
            }
            /* backward */
            for (size_t k = 0; k < NP; ++k) {
                Gt[k] = dhl ? dhl[((size_t)b * H + h) * NP + k] : 0.0;
                Ft[k] = 0.0;
            }
            for (int64_t t = L - 1; t >= 0; --t) {
                const double d = DT_AT(b, t, h);
                const double a = exp(d * A[h]);
                const int64_t c = t / S;
                const int last = (t == L - 1) || ((t + 1) % S == 0);
                const int first = (t % S) == 0;
                /* G_t = C_t^T dy_t + (a_{t+1} G_{t+1}, already in Gt) */
                for (int n = 0; n < N; ++n)
                    for (int p = 0; p < P; ++p)
                        Gt[(size_t)n * P + p] += CM_AT(b, t, g, n) * Y_AT(dy, b, t, h, p);
                /* F_t: dmem_c at the chunk's last token, carried inside it */
                if (last)
                    for (size_t k = 0; k < NP; ++k)
                        Ft[k] = dmem ? dmem[(((size_t)b * Mcap + c) * H + h) * NP + k] : 0.0;
                const double* Hp = Hs + (size_t)t * NP;        /* H_{t-1} */
                const double* Hc = Hs + (size_t)(t + 1) * NP;  /* H_t */
                const double* Dp = Ds + (size_t)t * NP;        /* D_{t-1} (not read at a chunk start) */
                double da = 0.0, din = 0.0;
                for (int n = 0; n < N; ++n) {
                    double db = 0.0, dc = 0.0;
                    for (int p = 0; p < P; ++p) {
                        const size_t k = (size_t)n * P + p;
                        const double lam = Gt[k] + Ft[k];
                        Y_AT(dx, b, t, h, p) += d * BM_AT(b, t, g, n) * lam;
                        db += lam * X_AT(b, t, h, p);
                        dc += Hc[k] * Y_AT(dy, b, t, h, p);
                        da += Gt[k] * Hp[k] + (first ? 0.0 : Ft[k] * Dp[k]);
                    }
                    dB[(((size_t)b * L + t) * G + g) * N + n] += d * db;
                    dC[(((size_t)b * L + t) * G + g) * N + n] += dc;
                    din += BM_AT(b, t, g, n) * db;
                }
                ddt[((size_t)b * L + t) * H + h] = din + da * a * A[h];
                dAb[(size_t)b * H + h] += da * a * d;
                /* carry to t - 1 */
                for (size_t k = 0; k < NP; ++k) {
                    Gt[k] *= a;
                    Ft[k] *= a;
                }
            }
            if (dh0)
                for (size_t k = 0; k < NP; ++k) dh0[((size_t)b * H + h) * NP + k] = Gt[k];
        }
        free(Hs);
        free(Ds);
        free(Gt);
        free(Ft);
    }
    for (int h = 0; h < H; ++h) {
        double s = 0.0;
        for (int64_t b = 0; b < B; ++b) s += dAb[(size_t)b * H + h];
        dA[h] = s;
    }
    free(dAb);
}

/* ------------------------------------------------------------------------ */
/* Sec. 3 state-memory attention + App. B.1 normalised score branch.         */
/* ------------------------------------------------------------------------ */

/* App. B.1: r_{c,n} = (P^{-1} sum_p dH[n,p]^2 + eps)^{-1/2}; r = 1 when the
 * score branch is not normalised (Alg. 1 as printed). */
static void inv_row_rms(const double* dH, int N, int P, double eps, int normalize, double* r) {
    for (int n = 0; n < N; ++n) {
        if (!normalize) {
            r[n] = 1.0;
            continue;
        }
        double ss = 0.0;
        for (int p = 0; p < P; ++p) ss += dH[(size_t)n * P + p] * dH[(size_t)n * P + p];
        r[n] = 1.0 / sqrt(ss / P + eps);
    }
}

/* RMSNorm of a length-D vector with optional weight (App. B.1). */
static void rms_normalise(const double* v, int D, double eps, const double* w, double* out) {
    double ss = 0.0;
    for (int k = 0; k < D; ++k) ss += v[k] * v[k];
    const double inv = 1.0 / sqrt(ss / D + eps);
    for (int k = 0; k < D; ++k) out[k] = v[k] * inv * (w ? w[k] : 1.0);
}

static double silu(double z) { return z / (1.0 + exp(-z)); }

/*
 * One query row (b, t, h): chunk index i = floor(t/S) (0-based form of
 * c(t) = ceil(t/S)); softmax over memories j = 0..i-1 (strictly earlier
 * chunks).  Empty history: R = 0 and LSE = -inf.  `rr` holds r for every
 * memory of this (b, h): rr[j*N + n].  Writes R[P], *lse and y[P].
 */
static void sma_row(int64_t B, int64_t L, int H, int G, int P, int N, int S, int64_t Mcap,
                    double eps, int normalize, int z_per_head, const double* q, const double* e,
                    const double* Cm, const double* qw, const double* ew, const double* mem,
                    const double* rr, const double* z, const double* y_ssd, int64_t b, int64_t t,
                    int h, double* R, double* lse, double* y, double* work) {
    (void)B;
    const int g = group_of(h, H, G);
    const int64_t i = t / S;
    const double* qt = q + ((size_t)b * L + t) * G * N + (size_t)g * N;
    const double* et = e + ((size_t)b * L + t) * G * P + (size_t)g * P;
    const double* ct = Cm + ((size_t)b * L + t) * G * N + (size_t)g * N;
    double* qbar = work;           /* N */
    double* ebar = qbar + N;       /* P */
    double* ell = ebar + P;        /* i logits */
    double* V = ell + (i > 0 ? i : 1); /* i*P values */

    for (int p = 0; p < P; ++p) R[p] = 0.0;
    if (i == 0) {
        *lse = -INFINITY;
    } else {
        if (normalize) {
            rms_normalise(qt, N, eps, qw, qbar);
            rms_normalise(et, P, eps, ew, ebar);
        } else {
            for (int n = 0; n < N; ++n) qbar[n] = qt[n];
            for (int p = 0; p < P; ++p) ebar[p] = et[p];
        }
        for (int64_t j = 0; j < i; ++j) {
            const double* dH = mem + (((size_t)b * Mcap + j) * H + h) * (size_t)N * P;
            const double* r = rr + (size_t)j * N;
            /* K_{t,j}[n] = r_j[n] * sum_p dH_j[n,p] Ebar_t[p];  l = Qbar . K / sqrt(N) */
            double l = 0.0;
            for (int n = 0; n < N; ++n) {
                double k = 0.0;
                for (int p = 0; p < P; ++p) k += dH[(size_t)n * P + p] * ebar[p];
                l += qbar[n] * (r[n] * k);
            }
            ell[j] = l / sqrt((double)N);
            /* V_{t,j}[p] = sum_n C_t[n] dH_j[n,p] */
            for (int p = 0; p < P; ++p) {
                double v = 0.0;
                for (int n = 0; n < N; ++n) v += ct[n] * dH[(size_t)n * P + p];
                V[(size_t)j * P + p] = v;
            }
        }
        /* explicit two-pass softmax over j < i */
        double m = -INFINITY;
        for (int64_t j = 0; j < i; ++j) m = ell[j] > m ? ell[j] : m;
        double d = 0.0;
        for (int64_t j = 0; j < i; ++j) d += exp(ell[j] - m);
        for (int64_t j = 0; j < i; ++j) {
            const double gw = exp(ell[j] - m) / d;
            for (int p = 0; p < P; ++p) R[p] += gw * V[(size_t)j * P + p];
        }
        *lse = m + log(d);
    }
    const double zz = z_per_head ? z[((size_t)b * L + t) * H + h] : z[(size_t)b * L + t];
    const double gate = silu(zz);
    for (int p = 0; p < P; ++p) y[p] = Y_AT(y_ssd, b, t, h, p) + gate * R[p];
}

static double* all_inv_rms(int64_t B, int H, int P, int N, int64_t Mcap, int64_t Mused,
                           double eps, int normalize, const double* mem) {
    double* rr = (double*)malloc(sizeof(double) * (size_t)B * H * (Mused > 0 ? Mused : 1) * N);
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b)
        for (int h = 0; h < H; ++h)
            for (int64_t j = 0; j < Mused; ++j)
                inv_row_rms(mem + (((size_t)b * Mcap + j) * H + h) * (size_t)N * P, N, P, eps,
                            normalize, rr + (((size_t)b * H + h) * Mused + j) * N);
    return rr;
}

/*
 * Full forward SMA + gate over every (b, t, h).  R may be NULL.
 * Memories 0..ceil(L/S)-1 of `mem` are read (only j < floor(t/S) matter).
 */
void dart_oracle_sma(int64_t B, int64_t L, int H, int G, int P, int N, int S, int64_t Mcap,
                     double eps, int normalize, int z_per_head, const double* q, const double* e,
                     const double* Cm, const double* qw, const double* ew, const double* mem,
                     const double* z, const double* y_ssd, double* y, double* lse, double* R) {
    const int64_t M = (L + S - 1) / S;
    double* rr = all_inv_rms(B, H, P, N, Mcap, M, eps, normalize, mem);
#pragma omp parallel
    {
        double* work = (double*)malloc(sizeof(double) * ((size_t)N + P + (M + 1) + (size_t)(M + 1) * P));
        double* Rrow = (double*)malloc(sizeof(double) * P);
#pragma omp for collapse(2) schedule(dynamic, 1)
        for (int64_t b = 0; b < B; ++b)
            for (int h = 0; h < H; ++h)
                for (int64_t t = 0; t < L; ++t) {
                    double l;
                    sma_row(B, L, H, G, P, N, S, Mcap, eps, normalize, z_per_head, q, e, Cm, qw,
                            ew, mem, rr + ((size_t)b * H + h) * M * N, z, y_ssd, b, t, h, Rrow,
                            &l, &Y_AT(y, b, t, h, 0), work);
                    lse[((size_t)b * L + t) * H + h] = l;
                    if (R)
                        for (int p = 0; p < P; ++p) Y_AT(R, b, t, h, p) = Rrow[p];
                }
        free(work);
        free(Rrow);
    }
    free(rr);
}

/*
 * The same definition evaluated only for a list of rows (b, t, h) given as
 * int64 triples; used to check sampled outputs at sizes where the full
 * oracle would take too long.  Outputs are packed: y_rows[k][P], lse_rows[k].
 */
void dart_oracle_sma_rows(int64_t B, int64_t L, int H, int G, int P, int N, int S, int64_t Mcap,
                          double eps, int normalize, int z_per_head, const double* q,
                          const double* e, const double* Cm, const double* qw, const double* ew,
                          const double* mem, const double* z, const double* y_ssd,
                          int64_t nrows, const int64_t* rows, double* y_rows, double* lse_rows) {
    const int64_t M = (L + S - 1) / S;
#pragma omp parallel
    {
        double* work = (double*)malloc(sizeof(double) * ((size_t)N + P + (M + 1) + (size_t)(M + 1) * P));
        double* Rrow = (double*)malloc(sizeof(double) * P);
        double* rr = (double*)malloc(sizeof(double) * (size_t)(M > 0 ? M : 1) * N);
#pragma omp for schedule(dynamic, 1)
        for (int64_t k = 0; k < nrows; ++k) {
            const int64_t b = rows[3 * k], t = rows[3 * k + 1];
            const int h = (int)rows[3 * k + 2];
            const int64_t i = t / S;
            for (int64_t j = 0; j < i; ++j)
                inv_row_rms(mem + (((size_t)b * Mcap + j) * H + h) * (size_t)N * P, N, P, eps,
                            normalize, rr + (size_t)j * N);
            sma_row(B, L, H, G, P, N, S, Mcap, eps, normalize, z_per_head, q, e, Cm, qw, ew, mem,
                    rr, z, y_ssd, b, t, h, Rrow, &lse_rows[k], y_rows + (size_t)k * P, work);
        }
        free(work);
        free(Rrow);
        free(rr);
    }
}

/* ------------------------------------------------------------------------ */
/* Backward of the SMA forward above (the loss is sum_t dy_t . y_t), by       */
/* recomputing each row's logits and recovering the softmax weights exactly  */
/* (App. C: scores recomputed, probabilities exp(l - LSE); here the exact    */
/* softmax).  Differentiating the definitions of Sec. 3 and App. B.1:        */
/*   y = y_ssd + SiLU(z) R:   dR = SiLU(z) dy,  dz = SiLU'(z) (R . dy),      */
/*   R = sum_j w_j V_j:       dw_j = dR . V_j,  dl_j = w_j (dw_j - dR . R),  */
/*                            dV_j = w_j dR                                  */
/*   V_j = C dH_j:            dC += dH_j dV_j,  ddH_j += C (x) dV_j          */
/*   l_j = Qbar . K_j / sqrt(N), K_j = r_j (.) (dH_j Ebar):                  */
/*     dQbar += dl_j K_j / sqrt(N),  dA_j = dl_j Qbar (.) r_j / sqrt(N),     */
/*     ddH_j += dA_j (x) Ebar,  dEbar += dH_j^T dA_j,                        */
/*     dr_j += dl_j Qbar (.) (dH_j Ebar) / sqrt(N)                           */
/*   r_j[n] = (P^-1 sum_p dH_j[n,p]^2 + eps)^-1/2:                           */
/*     ddH_j[n,p] -= dr_j[n] r_j[n]^3 dH_j[n,p] / P                          */
/*   Qbar = RMSNorm(q) w:  dq = inv u - q inv^3 (u . q) / N, u = dQbar (.) w */
/*   (and Ebar likewise).  The norm weights are constants here.             */
/* q, e, C gradients sum over the heads of their group; dz sums over heads   */
/* when one gate serves every head of a token.  Outputs are overwritten.     */
/* ------------------------------------------------------------------------ */
static double silu_grad(double z) {
    const double s = 1.0 / (1.0 + exp(-z));
    return s * (1.0 + z * (1.0 - s));
}

static void rms_normalise_bwd(const double* v, int D, double eps, const double* w,
                              const double* dout, double* dv) {
    double ss = 0.0;
    for (int k = 0; k < D; ++k) ss += v[k] * v[k];
    const double inv = 1.0 / sqrt(ss / D + eps);
    double uv = 0.0;
    for (int k = 0; k < D; ++k) uv += dout[k] * (w ? w[k] : 1.0) * v[k];
    for (int k = 0; k < D; ++k)
        dv[k] += dout[k] * (w ? w[k] : 1.0) * inv - v[k] * inv * inv * inv * uv / D;
}

void dart_oracle_sma_bwd(int64_t B, int64_t L, int H, int G, int P, int N, int S, int64_t Mcap,
                         double eps, int normalize, int z_per_head,
                         const double* q, const double* e, const double* Cm, const double* qw,
                         const double* ew, const double* mem, const double* z, const double* dy,
                         double* dq, double* de, double* dC, double* dmem, double* dz) {
    const int64_t M = (L + S - 1) / S;
    const double isn = 1.0 / sqrt((double)N);
    double* rr = all_inv_rms(B, H, P, N, Mcap, M, eps, normalize, mem);
    for (size_t k = 0; k < (size_t)B * L * G * N; ++k) dq[k] = 0.0, dC[k] = 0.0;
    for (size_t k = 0; k < (size_t)B * L * G * P; ++k) de[k] = 0.0;
    for (size_t k = 0; k < (size_t)B * Mcap * H * N * P; ++k) dmem[k] = 0.0;
    for (size_t k = 0; k < (size_t)B * L * (z_per_head ? H : 1); ++k) dz[k] = 0.0;
    /* rows of one batch entry touch only that entry's outputs */
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        double* drr = (double*)calloc((size_t)H * (M > 0 ? M : 1) * N, sizeof(double));
        double* qbar = (double*)malloc(sizeof(double) * N);
        double* ebar = (double*)malloc(sizeof(double) * P);
        double* ell = (double*)malloc(sizeof(double) * (M + 1));
        double* w = (double*)malloc(sizeof(double) * (M + 1));
        double* Vj = (double*)malloc(sizeof(double) * (size_t)(M + 1) * P);
        double* Aj = (double*)malloc(sizeof(double) * (size_t)(M + 1) * N);
        double* R = (double*)malloc(sizeof(double) * P);
        double* dR = (double*)malloc(sizeof(double) * P);
        double* dqbar = (double*)malloc(sizeof(double) * N);
        double* debar = (double*)malloc(sizeof(double) * P);
        for (int h = 0; h < H; ++h) {
            const int g = group_of(h, H, G);
            const double* rbh = rr + ((size_t)b * H + h) * M * N;
            for (int64_t t = 0; t < L; ++t) {
                const int64_t i = t / S;
                if (i == 0) continue; /* no history: y = y_ssd, nothing flows back */
                const double* qt = q + ((size_t)b * L + t) * G * N + (size_t)g * N;
                const double* et = e + ((size_t)b * L + t) * G * P + (size_t)g * P;
                const double* ct = Cm + ((size_t)b * L + t) * G * N + (size_t)g * N;
                if (normalize) {
                    rms_normalise(qt, N, eps, qw, qbar);
                    rms_normalise(et, P, eps, ew, ebar);
                } else {
                    for (int n = 0; n < N; ++n) qbar[n] = qt[n];
                    for (int p = 0; p < P; ++p) ebar[p] = et[p];
                }
                /* recompute logits and values */
                for (int64_t j = 0; j < i; ++j) {
                    const double* dH = mem + (((size_t)b * Mcap + j) * H + h) * (size_t)N * P;
                    const double* r = rbh + (size_t)j * N;
                    double l = 0.0;
                    for (int n = 0; n < N; ++n) {
                        double a = 0.0;
                        for (int p = 0; p < P; ++p) a += dH[(size_t)n * P + p] * ebar[p];
                        Aj[(size_t)j * N + n] = a;
                        l += qbar[n] * r[n] * a;
                    }
                    ell[j] = l * isn;
                    for (int p = 0; p < P; ++p) {
                        double v = 0.0;
                        for (int n = 0; n < N; ++n) v += ct[n] * dH[(size_t)n * P + p];
                        Vj[(size_t)j * P + p] = v;
                    }
                }
                double m = -INFINITY;
                for (int64_t j = 0; j < i; ++j) m = ell[j] > m ? ell[j] : m;
                double d = 0.0;
                for (int64_t j = 0; j < i; ++j) d += exp(ell[j] - m);
                for (int p = 0; p < P; ++p) R[p] = 0.0;
                for (int64_t j = 0; j < i; ++j) {
                    w[j] = exp(ell[j] - m) / d;
                    for (int p = 0; p < P; ++p) R[p] += w[j] * Vj[(size_t)j * P + p];
                }
                /* gate */
                const double* dyt = dy + (((size_t)b * L + t) * H + h) * P;
                const size_t zi = z_per_head ? ((size_t)b * L + t) * H + h : (size_t)b * L + t;
                const double gate = silu(z[zi]);
                double rdy = 0.0, D = 0.0;
                for (int p = 0; p < P; ++p) {
                    rdy += R[p] * dyt[p];
                    dR[p] = gate * dyt[p];
                    D += dR[p] * R[p];
                }
                dz[zi] += silu_grad(z[zi]) * rdy;
                for (int n = 0; n < N; ++n) dqbar[n] = 0.0;
                for (int p = 0; p < P; ++p) debar[p] = 0.0;
                double* dct = dC + ((size_t)b * L + t) * G * N + (size_t)g * N;
                for (int64_t j = 0; j < i; ++j) {
                    const double* dH = mem + (((size_t)b * Mcap + j) * H + h) * (size_t)N * P;
                    double* ddH = dmem + (((size_t)b * Mcap + j) * H + h) * (size_t)N * P;
                    const double* r = rbh + (size_t)j * N;
                    double* dr = drr + ((size_t)h * M + j) * N;
                    double dw = 0.0;
                    for (int p = 0; p < P; ++p) dw += dR[p] * Vj[(size_t)j * P + p];
                    const double dl = w[j] * (dw - D);
                    for (int n = 0; n < N; ++n) {
                        const double a = Aj[(size_t)j * N + n];
                        dqbar[n] += dl * r[n] * a * isn;
                        dr[n] += dl * qbar[n] * a * isn;
                        const double dA = dl * qbar[n] * r[n] * isn;
                        double dc = 0.0;
                        for (int p = 0; p < P; ++p) {
                            const double dV = w[j] * dR[p];
                            dc += dV * dH[(size_t)n * P + p];
                            ddH[(size_t)n * P + p] += ct[n] * dV + dA * ebar[p];
                            debar[p] += dA * dH[(size_t)n * P + p];
                        }
                        dct[n] += dc;
                    }
                }
                double* dqt = dq + ((size_t)b * L + t) * G * N + (size_t)g * N;
                double* det = de + ((size_t)b * L + t) * G * P + (size_t)g * P;
                if (normalize) {
                    rms_normalise_bwd(qt, N, eps, qw, dqbar, dqt);
                    rms_normalise_bwd(et, P, eps, ew, debar, det);
                } else {
                    for (int n = 0; n < N; ++n) dqt[n] += dqbar[n];
                    for (int p = 0; p < P; ++p) det[p] += debar[p];
                }
            }
            /* through r_j = (mean_p dH_j^2 + eps)^-1/2 */
            if (normalize)
                for (int64_t j = 0; j < M; ++j) {
                    const double* dH = mem + (((size_t)b * Mcap + j) * H + h) * (size_t)N * P;
                    double* ddH = dmem + (((size_t)b * Mcap + j) * H + h) * (size_t)N * P;
                    const double* r = rbh + (size_t)j * N;
                    const double* dr = drr + ((size_t)h * M + j) * N;
                    for (int n = 0; n < N; ++n) {
                        const double c = dr[n] * r[n] * r[n] * r[n] / P;
                        for (int p = 0; p < P; ++p) ddH[(size_t)n * P + p] -= c * dH[(size_t)n * P + p];
                    }
                }
        }
        free(drr);
        free(qbar);
        free(ebar);
        free(ell);
        free(w);
        free(Vj);
        free(Aj);
        free(R);
        free(dR);
        free(dqbar);
        free(debar);
    }
    free(rr);
}

/* ------------------------------------------------------------------------ */
/* Autoregressive decode step for token `pos` (0-based) of every sequence.   */
/* x [B][H][P], dt [B][H], Bm/Cm/q [B][G][N], e [B][G][P], z [B][H] or [B].  */
/* h_state, chunk_acc [B][H][N][P] and mem [B][Mcap][H][N][P] are in/out;    */
/* y [B][H][P] is out.                                                       */
/* ------------------------------------------------------------------------ */
int dart_oracle_decode_step(int64_t B, int H, int G, int P, int N, int S, int64_t Mcap,
                            int64_t pos, double eps, int normalize, int z_per_head,
                            const double* x, const double* dt, const double* A,
                            const double* Bm, const double* Cm, const double* q, const double* e,
                            const double* qw, const double* ew, const double* z,
                            double* h_state, double* chunk_acc, double* mem, double* y) {
    const int64_t m = pos / S; /* completed chunks before this token's chunk */
    if (pos < 0 || m > Mcap || (pos % S == S - 1 && m >= Mcap)) return 1; /* no room */
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b) {
        for (int h = 0; h < H; ++h) {
            const int g = group_of(h, H, G);
            const double d = dt[(size_t)b * H + h];
            const double a = exp(d * A[h]);
            const double* xb = x + ((size_t)b * H + h) * P;
            const double* bb = Bm + ((size_t)b * G + g) * N;
            const double* cb = Cm + ((size_t)b * G + g) * N;
            const double* qb = q + ((size_t)b * G + g) * N;
            const double* eb = e + ((size_t)b * G + g) * P;
            double* hs = h_state + ((size_t)b * H + h) * (size_t)N * P;
            double* ca = chunk_acc + ((size_t)b * H + h) * (size_t)N * P;
            double* yb = y + ((size_t)b * H + h) * P;
            /* 1. a new chunk starts with an empty running contribution */
            if (pos % S == 0)
                for (size_t k = 0; k < (size_t)N * P; ++k) ca[k] = 0.0;
            /* 2. recurrent state and running chunk contribution */
            for (int n = 0; n < N; ++n)
                for (int p = 0; p < P; ++p) {
                    const double u = d * bb[n] * xb[p];
                    hs[(size_t)n * P + p] = a * hs[(size_t)n * P + p] + u;
                    ca[(size_t)n * P + p] = a * ca[(size_t)n * P + p] + u;
                }
            /* 3. SSM readout C_t H_t */
            double* ysd = (double*)malloc(sizeof(double) * P);
            for (int p = 0; p < P; ++p) {
                double acc = 0.0;
                for (int n = 0; n < N; ++n) acc += cb[n] * hs[(size_t)n * P + p];
                ysd[p] = acc;
            }
            /* 4. SMA over the m cached memories (explicit two-pass softmax) */
            double* R = (double*)calloc((size_t)P, sizeof(double));
            if (m > 0) {
                double* qbar = (double*)malloc(sizeof(double) * N);
                double* ebar = (double*)malloc(sizeof(double) * P);
                double* ell = (double*)malloc(sizeof(double) * m);
                double* V = (double*)malloc(sizeof(double) * (size_t)m * P);
                double* r = (double*)malloc(sizeof(double) * N);
                if (normalize) {
                    rms_normalise(qb, N, eps, qw, qbar);
                    rms_normalise(eb, P, eps, ew, ebar);
                } else {
                    for (int n = 0; n < N; ++n) qbar[n] = qb[n];
                    for (int p = 0; p < P; ++p) ebar[p] = eb[p];
                }
                for (int64_t j = 0; j < m; ++j) {
                    const double* dH = mem + (((size_t)b * Mcap + j) * H + h) * (size_t)N * P;
                    inv_row_rms(dH, N, P, eps, normalize, r);
                    double l = 0.0;
                    for (int n = 0; n < N; ++n) {
                        double k = 0.0;
                        for (int p = 0; p < P; ++p) k += dH[(size_t)n * P + p] * ebar[p];
                        l += qbar[n] * (r[n] * k);
                    }
                    ell[j] = l / sqrt((double)N);
                    for (int p = 0; p < P; ++p) {
                        double v = 0.0;
                        for (int n = 0; n < N; ++n) v += cb[n] * dH[(size_t)n * P + p];
                        V[(size_t)j * P + p] = v;
                    }
                }
                double mx = -INFINITY;
                for (int64_t j = 0; j < m; ++j) mx = ell[j] > mx ? ell[j] : mx;
                double den = 0.0;
                for (int64_t j = 0; j < m; ++j) den += exp(ell[j] - mx);
                for (int64_t j = 0; j < m; ++j) {
                    const double gw = exp(ell[j] - mx) / den;
                    for (int p = 0; p < P; ++p) R[p] += gw * V[(size_t)j * P + p];
                }
                free(qbar);
                free(ebar);
                free(ell);
                free(V);
                free(r);
            }
            /* 5. gate */
            const double zz = z_per_head ? z[(size_t)b * H + h] : z[b];
            const double gate = silu(zz);
            for (int p = 0; p < P; ++p) yb[p] = ysd[p] + gate * R[p];
            free(ysd);
            free(R);
            /* 6. the token closes its chunk: the running contribution becomes memory m */
            if (pos % S == S - 1) {
                double* dst = mem + (((size_t)b * Mcap + m) * H + h) * (size_t)N * P;
                for (size_t k = 0; k < (size_t)N * P; ++k) dst[k] = ca[k];
            }
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* The block around the path (Table 8 context: convolution width 4 and      */
/* RMSNorm; the remaining conventions are those of the Mamba-2 block DART   */
/* builds on).                                                              */
/*                                                                          */
/* Causal depthwise convolution of width 4 over the token axis with bias    */
/* and SiLU: out[t][c] = SiLU(bias[c] + sum_{k=0..3} w[c][k] in[t-3+k][c]),  */
/* where in[t] for t < 0 is the carried state (st_in[c][3 + t], zeros when  */
/* absent).  st_out receives the last three inputs in token order (the     */
/* decode cache of the convolution).  in rows have `stride` elements, the   */
/* channels the first C of them.                                           */
/* ------------------------------------------------------------------------ */
void dart_oracle_conv1d_silu(int64_t B, int64_t L, int C, int64_t stride, const double* in,
                             const double* w, const double* bias, const double* st_in,
                             double* out, double* st_out) {
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b) {
        for (int c = 0; c < C; ++c) {
            for (int64_t t = 0; t < L; ++t) {
                double acc = bias ? bias[c] : 0.0;
                for (int k = 0; k < 4; ++k) {
                    const int64_t s = t - 3 + k;
                    double v;
                    if (s >= 0)
                        v = in[((size_t)b * L + s) * stride + c];
                    else
                        v = st_in ? st_in[((size_t)b * C + c) * 3 + (3 + s)] : 0.0;
                    acc += w[(size_t)c * 4 + k] * v;
                }
                out[((size_t)b * L + t) * C + c] = silu(acc);
            }
            if (st_out)
                for (int i = 0; i < 3; ++i) {
                    const int64_t s = L - 3 + i;
                    double v;
                    if (s >= 0)
                        v = in[((size_t)b * L + s) * stride + c];
                    else
                        v = st_in ? st_in[((size_t)b * C + c) * 3 + (3 + s)] : 0.0;
                    st_out[((size_t)b * C + c) * 3 + i] = v;
                }
        }
    }
}

/* Step size from the projection: dt = softplus(raw + bias[h]) (log1p(exp)). */
void dart_oracle_dt_softplus(int64_t rows, int H, const double* raw, const double* bias,
                             double* dt) {
    for (int64_t r = 0; r < rows; ++r)
        for (int h = 0; h < H; ++h) {
            const double v = raw[(size_t)r * H + h] + (bias ? bias[h] : 0.0);
            dt[(size_t)r * H + h] = v > 30.0 ? v + log1p(exp(-v)) : log1p(exp(v));
        }
}

/* Gated RMSNorm ahead of the output projection: with u = y (.) SiLU(z),     */
/* out = u / sqrt(mean_{group}(u^2) + eps) * w over consecutive groups of   */
/* `group` channels of each row (D channels, D % group == 0).              */
void dart_oracle_gated_rmsnorm(int64_t rows, int D, int group, double eps, const double* y,
                               const double* z, const double* w, double* out) {
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r) {
        for (int g0 = 0; g0 < D; g0 += group) {
            double ss = 0.0;
            for (int k = g0; k < g0 + group; ++k) {
                const double u = y[(size_t)r * D + k] * silu(z[(size_t)r * D + k]);
                ss += u * u;
            }
            const double inv = 1.0 / sqrt(ss / group + eps);
            for (int k = g0; k < g0 + group; ++k) {
                const double u = y[(size_t)r * D + k] * silu(z[(size_t)r * D + k]);
                out[(size_t)r * D + k] = u * inv * (w ? w[k] : 1.0);
            }
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Backward of the three block definitions above (chain rule, literal loops) */
/* for a loss whose gradient with respect to the output is dout.             */
/* ------------------------------------------------------------------------ */

/* Convolution: u[t] = bias + sum_k w[k] in[t-3+k] (in[s<0] from the carried */
/* state), out = SiLU(u).  du = dout SiLU'(u); every input term of u gets    */
/* du times its weight; the weights get du times their input.               */
void dart_oracle_conv1d_silu_bwd(int64_t B, int64_t L, int C, int64_t stride, const double* in,
                                 const double* w, const double* bias, const double* st_in,
                                 const double* dout, double* din, double* dw, double* db,
                                 double* dst) {
    for (size_t k = 0; k < (size_t)B * L * C; ++k) din[k] = 0.0;
    for (size_t k = 0; k < (size_t)C * 4; ++k) dw[k] = 0.0;
    for (int c = 0; c < C; ++c) db[c] = 0.0;
    for (size_t k = 0; k < (size_t)B * C * 3; ++k) dst[k] = 0.0;
    for (int64_t b = 0; b < B; ++b)
        for (int c = 0; c < C; ++c)
            for (int64_t t = 0; t < L; ++t) {
                double u = bias ? bias[c] : 0.0;
                for (int k = 0; k < 4; ++k) {
                    const int64_t s = t - 3 + k;
                    const double v = s >= 0 ? in[((size_t)b * L + s) * stride + c]
                                            : (st_in ? st_in[((size_t)b * C + c) * 3 + (3 + s)] : 0.0);
                    u += w[(size_t)c * 4 + k] * v;
                }
                const double sg = 1.0 / (1.0 + exp(-u));
                const double du = dout[((size_t)b * L + t) * C + c] * sg * (1.0 + u * (1.0 - sg));
                db[c] += du;
                for (int k = 0; k < 4; ++k) {
                    const int64_t s = t - 3 + k;
                    const double v = s >= 0 ? in[((size_t)b * L + s) * stride + c]
                                            : (st_in ? st_in[((size_t)b * C + c) * 3 + (3 + s)] : 0.0);
                    dw[(size_t)c * 4 + k] += du * v;
                    if (s >= 0)
                        din[((size_t)b * L + s) * C + c] += du * w[(size_t)c * 4 + k];
                    else
                        dst[((size_t)b * C + c) * 3 + (3 + s)] += du * w[(size_t)c * 4 + k];
                }
            }
}

/* Step sizes: dt = softplus(raw + bias): d raw = ddt sigmoid(raw + bias),   */
/* d bias = its sum over rows.                                              */
void dart_oracle_dt_softplus_bwd(int64_t rows, int H, const double* raw, const double* bias,
                                 const double* ddt, double* draw, double* dbias) {
    for (int h = 0; h < H; ++h) dbias[h] = 0.0;
    for (int64_t r = 0; r < rows; ++r)
        for (int h = 0; h < H; ++h) {
            const double v = raw[(size_t)r * H + h] + (bias ? bias[h] : 0.0);
            const double g = ddt[(size_t)r * H + h] / (1.0 + exp(-v));
            draw[(size_t)r * H + h] = g;
            dbias[h] += g;
        }
}

/* Gated RMSNorm: out_k = u_k inv w_k, u = y SiLU(z), inv = (mean u^2 +     */
/* eps)^-1/2 over the group.  d u_k = inv w_k dout_k - u_k inv^3 (sum_j     */
/* w_j dout_j u_j) / group; dy = du SiLU(z); dz = du y SiLU'(z);            */
/* dw_k = sum over rows of dout_k u_k inv.                                  */
void dart_oracle_gated_rmsnorm_bwd(int64_t rows, int D, int group, double eps, const double* y,
                                   const double* z, const double* w, const double* dout,
                                   double* dy, double* dz, double* dw) {
    for (int k = 0; k < D; ++k) dw[k] = 0.0;
    for (int64_t r = 0; r < rows; ++r)
        for (int g0 = 0; g0 < D; g0 += group) {
            double ss = 0.0, gu = 0.0;
            for (int k = g0; k < g0 + group; ++k) {
                const double u = y[(size_t)r * D + k] * silu(z[(size_t)r * D + k]);
                ss += u * u;
                gu += (w ? w[k] : 1.0) * dout[(size_t)r * D + k] * u;
            }
            const double inv = 1.0 / sqrt(ss / group + eps);
            for (int k = g0; k < g0 + group; ++k) {
                const double zz = z[(size_t)r * D + k];
                const double u = y[(size_t)r * D + k] * silu(zz);
                const double du = inv * (w ? w[k] : 1.0) * dout[(size_t)r * D + k] -
                                  u * inv * inv * inv * gu / group;
                dy[(size_t)r * D + k] = du * silu(zz);
                dz[(size_t)r * D + k] = du * y[(size_t)r * D + k] * silu_grad(zz);
                dw[k] += dout[(size_t)r * D + k] * u * inv;
            }
        }
}
