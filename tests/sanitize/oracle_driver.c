/* Runs every function of the CPU oracle (oracle/dart_oracle.c) on small
 * shapes -- ragged chunks, two groups, a memory capacity above the chunk
 * count, the decode step over a whole sequence -- with every buffer allocated
 * at its exact size, so that an AddressSanitizer / UndefinedBehaviorSanitizer
 * build of the oracle reports any out-of-bounds access or undefined
 * operation.  Test infrastructure: built and run by tests/test_sanitizers.py. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void dart_oracle_ssd_recurrence(int64_t, int64_t, int, int, int, int, const double*, const double*,
                                const double*, const double*, const double*, const double*, double*,
                                double*);
void dart_oracle_chunk_memories(int64_t, int64_t, int, int, int, int, int, int64_t, const double*,
                                const double*, const double*, const double*, double*);
void dart_oracle_ssd_bwd(int64_t, int64_t, int, int, int, int, int, int64_t, const double*,
                         const double*, const double*, const double*, const double*, const double*,
                         const double*, const double*, const double*, double*, double*, double*,
                         double*, double*, double*);
void dart_oracle_sma(int64_t, int64_t, int, int, int, int, int, int64_t, double, int, int,
                     const double*, const double*, const double*, const double*, const double*,
                     const double*, const double*, const double*, double*, double*, double*);
void dart_oracle_sma_rows(int64_t, int64_t, int, int, int, int, int, int64_t, double, int, int,
                          const double*, const double*, const double*, const double*, const double*,
                          const double*, const double*, const double*, int64_t, const int64_t*,
                          double*, double*);
void dart_oracle_sma_bwd(int64_t, int64_t, int, int, int, int, int, int64_t, double, int, int,
                         const double*, const double*, const double*, const double*, const double*,
                         const double*, const double*, const double*, double*, double*, double*,
                         double*, double*);
int dart_oracle_decode_step(int64_t, int, int, int, int, int, int64_t, int64_t, double, int, int,
                            const double*, const double*, const double*, const double*,
                            const double*, const double*, const double*, const double*,
                            const double*, const double*, double*, double*, double*, double*);
void dart_oracle_conv1d_silu(int64_t, int64_t, int, int64_t, const double*, const double*,
                             const double*, const double*, double*, double*);
void dart_oracle_dt_softplus(int64_t, int, const double*, const double*, double*);
void dart_oracle_gated_rmsnorm(int64_t, int, int, double, const double*, const double*,
                               const double*, double*);
void dart_oracle_conv1d_silu_bwd(int64_t, int64_t, int, int64_t, const double*, const double*,
                                 const double*, const double*, const double*, double*, double*,
                                 double*, double*);
void dart_oracle_dt_softplus_bwd(int64_t, int, const double*, const double*, const double*,
                                 double*, double*);
void dart_oracle_gated_rmsnorm_bwd(int64_t, int, int, double, const double*, const double*,
                                   const double*, const double*, double*, double*, double*);

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static double uni(void) { /* xorshift64*, uniform in [-1, 1) */
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return (double)((rng_state * 0x2545F4914F6CDD1Dull) >> 11) * (2.0 / 9007199254740992.0) - 1.0;
}
static double* buf(size_t n, double scale, double shift) {
    double* p = (double*)malloc(n * sizeof(double));
    if (!p) abort();
    for (size_t i = 0; i < n; ++i) p[i] = shift + scale * uni();
    return p;
}
static double* out(size_t n) { return buf(n, 0.0, 0.0); }

int main(void) {
    const int64_t B = 2, L = 150;
    const int H = 4, G = 2, P = 8, N = 6, S = 32;
    const int64_t M = (L + S - 1) / S, Mcap = M + 2;
    double* x = buf(B * L * H * P, 1.0, 0.0);
    double* dt = buf(B * L * H, 0.04, 0.05);
    double* A = buf(H, 1.0, -2.0);
    double* Bm = buf(B * L * G * N, 0.4, 0.0);
    double* Cm = buf(B * L * G * N, 0.4, 0.0);
    double* h0 = buf(B * H * N * P, 0.1, 0.0);
    double* q = buf(B * L * G * N, 0.5, 0.0);
    double* e = buf(B * L * G * P, 0.5, 0.0);
    double* qw = buf(N, 0.2, 1.0);
    double* ew = buf(P, 0.2, 1.0);
    double* zh = buf(B * L * H, 1.0, 0.0);
    double* zt = buf(B * L, 1.0, 0.0);
    double* dy = buf(B * L * H * P, 0.5, 0.0);

    double* y = out(B * L * H * P);
    double* hl = out(B * H * N * P);
    dart_oracle_ssd_recurrence(B, L, H, G, P, N, x, dt, A, Bm, Cm, h0, y, hl);
    dart_oracle_ssd_recurrence(B, L, H, G, P, N, x, dt, A, Bm, Cm, NULL, y, NULL);
    double* mem = out(B * Mcap * H * N * P);
    dart_oracle_chunk_memories(B, L, H, G, P, N, S, Mcap, x, dt, A, Bm, mem);

    double* dmem = buf(B * Mcap * H * N * P, 0.5, 0.0);
    double* dhl = buf(B * H * N * P, 0.5, 0.0);
    double *dx = out(B * L * H * P), *ddt = out(B * L * H), *dA = out(H);
    double *dB = out(B * L * G * N), *dC = out(B * L * G * N), *dh0 = out(B * H * N * P);
    dart_oracle_ssd_bwd(B, L, H, G, P, N, S, Mcap, x, dt, A, Bm, Cm, h0, dy, dmem, dhl, dx, ddt, dA,
                        dB, dC, dh0);
    dart_oracle_ssd_bwd(B, L, H, G, P, N, S, Mcap, x, dt, A, Bm, Cm, NULL, dy, NULL, NULL, dx, ddt,
                        dA, dB, dC, dh0);

    double* ys = out(B * L * H * P);
    double* lse = out(B * L * H);
    double* R = out(B * L * H * P);
    for (int zp = 0; zp < 2; ++zp)
        for (int nz = 0; nz < 2; ++nz)
            dart_oracle_sma(B, L, H, G, P, N, S, Mcap, 1e-6, nz, zp, q, e, Cm, nz ? qw : NULL,
                            nz ? ew : NULL, mem, zp ? zh : zt, y, ys, lse, R);
    /* sampled rows as (b, t, h) triples: first token, chunk edges, last token */
    const int64_t rows[15] = {0, 0, 0, 0, 31, 1, 1, 32, 2, 1, 149, 3, 0, 128, 2};
    double* yr = out(5 * P);
    double* lr = out(5);
    dart_oracle_sma_rows(B, L, H, G, P, N, S, Mcap, 1e-6, 1, 1, q, e, Cm, qw, ew, mem, zh, y, 5, rows,
                         yr, lr);
    double *dq = out(B * L * G * N), *de = out(B * L * G * P), *dCs = out(B * L * G * N);
    double *dm = out(B * Mcap * H * N * P), *dz = out(B * L * H);
    dart_oracle_sma_bwd(B, L, H, G, P, N, S, Mcap, 1e-6, 1, 1, q, e, Cm, qw, ew, mem, zh, dy, dq, de,
                        dCs, dm, dz);

    /* the decode step over the whole sequence, then one step past the cache */
    double* hs = out(B * H * N * P);
    double* ca = out(B * H * N * P);
    double* cache = out(B * Mcap * H * N * P);
    double* yt = out(B * H * P);
    double *xs = out(B * H * P), *dts = out(B * H), *bs = out(B * G * N), *cs = out(B * G * N);
    double *qs = out(B * G * N), *es = out(B * G * P), *zs = out(B * H);
    for (int64_t t = 0; t < L; ++t) {
        for (int64_t b = 0; b < B; ++b) {
            for (int i = 0; i < H * P; ++i) xs[b * H * P + i] = x[(b * L + t) * H * P + i];
            for (int i = 0; i < H; ++i) {
                dts[b * H + i] = dt[(b * L + t) * H + i];
                zs[b * H + i] = zh[(b * L + t) * H + i];
            }
            for (int i = 0; i < G * N; ++i) {
                bs[b * G * N + i] = Bm[(b * L + t) * G * N + i];
                cs[b * G * N + i] = Cm[(b * L + t) * G * N + i];
                qs[b * G * N + i] = q[(b * L + t) * G * N + i];
            }
            for (int i = 0; i < G * P; ++i) es[b * G * P + i] = e[(b * L + t) * G * P + i];
        }
        if (dart_oracle_decode_step(B, H, G, P, N, S, Mcap, t, 1e-6, 1, 1, xs, dts, A, bs, cs, qs, es,
                                    qw, ew, zs, hs, ca, cache, yt) != 0)
            return 2;
    }
    if (dart_oracle_decode_step(B, H, G, P, N, S, 1, S - 1 + S, 1e-6, 1, 1, xs, dts, A, bs, cs, qs,
                                es, qw, ew, zs, hs, ca, cache, yt) == 0)
        return 3; /* a step beyond the cache must be refused */

    /* block kernels: conv over a strided channel slice, softplus, gated norm */
    const int C = 10;
    const int64_t stride = 13;
    double* cin = buf(B * L * stride, 1.0, 0.0);
    double* cw = buf(C * 4, 0.5, 0.0);
    double* cb = buf(C, 0.1, 0.0);
    double* cst = buf(B * C * 3, 0.5, 0.0);
    double *cout = out(B * L * C), *cst2 = out(B * C * 3);
    dart_oracle_conv1d_silu(B, L, C, stride, cin, cw, cb, cst, cout, cst2);
    dart_oracle_conv1d_silu(B, L, C, stride, cin, cw, NULL, NULL, cout, NULL);
    double* dout = buf(B * L * C, 1.0, 0.0);
    double *din = out(B * L * stride), *dw = out(C * 4), *db = out(C), *dst = out(B * C * 3);
    dart_oracle_conv1d_silu_bwd(B, L, C, stride, cin, cw, cb, cst, dout, din, dw, db, dst);
    double* raw = buf(B * L * H, 2.0, 0.0);
    double* dtb = buf(H, 0.5, 0.0);
    double* dto = out(B * L * H);
    dart_oracle_dt_softplus(B * L, H, raw, dtb, dto);
    double *draw = out(B * L * H), *dbias = out(H);
    dart_oracle_dt_softplus_bwd(B * L, H, raw, dtb, dy, draw, dbias);
    const int D = 12, grp = 4;
    double* gy = buf(B * L * D, 1.0, 0.0);
    double* gz = buf(B * L * D, 1.0, 0.0);
    double* gw = buf(D, 0.2, 1.0);
    double* go = out(B * L * D);
    dart_oracle_gated_rmsnorm(B * L, D, grp, 1e-6, gy, gz, gw, go);
    dart_oracle_gated_rmsnorm(B * L, D, D, 1e-6, gy, gz, NULL, go);
    double* gd = buf(B * L * D, 1.0, 0.0);
    double *gdy = out(B * L * D), *gdz = out(B * L * D), *gdw = out(D);
    dart_oracle_gated_rmsnorm_bwd(B * L, D, grp, 1e-6, gy, gz, gw, gd, gdy, gdz, gdw);

    double chk = 0.0;
    for (size_t i = 0; i < (size_t)(B * L * H * P); ++i) chk += ys[i] + dx[i];
    printf("oracle driver ok %.6e\n", chk);
    return 0;
}
