/* Host-side checks of the C ABI (include/dart.h) run under AddressSanitizer /
 * UndefinedBehaviorSanitizer (or ThreadSanitizer) without a GPU: workspace
 * sizing for tuned and generic shapes, rejection of malformed arguments before
 * any launch, and the profiling calls hammered from several threads (their
 * shared totals sit behind one lock).  Pointers are never dereferenced by the
 * validation paths exercised here.  Test infrastructure: built and run by
 * tests/test_sanitizers.py. */
#include <pthread.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "dart.h"

static int failures = 0;
#define CHECK(cond)                                                              \
    do {                                                                         \
        if (!(cond)) {                                                           \
            fprintf(stderr, "check failed at line %d: %s (%s)\n", __LINE__, #cond, \
                    dart_last_error());                                          \
            ++failures;                                                          \
        }                                                                        \
    } while (0)

static dart_dims dims(int64_t B, int64_t L, int H, int G, int P, int N, int S, int dtype, int64_t mcap) {
    dart_dims d;
    memset(&d, 0, sizeof(d));
    d.batch = B;
    d.seqlen = L;
    d.nheads = H;
    d.ngroups = G;
    d.headdim = P;
    d.dstate = N;
    d.chunk = S;
    d.dtype = dtype;
    d.mem_capacity = mcap;
    return d;
}

#define P1 ((void*)(uintptr_t)4096)

static dart_status scan(const dart_dims* d, int null_arg, size_t nbytes) {
    void* p[8] = {P1, P1, P1, P1, P1, P1, P1, P1}; /* x dt A Bm Cm y mem ws */
    if (null_arg >= 0) p[null_arg] = NULL;
    return dart_ssd_chunk_scan(d, p[0], p[1], p[2], p[3], p[4], NULL, p[5], p[6], NULL, p[7], nbytes, NULL);
}

static void* hammer(void* arg) {
    const int id = (int)(intptr_t)arg;
    char name[32];
    for (int i = 0; i < 20000; ++i) {
        snprintf(name, sizeof(name), "k_%d_%d", id, i % 7);
        dart_profile_enable(i & 1);
        dart_profile_filter((i % 3) ? name : NULL);
        const int n = dart_profile_count();
        if (n > 0) (void)dart_profile_total_ms(n - 1);
        (void)dart_profile_launches(0);
        if (i % 97 == 0) dart_profile_reset();
        (void)dart_status_string((dart_status)(i % 4));
    }
    return NULL;
}

int main(int argc, char** argv) {
    const int threads_only = argc > 1 && strcmp(argv[1], "threads") == 0;
    if (!threads_only) {
        CHECK(strcmp(dart_status_string(DART_OK), "DART_OK") == 0);
        /* workspace sizing: tuned and generic shapes, both storage types */
        const int NS[5][2] = {{64, 64}, {128, 256}, {16, 16}, {128, 48}, {32, 1}};
        for (int k = 0; k < 5; ++k)
            for (int dt = 0; dt < 2; ++dt) {
                dart_dims d = dims(2, 300, 4, 2, 64, NS[k][0], NS[k][1], dt, 0);
                CHECK(dart_scan_workspace_bytes(&d) > 0);
                CHECK(dart_ssd_bwd_workspace_bytes(&d) > 0);
                CHECK(dart_sma_bwd_workspace_bytes(&d) > 0);
                (void)dart_sma_workspace_bytes(&d);
                dart_dims dd = dims(2, 0, 4, 2, 64, NS[k][0], NS[k][1], dt, 40);
                CHECK(dart_decode_workspace_bytes(&dd) > 0);
            }
        dart_dims bad = dims(2, 512, 4, 1, 48, 64, 64, 1, 0);
        CHECK(dart_scan_workspace_bytes(&bad) == 0);
        /* malformed dimensions */
        dart_dims d = dims(2, 512, 4, 1, 64, 64, 64, 1, 0);
        dart_dims v;
        v = d; v.batch = 0;          CHECK(scan(&v, -1, (size_t)1 << 40) == DART_ERR_INVALID_ARG);
        v = d; v.seqlen = 0;         CHECK(scan(&v, -1, (size_t)1 << 40) == DART_ERR_INVALID_ARG);
        v = d; v.ngroups = 2; v.nheads = 3; CHECK(scan(&v, -1, (size_t)1 << 40) == DART_ERR_INVALID_ARG);
        v = d; v.dtype = 7;          CHECK(scan(&v, -1, (size_t)1 << 40) == DART_ERR_INVALID_ARG);
        v = d; v.headdim = 128;      CHECK(scan(&v, -1, (size_t)1 << 40) == DART_ERR_UNSUPPORTED);
        v = d; v.dstate = 48;        CHECK(scan(&v, -1, (size_t)1 << 40) == DART_ERR_UNSUPPORTED);
        v = d; v.chunk = 8192;       CHECK(scan(&v, -1, (size_t)1 << 40) == DART_ERR_UNSUPPORTED);
        v = d; v.mem_capacity = 3;   CHECK(scan(&v, -1, (size_t)1 << 40) == DART_ERR_INVALID_ARG);
        v = d; v.batch = (int64_t)1 << 62; CHECK(scan(&v, -1, (size_t)1 << 40) != DART_OK);
        for (int k = 0; k < 8; ++k) CHECK(scan(&d, k, (size_t)1 << 40) == DART_ERR_INVALID_ARG);
        CHECK(scan(&d, -1, dart_scan_workspace_bytes(&d) - 1) == DART_ERR_INVALID_ARG);
        /* SMA options and partial aliasing */
        dart_sma_opts o = {0.0f, NULL, NULL, 1, 1};
        CHECK(dart_sma_fwd(&d, &o, P1, P1, P1, P1, P1, P1, P1, NULL, P1, (size_t)1 << 40, NULL) ==
              DART_ERR_INVALID_ARG);
        o.eps = 1e-6f;
        o.normalize = 2;
        CHECK(dart_sma_fwd(&d, &o, P1, P1, P1, P1, P1, P1, P1, NULL, P1, (size_t)1 << 40, NULL) ==
              DART_ERR_INVALID_ARG);
        o.normalize = 1;
        CHECK(dart_sma_fwd(&d, &o, P1, P1, P1, P1, P1, (void*)4096, (void*)4098, NULL, P1,
                           (size_t)1 << 40, NULL) == DART_ERR_INVALID_ARG);
        /* decode: bad positions, cache overflow, small workspace */
        dart_dims dd = dims(2, 0, 4, 1, 64, 64, 64, 1, 4);
        void* q = P1;
        CHECK(dart_decode_step(&dd, &o, -1, q, q, q, q, q, q, q, q, q, q, q, q, q, (size_t)1 << 40, NULL) ==
              DART_ERR_INVALID_ARG);
        CHECK(dart_decode_step(&dd, &o, 319, q, q, q, q, q, q, q, q, q, q, q, q, q, (size_t)1 << 40, NULL) ==
              DART_ERR_INVALID_ARG);
        CHECK(dart_decode_step(&dd, &o, 10, q, q, q, q, q, q, q, q, q, q, q, q, q,
                               dart_decode_workspace_bytes(&dd) - 1, NULL) == DART_ERR_INVALID_ARG);
        dart_dims huge = dims(4096, 0, 64, 1, 64, 64, 64, 1, 4);
        CHECK(dart_decode_step_noalloc(&huge, &o, 64, q, q, q, q, q, q, q, q, q, q, q, q, NULL) ==
              DART_ERR_UNSUPPORTED);
        CHECK(dart_decode_handoff(&dd, NULL, q, q, q, q, NULL) == DART_ERR_INVALID_ARG);
        /* backward entry points */
        for (int k = 0; k < 13; ++k) {
            void* p[13];
            for (int i = 0; i < 13; ++i) p[i] = P1;
            p[k] = NULL;
            CHECK(dart_sma_bwd(&d, &o, p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7], p[8], p[9], p[10],
                               p[11], p[12], (size_t)1 << 40, NULL) == DART_ERR_INVALID_ARG);
        }
        CHECK(dart_ssd_bwd(&d, NULL, P1, P1, P1, P1, NULL, P1, NULL, NULL, P1, P1, P1, P1, P1, NULL, P1,
                           (size_t)1 << 40, NULL) == DART_ERR_INVALID_ARG);
        /* block kernels */
        CHECK(dart_conv1d_silu(0, 8, 4, 4, 1, P1, P1, NULL, NULL, NULL, P1, NULL) == DART_ERR_INVALID_ARG);
        CHECK(dart_conv1d_silu(1, 33, 4, 4, 1, P1, P1, NULL, (float*)8, (float*)8, P1, NULL) ==
              DART_ERR_INVALID_ARG);
        CHECK(dart_dt_softplus(4, 3, 2, 1, P1, NULL, P1, NULL) == DART_ERR_INVALID_ARG);
        CHECK(dart_gated_rmsnorm(2, 64, 24, 1, (void*)16, (void*)16, 64, NULL, 1e-6f, (void*)16, NULL) ==
              DART_ERR_INVALID_ARG);
        CHECK(dart_gated_rmsnorm(2, 64, 64, 1, (void*)16, (void*)16, 64, NULL, 0.0f, (void*)16, NULL) ==
              DART_ERR_INVALID_ARG);
    }
    /* profiling calls from several threads */
    pthread_t th[4];
    for (int i = 0; i < 4; ++i) pthread_create(&th[i], NULL, hammer, (void*)(intptr_t)i);
    for (int i = 0; i < 4; ++i) pthread_join(th[i], NULL);
    dart_profile_reset();
    CHECK(dart_profile_count() == 0);
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("abi driver ok\n");
    return 0;
}
