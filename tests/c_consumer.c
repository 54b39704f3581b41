/*
 * A plain C program that uses libgem through include/gem.h only: the master
 * for a small diagonal quadratic, a simulated schedule, fused passes, single
 * commits of a device update, a checkpoint round trip, and the read-back.
 * It prints the clock and theta as hexadecimal bit patterns, one per line,
 * for tests/test_c_consumer.py to compare with the oracle.
 *
 * Usage: c_consumer P n T K out_checkpoint_path
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../include/gem.h"

/* The HIP runtime, through its C entry points only. */
extern int hipMalloc(void** ptr, size_t size);
extern int hipMemcpy(void* dst, const void* src, size_t size, int kind);
extern int hipFree(void* ptr);

#define CHECK(call)                                                              \
    do {                                                                         \
        int rc_ = (call);                                                        \
        if (rc_ != GEM_OK) {                                                     \
            fprintf(stderr, "%s failed: %s (%d) [%s]\n", #call, gem_strerror(rc_), \
                    rc_, gem_last_error());                                      \
            return 1;                                                            \
        }                                                                        \
    } while (0)

int main(int argc, char** argv)
{
    if (argc != 6) {
        fprintf(stderr, "usage: %s P n T K checkpoint\n", argv[0]);
        return 2;
    }
    const int64_t P = atoll(argv[1]);
    const int32_t n = atoi(argv[2]);
    const int64_t T = atoll(argv[3]);
    const int32_t K = atoi(argv[4]);
    const char* ckpt = argv[5];

    float* h = malloc(sizeof(float) * (size_t)P);
    float* ts = malloc(sizeof(float) * (size_t)P);
    float* upd = malloc(sizeof(float) * (size_t)P);
    float* theta = malloc(sizeof(float) * (size_t)P);
    int32_t* worker = malloc(sizeof(int32_t) * (size_t)T);
    int32_t* tau = malloc(sizeof(int32_t) * (size_t)T);
    if (!h || !ts || !upd || !theta || !worker || !tau) return 1;
    for (int64_t i = 0; i < P; ++i) {
        h[i] = 0.001f + (float)(i % 97) / 97.0f;     /* in [1e-3, 1] */
        ts[i] = (float)(i % 13) / 6.0f - 1.0f;
        upd[i] = (float)((i * 7) % 11 - 5) * 1e-3f;
    }

    gem_hyperparams hp;
    CHECK(gem_hyperparams_default(&hp));
    gem_t* g = NULL;
    CHECK(gem_create(P, n, &hp, NULL, &g));
    gem_sim_params sp;
    memset(&sp, 0, sizeof(sp));
    sp.lr = 0.01f;
    sp.sigma = 0.1f;
    sp.seed = 20180522u;
    sp.update_dtype = GEM_F32;
    CHECK(gem_set_quadratic(g, h, ts, &sp));

    gem_schedule_law law;
    memset(&law, 0, sizeof(law));
    law.law = GEM_LAW_EXP;
    CHECK(gem_schedule_make(n, T, &law, 7u, GEM_PULL_POST_COMMIT, worker, tau));
    CHECK(gem_sim_run(g, worker, tau, T, K));

    /* Two single commits of a caller update from device memory (staleness
     * comes from the library's own bookkeeping). */
    void* d_upd = NULL;
    if (hipMalloc(&d_upd, sizeof(float) * (size_t)P) != 0) return 1;
    if (hipMemcpy(d_upd, upd, sizeof(float) * (size_t)P, 1 /* host to device */) != 0) return 1;
    CHECK(gem_commit(g, (const float*)d_upd, 0));
    CHECK(gem_commit(g, (const float*)d_upd, n - 1));

    /* Checkpoint round trip into a second master. */
    CHECK(gem_save(g, ckpt));
    gem_t* g2 = NULL;
    CHECK(gem_create(P, n, &hp, NULL, &g2));
    CHECK(gem_load(g2, ckpt));
    CHECK(gem_destroy(g));

    /* A bad call changes nothing and names its error. */
    if (gem_commit(g2, (const float*)d_upd, n) != GEM_EWORKER) return 1;

    int64_t t = 0;
    CHECK(gem_clock(g2, &t));
    CHECK(gem_read_theta(g2, theta, 0));
    CHECK(gem_destroy(g2));
    hipFree(d_upd);

    printf("%lld\n", (long long)t);
    for (int64_t i = 0; i < P; ++i) {
        uint32_t b;
        memcpy(&b, &theta[i], 4);
        printf("%08x\n", b);
    }
    free(h); free(ts); free(upd); free(theta); free(worker); free(tau);
    return 0;
}
