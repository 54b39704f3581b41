/*
 * Exercises every entry point of the CPU oracle (test infrastructure) under
 * AddressSanitizer and UndefinedBehaviorSanitizer: the schedule for every
 * law, simulated runs in every mode with diagnostics, traces and histograms,
 * given updates, the segment-norm variant and the rejected inputs.  Built
 * and run by tests/test_sanitizers.py; exits non-zero on any failure.
 */
#include "../oracle/gem_oracle.c"

#include <stdio.h>

#define CHECK(cond)                                                        \
    do {                                                                   \
        if (!(cond)) {                                                     \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
            return 1;                                                      \
        }                                                                  \
    } while (0)

enum { P = 1300, N = 5, T = 120 };

static float h[P], ts[P], theta[P], S[N * P], M[N * P];
static int64_t pc[N], idx[P];
static int32_t worker[T], tau[T];

static void reset_state(void)
{
    memset(theta, 0, sizeof(theta));
    memset(S, 0, sizeof(S));
    memset(M, 0, sizeof(M));
    memset(pc, 0, sizeof(pc));
}

static or_config config(int mode)
{
    or_config c;
    memset(&c, 0, sizeof(c));
    c.P = P;
    c.n = N;
    c.lr = 0.01f;
    c.sigma = 0.1f;
    c.momentum = 0.9f;
    c.eps = 1e-16f;
    c.kappa = 1.0f;
    c.seed = 42;
    switch (mode) {
    case 1: c.pi_mode = OR_PI_LITERAL; break;
    case 2: c.kappa = 3.0f; c.kappa_mode = OR_KAPPA_SQRT; break;
    case 3: c.pull_mode = OR_PULL_PRE; break;
    case 4: c.rule = OR_RULE_DOWNPOUR; break;
    case 5: c.rule = OR_RULE_ADAPTIVE; break;
    case 6: c.bf16 = 1; break;
    case 7: c.proxy = OR_PROXY_GLOBAL; break;
    default: break;
    }
    return c;
}

int main(void)
{
    for (int i = 0; i < P; ++i) {
        h[i] = 1e-3f + (float)i / (float)P;
        ts[i] = (float)((i * 37) % 101) / 50.0f - 1.0f;
        idx[i] = i;
    }
    /* Schedules: every law and pull mode. */
    for (int law = 0; law <= 3; ++law)
        for (int pull = 0; pull <= 1; ++pull)
            CHECK(or_schedule(N, T, law, law == 3 ? 1.5 : 0.8, law == 3 ? 1.0 / 3 : 1.2, 7, pull,
                              worker, tau) == OR_OK);
    CHECK(or_schedule(0, T, 0, 0, 0, 7, 0, worker, tau) != OR_OK);

    static or_commit_diag diag[T];
    static float trace[T * P * 4];
    static uint32_t hist[T * OR_PI_BINS];
    for (int mode = 0; mode <= 7; ++mode) {
        or_config c = config(mode);
        CHECK(or_schedule(N, T, 0, 0, 0, 11, c.pull_mode, worker, tau) == OR_OK);
        reset_state();
        memset(hist, 0, sizeof(hist));
        CHECK(or_run(&c, idx, P, h, ts, theta, S, M, pc, 0, worker, tau, T, diag, trace, hist, 0,
                     NULL) == OR_OK);
        /* per-segment histograms */
        {
            static uint32_t seg_hist[T * 4 * OR_PI_BINS];
            int64_t hseg[5] = {0, 1, 700, 1024, P};
            reset_state();
            CHECK(or_run(&c, idx, P, h, ts, theta, S, M, pc, 0, worker, tau, T, NULL, NULL,
                         seg_hist, 4, hseg) == OR_OK);
        }
        /* a subset run from the start */
        reset_state();
        CHECK(or_run(&c, idx + 100, 50, h + 100, ts + 100, theta, S, M, pc, 0, worker, tau, T / 2,
                     NULL, NULL, NULL, 0, NULL) == OR_OK);
    }
    /* Rejected schedules leave the state alone. */
    {
        or_config c = config(0);
        reset_state();
        int32_t bad_w[2] = {0, N};
        CHECK(or_run(&c, idx, P, h, ts, theta, S, M, pc, 0, bad_w, NULL, 2, NULL, NULL, NULL, 0,
                     NULL) == OR_EWORKER);
        int32_t w2[2] = {1, 1}, t2[2] = {0, 5};
        CHECK(or_run(&c, idx, P, h, ts, theta, S, M, pc, 0, w2, t2, 2, NULL, NULL, NULL, 0,
                     NULL) == OR_ESTALE);
        for (int i = 0; i < P; ++i) CHECK(theta[i] == 0.0f);
    }
    /* Given updates, binary32 and bfloat16. */
    {
        static float d[8 * P];
        static uint16_t db[8 * P];
        for (int i = 0; i < 8 * P; ++i) {
            d[i] = (float)((i * 13) % 29 - 14) * 1e-3f;
            db[i] = (uint16_t)(or_float_to_bits(or_round_bf16(d[i])) >> 16);
        }
        or_config c = config(0);
        CHECK(or_schedule(N, 8, 0, 0, 0, 3, 0, worker, tau) == OR_OK);
        reset_state();
        CHECK(or_commit_given(&c, P, theta, S, M, pc, 0, worker, tau, 8, d, NULL, diag, trace, hist) == OR_OK);
        reset_state();
        CHECK(or_commit_given(&c, P, theta, S, M, pc, 0, worker, NULL, 8, NULL, db, NULL, NULL, NULL) == OR_OK);
        /* Segment norms with given updates. */
        int64_t seg[4] = {0, 1, 1024, P};
        static float pi_out[8 * 3];
        reset_state();
        CHECK(or_run_segments(&c, 3, seg, NULL, NULL, theta, S, M, pc, 0, worker, tau, 8, d, NULL,
                              pi_out, NULL, diag) == OR_OK);
        reset_state();
        CHECK(or_run_segments(&c, 3, seg, NULL, NULL, theta, S, M, pc, 0, worker, tau, 8, NULL, db,
                              NULL, NULL, NULL) == OR_OK);
    }
    /* Segment norms with generated updates, every supported mode. */
    for (int mode = 0; mode <= 7; ++mode) {
        if (mode == 4 || mode == 5) continue;   /* GEM rule only */
        or_config c = config(mode);
        CHECK(or_schedule(N, 40, 0, 0, 0, 5, c.pull_mode, worker, tau) == OR_OK);
        int64_t seg[6] = {0, 17, 1024, 1025, 1200, P};
        static float pi_out[40 * 5];
        static float tr3[40 * P * 3];
        reset_state();
        CHECK(or_run_segments(&c, 5, seg, h, ts, theta, S, M, pc, 0, worker, tau, 40, NULL, NULL,
                              pi_out, tr3, diag) == OR_OK);
    }
    {
        or_config c = config(0);
        int64_t bad1[3] = {0, 0, P}, bad2[2] = {1, P}, good[2] = {0, P};
        CHECK(or_run_segments(&c, 2, bad1, h, ts, theta, S, M, pc, 0, worker, tau, 1, NULL, NULL,
                              NULL, NULL, NULL) == OR_EINVAL);
        CHECK(or_run_segments(&c, 1, bad2, h, ts, theta, S, M, pc, 0, worker, tau, 1, NULL, NULL,
                              NULL, NULL, NULL) == OR_EINVAL);
        c.rule = OR_RULE_DOWNPOUR;
        CHECK(or_run_segments(&c, 1, good, h, ts, theta, S, M, pc, 0, worker, tau, 1, NULL, NULL,
                              NULL, NULL, NULL) == OR_EINVAL);
    }
    CHECK(or_sumsq(h, 5, 5) == 0.0);
    CHECK(or_loss(theta, h, ts, P) >= 0.0);
    printf("sanitized oracle run: ok\n");
    return 0;
}
