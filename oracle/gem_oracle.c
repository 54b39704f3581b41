/*
 * gem_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded CPU reference for Gradient Energy Matching
 * (Hermans & Louppe, "Gradient Energy Matching for Distributed Asynchronous
 * Gradient Descent", arXiv 1805.08469) and for the simulated asynchronous
 * system that feeds it.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load this library.  It shares no
 * code, header, table or constant generator with the HIP library; both sides
 * implement the same written numerics from their published definitions.
 *
 * What it computes (paper references are to sections, equations and Alg. 1):
 *   - the master commit theta_{t+1} = theta_t + Psi(dtheta_t)        (eq. 3)
 *     with Psi the GEM rescaling of Alg. 1:
 *       m   <- mu*m + dtheta                  (Alg. 1, Psi_GEM; eq. 23)
 *       pi  <- (|m| - |theta - s|) / (|dtheta| + eps)   (Alg. 1; eq. 18)
 *       Psi  = pi (.) dtheta                  (Alg. 1)
 *     where s = theta_{t - tau_t} is the committing worker's snapshot
 *     (eq. 2) and m is that worker's own first-moment estimate (Sec. 3.3).
 *   - the worker update dtheta = -eta * grad L(s)   (notation table) for a
 *     diagonal quadratic L = 1/2 sum h_i (theta_i - theta*_i)^2 whose gradient
 *     carries additive Gaussian noise sigma * xi(seed, t, i).
 *   - the queuing schedule that says which worker commits at each global
 *     clock t and with what staleness tau_t (Sec. 1, eq. 2).
 *
 * Floating point: the workloads fix fp32 parameters and fp32 (or bf16)
 * updates, so every step is evaluated in IEEE binary32 with round-to-nearest-
 * even, in the order written below, with fmaf() only where it is written and
 * no contraction anywhere (build with -ffp-contract=off).  Diagnostics that
 * sum over elements accumulate in binary64.
 *
 * Readings where the paper is silent (all listed in the design notes):
 *   - the snapshot is taken right after the worker's own commit (post-commit
 *     pull), so tau counts the other workers' commits in between and n=1
 *     means zero staleness; Alg. 1's literal pre-commit pull is a mode;
 *   - pi is clamped at zero (CLAMP0) unless the LITERAL mode is requested;
 *   - m is per worker (a global m is a mode); kappa enters as kappa*|m|
 *     (LINEAR, appendix B, last form) or sqrt(kappa)*|m| (SQRT, appendix B,
 *     first form).
 *
 * What pins it (the test suite, against things other than this file):
 * hand traces in exact dyadic arithmetic and the Psi-level cases; the n = 1
 * reductions to SGD (bit for bit) and to the heavy-ball closed form; eqs.
 * (12)-(13) as invariants of every element-commit; Philox against numpy's
 * independent Philox4x64 and published known answers; ln, sin and cos
 * exhaustively against binary64 libm; the schedule's staleness law (Sec. 1)
 * and the per-worker mean laws (Kolmogorov-Smirnov); one-element segments
 * against the element-wise commit; segment factors against exactly rounded
 * norms; the energy sums (eqs. 11, 22) and clamp counts recomputed from the
 * states around each commit, eq. 13 for one worker and eq. 12 for clamped
 * commits; the loss on exact cases and along the SGD closed form.
 * Parity unpinned:
 * the paper prints no trajectory at n > 1, so beyond those invariants and
 * special cases nothing but device == oracle equality pins such runs.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* Philox4xW-10, Salmon, Moraes, Dror & Shaw, "Parallel random numbers: as    */
/* easy as 1, 2, 3", SC'11.  Round: (hi,lo) products of words 0 and 2 with   */
/* the two multipliers; out = (hi1^c1^k0, lo1, hi0^c3^k1, lo0).  The key is   */
/* bumped by the Weyl constants between rounds.                               */
/* ------------------------------------------------------------------------- */
#define OR_PHILOX_M32_0 0xD2511F53u
#define OR_PHILOX_M32_1 0xCD9E8D57u
#define OR_PHILOX_W32_0 0x9E3779B9u /* golden ratio: floor(2^32 * (sqrt(5)-1)/2) */
#define OR_PHILOX_W32_1 0xBB67AE85u /* floor(2^32 * (sqrt(3)-1)) */

#define OR_PHILOX_M64_0 0xD2E7470EE14C6C93ull
#define OR_PHILOX_M64_1 0xCA5A826395121157ull
#define OR_PHILOX_W64_0 0x9E3779B97F4A7C15ull
#define OR_PHILOX_W64_1 0xBB67AE8584CAA73Bull

void or_philox4x32(const uint32_t ctr[4], const uint32_t key[2], int rounds,
                   uint32_t out[4])
{
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int r = 0; r < rounds; ++r) {
        if (r > 0) {
            k0 += OR_PHILOX_W32_0;
            k1 += OR_PHILOX_W32_1;
        }
        uint64_t p0 = (uint64_t)OR_PHILOX_M32_0 * (uint64_t)c0;
        uint64_t p1 = (uint64_t)OR_PHILOX_M32_1 * (uint64_t)c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* The 64-bit-word member of the same family; used only to pin the round and
 * key-schedule structure against an independent implementation. */
void or_philox4x64(const uint64_t ctr[4], const uint64_t key[2], int rounds,
                   uint64_t out[4])
{
    uint64_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint64_t k0 = key[0], k1 = key[1];
    for (int r = 0; r < rounds; ++r) {
        if (r > 0) {
            k0 += OR_PHILOX_W64_0;
            k1 += OR_PHILOX_W64_1;
        }
        unsigned __int128 p0 = (unsigned __int128)OR_PHILOX_M64_0 * c0;
        unsigned __int128 p1 = (unsigned __int128)OR_PHILOX_M64_1 * c2;
        uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
        uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
        uint64_t n0 = hi1 ^ c1 ^ k0;
        uint64_t n1 = lo1;
        uint64_t n2 = hi0 ^ c3 ^ k1;
        uint64_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

uint32_t or_philox_weyl32(int which) { return which ? OR_PHILOX_W32_1 : OR_PHILOX_W32_0; }
uint64_t or_philox_weyl64(int which) { return which ? OR_PHILOX_W64_1 : OR_PHILOX_W64_0; }

/* ------------------------------------------------------------------------- */
/* Gaussian noise: Box & Muller (1958), r = sqrt(-2 ln u1),                   */
/* xi = r cos(2 pi u2) and r sin(2 pi u2), with ln, sin and cos evaluated by  */
/* textbook series in a fixed binary32 operation order so that any IEEE       */
/* implementation of the same steps gives the same bits.                      */
/* ------------------------------------------------------------------------- */

static float or_bits_to_float(uint32_t b) { float f; memcpy(&f, &b, 4); return f; }
static uint32_t or_float_to_bits(float f) { uint32_t b; memcpy(&b, &f, 4); return b; }

/* ln 2 split: LN2_HI = 0x1.62e4p-1 has 15 significant bits, so e*LN2_HI is
 * exact for |e| < 512; LN2_LO is ln 2 - LN2_HI rounded to binary32. */
#define OR_LN2_HI 0x1.62e4p-1f
#define OR_LN2_LO 0x1.7f7d1cp-20f

float or_ln2_lo(void) { return OR_LN2_LO; }

/* Natural log of a normal binary32 u in (0, 1].  u = 2^e * f with f in
 * (sqrt(1/2), sqrt(2)], ln f = 2 atanh(s), s = (f-1)/(f+1) (Abramowitz &
 * Stegun 4.1.27), the series truncated after the s^9 term. */
float or_log_unit(float u)
{
    uint32_t b = or_float_to_bits(u);
    int32_t e = (int32_t)((b >> 23) & 0xFFu) - 127;
    uint32_t mant = b & 0x7FFFFFu;
    uint32_t fb;
    if (mant > 0x3504F3u) {          /* 1.mant > sqrt(2) rounded to binary32 */
        fb = mant | (126u << 23);    /* f = 1.mant / 2 */
        e += 1;
    } else {
        fb = mant | (127u << 23);    /* f = 1.mant */
    }
    float f = or_bits_to_float(fb);
    float num = f - 1.0f;
    float den = f + 1.0f;
    float s = num / den;
    float z = s * s;
    float p = 1.0f / 9.0f;
    p = fmaf(p, z, 1.0f / 7.0f);
    p = fmaf(p, z, 1.0f / 5.0f);
    p = fmaf(p, z, 1.0f / 3.0f);
    p = p * z;
    float s2 = s + s;
    float lnf = fmaf(s2, p, s2);
    float ef = (float)e;
    float r = fmaf(ef, OR_LN2_LO, lnf);
    r = fmaf(ef, OR_LN2_HI, r);
    return r;
}

/* sin and cos of 2*pi*k/2^24 for an integer k in [0, 2^24).  The reduction
 * to the nearest quarter turn is done on the integer (exact); the remaining
 * angle x in [-pi/4, pi/4) is evaluated with the Taylor series of sin (to
 * x^9) and cos (to x^10). */
void or_sincos_turn24(uint32_t k, float* sin_out, float* cos_out)
{
    uint32_t j = (k + 0x200000u) >> 22;              /* nearest quarter turn, 0..4 */
    int32_t rem = (int32_t)k - (int32_t)(j << 22);   /* in [-2^21, 2^21) */
    const float two_pi_2m24 = 6.28318530717958647692f * 0x1p-24f;
    float x = (float)rem * two_pi_2m24;
    float x2 = x * x;

    float ps = 1.0f / 362880.0f;
    ps = fmaf(ps, x2, -1.0f / 5040.0f);
    ps = fmaf(ps, x2, 1.0f / 120.0f);
    ps = fmaf(ps, x2, -1.0f / 6.0f);
    ps = ps * x2;
    float sx = fmaf(x, ps, x);

    float pc = -1.0f / 3628800.0f;
    pc = fmaf(pc, x2, 1.0f / 40320.0f);
    pc = fmaf(pc, x2, -1.0f / 720.0f);
    pc = fmaf(pc, x2, 1.0f / 24.0f);
    pc = fmaf(pc, x2, -0.5f);
    float cx = fmaf(pc, x2, 1.0f);

    switch (j & 3u) {
    case 0: *sin_out = sx;  *cos_out = cx;  break;
    case 1: *sin_out = cx;  *cos_out = -sx; break;
    case 2: *sin_out = -sx; *cos_out = -cx; break;
    default: *sin_out = -cx; *cos_out = sx; break;
    }
}

/* Box-Muller pair from two 32-bit words: u1 = ((xa>>8)+1) 2^-24 in (0,1],
 * u2 = (xb>>8) 2^-24 in [0,1). */
void or_box_muller(uint32_t xa, uint32_t xb, float* z_cos, float* z_sin)
{
    float u1 = (float)((xa >> 8) + 1u) * 0x1p-24f;
    float l = or_log_unit(u1);
    float r = sqrtf(-2.0f * l);
    float sn, cs;
    or_sincos_turn24(xb >> 8, &sn, &cs);
    *z_cos = r * cs;
    *z_sin = r * sn;
}

/* Standard normal xi(seed, t, i): one Philox4x32-10 call with key
 * (seed lo, seed hi) and counter (q lo, q hi, t, 0), q = i >> 2, serves the
 * four elements 4q..4q+3 as (r0 cos, r0 sin, r2 cos, r2 sin). */
float or_normal(uint64_t seed, uint32_t t, int64_t i)
{
    uint64_t q = (uint64_t)i >> 2;
    uint32_t ctr[4] = {(uint32_t)q, (uint32_t)(q >> 32), t, 0u};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t x[4];
    or_philox4x32(ctr, key, 10, x);
    int lane = (int)(i & 3);
    float zc, zs;
    if (lane < 2) or_box_muller(x[0], x[1], &zc, &zs);
    else or_box_muller(x[2], x[3], &zc, &zs);
    return (lane & 1) ? zs : zc;
}

void or_normals(uint64_t seed, uint32_t t, int64_t i0, int64_t count, float* out)
{
    for (int64_t k = 0; k < count; ++k) out[k] = or_normal(seed, t, i0 + k);
}

/* Round a binary32 value to bfloat16, nearest-even, and widen it back. */
float or_round_bf16(float x)
{
    uint32_t b = or_float_to_bits(x);
    if ((b & 0x7FFFFFFFu) > 0x7F800000u) {
        b = (b | 0x00400000u) & 0xFFFF0000u; /* quiet NaN */
    } else {
        b = (b + 0x7FFFu + ((b >> 16) & 1u)) & 0xFFFF0000u;
    }
    return or_bits_to_float(b);
}

/* ------------------------------------------------------------------------- */
/* Queuing schedule (Sec. 1: asynchronous workers and staleness, eq. 2).      */
/* All n workers pull theta_0 at clock 0 and start a job; worker w's k-th job */
/* lasts c_{w,k}.  The next commit belongs to the worker whose job ends       */
/* first (ties to the lower id); that worker then pulls and starts its next   */
/* job.  tau_t = t - (clock of w's last pull).                                */
/* ------------------------------------------------------------------------- */
enum { OR_LAW_EXP = 0, OR_LAW_EXP_UNIFORM_MEAN = 1, OR_LAW_EXP_LOGNORMAL_MEAN = 2,
       OR_LAW_PARETO = 3 };
enum { OR_PULL_POST = 0, OR_PULL_PRE = 1 };

/* 53-bit uniform in (0, 1] from two Philox words. */
static double or_u53_open0(uint32_t a, uint32_t b)
{
    uint64_t v = ((uint64_t)(a >> 11) << 32) | (uint64_t)b;
    return (double)(v + 1u) * 0x1p-53;
}
/* 53-bit uniform in [0, 1). */
static double or_u53_closed0(uint32_t a, uint32_t b)
{
    uint64_t v = ((uint64_t)(a >> 11) << 32) | (uint64_t)b;
    return (double)v * 0x1p-53;
}

static void or_sched_draw(uint64_t seed, uint32_t w, uint64_t k, uint32_t tag, uint32_t x[4])
{
    uint32_t ctr[4] = {w, (uint32_t)k, (uint32_t)(k >> 32), tag};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    or_philox4x32(ctr, key, 10, x);
}

/* Mean compute time of worker w under the law (tag 2 draws). */
double or_worker_mean(int32_t law, double p0, double p1, uint64_t seed, int32_t w)
{
    uint32_t x[4];
    or_sched_draw(seed, (uint32_t)w, 0, 2u, x);
    if (law == OR_LAW_EXP_UNIFORM_MEAN) {
        return p0 + (p1 - p0) * or_u53_closed0(x[0], x[1]);
    }
    if (law == OR_LAW_EXP_LOGNORMAL_MEAN) {
        double u1 = or_u53_open0(x[0], x[1]);
        double u2 = or_u53_closed0(x[2], x[3]);
        double z = sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2);
        return exp(p0 + p1 * z);
    }
    return 1.0;
}

/* Duration of job k of worker w (tag 1 draws). */
double or_job_time(int32_t law, double p0, double p1, double mean_w, uint64_t seed,
                   int32_t w, int64_t k)
{
    uint32_t x[4];
    or_sched_draw(seed, (uint32_t)w, (uint64_t)k, 1u, x);
    double u = or_u53_open0(x[0], x[1]);
    if (law == OR_LAW_PARETO) {
        /* p0 = alpha, p1 = x_m */
        return p1 * pow(u, -1.0 / p0);
    }
    return -mean_w * log(u);
}

int or_schedule(int32_t n, int64_t T, int32_t law, double p0, double p1, uint64_t seed,
                int32_t pull_mode, int32_t* worker, int32_t* tau)
{
    if (n <= 0 || T < 0) return -1;
    double* finish = (double*)malloc(sizeof(double) * (size_t)n);
    double* mean = (double*)malloc(sizeof(double) * (size_t)n);
    int64_t* jobs = (int64_t*)malloc(sizeof(int64_t) * (size_t)n);
    int64_t* pulled = (int64_t*)malloc(sizeof(int64_t) * (size_t)n);
    if (!finish || !mean || !jobs || !pulled) {
        free(finish); free(mean); free(jobs); free(pulled);
        return -2;
    }
    for (int32_t w = 0; w < n; ++w) {
        mean[w] = or_worker_mean(law, p0, p1, seed, w);
        finish[w] = or_job_time(law, p0, p1, mean[w], seed, w, 0);
        jobs[w] = 1;
        pulled[w] = 0;
    }
    for (int64_t t = 0; t < T; ++t) {
        int32_t best = 0;
        for (int32_t w = 1; w < n; ++w)
            if (finish[w] < finish[best]) best = w;
        worker[t] = best;
        tau[t] = (int32_t)(t - pulled[best]);
        pulled[best] = (pull_mode == OR_PULL_PRE) ? t : t + 1;
        finish[best] = finish[best] + or_job_time(law, p0, p1, mean[best], seed, best, jobs[best]);
        jobs[best] += 1;
    }
    free(finish); free(mean); free(jobs); free(pulled);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* The master commit.                                                         */
/* ------------------------------------------------------------------------- */
enum { OR_PI_CLAMP0 = 0, OR_PI_LITERAL = 1 };
enum { OR_KAPPA_LINEAR = 0, OR_KAPPA_SQRT = 1 };
enum { OR_RULE_GEM = 0, OR_RULE_DOWNPOUR = 1, OR_RULE_ADAPTIVE = 2 };
enum { OR_OK = 0, OR_EINVAL = -1, OR_ENOMEM = -2, OR_EWORKER = -3, OR_ESTALE = -4 };
/* Proxy estimate: each worker's own first moment (Sec. 3.3), or one moment
 * shared by all workers and refreshed by every commit -- the global proxy the
 * conclusion (Sec. 6) proposes as future work; it is then the velocity of
 * sequential momentum SGD (eq. 14) driven by all the committed updates. */
enum { OR_PROXY_LOCAL = 0, OR_PROXY_GLOBAL = 1 };

typedef struct {
    int64_t P;        /* total parameter count; noise is keyed by global index */
    int32_t n;        /* number of workers */
    float lr;         /* eta */
    float sigma;      /* gradient noise standard deviation */
    float momentum;   /* mu */
    float eps;        /* epsilon of Alg. 1 */
    float kappa;      /* proxy energy amplification (appendix B) */
    int32_t pi_mode;
    int32_t kappa_mode;
    int32_t pull_mode;
    int32_t rule;
    int32_t bf16;     /* round each update to bfloat16 before it is committed */
    int32_t proxy;    /* OR_PROXY_LOCAL: m per worker; OR_PROXY_GLOBAL: one m in row 0 */
    uint64_t seed;
} or_config;

/* Histogram of the applied scale factor of one commit (the per-parameter pi
 * whose median Sec. 4 follows over time).  Bin 0: pi <= 0 or NaN (clamped);
 * bin 1: 0 < pi < 2^-20; bins 2 + 16 o + f for 2^(o-20) (1 + f/16) <= pi
 * < 2^(o-20) (1 + (f+1)/16), o in [0, 40), f in [0, 16); bin 642: pi >= 2^20. */
#define OR_PI_BINS 643

int or_pi_bin(float pi)
{
    if (!(pi > 0.0f)) return 0;
    uint32_t b = or_float_to_bits(pi);
    int32_t octave = (int32_t)((b >> 23) & 0xFFu) - 127 + 20;
    if (octave < 0) return 1;
    if (octave >= 40) return OR_PI_BINS - 1;
    return 2 + octave * 16 + (int32_t)((b >> 19) & 0xFu);
}

typedef struct {
    double sum_ek;        /* sum_i 1/2 (theta_{t+1} - s)^2      (eq. 11) */
    double sum_proxy;     /* sum_i 1/2 (k_eff m)^2              (eq. 22) */
    int64_t n_clamped;    /* elements whose raw pi was negative or NaN */
    int64_t pad;
} or_commit_diag;

/* kappa as it multiplies |m|: kappa itself, or sqrt(kappa) (binary32). */
static float or_k_eff(const or_config* c)
{
    return (c->kappa_mode == OR_KAPPA_SQRT) ? sqrtf(c->kappa) : c->kappa;
}

/* One element of one commit.  theta, m_w and s_w are updated in place;
 * d is the (possibly bf16-rounded) update; trace, if given, receives
 * (a, pi, d, m). */
static void or_commit_element(const or_config* c, float k_eff, int32_t tau, float d,
                              float* theta, float* m_w, float* s_w,
                              or_commit_diag* dg, float* trace, uint32_t* hist)
{
    float th = *theta;
    float s = *s_w;
    /* Alg. 1 Psi_GEM, first line: the worker's first moment, eq. (23). */
    float m = fmaf(c->momentum, *m_w, d);
    /* theta_t - s_t: the collective drift since the worker's pull (eq. 16). */
    float a = th - s;
    float pi_raw = 0.0f, pi = 0.0f, psi, scale;
    if (c->rule == OR_RULE_GEM) {
        /* Alg. 1, second line, with kappa per appendix B. */
        float num = k_eff * fabsf(m) - fabsf(a);
        float den = fabsf(d) + c->eps;
        pi_raw = num / den;
        if (c->pi_mode == OR_PI_CLAMP0) pi = (pi_raw > 0.0f) ? pi_raw : 0.0f;
        else pi = pi_raw;
        /* Alg. 1, third line, and eq. (3). */
        th = fmaf(pi, d, th);
        scale = pi;
    } else if (c->rule == OR_RULE_DOWNPOUR) {
        th = th + d;                                   /* eq. (1) */
        scale = 1.0f;
    } else {
        psi = d / (float)(tau + 1);                    /* dtheta / (tau + 1) */
        th = th + psi;
        scale = 1.0f / (float)(tau + 1);
    }
    if (hist) hist[or_pi_bin(scale)] += 1u;
    if (dg) {
        double e = (double)th - (double)s;
        double km = (double)k_eff * (double)m;
        dg->sum_ek += 0.5 * e * e;
        dg->sum_proxy += 0.5 * km * km;
        if (c->rule == OR_RULE_GEM && !(pi_raw >= 0.0f)) dg->n_clamped += 1;
    }
    if (trace) {
        trace[0] = a; trace[1] = pi; trace[2] = d; trace[3] = m;
    }
    *m_w = m;
    /* Pull: post-commit takes theta_{t+1}; Alg. 1's literal order takes theta_t. */
    *s_w = (c->pull_mode == OR_PULL_PRE) ? *theta : th;
    *theta = th;
}

static int or_check_schedule(const or_config* c, const int64_t* pc_in, int64_t t0,
                             const int32_t* worker, const int32_t* tau, int64_t T)
{
    int64_t* pc = (int64_t*)malloc(sizeof(int64_t) * (size_t)c->n);
    if (!pc) return OR_ENOMEM;
    memcpy(pc, pc_in, sizeof(int64_t) * (size_t)c->n);
    int rc = OR_OK;
    for (int64_t j = 0; j < T; ++j) {
        int32_t w = worker[j];
        if (w < 0 || w >= c->n) { rc = OR_EWORKER; break; }
        int64_t t = t0 + j;
        if (tau && (int64_t)tau[j] != t - pc[w]) { rc = OR_ESTALE; break; }
        pc[w] = (c->pull_mode == OR_PULL_PRE) ? t : t + 1;
    }
    free(pc);
    return rc;
}

/*
 * Simulated run: T commits starting at global clock t0 on the element subset
 * idx[0..cnt).  For commit j the worker is w = worker[j]; its update is
 * computed at its snapshot: dtheta = -eta (h (s - theta*) + sigma xi(seed, t, i)).
 * State arrays: theta[cnt], S[n*cnt], M[n*cnt] (row w at w*cnt), pc[n].
 * diag, if given, has T entries; trace, if given, has T*cnt*4 floats;
 * pi_hist, if given, has T*OR_PI_BINS counts (added to); with hist_nseg > 0
 * segments [hist_seg_off[s], hist_seg_off[s+1]) of the global index it has
 * T*hist_nseg*OR_PI_BINS, commit-major, each element counted in its
 * segment's histogram (the per-tensor statistics of the supplementary
 * figures).
 */
int or_run(const or_config* c, const int64_t* idx, int64_t cnt,
           const float* h, const float* ts,
           float* theta, float* S, float* M, int64_t* pc, int64_t t0,
           const int32_t* worker, const int32_t* tau, int64_t T,
           or_commit_diag* diag, float* trace, uint32_t* pi_hist,
           int32_t hist_nseg, const int64_t* hist_seg_off)
{
    if (!c || c->n <= 0 || cnt < 0 || T < 0) return OR_EINVAL;
    if (hist_nseg < 0 || (hist_nseg > 0 && !hist_seg_off)) return OR_EINVAL;
    int rc = or_check_schedule(c, pc, t0, worker, tau, T);
    if (rc) return rc;
    const float k_eff = or_k_eff(c);
    const float neg_lr = -c->lr;
    for (int64_t j = 0; j < T; ++j) {
        const int32_t w = worker[j];
        const int64_t t = t0 + j;
        const int32_t tj = (int32_t)(t - pc[w]);
        or_commit_diag* dg = diag ? &diag[j] : NULL;
        if (dg) memset(dg, 0, sizeof(*dg));
        const int64_t mrow = (c->proxy == OR_PROXY_GLOBAL) ? 0 : w;
        for (int64_t k = 0; k < cnt; ++k) {
            float* s_w = &S[(int64_t)w * cnt + k];
            float* m_w = &M[mrow * cnt + k];
            const float s = *s_w;
            /* Stale gradient at the snapshot (notation table: dtheta = -eta grad L(s_t)). */
            float xi = or_normal(c->seed, (uint32_t)t, idx[k]);
            float noise = c->sigma * xi;
            float diff = s - ts[k];
            float g = fmaf(h[k], diff, noise);
            float d = neg_lr * g;
            if (c->bf16) d = or_round_bf16(d);
            uint32_t* hist = NULL;
            if (pi_hist && hist_nseg == 0) hist = &pi_hist[j * OR_PI_BINS];
            if (pi_hist && hist_nseg > 0) {
                int32_t sg = 0;   /* the segment holding global index idx[k] */
                while (sg + 1 < hist_nseg && hist_seg_off[sg + 1] <= idx[k]) ++sg;
                hist = &pi_hist[(j * hist_nseg + sg) * OR_PI_BINS];
            }
            or_commit_element(c, k_eff, tj, d, &theta[k], m_w, s_w, dg,
                              trace ? &trace[(j * cnt + k) * 4] : NULL, hist);
        }
        pc[w] = (c->pull_mode == OR_PULL_PRE) ? t : t + 1;
    }
    return OR_OK;
}

/*
 * Commits of given updates (the gem_commit / gem_commit_batch semantics):
 * K commits starting at clock t0 on all P elements; update j is d[j*P ..]
 * (binary32) or db[j*P ..] (bfloat16 bit patterns) when d is NULL.
 * trace, if given, has K*P*4 floats (a, pi, d, m); pi_hist as in or_run.
 */
int or_commit_given(const or_config* c, int64_t P, float* theta, float* S, float* M,
                    int64_t* pc, int64_t t0, const int32_t* worker, const int32_t* tau,
                    int64_t K, const float* d, const uint16_t* db, or_commit_diag* diag,
                    float* trace, uint32_t* pi_hist)
{
    if (!c || c->n <= 0 || P < 0 || K < 0 || (!d && !db)) return OR_EINVAL;
    int rc = or_check_schedule(c, pc, t0, worker, tau, K);
    if (rc) return rc;
    const float k_eff = or_k_eff(c);
    for (int64_t j = 0; j < K; ++j) {
        const int32_t w = worker[j];
        const int64_t t = t0 + j;
        const int32_t tj = (int32_t)(t - pc[w]);
        or_commit_diag* dg = diag ? &diag[j] : NULL;
        if (dg) memset(dg, 0, sizeof(*dg));
        const int64_t mrow = (c->proxy == OR_PROXY_GLOBAL) ? 0 : w;
        for (int64_t i = 0; i < P; ++i) {
            float di;
            if (d) di = d[j * P + i];
            else di = or_bits_to_float((uint32_t)db[j * P + i] << 16);
            or_commit_element(c, k_eff, tj, di, &theta[i], &M[mrow * P + i],
                              &S[(int64_t)w * P + i], dg,
                              trace ? &trace[(j * P + i) * 4] : NULL,
                              pi_hist ? &pi_hist[j * OR_PI_BINS] : NULL);
        }
        pc[w] = (c->pull_mode == OR_PULL_PRE) ? t : t + 1;
    }
    return OR_OK;
}

/* ------------------------------------------------------------------------- */
/* Segment-norm scale factors.                                                */
/*                                                                            */
/* Eq. (18) divides absolute values element by element.  The same energy      */
/* argument (eqs. 11-13, triangle inequality) holds with Euclidean norms over */
/* any block of parameters, which gives one scale factor per segment of the   */
/* parameter vector (a tensor, or the whole vector for a global norm):       */
/*   pi_T = (k_eff ||m_T|| - ||theta_T - s_T||) / (||dtheta_T|| + eps),       */
/* applied as theta_i <- theta_i + pi_T dtheta_i for i in T.  With segments  */
/* of one element the norms are absolute values and this is eq. (18).        */
/*                                                                            */
/* A sum of squares over a segment is a sum of many terms, so its order is   */
/* part of the definition:                                                    */
/*   - every term x_i^2 of binary32 x_i is formed exactly in binary64;       */
/*   - indices are split into aligned blocks of 2^18 (block b holds          */
/*     i = 2^18 b .. 2^18 b + 2^18 - 1); terms outside the segment count as   */
/*     zero;                                                                  */
/*   - a block's terms are added by the adjacent-pairs binary tree: (0+1),   */
/*     (2+3), ..., then ((0+1)+(2+3)), and so on up to one value;             */
/*   - the block values are added, in increasing b, to a running total that  */
/*     starts at zero.                                                        */
/* The norm is the binary64 square root of that total, rounded to binary32;  */
/* pi_T then follows the binary32 steps of or_commit_element.                */
/* ------------------------------------------------------------------------- */
#define OR_SEG_BLOCK (1 << 18)

/* The adjacent-pairs tree over the aligned index range [base, base + len),
 * len a power of two: the sum of its two halves, each added the same way; one
 * index gives its term.  A subtree with no index in [lo, hi) is zero, and
 * adding zero is exact, so such subtrees are not visited. */
static double or_tree(const float* x, int64_t lo, int64_t hi, int64_t base, int64_t len)
{
    if (base >= hi || base + len <= lo) return 0.0;
    if (len == 1) return (double)x[base] * (double)x[base];
    const int64_t half = len / 2;
    return or_tree(x, lo, hi, base, half) + or_tree(x, lo, hi, base + half, half);
}

double or_sumsq(const float* x, int64_t lo, int64_t hi)
{
    double total = 0.0;
    if (hi <= lo) return 0.0;
    for (int64_t b = lo / OR_SEG_BLOCK; b * OR_SEG_BLOCK < hi; ++b)
        total = total + or_tree(x, lo, hi, b * OR_SEG_BLOCK, OR_SEG_BLOCK);
    return total;
}

static float or_norm(const float* x, int64_t lo, int64_t hi)
{
    return (float)sqrt(or_sumsq(x, lo, hi));
}

/*
 * T commits on all P = c->P elements with one scale factor per segment
 * [seg_off[k], seg_off[k+1]), seg_off[0] = 0 < ... < seg_off[nseg] = P.
 * Updates are generated at the snapshots as in or_run when d and db are both
 * NULL, else given as in or_commit_given.  GEM rule only.  pi_out, if given,
 * receives the applied pi of every segment of every commit (T * nseg);
 * trace, if given, (a, d, m) of every element of every commit (T * P * 3);
 * diag, if given, the energies of each commit as in or_run (T entries), with
 * n_clamped counting the elements of segments whose raw pi was negative or
 * NaN.
 */
int or_run_segments(const or_config* c, int32_t nseg, const int64_t* seg_off,
                    const float* h, const float* ts, float* theta, float* S, float* M,
                    int64_t* pc, int64_t t0, const int32_t* worker, const int32_t* tau,
                    int64_t T, const float* d, const uint16_t* db, float* pi_out, float* trace,
                    or_commit_diag* diag)
{
    if (!c || c->n <= 0 || c->P < 0 || T < 0 || nseg < 1 || !seg_off) return OR_EINVAL;
    if (c->rule != OR_RULE_GEM) return OR_EINVAL;
    if (seg_off[0] != 0 || seg_off[nseg] != c->P) return OR_EINVAL;
    for (int32_t k = 0; k < nseg; ++k)
        if (seg_off[k + 1] <= seg_off[k]) return OR_EINVAL;
    if (!d && !db && (!h || !ts)) return OR_EINVAL;
    int rc = or_check_schedule(c, pc, t0, worker, tau, T);
    if (rc) return rc;
    const int64_t P = c->P;
    float* dv = (float*)malloc(sizeof(float) * (size_t)(P > 0 ? P : 1));
    float* mv = (float*)malloc(sizeof(float) * (size_t)(P > 0 ? P : 1));
    float* av = (float*)malloc(sizeof(float) * (size_t)(P > 0 ? P : 1));
    if (!dv || !mv || !av) { free(dv); free(mv); free(av); return OR_ENOMEM; }
    const float k_eff = or_k_eff(c);
    const float neg_lr = -c->lr;
    for (int64_t j = 0; j < T; ++j) {
        const int32_t w = worker[j];
        const int64_t t = t0 + j;
        const int64_t mrow = (c->proxy == OR_PROXY_GLOBAL) ? 0 : w;
        float* s_row = &S[(int64_t)w * P];
        float* m_row = &M[mrow * P];
        or_commit_diag* dg = diag ? &diag[j] : NULL;
        if (dg) memset(dg, 0, sizeof(*dg));
        /* The update, the refreshed first moment (Alg. 1, eq. 23) and the
         * drift theta_t - s_t (eq. 16), element by element. */
        for (int64_t i = 0; i < P; ++i) {
            float di;
            if (d) {
                di = d[j * P + i];
            } else if (db) {
                di = or_bits_to_float((uint32_t)db[j * P + i] << 16);
            } else {
                float xi = or_normal(c->seed, (uint32_t)t, i);
                float g = fmaf(h[i], s_row[i] - ts[i], c->sigma * xi);
                di = neg_lr * g;
                if (c->bf16) di = or_round_bf16(di);
            }
            dv[i] = di;
            mv[i] = fmaf(c->momentum, m_row[i], di);
            av[i] = theta[i] - s_row[i];
        }
        if (trace)
            for (int64_t i = 0; i < P; ++i) {
                trace[(j * P + i) * 3 + 0] = av[i];
                trace[(j * P + i) * 3 + 1] = dv[i];
                trace[(j * P + i) * 3 + 2] = mv[i];
            }
        for (int32_t k = 0; k < nseg; ++k) {
            const int64_t lo = seg_off[k], hi = seg_off[k + 1];
            /* Eq. (18) with norms over the segment. */
            float num = k_eff * or_norm(mv, lo, hi) - or_norm(av, lo, hi);
            float den = or_norm(dv, lo, hi) + c->eps;
            const float pi_raw = num / den;
            float pi = pi_raw;
            if (c->pi_mode == OR_PI_CLAMP0) pi = (pi > 0.0f) ? pi : 0.0f;
            if (pi_out) pi_out[j * nseg + k] = pi;
            if (dg && !(pi_raw >= 0.0f)) dg->n_clamped += hi - lo;
            for (int64_t i = lo; i < hi; ++i) {
                const float th_old = theta[i];
                const float th_new = fmaf(pi, dv[i], th_old);   /* eq. (3) */
                if (dg) {
                    /* E_k (eq. 11) against the committing worker's snapshot
                     * and the proxy energy (eq. 22), as in or_commit_element. */
                    const double e = (double)th_new - (double)s_row[i];
                    const double km = (double)k_eff * (double)mv[i];
                    dg->sum_ek += 0.5 * e * e;
                    dg->sum_proxy += 0.5 * km * km;
                }
                m_row[i] = mv[i];
                s_row[i] = (c->pull_mode == OR_PULL_PRE) ? th_old : th_new;
                theta[i] = th_new;
            }
        }
        pc[w] = (c->pull_mode == OR_PULL_PRE) ? t : t + 1;
    }
    free(dv); free(mv); free(av);
    return OR_OK;
}

/* Loss of the diagonal quadratic, 1/2 sum h (theta - theta*)^2, in binary64. */
double or_loss(const float* theta, const float* h, const float* ts, int64_t cnt)
{
    double acc = 0.0;
    for (int64_t k = 0; k < cnt; ++k) {
        double e = (double)theta[k] - (double)ts[k];
        acc += 0.5 * (double)h[k] * e * e;
    }
    return acc;
}

/* ------------------------------------------------------------------------- */
/* Array helpers for the test suite (element-wise loops over the above).     */
/* ------------------------------------------------------------------------- */
void or_log_unit_array(const float* u, float* out, int64_t n)
{
    for (int64_t k = 0; k < n; ++k) out[k] = or_log_unit(u[k]);
}

void or_sincos_turn24_array(const uint32_t* k24, float* s, float* c, int64_t n)
{
    for (int64_t k = 0; k < n; ++k) or_sincos_turn24(k24[k], &s[k], &c[k]);
}

void or_round_bf16_array(const float* x, float* out, int64_t n)
{
    for (int64_t k = 0; k < n; ++k) out[k] = or_round_bf16(x[k]);
}

void or_normals_at(uint64_t seed, uint32_t t, const int64_t* idx, int64_t count, float* out)
{
    for (int64_t k = 0; k < count; ++k) out[k] = or_normal(seed, t, idx[k]);
}

void or_pi_bin_array(const float* pi, int32_t* out, int64_t n)
{
    for (int64_t k = 0; k < n; ++k) out[k] = or_pi_bin(pi[k]);
}
