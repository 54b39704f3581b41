/*
 * gem.h -- C ABI of libgem: the master-side commit of Gradient Energy Matching
 * (GEM; Hermans & Louppe, "Gradient Energy Matching for Distributed
 * Asynchronous Gradient Descent", arXiv 1805.08469) on one AMD MI355X (gfx950).
 *
 * The master holds the central variable theta[P].  Each of n workers holds a
 * snapshot S[w] of theta taken at its last pull (the s_t = theta_{t - tau_t}
 * of eq. 2) and its own first-moment estimate M[w] (Sec. 3.3, eq. 23).  A
 * commit of update dtheta by worker w at global clock t applies, elementwise
 * (Alg. 1, Psi_GEM; eqs. 3, 16-18):
 *
 *     m      = mu * M[w] + dtheta
 *     pi     = (kappa_eff * |m| - |theta - S[w]|) / (|dtheta| + eps)
 *     pi     = max(pi, 0)                 (default; GEM_PI_LITERAL keeps it)
 *     theta  = theta + pi * dtheta
 *     M[w]   = m;   S[w] = theta          (the worker pulls after committing)
 *
 * Conventions for every entry point:
 *   - Return value: GEM_OK (0) or a negative GEM_E* code; gem_strerror()
 *     names it.  Arguments are validated before any work is queued, so a
 *     failed call has changed nothing.
 *   - Device pointers are HIP device addresses on the handle's device; host
 *     pointers are ordinary process memory.  Sizes are element counts.
 *   - Work is queued on the handle's HIP stream in call order.  Calls that
 *     return data to the host (gem_read_*, gem_gather, gem_diag, gem_save)
 *     synchronise that stream; the others return once the work is queued.
 *   - A handle is not thread-safe: calls on one handle must not overlap.
 *   - The library owns theta, S, M and the problem arrays (hipMalloc'd at
 *     create / set time, freed by gem_destroy).  Caller buffers passed in
 *     (updates) are only read and must stay valid until the stream reaches
 *     the queued work.
 */
#ifndef LIBGEM_GEM_H
#define LIBGEM_GEM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- return codes ------------------------------------------------------- */
#define GEM_OK        0
#define GEM_EINVAL   (-1)  /* bad argument: null pointer, size out of range, bad enum */
#define GEM_ENOMEM   (-2)  /* device or host allocation failed */
#define GEM_EWORKER  (-3)  /* worker id not in [0, n) */
#define GEM_ESTALE   (-4)  /* a staleness value disagrees with the pull bookkeeping */
#define GEM_EDTYPE   (-5)  /* unknown update dtype */
#define GEM_EHIP     (-6)  /* a HIP runtime call failed */
#define GEM_ESTATE   (-7)  /* the call needs set-up that has not happened (no problem set) */
#define GEM_EIO      (-8)  /* checkpoint file could not be read or written, or does not match */
#define GEM_EALIGN   (-9)  /* a device buffer is not aligned as required */
#define GEM_ESCRATCH (-10) /* the request does not fit the fixed device scratch */

/* ---- enums --------------------------------------------------------------- */
enum { GEM_F32 = 0, GEM_BF16 = 1 };                        /* update element type */
enum { GEM_PI_CLAMP0 = 0, GEM_PI_LITERAL = 1 };            /* sign handling of pi */
enum { GEM_KAPPA_LINEAR = 0, GEM_KAPPA_SQRT = 1 };         /* appendix B forms    */
enum { GEM_PULL_POST_COMMIT = 0, GEM_PULL_PRE_COMMIT = 1 };/* when S[w] is taken  */
enum { GEM_RULE_GEM = 0, GEM_RULE_DOWNPOUR = 1, GEM_RULE_ADAPTIVE = 2 };
enum { GEM_PROXY_LOCAL = 0, GEM_PROXY_GLOBAL = 1 };        /* where m lives       */
enum { GEM_PI_ELEMENT = 0, GEM_PI_SEGMENT = 1 };           /* scope of one pi     */
enum { GEM_CACHE_AUTO = 0, GEM_CACHE_KEEP = 1, GEM_CACHE_STREAM = 2 };  /* see gem_set_cache_policy */
enum { GEM_LAW_EXP = 0, GEM_LAW_EXP_UNIFORM_MEAN = 1, GEM_LAW_EXP_LOGNORMAL_MEAN = 2,
       GEM_LAW_PARETO = 3 };
enum { GEM_SNAPSHOT = 0, GEM_MOMENT = 1 };

/* Largest number of commits one fused pass applies; longer batches are split. */
#define GEM_K_MAX 32

/* Largest P (and gem_gather count): launches run one thread per element or
 * index, and 2^31 of them keep every grid within one dispatch. */
#define GEM_P_MAX (INT64_C(1) << 31)

/* ---- parameter blocks ----------------------------------------------------- */
typedef struct gem_handle gem_t;

/* Commit rule.  Alg. 1 defaults: momentum 0.9, eps 1e-16.  kappa (appendix B)
 * scales the proxy energy; 1 reproduces Alg. 1.  pull_mode POST_COMMIT takes
 * the snapshot after the worker's own commit (so tau counts only the other
 * workers' commits, eq. 2); PRE_COMMIT is Alg. 1's literal Worker order (pull,
 * commit, keep the pulled theta_t).  rule selects GEM or the two baselines of
 * Sec. 4: DOWNPOUR (commit dtheta unchanged, eq. 1) and adaptive staleness
 * (commit dtheta / (tau + 1)).  proxy_mode LOCAL keeps one first moment per
 * worker (Sec. 3.3); GLOBAL keeps one moment shared by all workers, refreshed
 * by every commit (the global proxy of Sec. 6), stored as worker 0's moment
 * (gem_read_state(g, 0, GEM_MOMENT, ...) returns it).
 * pi_scope ELEMENT computes pi per parameter from absolute values (eq. 18);
 * SEGMENT computes one pi per segment of the parameter vector from Euclidean
 * norms over the segment (see gem_set_segments; GEM rule only).
 * momentum must be finite; eps finite and > 0 (it keeps the denominator
 * |dtheta| + eps of Alg. 1 away from zero, so an update of exactly zero
 * leaves theta unchanged); kappa finite and > 0 in both forms.  Calls that
 * take a gem_hyperparams return GEM_EINVAL otherwise. */
typedef struct {
    float momentum;
    float eps;
    float kappa;
    int32_t pi_mode;
    int32_t kappa_mode;
    int32_t pull_mode;
    int32_t rule;
    int32_t proxy_mode;
    int32_t pi_scope;
} gem_hyperparams;

/* Stale-gradient generator of the simulated workers: a worker whose snapshot
 * is s sends dtheta = -lr * (h (s - theta*) + sigma * xi(seed, t, i)), the SGD
 * update of the notation table for the diagonal quadratic
 * L = 1/2 sum h_i (theta_i - theta*_i)^2 with Gaussian gradient noise;
 * xi is Philox4x32-10 + Box-Muller keyed by (seed, commit clock t, index i).
 * update_dtype GEM_BF16 rounds each dtheta to bfloat16 (nearest-even) before
 * it is committed. */
typedef struct {
    float lr;
    float sigma;
    uint64_t seed;
    int32_t update_dtype;
    int32_t reserved;
} gem_sim_params;

/* Compute-time law of the simulated workers (see gem_schedule_make). */
typedef struct {
    int32_t law;
    int32_t reserved;
    double p0;
    double p1;
} gem_schedule_law;

typedef struct {
    double loss;          /* 1/2 sum_i h_i (theta_i - theta*_i)^2 now (0 without a problem) */
    double sum_ek;        /* sum over element-commits of 1/2 (theta_{t+1} - s)^2 (eq. 11) */
    double sum_proxy;     /* sum over element-commits of 1/2 (kappa_eff m)^2 (eq. 22) */
    int64_t n_clamped;    /* element-commits whose raw pi was negative or NaN */
    int64_t n_elem_commits;
    int64_t n_commits;
} gem_diag_t;

/* Work counters since gem_create (or the last gem_stats_reset). */
typedef struct {
    int64_t commits;      /* commits applied */
    int64_t passes;       /* fused kernel launches */
    double alg_bytes;     /* algorithmic HBM bytes of those launches (see below) */
} gem_stats_t;

/* ---- library -------------------------------------------------------------- */

/* Text for a return code; never NULL. */
const char* gem_strerror(int code);

/* Detail of the last GEM_EHIP returned on the calling thread: the HIP call
 * that failed and its error string ("" if none).  Never NULL; valid until the
 * thread's next libgem call. */
const char* gem_last_error(void);

/* Fill hp with Alg. 1's defaults: momentum 0.9, eps 1e-16, kappa 1, CLAMP0,
 * LINEAR, POST_COMMIT, GEM, LOCAL, ELEMENT.  Returns GEM_EINVAL if hp is NULL. */
int gem_hyperparams_default(gem_hyperparams* hp);

/* Create a master for P parameters and n workers on the current HIP device.
 * theta = 0, every S[w] = 0, every M[w] = 0, clock t = 0, all pull clocks 0
 * (all workers pulled theta_0 at clock 0 with m = 0: Alg. 1 Worker start-up).
 * hp may be NULL (defaults).  stream is the hipStream_t all of the handle's
 * work is queued on; NULL means the device's null stream (torch's default
 * stream), so work is ordered with other blocking-stream work.  The stream
 * must outlive the handle.  Device memory: 1 + 2n rows of P floats (2 more
 * once a problem is set), each row padded to a multiple of 64 elements.
 * Errors: EINVAL (P < 1, P > GEM_P_MAX, n < 1, out NULL, bad enum or
 * hyper-parameter value), ENOMEM
 * (including sizes whose byte count does not fit 64 bits), EHIP. */
int gem_create(int64_t P, int32_t n, const gem_hyperparams* hp, void* stream, gem_t** out);

/* Free all device memory (after the stream drains) and the handle. */
int gem_destroy(gem_t* g);

/* Set theta_0 from P floats (host, or device if in_is_device) and restart:
 * S[w] = theta_0, M[w] = 0, t = 0, pull clocks 0, diagnostics cleared. */
int gem_set_theta(gem_t* g, const float* theta0, int32_t in_is_device);

/* Provide the simulated workers' problem: h[P] and theta_star[P] on the host
 * (copied to the device) and the generator parameters.  Needed by
 * gem_generate, gem_sim_run and the loss.  Errors: EINVAL, EDTYPE, ENOMEM. */
int gem_set_quadratic(gem_t* g, const float* h, const float* theta_star,
                      const gem_sim_params* sp);

/* One commit (eq. 3 with Alg. 1's Psi) of the P-float update dtheta_dev (device,
 * 16-byte aligned) by worker_id at the current clock t; then t += 1.
 * Errors: EWORKER, EINVAL (NULL), EALIGN. */
int gem_commit(gem_t* g, const float* dtheta_dev, int32_t worker_id);

/* K queued commits, applied in order at clocks t..t+K-1, bit-identical to K
 * calls of gem_commit (including a worker that appears twice: its second
 * update sees the snapshot it pulled after its first).  dthetas_dev is a host
 * array of K device pointers to P elements of dtype (F32: 16-byte aligned;
 * BF16: 8-byte aligned bfloat16 bit patterns).  staleness, if not NULL, gives
 * each commit's tau (eq. 2) and must equal t_j - pull clock of its worker;
 * otherwise nothing is applied and ESTALE is returned.  Passes of up to
 * GEM_K_MAX commits stream theta once and each distinct worker's S and M rows
 * once (under GEM_PI_SEGMENT each commit is applied on its own; see
 * gem_set_segments). */
int gem_commit_batch(gem_t* g, int32_t K, const void* const* dthetas_dev, int32_t dtype,
                     const int32_t* worker_ids, const int32_t* staleness);

/* The stale-gradient generator alone: write into out_dev (device, P elements
 * of dtype, aligned as for gem_commit_batch) the update worker_id would send
 * for the commit at the current clock t, computed at its snapshot S[w].
 * Needs gem_set_quadratic.  Errors: ESTATE, EWORKER, EDTYPE, EALIGN. */
int gem_generate(gem_t* g, int32_t worker_id, void* out_dev, int32_t dtype);

/* Queuing schedule of the simulated asynchronous system (Sec. 1, eq. 2),
 * host only.  Every worker pulls theta_0 and starts a job at time 0; job k of
 * worker w lasts c_{w,k} drawn from the law (Philox4x32-10 keyed by seed); the
 * next commit belongs to the worker whose job ends first (ties to the lower
 * id), which then pulls and starts its next job.  Writes worker[T] and
 * tau[T] = t - (clock of the worker's last pull), the pull being at t+1 after
 * a commit at t (POST_COMMIT) or at t (PRE_COMMIT).  Laws: EXP (mean 1),
 * EXP_UNIFORM_MEAN (mean_w ~ U[p0, p1]), EXP_LOGNORMAL_MEAN (mean_w =
 * exp(p0 + p1 z)), PARETO (shape p0, scale p1).  Errors: EINVAL. */
int gem_schedule_make(int32_t n, int64_t T, const gem_schedule_law* law, uint64_t seed,
                      int32_t pull_mode, int32_t* worker, int32_t* tau);

/* Simulated run of T commits: commit j is by worker[j] (host array) with
 * staleness tau[j] (host array, may be NULL, else checked like
 * gem_commit_batch), its update generated at the worker's snapshot (see
 * gem_sim_params), all fused into passes of at most K commits (1 <= K <=
 * GEM_K_MAX) that keep theta and the pass's (s, m) pairs in registers (under
 * GEM_PI_SEGMENT K is checked but each commit is applied on its own).  Needs
 * gem_set_quadratic.  Errors: ESTATE, EINVAL, EWORKER, ESTALE. */
int gem_sim_run(gem_t* g, const int32_t* worker, const int32_t* tau, int64_t T, int32_t K);

/* Copy theta (P floats) to out (host, or device if out_is_device). */
int gem_read_theta(gem_t* g, float* out, int32_t out_is_device);

/* Copy worker w's snapshot (which = GEM_SNAPSHOT) or moment (GEM_MOMENT) row,
 * P elements, to out (device memory of any alignment if out_is_device, else
 * host memory); synchronises.  A host copy goes through a temporary device row
 * of P elements: GEM_ENOMEM if it cannot be allocated. */
int gem_read_state(gem_t* g, int32_t w, int32_t which, float* out, int32_t out_is_device);

/* Gather theta[idx[k]] into theta_out[k] and S[w][idx[k]], M[w][idx[k]] into
 * S_out[w * count + k], M_out[w * count + k] (all host; any output may be
 * NULL).  idx is a host array of count indices in [0, P); count at most
 * GEM_P_MAX (EINVAL above).  ENOMEM if the device staging cannot be allocated. */
int gem_gather(gem_t* g, const int64_t* idx, int64_t count, float* theta_out, float* S_out,
               float* M_out);

/* gem_gather for callers that cannot allocate memory (code under HIP graph
 * capture, serving loops, harnesses that forbid allocation): the same outputs,
 * bit for bit, staged through a fixed device scratch of GEM_SCRATCH_BYTES
 * that the library holds on each GPU it runs on until the process ends,
 * instead of buffers allocated per call.  The call allocates nothing, on the
 * device or the host.  The indices and the gathered values must fit the
 * scratch: count * (8 + 4 * (1 + 2 n)) <= GEM_SCRATCH_BYTES, else
 * GEM_ESCRATCH and nothing is done (count <= 5165 at n = 100).  Other errors
 * as gem_gather.  All handles on one GPU share its scratch: calls that
 * overlap on one GPU (handles used from several threads, or on streams that
 * run concurrently) race and must be serialised by the caller.  The scratch
 * keeps the last call's contents; nothing in it needs to start at zero.
 * Synchronises the handle's stream. */
#define GEM_SCRATCH_BYTES (4 << 20)
int gem_gather_static(gem_t* g, const int64_t* idx, int64_t count, float* theta_out,
                      float* S_out, float* M_out);

/* The handle's sizes: P parameters and n workers (what every host buffer of
 * P or n elements passed to or filled by the calls here must hold).
 * GEM_EINVAL for a NULL argument. */
int gem_dims(gem_t* g, int64_t* P, int32_t* n);

/* Current global clock t (commits applied since the last restart). */
int gem_clock(gem_t* g, int64_t* t);

/* Pull clocks of all n workers into out[n] (host). */
int gem_pull_clocks(gem_t* g, int64_t* out);

/* Restart worker w as a fresh Alg. 1 Worker: m_w = 0, S[w] = theta, pull
 * clock = t (a worker that failed and came back).  With the GLOBAL proxy the
 * shared moment belongs to the master and is kept; only the pull happens. */
int gem_reset_worker(gem_t* g, int32_t w);

/* Diagnostics (eq. 11 and eq. 22 energies, clamp count) off the timed path:
 * while enabled, commits run an instrumented kernel variant that accumulates
 * into the handle; gem_diag adds the current loss.  gem_diag_reset zeroes
 * the accumulators. */
int gem_diag_enable(gem_t* g, int32_t on);
int gem_diag_reset(gem_t* g);
int gem_diag(gem_t* g, gem_diag_t* out);

/*
 * Segments for pi_scope GEM_PI_SEGMENT: count >= 1 segments
 * [offsets[k], offsets[k+1]) of the parameter vector, offsets a host array of
 * count + 1 values with offsets[0] = 0 < offsets[1] < ... < offsets[count] = P
 * (for instance the tensors of a model; one segment [0, P) gives a global
 * norm, the default).  A commit by worker w then applies, for each segment T
 * (eqs. 11-13 and 18 with the absolute values replaced by norms over T):
 *
 *     m     = mu * M[w] + dtheta                        (every element)
 *     pi_T  = (kappa_eff ||m_T|| - ||theta_T - S[w]_T||) / (||dtheta_T|| + eps)
 *     theta = theta + pi_T * dtheta                     (every element of T)
 *
 * with pi_mode as for element-wise pi.  A sum of squares is taken in
 * binary64 in a fixed order (exact squares; aligned blocks of 2^18 indices
 * added by the adjacent-pairs tree, then the blocks in increasing order), the
 * norm is its binary64 square root rounded to binary32, and pi_T follows in
 * binary32; segments of one element give element-wise GEM bit for bit.
 * Each commit is one streaming launch plus one small reduction launch (a
 * commit's pi needs every element of its segment first), so commits are not
 * fused.  pi histograms record each segment's factor once per element (one
 * bin per segment holding its size); the diagnostics count the elements of
 * segments whose raw pi was negative or NaN as clamped.
 * The offsets are copied; the call may be made at any time between commits.
 * GEM_EINVAL for a malformed table.
 */
int gem_set_segments(gem_t* g, const int64_t* offsets, int32_t count);

/* Histogram, for each recorded commit, of the scale factor it applied to
 * each parameter: pi for GEM (Sec. 4 follows its per-parameter median over
 * time), 1 for DOWNPOUR, 1/(tau + 1) for adaptive staleness.  Bins (on the
 * binary32 value): 0: factor <= 0 or NaN (a clamped pi is 0); 1: below 2^-20;
 * 2 + 16 o + f: 2^(o-20) (1 + f/16) <= factor < 2^(o-20) (1 + (f+1)/16) for o
 * in [0, 40), f in [0, 16); GEM_PI_BINS - 1: 2^20 and above.
 * gem_pi_hist_start allocates room for `capacity` commits (capacity >= 1) and
 * records the commits that follow, up to capacity, through the instrumented
 * kernel variant (off the timed path).  gem_pi_hist_read copies the recorded
 * histograms -- commit-major, GEM_PI_BINS uint32 counts over the P parameters
 * each -- for at most max_commits commits into out (host), sets *commits to
 * the number recorded, and stops recording.  Errors: EINVAL (also a capacity
 * whose byte count does not fit 64 bits), ENOMEM, ESTATE (read without a
 * recording).
 * gem_pi_hist_start_segments records one histogram per segment of the
 * partition set by gem_set_segments (one segment if none): the per-tensor
 * median pi of the paper's supplementary figures.  Each recorded commit is
 * then nseg * GEM_PI_BINS counts, segment-major, and out must hold
 * max_commits * nseg * GEM_PI_BINS.  gem_set_segments returns GEM_EINVAL
 * while such a recording runs; gem_load ends it. */
#define GEM_PI_BINS 643
int gem_pi_hist_start(gem_t* g, int64_t capacity);
int gem_pi_hist_start_segments(gem_t* g, int64_t capacity);
int gem_pi_hist_read(gem_t* g, uint32_t* out, int64_t max_commits, int64_t* commits);

/* Work counters.  alg_bytes counts, per pass over P' (P padded to 64) elements:
 * theta read and written, h and theta* read (simulated runs), each distinct
 * worker's S and M rows read and written once (GLOBAL proxy: its S row, plus
 * the shared moment read and written once), and caller updates read -- 4
 * bytes per float, 2 per bfloat16.  Under GEM_PI_SEGMENT every commit is one
 * pass and counts 32 bytes per element (generated updates: theta read, the
 * committing and the pending worker's snapshot read, the pull written, M
 * read and written, h and theta* read) or 28 / 24 (given f32 / bf16 updates,
 * each read twice); with GEM_PULL_PRE_COMMIT theta is also written (4 more).
 * With post-commit pulls the pull of each commit is theta itself, so the
 * next launch reads theta from that snapshot row and only a run's last
 * launch writes the theta array. */
int gem_stats(gem_t* g, gem_stats_t* out);
int gem_stats_reset(gem_t* g);

/* Checkpoint: write / read theta, S, M, pull clocks, t, hyper-parameters,
 * the problem (if set) and the segment partition (if set) to a host file.
 * Load requires a handle of the same P and n, and checks the whole file
 * (size, partition, clocks: 0 <= each pull clock <= t < 2^32) before it
 * changes any state.  Resume is bit-exact: noise
 * is a function of (seed, t, i).  GEM_EIO for an unreadable, foreign or
 * truncated file; GEM_ENOMEM (before any file or state is touched) when the
 * device row of P' elements that stages S and M cannot be allocated.  The file
 * holds each row as P contiguous floats, whatever the device layout. */
int gem_save(gem_t* g, const char* path);
int gem_load(gem_t* g, const char* path);

/* Cache policy of the fused pass's memory accesses (theta, h, theta* and the
 * snapshot and moment rows).  GEM_CACHE_STREAM marks them non-temporal: every
 * chunk a pass touches is read once and written once, and over a state much
 * larger than the caches that makes passes 7-12% faster on MI355X.
 * GEM_CACHE_KEEP uses the default policy, under which a state that fits the
 * 256 MiB Infinity Cache stays there between passes (streaming it is 14-24%
 * slower).  GEM_CACHE_AUTO (the default) streams when theta, h, theta* and
 * the snapshot and moment table together exceed 256 MiB.  Results are the
 * same bits under every policy.  The diagnostic passes keep the default
 * policy; so do the per-segment scope's loads of h and theta*, which every
 * commit reads: with the other streams non-temporal the Infinity Cache keeps
 * them between commits.  GEM_EINVAL for another value. */
int gem_set_cache_policy(gem_t* g, int32_t policy);

/* Wait for all queued work of the handle. */
int gem_sync(gem_t* g);

/* Device-to-device float copy of count elements (16-byte aligned), the
 * bandwidth reference the benchmark scales counters with.  Queued on stream
 * (hipStream_t or NULL). */
int gem_copy_f32(const float* src, float* dst, int64_t count, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* LIBGEM_GEM_H */
