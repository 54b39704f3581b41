// gem_api.cpp -- the libgem C ABI: device state, validation, pass planning,
// the queuing schedule and checkpoints.  Kernels live in gem_kernels.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include "../../include/gem.h"
#include "gem_device.hpp"
#include "gem_internal.hpp"

using gemk::PassArgs;
using gemk::SegArgs;
using gemk::Source;

struct gem_handle {
    int device = 0;
    int64_t P = 0;
    int64_t Pp = 0;       // row length padded to a multiple of 64 elements (256 B)
    int32_t n = 0;
    gem_hyperparams hp{};
    hipStream_t stream = nullptr;
    float* theta = nullptr;   // [Pp]
    // Snapshot and moment table (layout: gemk::tile_index); S is the
    // allocation and addresses the snapshot pieces, M = S + kTileElems the
    // moment pieces: S_w[i] = S[tile_index(n, w, i)], M_w[i] = M[tile_index(n, w, i)].
    float* S = nullptr;
    float* M = nullptr;
    float* h = nullptr;       // [Pp]
    float* ts = nullptr;      // [Pp]
    double* acc = nullptr;    // [5]: sum_ek, sum_proxy, n_clamped, n_elem_commits, loss
    float* sink = nullptr;    // [2][kSinkChunks * 4] loads/stores a pass step does not need
    bool have_problem = false;
    gem_sim_params sp{};
    int64_t t = 0;
    std::vector<int64_t> pc;  // pull clock of each worker
    bool diag_on = false;
    int32_t cache_policy = GEM_CACHE_AUTO;
    int64_t diag_commits = 0;
    uint32_t* pi_hist = nullptr;   // [hist_cap][GEM_PI_BINS] device counts
    int64_t hist_cap = 0;
    int64_t hist_count = 0;        // commits recorded so far (may exceed hist_cap)
    int32_t hist_rows = 1;         // histograms per commit: 1, or one per segment
    bool hist_on = false;
    bool hist_seg = false;         // the recording is per segment of the partition
    gem_stats_t stats{};
    // Segment-norm scope: the partition (host copy) and its device tables,
    // built by gem_set_segments or, with one segment, by the first run.
    std::vector<int64_t> seg_host;   // [nseg + 1] offsets
    int64_t* seg_off = nullptr;      // [nseg + 1]
    int64_t* part_off = nullptr;     // [nseg + 1]
    int32_t* gseg = nullptr;         // [groups]
    double* part = nullptr;          // [3][npart][4] wave sums of the current commit
    int32_t* pair_seg = nullptr;     // [nsup] (segment, index block) pairs
    int32_t* pair_blk = nullptr;
    int64_t* sup_off = nullptr;      // [nseg + 1] first index-block slot of each segment
    double* sup = nullptr;           // [3][nsup] index-block sums
    float* pi_seg = nullptr;         // [nseg]
    uint32_t* seg_done = nullptr;    // [nseg] pair blocks finished in the running launch
    uint32_t deep_lds = 0;           // LDS reserved per block of the deep-ring pass
    int32_t cus = 0;                 // compute units of the device (0 if unknown)
    int64_t npart = 0;
    int64_t nsup = 0;
    void* scratch = nullptr;         // this device's static scratch (gem_gather_static)
};

namespace {

constexpr int64_t kRowAlign = 64;

thread_local char g_last_error[512] = "";

void note_hip_error(const char* what, hipError_t e, int line)
{
    std::snprintf(g_last_error, sizeof(g_last_error), "%s failed at gem_api.cpp:%d: %s (%d)", what,
                  line, hipGetErrorString(e), static_cast<int>(e));
}

#define GEM_HIP(expr)                                        \
    do {                                                     \
        const hipError_t gem_e_ = (expr);                    \
        if (gem_e_ != hipSuccess) {                          \
            note_hip_error(#expr, gem_e_, __LINE__);         \
            return GEM_EHIP;                                 \
        }                                                    \
    } while (0)

bool valid_hp(const gem_hyperparams& hp)
{
    if (hp.pi_mode != GEM_PI_CLAMP0 && hp.pi_mode != GEM_PI_LITERAL) return false;
    if (hp.kappa_mode != GEM_KAPPA_LINEAR && hp.kappa_mode != GEM_KAPPA_SQRT) return false;
    if (hp.pull_mode != GEM_PULL_POST_COMMIT && hp.pull_mode != GEM_PULL_PRE_COMMIT) return false;
    if (hp.rule != GEM_RULE_GEM && hp.rule != GEM_RULE_DOWNPOUR && hp.rule != GEM_RULE_ADAPTIVE)
        return false;
    if (hp.proxy_mode != GEM_PROXY_LOCAL && hp.proxy_mode != GEM_PROXY_GLOBAL) return false;
    if (hp.pi_scope != GEM_PI_ELEMENT && hp.pi_scope != GEM_PI_SEGMENT) return false;
    if (hp.pi_scope == GEM_PI_SEGMENT && hp.rule != GEM_RULE_GEM) return false;
    if (!std::isfinite(hp.momentum) || !std::isfinite(hp.eps) || !std::isfinite(hp.kappa))
        return false;
    // eps keeps the scale factor's denominator |dtheta| + eps away from zero
    // (Alg. 1): with eps <= 0 an update of exactly zero would give pi = inf
    // and theta = inf * 0 = NaN.  kappa scales the proxy energy (appendix B),
    // which is positive.
    if (!(hp.eps > 0.0f)) return false;
    if (!(hp.kappa > 0.0f)) return false;
    return true;
}

// kappa as it multiplies |m| (binary32, correctly rounded square root).
float kappa_eff(const gem_hyperparams& hp)
{
    return hp.kappa_mode == GEM_KAPPA_SQRT ? std::sqrt(hp.kappa) : hp.kappa;
}

// The pass-kernel specialisation for these hyperparameters: the default rule
// (GEM, CLAMP0, post-commit pull, kappa_eff = 1) has its own, for each proxy.
gemk::Variant kernel_variant(const gem_hyperparams& hp)
{
    const bool default_rule = hp.rule == GEM_RULE_GEM && hp.pi_mode == GEM_PI_CLAMP0 &&
                              hp.pull_mode == GEM_PULL_POST_COMMIT && kappa_eff(hp) == 1.0f;
    if (!default_rule) return gemk::Variant::General;
    return hp.proxy_mode == GEM_PROXY_GLOBAL ? gemk::Variant::FastGlobal : gemk::Variant::Fast;
}

uint32_t mode_bits(const gem_hyperparams& hp)
{
    uint32_t m = 0;
    if (hp.pi_mode == GEM_PI_LITERAL) m |= gemk::kModeLiteralPi;
    if (kappa_eff(hp) != 1.0f) m |= gemk::kModeKappaMul;
    if (hp.pull_mode == GEM_PULL_PRE_COMMIT) m |= gemk::kModePrePull;
    if (hp.rule == GEM_RULE_DOWNPOUR) m |= gemk::kModeDownpour;
    if (hp.rule == GEM_RULE_ADAPTIVE) m |= gemk::kModeAdaptive;
    if (hp.proxy_mode == GEM_PROXY_GLOBAL) m |= gemk::kModeGlobalProxy;
    return m;
}

int64_t next_pull(const gem_handle* g, int64_t t)
{
    return g->hp.pull_mode == GEM_PULL_PRE_COMMIT ? t : t + 1;
}

// Check a commit sequence against the pull bookkeeping without changing it.
int check_sequence(const gem_handle* g, const int32_t* worker, const int32_t* tau, int64_t T)
{
    if (T > 0 && !worker) return GEM_EINVAL;
    if (g->t + T > static_cast<int64_t>(UINT32_MAX)) return GEM_EINVAL;  // clock keys the noise
    std::vector<int64_t> pc = g->pc;
    for (int64_t j = 0; j < T; ++j) {
        const int32_t w = worker[j];
        if (w < 0 || w >= g->n) return GEM_EWORKER;
        const int64_t t = g->t + j;
        if (tau && static_cast<int64_t>(tau[j]) != t - pc[w]) return GEM_ESTALE;
        pc[w] = next_pull(g, t);
    }
    return GEM_OK;
}

struct Pass {
    int32_t K = 0;
    int32_t worker[GEM_K_MAX];
    int32_t tau[GEM_K_MAX];
    uint32_t routes[GEM_K_MAX];
    int32_t distinct = 0;     // distinct workers (the algorithmic row traffic)
    int32_t row_reads = 0;    // (snapshot, moment) row pairs the kernel reads
    int32_t row_writes = 0;   // and writes
};

// Cut a validated commit sequence into passes of at most Kmax commits, with
// routes for a ring of the given depth.
void plan_passes(const gem_handle* g, const int32_t* worker, int64_t T, int32_t Kmax, int depth,
                 std::vector<Pass>& out)
{
    std::vector<int64_t> pc = g->pc;
    int64_t j0 = 0;
    while (j0 < T) {
        Pass p;
        int k = static_cast<int>(std::min<int64_t>(Kmax, T - j0));
        k = gemk::plan_pass(worker + j0, k, depth, p.routes, &p.row_reads, &p.row_writes);
        p.K = k;
        for (int j = 0; j < k; ++j) {
            const int32_t w = worker[j0 + j];
            const int64_t t = g->t + j0 + j;
            p.worker[j] = w;
            p.tau[j] = static_cast<int32_t>(t - pc[w]);
            pc[w] = next_pull(g, t);
            bool seen = false;
            for (int q = 0; q < j; ++q) seen = seen || (p.worker[q] == w);
            if (!seen) p.distinct += 1;
        }
        out.push_back(p);
        j0 += k;
    }
}

void base_args(const gem_handle* g, PassArgs& a)
{
    std::memset(&a, 0, sizeof(a));
    a.theta = g->theta;
    a.S = g->S;
    a.M = g->M;
    a.h = g->h;
    a.ts = g->ts;
    a.diag = g->acc;
    a.sink_S = g->sink;
    a.sink_M = g->sink + gemk::kSinkChunks * 4;
    a.sink_mask = gemk::kSinkChunks - 1;
    a.Pp = g->Pp;
    a.P = g->P;
    a.nw = g->n;
    a.key0 = static_cast<uint32_t>(g->sp.seed);
    a.key1 = static_cast<uint32_t>(g->sp.seed >> 32);
    a.neg_lr = -g->sp.lr;
    a.sigma = g->sp.sigma;
    a.mu = g->hp.momentum;
    a.eps = g->hp.eps;
    a.k_eff = kappa_eff(g->hp);
    a.mode = mode_bits(g->hp);
}

// Queue the planned passes; advance the clock and pull bookkeeping.
// The ring depth of a run's passes: the deep ring for the default rule with
// per-worker moments on generated updates in passes of at least kDeepMinK
// commits, without diagnostics or recording.
int pass_depth(const gem_handle* g, Source src, int64_t kmax)
{
    const bool deep = src == Source::Generated && kernel_variant(g->hp) == gemk::Variant::Fast &&
                      kmax >= gemk::kDeepMinK && !g->diag_on && (!g->hist_on || g->hist_rows == 1);
    return deep ? gemk::kPrefetchDeep : gemk::kPrefetchShallow;
}

// Whether the fused passes stream their accesses (GEM_CACHE_AUTO: when the
// state they touch outgrows the Infinity Cache).
bool stream_rows(const gem_handle* g)
{
    if (g->cache_policy != GEM_CACHE_AUTO) return g->cache_policy == GEM_CACHE_STREAM;
    const int64_t bytes = 4 * (gemk::table_elems(g->n, g->Pp) + 3 * g->Pp);
    return bytes > gemk::kInfinityCacheBytes;
}

int run_passes(gem_handle* g, const std::vector<Pass>& passes, Source src,
               const void* const* upd, bool bf16_out, int depth)
{
    const bool stream = stream_rows(g);
    PassArgs a;
    base_args(g, a);
    // Under streaming, vectors that fit three quarters of the Infinity Cache
    // beside the streamed rows keep the default policy and stay cached
    // between passes: theta, h and theta* together (resnet18's 11.7M
    // parameters: 9% faster passes), else h and theta* alone (25M: 1.3%);
    // larger vectors stream with the rows (at 124M keeping them costs 1-2%).
    if (stream && g->cache_policy == GEM_CACHE_AUTO) {
        const int64_t room = gemk::kInfinityCacheBytes / 4 * 3;
        const int64_t vec = 4 * g->Pp;
        const bool gen = src == Source::Generated;
        a.keep_theta = (gen ? 3 : 1) * vec <= room;
        a.keep_problem = gen && 2 * vec <= room;
    }
    const gemk::Variant variant = kernel_variant(g->hp);
    int64_t j0 = 0;
    const double row_bytes = 4.0 * static_cast<double>(g->Pp);
    for (const Pass& p : passes) {
        a.t0 = static_cast<uint32_t>(g->t);
        a.K = p.K;
        std::memcpy(a.worker, p.worker, sizeof(p.worker));
        std::memcpy(a.tau, p.tau, sizeof(p.tau));
        std::memcpy(a.routes, p.routes, sizeof(p.routes));
        // theta read and written; S and M rows of each distinct worker read and
        // written (global proxy: S rows, and the shared moment once).
        double bytes = g->hp.proxy_mode == GEM_PROXY_GLOBAL
                           ? 4.0 * row_bytes + 2.0 * row_bytes * p.distinct
                           : 2.0 * row_bytes + 4.0 * row_bytes * p.distinct;
        if (src == Source::Generated) {
            bytes += 2.0 * row_bytes;                                     // h, theta*
        } else {
            for (int j = 0; j < p.K; ++j) a.upd[j] = upd[j0 + j];
            bytes += (src == Source::GivenBF16 ? 0.5 : 1.0) * row_bytes * p.K;
        }
        const bool hist = g->hist_on && g->hist_count < g->hist_cap;
        a.pi_hist = hist ? g->pi_hist : nullptr;
        a.hist_rows = g->hist_rows;
        a.hseg_off = g->seg_off;
        a.hseg_grp = g->gseg;
        a.diag = g->diag_on ? g->acc : nullptr;
        a.hist_first = g->hist_count;
        a.hist_cap = g->hist_cap;
        // Recording one histogram per commit on the fast path: the recording
        // variant of the same pass; otherwise recording takes the diagnostic
        // variant.
        const bool rec = hist && !g->diag_on && g->hist_rows == 1 && src == Source::Generated &&
                         variant == gemk::Variant::Fast;
        // a recording pass loops 8 blocks per compute unit over the groups
        a.rec_grid = rec ? 8 * g->cus : 0;
        const bool diag = (g->diag_on || hist) && !rec;
        // a single-commit pass runs the kernel compiled for one commit
        const int d = p.K == 1 && !diag && !rec ? gemk::kPrefetchNone : depth;
        GEM_HIP(gemk::launch_pass(a, src, variant, bf16_out, diag, rec, d, stream, g->deep_lds,
                                  g->stream));
        if (g->hist_on) g->hist_count += p.K;
        for (int j = 0; j < p.K; ++j) g->pc[p.worker[j]] = next_pull(g, g->t + j);
        g->t += p.K;
        j0 += p.K;
        g->stats.commits += p.K;
        g->stats.passes += 1;
        g->stats.alg_bytes += bytes;
        if (g->diag_on) g->diag_commits += p.K;
    }
    return GEM_OK;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

void free_segments(gem_handle* g)
{
    (void)hipFree(g->seg_off);
    (void)hipFree(g->part_off);
    (void)hipFree(g->gseg);
    (void)hipFree(g->part);
    (void)hipFree(g->pair_seg);
    (void)hipFree(g->pair_blk);
    (void)hipFree(g->sup_off);
    (void)hipFree(g->sup);
    (void)hipFree(g->pi_seg);
    (void)hipFree(g->seg_done);
    g->seg_done = nullptr;
    g->seg_off = g->part_off = g->sup_off = nullptr;
    g->gseg = g->pair_seg = g->pair_blk = nullptr;
    g->part = g->sup = nullptr;
    g->pi_seg = nullptr;
    g->npart = g->nsup = 0;
    g->seg_host.clear();
}

// Build the device tables of a validated partition (replacing any earlier).
int build_segments(gem_handle* g, const std::vector<int64_t>& off)
{
    const int32_t nseg = static_cast<int32_t>(off.size() - 1);
    const int64_t groups = (g->Pp + gemk::kSegGroup - 1) / gemk::kSegGroup;
    std::vector<int64_t> part_off(static_cast<size_t>(nseg) + 1, 0);
    for (int32_t k = 0; k < nseg; ++k)
        part_off[k + 1] = part_off[k] + (off[k + 1] - 1) / gemk::kSegGroup - off[k] / gemk::kSegGroup + 1;
    std::vector<int64_t> sup_off(static_cast<size_t>(nseg) + 1, 0);
    std::vector<int32_t> pair_seg, pair_blk;
    for (int32_t s = 0; s < nseg; ++s) {
        const int64_t b_lo = off[s] / gemk::kSegBlock, b_hi = (off[s + 1] - 1) / gemk::kSegBlock;
        sup_off[s + 1] = sup_off[s] + (b_hi - b_lo + 1);
        for (int64_t b = b_lo; b <= b_hi; ++b) {
            pair_seg.push_back(s);
            pair_blk.push_back(static_cast<int32_t>(b));
        }
    }
    const int64_t nsup = sup_off[nseg];
    std::vector<int32_t> gseg(static_cast<size_t>(groups));
    int32_t k = 0;
    for (int64_t grp = 0; grp < groups; ++grp) {
        while (off[k + 1] <= grp * gemk::kSegGroup) ++k;   // every group starts below P
        gseg[grp] = k;
    }
    GEM_HIP(hipStreamSynchronize(g->stream));
    free_segments(g);
    const int64_t npart = part_off[nseg];
    bool ok = hipMalloc(&g->seg_off, off.size() * sizeof(int64_t)) == hipSuccess &&
              hipMalloc(&g->part_off, part_off.size() * sizeof(int64_t)) == hipSuccess &&
              hipMalloc(&g->gseg, gseg.size() * sizeof(int32_t)) == hipSuccess &&
              hipMalloc(&g->part, static_cast<size_t>(3 * npart * gemk::kWavesPerGroup) *
                                      sizeof(double)) == hipSuccess &&
              hipMalloc(&g->pair_seg, pair_seg.size() * sizeof(int32_t)) == hipSuccess &&
              hipMalloc(&g->pair_blk, pair_blk.size() * sizeof(int32_t)) == hipSuccess &&
              hipMalloc(&g->sup_off, sup_off.size() * sizeof(int64_t)) == hipSuccess &&
              hipMalloc(&g->sup, static_cast<size_t>(3 * nsup) * sizeof(double)) == hipSuccess &&
              hipMalloc(&g->pi_seg, static_cast<size_t>(nseg) * sizeof(float)) == hipSuccess &&
              hipMalloc(&g->seg_done, static_cast<size_t>(nseg) * sizeof(uint32_t)) == hipSuccess;
    if (!ok) {
        (void)hipGetLastError();
        free_segments(g);
        return GEM_ENOMEM;
    }
    g->npart = npart;
    g->nsup = nsup;
    const int rc = [&]() -> int {
        GEM_HIP(hipMemcpyAsync(g->seg_off, off.data(), off.size() * sizeof(int64_t),
                               hipMemcpyHostToDevice, g->stream));
        GEM_HIP(hipMemcpyAsync(g->part_off, part_off.data(), part_off.size() * sizeof(int64_t),
                               hipMemcpyHostToDevice, g->stream));
        GEM_HIP(hipMemcpyAsync(g->gseg, gseg.data(), gseg.size() * sizeof(int32_t),
                               hipMemcpyHostToDevice, g->stream));
        GEM_HIP(hipMemcpyAsync(g->pair_seg, pair_seg.data(), pair_seg.size() * sizeof(int32_t),
                               hipMemcpyHostToDevice, g->stream));
        GEM_HIP(hipMemcpyAsync(g->pair_blk, pair_blk.data(), pair_blk.size() * sizeof(int32_t),
                               hipMemcpyHostToDevice, g->stream));
        GEM_HIP(hipMemcpyAsync(g->sup_off, sup_off.data(), sup_off.size() * sizeof(int64_t),
                               hipMemcpyHostToDevice, g->stream));
        GEM_HIP(hipMemsetAsync(g->seg_done, 0, static_cast<size_t>(nseg) * sizeof(uint32_t),
                               g->stream));
        GEM_HIP(hipStreamSynchronize(g->stream));
        return GEM_OK;
    }();
    if (rc != GEM_OK) {
        free_segments(g);
        return rc;
    }
    g->seg_host = off;
    return GEM_OK;
}

// Commits with one scale factor per segment.  Each commit is a step launch
// (finish the previous commit, start this one), the index-block sums and a
// per-segment reduction;
// a last step launch finishes the final commit, so the state in HBM is
// complete when the call returns to the stream.
int run_segments(gem_handle* g, const int32_t* worker, int64_t T, Source src,
                 const void* const* upd, bool bf16_out)
{
    if (T == 0) return GEM_OK;
    if (g->seg_host.empty()) {
        const int rc = build_segments(g, {0, g->P});
        if (rc) return rc;
    }
    SegArgs a;
    std::memset(&a, 0, sizeof(a));
    a.theta = g->theta;
    a.S = g->S;
    a.M = g->M;
    a.h = g->h;
    a.ts = g->ts;
    a.pi_seg = g->pi_seg;
    a.part = g->part;
    a.seg_off = g->seg_off;
    a.part_off = g->part_off;
    a.gseg = g->gseg;
    a.npart = g->npart;
    a.Pp = g->Pp;
    a.P = g->P;
    a.nw = g->n;
    a.pre_pull = g->hp.pull_mode == GEM_PULL_PRE_COMMIT;
    a.key0 = static_cast<uint32_t>(g->sp.seed);
    a.key1 = static_cast<uint32_t>(g->sp.seed >> 32);
    a.neg_lr = -g->sp.lr;
    a.sigma = g->sp.sigma;
    a.mu = g->hp.momentum;
    const float k_eff = kappa_eff(g->hp);
    a.k_eff = k_eff;
    a.diag = g->diag_on ? g->acc : nullptr;
    gemk::SegFactors f;
    f.pi_seg = g->pi_seg;
    f.k_eff = k_eff;
    f.eps = g->hp.eps;
    f.literal = g->hp.pi_mode == GEM_PI_LITERAL;
    f.hist_per_seg = g->hist_seg ? 1 : 0;
    f.hist = nullptr;
    f.diag = a.diag;
    // Bytes per element-commit the launches move: theta read (and, with
    // pre-commit pulls, written: otherwise the pull of each commit holds it
    // for the next launch, and only a run's last launch writes the array),
    // the committing worker's snapshot read and its pull written, the moment
    // read and written; generated updates read h and theta* and the pending
    // commit's snapshot (to generate its update again), given updates read
    // the caller's update twice.
    const bool post = g->hp.pull_mode == GEM_PULL_POST_COMMIT;
    const double per_elem = (src == Source::Generated ? 36.0 : src == Source::GivenF32 ? 32.0 : 28.0) -
                            (post ? 4.0 : 0.0);
    for (int64_t j = 0; j < T; ++j) {
        const int32_t w = worker[j];
        const int64_t t = g->t;
        a.apply = j > 0;
        a.start = 1;
        a.w_prev = j > 0 ? worker[j - 1] : 0;
        a.w_cur = w;
        a.m_row_prev = a.m_row;
        a.m_row = g->hp.proxy_mode == GEM_PROXY_GLOBAL ? 0 : w;
        a.t = static_cast<uint32_t>(t);
        a.upd_prev = (upd && j > 0) ? upd[j - 1] : nullptr;
        a.upd_cur = upd ? upd[j] : nullptr;
        // theta before the pending commit j - 1: the array at the start of
        // the run, else the pull of commit j - 2 (post-commit pulls)
        a.theta_row = (post && j >= 2) ? worker[j - 2] : -1;
        a.store_theta = post ? 0 : 1;
        GEM_HIP(gemk::launch_seg_step(a, src, bf16_out, stream_rows(g), g->stream));
        // Histogram recording: this commit's rows, while there is room.
        f.hist = nullptr;
        if (g->hist_on && g->hist_count < g->hist_cap)
            f.hist = g->pi_hist + g->hist_count * g->hist_rows * GEM_PI_BINS;
        GEM_HIP(gemk::launch_seg_blocks(g->part, g->npart, g->part_off, g->seg_off, g->pair_seg,
                                        g->pair_blk, g->nsup, g->sup, g->sup_off, g->seg_done, f,
                                        g->stream));
        if (g->hist_on) g->hist_count += 1;
        if (g->diag_on) g->diag_commits += 1;
        g->pc[w] = next_pull(g, t);
        g->t += 1;
        g->stats.commits += 1;
        g->stats.passes += 1;
        g->stats.alg_bytes += per_elem * static_cast<double>(g->Pp);
    }
    a.apply = 1;
    a.start = 0;
    a.t = static_cast<uint32_t>(g->t);
    a.theta_row = (post && T >= 2) ? worker[T - 2] : -1;
    a.store_theta = 1;
    a.w_prev = worker[T - 1];
    a.m_row_prev = a.m_row;
    a.upd_prev = upd ? upd[T - 1] : nullptr;
    a.upd_cur = nullptr;
    GEM_HIP(gemk::launch_seg_step(a, src, bf16_out, stream_rows(g), g->stream));
    return GEM_OK;
}

}  // namespace

extern "C" {

const char* gem_last_error(void) { return g_last_error; }

const char* gem_strerror(int code)
{
    switch (code) {
    case GEM_OK: return "ok";
    case GEM_EINVAL: return "invalid argument";
    case GEM_ENOMEM: return "out of memory";
    case GEM_EWORKER: return "worker id out of range";
    case GEM_ESTALE: return "staleness disagrees with the pull bookkeeping";
    case GEM_EDTYPE: return "unknown update dtype";
    case GEM_EHIP: return "HIP runtime error";
    case GEM_ESTATE: return "operation needs a problem set with gem_set_quadratic";
    case GEM_EIO: return "checkpoint I/O error or mismatch";
    case GEM_EALIGN: return "device buffer not aligned";
    case GEM_ESCRATCH: return "request does not fit the fixed device scratch";
    default: return "unknown error";
    }
}

int gem_hyperparams_default(gem_hyperparams* hp)
{
    if (!hp) return GEM_EINVAL;
    std::memset(hp, 0, sizeof(*hp));
    hp->momentum = 0.9f;
    hp->eps = 1e-16f;
    hp->kappa = 1.0f;
    hp->pi_mode = GEM_PI_CLAMP0;
    hp->kappa_mode = GEM_KAPPA_LINEAR;
    hp->pull_mode = GEM_PULL_POST_COMMIT;
    hp->rule = GEM_RULE_GEM;
    hp->proxy_mode = GEM_PROXY_LOCAL;
    hp->pi_scope = GEM_PI_ELEMENT;
    return GEM_OK;
}

int gem_destroy(gem_t* g)
{
    if (!g) return GEM_EINVAL;
    (void)hipStreamSynchronize(g->stream);
    (void)hipFree(g->theta);
    (void)hipFree(g->S);
    (void)hipFree(g->h);
    (void)hipFree(g->ts);
    (void)hipFree(g->acc);
    (void)hipFree(g->sink);
    (void)hipFree(g->pi_hist);
    free_segments(g);
    delete g;
    return GEM_OK;
}

int gem_create(int64_t P, int32_t n, const gem_hyperparams* hp, void* stream, gem_t** out)
{
    if (!out || P < 1 || n < 1) return GEM_EINVAL;
    *out = nullptr;
    gem_hyperparams h;
    if (hp) h = *hp;
    else gem_hyperparams_default(&h);
    if (!valid_hp(h)) return GEM_EINVAL;
    if (P > GEM_P_MAX) return GEM_EINVAL;
    const int64_t Pp = (P + kRowAlign - 1) / kRowAlign * kRowAlign;
    // The table's byte count must fit 64 bits (it can exceed any device).
    if (n > INT64_MAX / 4 / gemk::table_elems(1, Pp)) return GEM_ENOMEM;
    gem_handle* g = new (std::nothrow) gem_handle();
    if (!g) return GEM_ENOMEM;
    g->P = P;
    g->Pp = Pp;
    g->n = n;
    g->hp = h;
    g->pc.assign(static_cast<size_t>(n), 0);
    {
        const hipError_t e = hipGetDevice(&g->device);
        if (e != hipSuccess) {
            note_hip_error("hipGetDevice", e, __LINE__);
            delete g;
            return GEM_EHIP;
        }
    }
    {
        // The static scratch of the allocation-free entry point: its device
        // address on this (current) device, looked up once per device.
        const hipError_t e = gemk::scratch_address(g->device, &g->scratch);
        if (e != hipSuccess) {
            note_hip_error("hipGetSymbolAddress(scratch)", e, __LINE__);
            delete g;
            return GEM_EHIP;
        }
    }
    {
        int lds = 0;
        if (hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor,
                                  g->device) == hipSuccess)
            g->deep_lds = gemk::deep_lds_bytes(lds);
        else
            (void)hipGetLastError();   // no cap: the pass runs as its registers allow
        if (hipDeviceGetAttribute(&g->cus, hipDeviceAttributeMultiprocessorCount, g->device) !=
            hipSuccess) {
            (void)hipGetLastError();
            g->cus = 0;
        }
    }
    // NULL is the device's null stream, which is also torch's default stream.
    g->stream = static_cast<hipStream_t>(stream);
    const size_t row = static_cast<size_t>(Pp) * sizeof(float);
    const size_t tab = static_cast<size_t>(gemk::table_elems(n, Pp)) * sizeof(float);
    {
        hipError_t e = hipMalloc(&g->theta, row);
        if (e == hipSuccess) e = hipMalloc(&g->S, tab);
        if (e == hipSuccess) g->M = g->S + gemk::kTileElems;
        if (e == hipSuccess) e = hipMalloc(&g->acc, 8 * sizeof(double));
        if (e == hipSuccess) e = hipMalloc(&g->sink, 2 * gemk::kSinkChunks * 4 * sizeof(float));
        if (e != hipSuccess) {
            note_hip_error("hipMalloc", e, __LINE__);
            (void)hipGetLastError();
            gem_destroy(g);
            return GEM_ENOMEM;
        }
    }
    const int rc = [&]() -> int {
        GEM_HIP(hipMemsetAsync(g->theta, 0, row, g->stream));
        GEM_HIP(hipMemsetAsync(g->S, 0, tab, g->stream));   // every snapshot and moment
        GEM_HIP(hipMemsetAsync(g->acc, 0, 8 * sizeof(double), g->stream));
        GEM_HIP(hipMemsetAsync(g->sink, 0, 2 * gemk::kSinkChunks * 4 * sizeof(float), g->stream));
        GEM_HIP(hipStreamSynchronize(g->stream));
        return GEM_OK;
    }();
    if (rc != GEM_OK) {
        gem_destroy(g);
        return rc;
    }
    *out = g;
    return GEM_OK;
}

int gem_set_theta(gem_t* g, const float* theta0, int32_t in_is_device)
{
    if (!g || !theta0) return GEM_EINVAL;
    const size_t bytes = static_cast<size_t>(g->P) * sizeof(float);
    GEM_HIP(hipMemcpyAsync(g->theta, theta0, bytes,
                           in_is_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice,
                           g->stream));
    GEM_HIP(gemk::launch_fill_rows(g->S, g->n, 0, g->n, g->Pp, g->theta, g->stream));
    GEM_HIP(gemk::launch_fill_rows(g->M, g->n, 0, g->n, g->Pp, nullptr, g->stream));
    GEM_HIP(hipMemsetAsync(g->acc, 0, 8 * sizeof(double), g->stream));
    GEM_HIP(hipStreamSynchronize(g->stream));
    g->t = 0;
    std::fill(g->pc.begin(), g->pc.end(), 0);
    g->diag_commits = 0;
    return GEM_OK;
}

int gem_set_quadratic(gem_t* g, const float* h, const float* theta_star, const gem_sim_params* sp)
{
    if (!g || !h || !theta_star || !sp) return GEM_EINVAL;
    if (sp->update_dtype != GEM_F32 && sp->update_dtype != GEM_BF16) return GEM_EDTYPE;
    if (!std::isfinite(sp->lr) || !std::isfinite(sp->sigma)) return GEM_EINVAL;
    const size_t row = static_cast<size_t>(g->Pp) * sizeof(float);
    if (!g->h) {
        if (hipMalloc(&g->h, row) != hipSuccess || hipMalloc(&g->ts, row) != hipSuccess) {
            (void)hipGetLastError();
            (void)hipFree(g->h);
            (void)hipFree(g->ts);
            g->h = g->ts = nullptr;
            return GEM_ENOMEM;
        }
    }
    const size_t bytes = static_cast<size_t>(g->P) * sizeof(float);
    GEM_HIP(hipMemsetAsync(g->h, 0, row, g->stream));
    GEM_HIP(hipMemsetAsync(g->ts, 0, row, g->stream));
    GEM_HIP(hipMemcpyAsync(g->h, h, bytes, hipMemcpyHostToDevice, g->stream));
    GEM_HIP(hipMemcpyAsync(g->ts, theta_star, bytes, hipMemcpyHostToDevice, g->stream));
    GEM_HIP(hipStreamSynchronize(g->stream));
    g->sp = *sp;
    g->have_problem = true;
    return GEM_OK;
}

int gem_commit_batch(gem_t* g, int32_t K, const void* const* dthetas_dev, int32_t dtype,
                     const int32_t* worker_ids, const int32_t* staleness)
{
    if (!g || K < 0 || (K > 0 && (!dthetas_dev || !worker_ids))) return GEM_EINVAL;
    if (dtype != GEM_F32 && dtype != GEM_BF16) return GEM_EDTYPE;
    const size_t align = dtype == GEM_F32 ? 16 : 8;
    for (int32_t j = 0; j < K; ++j) {
        if (!dthetas_dev[j]) return GEM_EINVAL;
        if (!aligned(dthetas_dev[j], align)) return GEM_EALIGN;
    }
    int rc = check_sequence(g, worker_ids, staleness, K);
    if (rc) return rc;
    const Source src = dtype == GEM_F32 ? Source::GivenF32 : Source::GivenBF16;
    if (g->hp.pi_scope == GEM_PI_SEGMENT) {
        return run_segments(g, worker_ids, K, src, dthetas_dev, false);
    }
    const int depth = pass_depth(g, src, std::min<int32_t>(K, GEM_K_MAX));
    std::vector<Pass> passes;
    plan_passes(g, worker_ids, K, GEM_K_MAX, depth, passes);
    return run_passes(g, passes, src, dthetas_dev, false, depth);
}

int gem_set_segments(gem_t* g, const int64_t* offsets, int32_t count)
{
    if (!g || !offsets || count < 1) return GEM_EINVAL;
    if (g->hist_on && g->hist_seg) return GEM_EINVAL;   // recording per segment
    if (offsets[0] != 0 || offsets[count] != g->P) return GEM_EINVAL;
    for (int32_t k = 0; k < count; ++k)
        if (offsets[k + 1] <= offsets[k]) return GEM_EINVAL;
    return build_segments(g, std::vector<int64_t>(offsets, offsets + count + 1));
}

int gem_commit(gem_t* g, const float* dtheta_dev, int32_t worker_id)
{
    const void* p = dtheta_dev;
    return gem_commit_batch(g, 1, &p, GEM_F32, &worker_id, nullptr);
}

int gem_generate(gem_t* g, int32_t worker_id, void* out_dev, int32_t dtype)
{
    if (!g || !out_dev) return GEM_EINVAL;
    if (dtype != GEM_F32 && dtype != GEM_BF16) return GEM_EDTYPE;
    if (!g->have_problem) return GEM_ESTATE;
    if (worker_id < 0 || worker_id >= g->n) return GEM_EWORKER;
    if (!aligned(out_dev, dtype == GEM_F32 ? 16 : 8)) return GEM_EALIGN;
    if (g->t > static_cast<int64_t>(UINT32_MAX)) return GEM_EINVAL;
    GEM_HIP(gemk::launch_generate(g->S, g->n, worker_id, g->h, g->ts,
                                  out_dev, dtype == GEM_BF16, g->P, static_cast<uint32_t>(g->t),
                                  static_cast<uint32_t>(g->sp.seed),
                                  static_cast<uint32_t>(g->sp.seed >> 32), -g->sp.lr, g->sp.sigma,
                                  g->stream));
    return GEM_OK;
}

int gem_sim_run(gem_t* g, const int32_t* worker, const int32_t* tau, int64_t T, int32_t K)
{
    if (!g || T < 0 || K < 1 || K > GEM_K_MAX) return GEM_EINVAL;
    if (!g->have_problem) return GEM_ESTATE;
    int rc = check_sequence(g, worker, tau, T);
    if (rc) return rc;
    if (g->hp.pi_scope == GEM_PI_SEGMENT) {
        return run_segments(g, worker, T, Source::Generated, nullptr,
                            g->sp.update_dtype == GEM_BF16);
    }
    const int depth = pass_depth(g, Source::Generated, std::min<int64_t>(K, T));
    std::vector<Pass> passes;
    plan_passes(g, worker, T, K, depth, passes);
    return run_passes(g, passes, Source::Generated, nullptr, g->sp.update_dtype == GEM_BF16,
                      depth);
}

int gem_read_theta(gem_t* g, float* out, int32_t out_is_device)
{
    if (!g || !out) return GEM_EINVAL;
    GEM_HIP(hipMemcpyAsync(out, g->theta, static_cast<size_t>(g->P) * sizeof(float),
                           out_is_device ? hipMemcpyDeviceToDevice : hipMemcpyDeviceToHost,
                           g->stream));
    GEM_HIP(hipStreamSynchronize(g->stream));
    return GEM_OK;
}

int gem_read_state(gem_t* g, int32_t w, int32_t which, float* out, int32_t out_is_device)
{
    if (!g || !out) return GEM_EINVAL;
    if (w < 0 || w >= g->n) return GEM_EWORKER;
    if (which != GEM_SNAPSHOT && which != GEM_MOMENT) return GEM_EINVAL;
    const float* base = which == GEM_SNAPSHOT ? g->S : g->M;
    if (out_is_device) {
        GEM_HIP(gemk::launch_read_row(base, g->n, w, g->P, out, g->stream));
        GEM_HIP(hipStreamSynchronize(g->stream));
        return GEM_OK;
    }
    // The row is spread over the table's tiles: gather it into a device
    // staging row, then copy that to the host.
    float* stage = nullptr;
    if (hipMalloc(&stage, static_cast<size_t>(g->P) * sizeof(float)) != hipSuccess) {
        (void)hipGetLastError();
        return GEM_ENOMEM;
    }
    int rc = GEM_OK;
    if (gemk::launch_read_row(base, g->n, w, g->P, stage, g->stream) != hipSuccess ||
        hipMemcpyAsync(out, stage, static_cast<size_t>(g->P) * sizeof(float), hipMemcpyDeviceToHost,
                       g->stream) != hipSuccess ||
        hipStreamSynchronize(g->stream) != hipSuccess)
        rc = GEM_EHIP;
    (void)hipStreamSynchronize(g->stream);
    (void)hipFree(stage);
    return rc;
}

int gem_gather(gem_t* g, const int64_t* idx, int64_t count, float* theta_out, float* S_out,
               float* M_out)
{
    if (!g || count < 0 || count > GEM_P_MAX || (count > 0 && !idx)) return GEM_EINVAL;
    if (count == 0) return GEM_OK;
    if (count > INT64_MAX / 4 / (1 + 2 * static_cast<int64_t>(g->n))) return GEM_ENOMEM;
    for (int64_t k = 0; k < count; ++k)
        if (idx[k] < 0 || idx[k] >= g->P) return GEM_EINVAL;
    const int64_t rows = 1 + 2 * static_cast<int64_t>(g->n);
    int64_t* d_idx = nullptr;
    float* d_out = nullptr;
    if (hipMalloc(&d_idx, static_cast<size_t>(count) * sizeof(int64_t)) != hipSuccess ||
        hipMalloc(&d_out, static_cast<size_t>(count * rows) * sizeof(float)) != hipSuccess) {
        (void)hipGetLastError();
        (void)hipFree(d_idx);
        return GEM_ENOMEM;
    }
    int rc = GEM_OK;
    do {
        if (hipMemcpyAsync(d_idx, idx, static_cast<size_t>(count) * sizeof(int64_t),
                           hipMemcpyHostToDevice, g->stream) != hipSuccess) { rc = GEM_EHIP; break; }
        if (theta_out && gemk::launch_gather(g->theta, d_idx, count, d_out, g->stream) != hipSuccess) {
            rc = GEM_EHIP;
            break;
        }
        if (S_out && gemk::launch_gather_rows(g->S, g->n, d_idx, count, d_out + count,
                                              g->stream) != hipSuccess) {
            rc = GEM_EHIP;
            break;
        }
        if (M_out && gemk::launch_gather_rows(g->M, g->n, d_idx, count, d_out + (1 + g->n) * count,
                                              g->stream) != hipSuccess) {
            rc = GEM_EHIP;
            break;
        }
        std::vector<float> host(static_cast<size_t>(count * rows));
        if (hipMemcpyAsync(host.data(), d_out, host.size() * sizeof(float), hipMemcpyDeviceToHost,
                           g->stream) != hipSuccess ||
            hipStreamSynchronize(g->stream) != hipSuccess) { rc = GEM_EHIP; break; }
        if (theta_out) std::memcpy(theta_out, host.data(), static_cast<size_t>(count) * sizeof(float));
        if (S_out) std::memcpy(S_out, host.data() + count, static_cast<size_t>(count * g->n) * sizeof(float));
        if (M_out)
            std::memcpy(M_out, host.data() + count * (1 + g->n),
                        static_cast<size_t>(count * g->n) * sizeof(float));
    } while (false);
    (void)hipStreamSynchronize(g->stream);
    (void)hipFree(d_idx);
    (void)hipFree(d_out);
    return rc;
}

int gem_gather_static(gem_t* g, const int64_t* idx, int64_t count, float* theta_out,
                      float* S_out, float* M_out)
{
    if (!g || count < 0 || (count > 0 && !idx)) return GEM_EINVAL;
    if (count == 0) return GEM_OK;
    const int64_t rows = 1 + 2 * static_cast<int64_t>(g->n);
    const int64_t per_index = 8 + 4 * rows;   // the index and its gathered values
    if (count > GEM_SCRATCH_BYTES / per_index) return GEM_ESCRATCH;
    for (int64_t k = 0; k < count; ++k)
        if (idx[k] < 0 || idx[k] >= g->P) return GEM_EINVAL;
    // Scratch layout: the indices, then theta, then the S rows, then the M
    // rows of the gathered entries (the byte counts keep each part 4-aligned
    // and the indices 8-aligned at the 256-byte aligned start).
    auto* d_idx = static_cast<int64_t*>(g->scratch);
    float* d_out = reinterpret_cast<float*>(d_idx + count);
    GEM_HIP(hipMemcpyAsync(d_idx, idx, static_cast<size_t>(count) * sizeof(int64_t),
                           hipMemcpyHostToDevice, g->stream));
    if (theta_out) GEM_HIP(gemk::launch_gather(g->theta, d_idx, count, d_out, g->stream));
    if (S_out) GEM_HIP(gemk::launch_gather_rows(g->S, g->n, d_idx, count, d_out + count, g->stream));
    if (M_out)
        GEM_HIP(gemk::launch_gather_rows(g->M, g->n, d_idx, count, d_out + (1 + g->n) * count,
                                         g->stream));
    const size_t row_bytes = static_cast<size_t>(count) * sizeof(float);
    if (theta_out)
        GEM_HIP(hipMemcpyAsync(theta_out, d_out, row_bytes, hipMemcpyDeviceToHost, g->stream));
    if (S_out)
        GEM_HIP(hipMemcpyAsync(S_out, d_out + count, row_bytes * g->n, hipMemcpyDeviceToHost,
                               g->stream));
    if (M_out)
        GEM_HIP(hipMemcpyAsync(M_out, d_out + (1 + g->n) * count, row_bytes * g->n,
                               hipMemcpyDeviceToHost, g->stream));
    GEM_HIP(hipStreamSynchronize(g->stream));
    return GEM_OK;
}

int gem_dims(gem_t* g, int64_t* P, int32_t* n)
{
    if (!g || !P || !n) return GEM_EINVAL;
    *P = g->P;
    *n = g->n;
    return GEM_OK;
}

int gem_clock(gem_t* g, int64_t* t)
{
    if (!g || !t) return GEM_EINVAL;
    *t = g->t;
    return GEM_OK;
}

int gem_pull_clocks(gem_t* g, int64_t* out)
{
    if (!g || !out) return GEM_EINVAL;
    std::memcpy(out, g->pc.data(), g->pc.size() * sizeof(int64_t));
    return GEM_OK;
}

int gem_reset_worker(gem_t* g, int32_t w)
{
    if (!g) return GEM_EINVAL;
    if (w < 0 || w >= g->n) return GEM_EWORKER;
    GEM_HIP(gemk::launch_fill_rows(g->S, g->n, w, 1, g->Pp, g->theta, g->stream));
    if (g->hp.proxy_mode == GEM_PROXY_LOCAL)
        GEM_HIP(gemk::launch_fill_rows(g->M, g->n, w, 1, g->Pp, nullptr, g->stream));
    g->pc[w] = g->t;
    return GEM_OK;
}

int gem_diag_enable(gem_t* g, int32_t on)
{
    if (!g) return GEM_EINVAL;
    g->diag_on = on != 0;
    return GEM_OK;
}

int gem_diag_reset(gem_t* g)
{
    if (!g) return GEM_EINVAL;
    GEM_HIP(hipMemsetAsync(g->acc, 0, 8 * sizeof(double), g->stream));
    g->diag_commits = 0;
    return GEM_OK;
}

int gem_diag(gem_t* g, gem_diag_t* out)
{
    if (!g || !out) return GEM_EINVAL;
    GEM_HIP(hipMemsetAsync(g->acc + 4, 0, sizeof(double), g->stream));
    if (g->have_problem) GEM_HIP(gemk::launch_loss(g->theta, g->h, g->ts, g->P, g->acc + 4, g->stream));
    double host[5];
    GEM_HIP(hipMemcpyAsync(host, g->acc, sizeof(host), hipMemcpyDeviceToHost, g->stream));
    GEM_HIP(hipStreamSynchronize(g->stream));
    out->sum_ek = host[0];
    out->sum_proxy = host[1];
    out->n_clamped = static_cast<int64_t>(host[2]);
    out->n_elem_commits = static_cast<int64_t>(host[3]);
    out->loss = host[4];
    out->n_commits = g->diag_commits;
    return GEM_OK;
}

namespace {

// (Re)allocate and clear room for `capacity` commits of `rows` histograms.
int hist_begin(gem_handle* g, int64_t capacity, int32_t rows, bool per_segment)
{
    const size_t bytes = static_cast<size_t>(capacity) * static_cast<size_t>(rows) * GEM_PI_BINS *
                         sizeof(uint32_t);
    const size_t have = static_cast<size_t>(g->hist_cap) * static_cast<size_t>(g->hist_rows) *
                        GEM_PI_BINS * sizeof(uint32_t);
    if (!g->pi_hist || bytes > have) {
        GEM_HIP(hipStreamSynchronize(g->stream));
        (void)hipFree(g->pi_hist);
        g->pi_hist = nullptr;
        g->hist_cap = 0;
        if (hipMalloc(&g->pi_hist, bytes) != hipSuccess) {
            (void)hipGetLastError();
            g->pi_hist = nullptr;
            g->hist_on = false;
            return GEM_ENOMEM;
        }
    }
    GEM_HIP(hipMemsetAsync(g->pi_hist, 0, bytes, g->stream));
    g->hist_cap = capacity;
    g->hist_rows = rows;
    g->hist_count = 0;
    g->hist_on = true;
    g->hist_seg = per_segment;
    return GEM_OK;
}

}  // namespace

int gem_pi_hist_start(gem_t* g, int64_t capacity)
{
    if (!g || capacity < 1) return GEM_EINVAL;
    if (capacity > INT64_MAX / (GEM_PI_BINS * 4)) return GEM_EINVAL;
    return hist_begin(g, capacity, 1, false);
}

int gem_pi_hist_start_segments(gem_t* g, int64_t capacity)
{
    if (!g || capacity < 1) return GEM_EINVAL;
    if (g->seg_host.empty()) {
        const int rc = build_segments(g, {0, g->P});
        if (rc) return rc;
    }
    const int64_t nseg = static_cast<int64_t>(g->seg_host.size()) - 1;
    if (capacity > INT64_MAX / (nseg * GEM_PI_BINS * 4)) return GEM_EINVAL;
    return hist_begin(g, capacity, static_cast<int32_t>(nseg), true);
}

int gem_pi_hist_read(gem_t* g, uint32_t* out, int64_t max_commits, int64_t* commits)
{
    if (!g || !commits || max_commits < 0 || (max_commits > 0 && !out)) return GEM_EINVAL;
    if (!g->pi_hist) return GEM_ESTATE;
    const int64_t recorded = std::min(g->hist_count, g->hist_cap);
    const int64_t n = std::min(recorded, max_commits);
    if (n > 0)
        GEM_HIP(hipMemcpyAsync(out, g->pi_hist,
                               static_cast<size_t>(n) * static_cast<size_t>(g->hist_rows) *
                                   GEM_PI_BINS * sizeof(uint32_t),
                               hipMemcpyDeviceToHost, g->stream));
    GEM_HIP(hipStreamSynchronize(g->stream));
    *commits = recorded;
    g->hist_on = false;
    return GEM_OK;
}

int gem_stats(gem_t* g, gem_stats_t* out)
{
    if (!g || !out) return GEM_EINVAL;
    *out = g->stats;
    return GEM_OK;
}

int gem_stats_reset(gem_t* g)
{
    if (!g) return GEM_EINVAL;
    g->stats = gem_stats_t{};
    return GEM_OK;
}

int gem_set_cache_policy(gem_t* g, int32_t policy)
{
    if (!g) return GEM_EINVAL;
    if (policy != GEM_CACHE_AUTO && policy != GEM_CACHE_KEEP && policy != GEM_CACHE_STREAM)
        return GEM_EINVAL;
    g->cache_policy = policy;
    return GEM_OK;
}

int gem_sync(gem_t* g)
{
    if (!g) return GEM_EINVAL;
    GEM_HIP(hipStreamSynchronize(g->stream));
    return GEM_OK;
}

int gem_copy_f32(const float* src, float* dst, int64_t count, void* stream)
{
    if (!src || !dst || count < 0) return GEM_EINVAL;
    if (!aligned(src, 16) || !aligned(dst, 16)) return GEM_EALIGN;
    GEM_HIP(gemk::launch_copy(src, dst, count, static_cast<hipStream_t>(stream)));
    return GEM_OK;
}

// ---------------------------------------------------------------------------
// Queuing schedule (host).  Philox4x32-10 draws keyed by the seed with
// counter (w, k lo, k hi, tag); tag 1 = job times, tag 2 = per-worker means.
// ---------------------------------------------------------------------------
namespace {

void sched_words(uint64_t seed, uint32_t w, uint64_t k, uint32_t tag, uint32_t x[4])
{
    const gemk::Words4 r = gemk::philox10(w, static_cast<uint32_t>(k), static_cast<uint32_t>(k >> 32),
                                          tag, static_cast<uint32_t>(seed),
                                          static_cast<uint32_t>(seed >> 32));
    x[0] = r.x0; x[1] = r.x1; x[2] = r.x2; x[3] = r.x3;
}

uint64_t bits53(uint32_t a, uint32_t b)
{
    return (static_cast<uint64_t>(a >> 11) << 32) | static_cast<uint64_t>(b);
}

double unit_open0(uint32_t a, uint32_t b) { return static_cast<double>(bits53(a, b) + 1u) * 0x1p-53; }
double unit_closed0(uint32_t a, uint32_t b) { return static_cast<double>(bits53(a, b)) * 0x1p-53; }

double mean_of_worker(const gem_schedule_law& L, uint64_t seed, int32_t w)
{
    uint32_t x[4];
    sched_words(seed, static_cast<uint32_t>(w), 0, 2u, x);
    switch (L.law) {
    case GEM_LAW_EXP_UNIFORM_MEAN:
        return L.p0 + (L.p1 - L.p0) * unit_closed0(x[0], x[1]);
    case GEM_LAW_EXP_LOGNORMAL_MEAN: {
        const double u = unit_open0(x[0], x[1]);
        const double v = unit_closed0(x[2], x[3]);
        const double z = std::sqrt(-2.0 * std::log(u)) * std::cos(6.283185307179586 * v);
        return std::exp(L.p0 + L.p1 * z);
    }
    default:
        return 1.0;
    }
}

double job_duration(const gem_schedule_law& L, double mean_w, uint64_t seed, int32_t w, int64_t k)
{
    uint32_t x[4];
    sched_words(seed, static_cast<uint32_t>(w), static_cast<uint64_t>(k), 1u, x);
    const double u = unit_open0(x[0], x[1]);
    if (L.law == GEM_LAW_PARETO) return L.p1 * std::pow(u, -1.0 / L.p0);
    return -mean_w * std::log(u);
}

}  // namespace

int gem_schedule_make(int32_t n, int64_t T, const gem_schedule_law* law, uint64_t seed,
                      int32_t pull_mode, int32_t* worker, int32_t* tau)
{
    if (n < 1 || T < 0 || !law || (T > 0 && (!worker || !tau))) return GEM_EINVAL;
    if (pull_mode != GEM_PULL_POST_COMMIT && pull_mode != GEM_PULL_PRE_COMMIT) return GEM_EINVAL;
    if (law->law < GEM_LAW_EXP || law->law > GEM_LAW_PARETO) return GEM_EINVAL;
    if (law->law == GEM_LAW_PARETO && !(law->p0 > 0.0 && law->p1 > 0.0)) return GEM_EINVAL;
    std::vector<double> mean(static_cast<size_t>(n)), finish(static_cast<size_t>(n));
    std::vector<int64_t> jobs(static_cast<size_t>(n), 1), pulled(static_cast<size_t>(n), 0);
    for (int32_t w = 0; w < n; ++w) {
        mean[w] = mean_of_worker(*law, seed, w);
        finish[w] = job_duration(*law, mean[w], seed, w, 0);
    }
    for (int64_t t = 0; t < T; ++t) {
        int32_t best = 0;
        for (int32_t w = 1; w < n; ++w)
            if (finish[w] < finish[best]) best = w;
        worker[t] = best;
        const int64_t st = t - pulled[best];
        if (st > INT32_MAX) return GEM_EINVAL;
        tau[t] = static_cast<int32_t>(st);
        pulled[best] = pull_mode == GEM_PULL_PRE_COMMIT ? t : t + 1;
        finish[best] = finish[best] + job_duration(*law, mean[best], seed, best, jobs[best]);
        jobs[best] += 1;
    }
    return GEM_OK;
}

// ---------------------------------------------------------------------------
// Checkpoints: a small header, then theta, S rows, M rows (P floats each),
// the pull clocks, if set h and theta*, and if set the nseg + 1 segment
// offsets.
// ---------------------------------------------------------------------------
namespace {

struct CkptHeader {
    char magic[8];
    int64_t P;
    int32_t n;
    int32_t have_problem;
    int64_t t;
    gem_hyperparams hp;
    gem_sim_params sp;
    int64_t nseg;         // segments of the partition, 0 if none was set
};

constexpr char kCkptMagic[8] = {'G', 'E', 'M', 'C', 'K', 'P', 'T', '2'};

int write_rows(gem_handle* g, FILE* f, const float* dev, int64_t rows, std::vector<float>& buf)
{
    for (int64_t r = 0; r < rows; ++r) {
        GEM_HIP(hipMemcpyAsync(buf.data(), dev + r * g->Pp, static_cast<size_t>(g->P) * sizeof(float),
                               hipMemcpyDeviceToHost, g->stream));
        GEM_HIP(hipStreamSynchronize(g->stream));
        if (std::fwrite(buf.data(), sizeof(float), static_cast<size_t>(g->P), f) !=
            static_cast<size_t>(g->P))
            return GEM_EIO;
    }
    return GEM_OK;
}

int read_rows(gem_handle* g, FILE* f, float* dev, int64_t rows, std::vector<float>& buf)
{
    for (int64_t r = 0; r < rows; ++r) {
        if (std::fread(buf.data(), sizeof(float), static_cast<size_t>(g->P), f) !=
            static_cast<size_t>(g->P))
            return GEM_EIO;
        GEM_HIP(hipMemcpyAsync(dev + r * g->Pp, buf.data(), static_cast<size_t>(g->P) * sizeof(float),
                               hipMemcpyHostToDevice, g->stream));
        GEM_HIP(hipStreamSynchronize(g->stream));
    }
    return GEM_OK;
}

// Rows of the table pieces at base (g->S or g->M), one worker after another,
// through a device staging row of Pp elements.
int write_table(gem_handle* g, FILE* f, const float* base, float* stage, std::vector<float>& buf)
{
    for (int32_t w = 0; w < g->n; ++w) {
        GEM_HIP(gemk::launch_read_row(base, g->n, w, g->P, stage, g->stream));
        GEM_HIP(hipMemcpyAsync(buf.data(), stage, static_cast<size_t>(g->P) * sizeof(float),
                               hipMemcpyDeviceToHost, g->stream));
        GEM_HIP(hipStreamSynchronize(g->stream));
        if (std::fwrite(buf.data(), sizeof(float), static_cast<size_t>(g->P), f) !=
            static_cast<size_t>(g->P))
            return GEM_EIO;
    }
    return GEM_OK;
}

// The staging row's padding [P, Pp) is zero, so each row's padding stays zero.
int read_table(gem_handle* g, FILE* f, float* base, float* stage, std::vector<float>& buf)
{
    for (int32_t w = 0; w < g->n; ++w) {
        if (std::fread(buf.data(), sizeof(float), static_cast<size_t>(g->P), f) !=
            static_cast<size_t>(g->P))
            return GEM_EIO;
        GEM_HIP(hipMemcpyAsync(stage, buf.data(), static_cast<size_t>(g->P) * sizeof(float),
                               hipMemcpyHostToDevice, g->stream));
        GEM_HIP(gemk::launch_fill_rows(base, g->n, w, 1, g->Pp, stage, g->stream));
        GEM_HIP(hipStreamSynchronize(g->stream));
    }
    return GEM_OK;
}

// A zeroed device row of Pp elements for checkpoint I/O, or null.
float* staging_row(gem_handle* g)
{
    float* stage = nullptr;
    const size_t bytes = static_cast<size_t>(g->Pp) * sizeof(float);
    if (hipMalloc(&stage, bytes) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
    }
    if (hipMemsetAsync(stage, 0, bytes, g->stream) != hipSuccess) {
        (void)hipGetLastError();
        (void)hipFree(stage);
        return nullptr;
    }
    return stage;
}

}  // namespace

int gem_save(gem_t* g, const char* path)
{
    if (!g || !path) return GEM_EINVAL;
    GEM_HIP(hipStreamSynchronize(g->stream));
    float* stage = staging_row(g);
    if (!stage) return GEM_ENOMEM;
    FILE* f = std::fopen(path, "wb");
    if (!f) {
        (void)hipStreamSynchronize(g->stream);
        (void)hipFree(stage);
        return GEM_EIO;
    }
    CkptHeader hd;
    std::memset(&hd, 0, sizeof(hd));
    std::memcpy(hd.magic, kCkptMagic, 8);
    hd.P = g->P;
    hd.n = g->n;
    hd.have_problem = g->have_problem ? 1 : 0;
    hd.t = g->t;
    hd.hp = g->hp;
    hd.sp = g->sp;
    hd.nseg = g->seg_host.empty() ? 0 : static_cast<int64_t>(g->seg_host.size()) - 1;
    std::vector<float> buf(static_cast<size_t>(g->P));
    int rc = std::fwrite(&hd, sizeof(hd), 1, f) == 1 ? GEM_OK : GEM_EIO;
    if (!rc) rc = write_rows(g, f, g->theta, 1, buf);
    if (!rc) rc = write_table(g, f, g->S, stage, buf);
    if (!rc) rc = write_table(g, f, g->M, stage, buf);
    if (!rc && std::fwrite(g->pc.data(), sizeof(int64_t), g->pc.size(), f) != g->pc.size()) rc = GEM_EIO;
    if (!rc && g->have_problem) rc = write_rows(g, f, g->h, 1, buf);
    if (!rc && g->have_problem) rc = write_rows(g, f, g->ts, 1, buf);
    if (!rc && hd.nseg > 0 &&
        std::fwrite(g->seg_host.data(), sizeof(int64_t), g->seg_host.size(), f) != g->seg_host.size())
        rc = GEM_EIO;
    if (std::fclose(f) != 0 && !rc) rc = GEM_EIO;
    (void)hipStreamSynchronize(g->stream);
    (void)hipFree(stage);
    return rc;
}

int gem_load(gem_t* g, const char* path)
{
    if (!g || !path) return GEM_EINVAL;
    FILE* f = std::fopen(path, "rb");
    if (!f) return GEM_EIO;
    CkptHeader hd;
    int rc = std::fread(&hd, sizeof(hd), 1, f) == 1 ? GEM_OK : GEM_EIO;
    if (!rc && (std::memcmp(hd.magic, kCkptMagic, 8) != 0 || hd.P != g->P || hd.n != g->n ||
                hd.nseg < 0 || hd.nseg > g->P))
        rc = GEM_EIO;
    if (!rc && !valid_hp(hd.hp)) rc = GEM_EIO;
    std::vector<int64_t> seg;
    std::vector<int64_t> pc(static_cast<size_t>(g->n));
    if (!rc) {
        // The whole file must be there, and the partition valid, before any
        // state is overwritten.
        const int64_t rows = 1 + 2 * static_cast<int64_t>(g->n) + (hd.have_problem ? 2 : 0);
        const int64_t body = static_cast<int64_t>(sizeof(hd)) + rows * g->P * 4 + 8 * static_cast<int64_t>(g->n);
        const int64_t want = body + (hd.nseg > 0 ? 8 * (hd.nseg + 1) : 0);
        if (std::fseek(f, 0, SEEK_END) != 0 || std::ftell(f) != want) rc = GEM_EIO;
        // The clocks: 0 <= pull clock <= t <= 2^32 - 1 (t keys the noise).
        if (!rc && (hd.t < 0 || hd.t > static_cast<int64_t>(UINT32_MAX))) rc = GEM_EIO;
        if (!rc) {
            const int64_t pc_at = static_cast<int64_t>(sizeof(hd)) +
                                  (1 + 2 * static_cast<int64_t>(g->n)) * g->P * 4;
            if (std::fseek(f, static_cast<long>(pc_at), SEEK_SET) != 0 ||
                std::fread(pc.data(), sizeof(int64_t), pc.size(), f) != pc.size())
                rc = GEM_EIO;
            for (size_t w = 0; !rc && w < pc.size(); ++w)
                if (pc[w] < 0 || pc[w] > hd.t) rc = GEM_EIO;
        }
        if (!rc && hd.nseg > 0) {
            seg.resize(static_cast<size_t>(hd.nseg) + 1);
            if (std::fseek(f, static_cast<long>(body), SEEK_SET) != 0 ||
                std::fread(seg.data(), sizeof(int64_t), seg.size(), f) != seg.size())
                rc = GEM_EIO;
            if (!rc && (seg.front() != 0 || seg.back() != g->P)) rc = GEM_EIO;
            for (size_t k = 0; !rc && k + 1 < seg.size(); ++k)
                if (seg[k + 1] <= seg[k]) rc = GEM_EIO;
        }
        if (!rc && std::fseek(f, static_cast<long>(sizeof(hd)), SEEK_SET) != 0) rc = GEM_EIO;
    }
    float* stage = nullptr;
    if (!rc) {
        stage = staging_row(g);
        if (!stage) rc = GEM_ENOMEM;
    }
    if (!rc && g->hist_on && g->hist_seg)
        g->hist_on = false;   // the partition under a per-segment recording may change
    if (!rc && !seg.empty()) rc = build_segments(g, seg);
    if (!rc && hd.have_problem && !g->h) {
        if (hipMalloc(&g->h, static_cast<size_t>(g->Pp) * sizeof(float)) != hipSuccess ||
            hipMalloc(&g->ts, static_cast<size_t>(g->Pp) * sizeof(float)) != hipSuccess) {
            (void)hipGetLastError();
            rc = GEM_ENOMEM;
        } else {
            (void)hipMemsetAsync(g->h, 0, static_cast<size_t>(g->Pp) * sizeof(float), g->stream);
            (void)hipMemsetAsync(g->ts, 0, static_cast<size_t>(g->Pp) * sizeof(float), g->stream);
        }
    }
    std::vector<float> buf(static_cast<size_t>(g->P));
    if (!rc) rc = read_rows(g, f, g->theta, 1, buf);
    if (!rc) rc = read_table(g, f, g->S, stage, buf);
    if (!rc) rc = read_table(g, f, g->M, stage, buf);
    // the pull clocks, read and checked above
    if (!rc && std::fseek(f, static_cast<long>(8 * pc.size()), SEEK_CUR) != 0) rc = GEM_EIO;
    if (!rc && hd.have_problem) rc = read_rows(g, f, g->h, 1, buf);
    if (!rc && hd.have_problem) rc = read_rows(g, f, g->ts, 1, buf);
    std::fclose(f);
    (void)hipStreamSynchronize(g->stream);
    (void)hipFree(stage);
    if (rc) return rc;
    if (seg.empty() && !g->seg_host.empty()) {
        GEM_HIP(hipStreamSynchronize(g->stream));
        free_segments(g);   // the saved run used the default single segment
    }
    g->hp = hd.hp;
    g->sp = hd.sp;
    g->have_problem = hd.have_problem != 0;
    g->t = hd.t;
    g->pc = pc;
    return GEM_OK;
}

}  // extern "C"
