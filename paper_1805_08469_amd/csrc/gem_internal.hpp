// gem_internal.hpp -- pieces shared by the libgem host code and its kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/gem.h"
#include "gem_layout.hpp"
#include "gem_plan.hpp"

namespace gemk {

static_assert(kPlanMaxK == GEM_K_MAX, "the planner handles whole passes");

// Size of the sink rows, in 16-byte chunks (power of two); small enough to
// stay resident in each XCD's L2.
constexpr int64_t kSinkChunks = 4096;

// Runtime mode bits for the general kernel variant.
enum : uint32_t {
    kModeLiteralPi = 1u << 0,
    kModeKappaMul = 1u << 1,     // multiply |m| by k_eff (kappa != 1 or SQRT form)
    kModePrePull = 1u << 2,
    kModeDownpour = 1u << 3,
    kModeAdaptive = 1u << 4,
    kModeGlobalProxy = 1u << 5,  // one moment (worker 0's) shared by all workers
};

// Kernel argument block of one fused pass: K <= GEM_K_MAX commits at clocks
// t0 .. t0 + K - 1 over the padded parameter vector.
struct PassArgs {
    float* theta;            // [Pp]
    float* S;                // the table: S_w[i] at S[tile_index(nw, w, i)]
    float* M;                // S + kTileElems: M_w[i] at M[tile_index(nw, w, i)]
    const float* h;          // [Pp]   (generated updates only)
    const float* ts;         // [Pp]   theta*
    double* diag;            // [4] accumulators, or null (diagnostic variant only)
    uint32_t* pi_hist;       // [hist_cap][hist_rows][GEM_PI_BINS] or null (diagnostic variant only)
    int64_t hist_first;      // recording index of this pass's first commit
    int64_t hist_cap;
    // Per-segment histograms: hist_rows = number of segments, each element
    // counted in its segment's row; hist_rows = 1: one histogram per commit.
    const int64_t* hseg_off; // [hist_rows + 1] segment offsets (per-segment mode)
    const int32_t* hseg_grp; // [groups] segment of each 1024-element group's first element
    int32_t hist_rows;
    int32_t rec_grid;        // blocks of a recording pass (0: one per group of 1024 elements)
    float* sink_S;           // [kSinkChunks * 4] target of loads/stores a step does not need
    float* sink_M;
    int64_t sink_mask;       // kSinkChunks - 1
    int64_t Pp;              // padded row length, a multiple of 64
    int64_t P;               // true length
    int64_t nw;              // workers (the table's worker stride)
    uint32_t key0, key1;     // noise seed
    uint32_t t0;             // clock of the pass's first commit
    int32_t K;
    float neg_lr, sigma, mu, eps, k_eff;
    uint32_t mode;
    // Streaming passes (NT) still read theta (keep_theta) or h and theta*
    // (keep_problem) with the default policy when those vectors fit the
    // Infinity Cache beside the streamed rows, which then serves them from
    // one pass to the next.
    uint8_t keep_theta, keep_problem, pad_[2];
    int32_t worker[GEM_K_MAX];
    int32_t tau[GEM_K_MAX];  // staleness (adaptive-staleness rule only)
    // 32-bit so that a uniform per-commit read is a scalar load: gfx9 has no
    // scalar byte load, and a vector one would wait on every outstanding
    // memory operation of the wave.
    uint32_t routes[GEM_K_MAX];
    const void* upd[GEM_K_MAX];  // caller updates (given-update variants)
};

enum class Source { Generated = 0, GivenF32 = 1, GivenBF16 = 2 };

// Segment-norm scale factors.  A sum of squares is the adjacent-pairs tree
// over aligned blocks of kSegBlock indices, then the blocks in order.  The
// step kernel forms the tree's lower levels, one aligned group of
// kSegGroup = 4 * 256 indices per thread block; seg_blocks_kernel the upper
// levels, 256 groups per index block.
constexpr int64_t kSegGroup = 1024;
constexpr int64_t kSegBlock = 1 << 18;
// The step kernel writes one partial sum per wave (256 indices); a group's
// four follow each other in the partial-sum array.
constexpr int64_t kWavesPerGroup = 4;

// One launch of the segment step kernel: finish the pending commit (apply its
// per-segment factors and pull) and/or start commit t (form d, m and the
// drift, store m, and write the group sums of squares of the drift, m and d
// for every segment the group touches).
struct SegArgs {
    float* theta;             // [Pp]
    float* S;                 // the table's snapshot pieces (as in PassArgs)
    float* M;                 // S + kTileElems: its moment pieces
    const float* h;           // [Pp]   (generated updates)
    const float* ts;          // [Pp]
    const void* upd_prev;     // caller update of the pending commit (given updates)
    const void* upd_cur;      // caller update of commit t (given updates)
    const float* pi_seg;      // [nseg] factors of the pending commit
    double* part;             // [3][npart][4] wave sums of squares of commit t: drift, m, d
    const int64_t* seg_off;   // [nseg + 1]
    const int64_t* part_off;  // [nseg + 1] first group-sum slot of each segment
    const int32_t* gseg;      // [groups] segment holding each group's first element
    int64_t npart;
    int64_t Pp, P;
    int64_t nw;               // workers (the table's worker stride)
    int32_t apply;            // finish the pending commit
    int32_t start;            // start commit t
    int32_t w_prev;           // worker of the pending commit
    int32_t w_cur;            // worker of commit t
    int32_t m_row;            // worker whose moment commit t refreshes
    int32_t m_row_prev;       // worker whose moment the pending commit refreshed (diagnostics)
    int32_t pre_pull;         // the snapshot keeps the pre-commit theta
    // Where theta before the pending commit is read from: -1 for the theta
    // array, else this worker's snapshot row (with post-commit pulls the
    // previous commit's worker pulled exactly that theta, so the array need
    // not be written between the launches of a run).
    int32_t theta_row;
    int32_t store_theta;      // write theta to the theta array (a run's last launch)
    double* diag;             // [4] accumulators, or null (diagnostic variant)
    float k_eff;              // kappa as it multiplies the moment (diagnostics)
    uint32_t t;               // clock of commit t; the pending commit's is t - 1
    uint32_t key0, key1;
    float neg_lr, sigma, mu;
};

// Pass-kernel specialisations.  Fast and FastGlobal take the default rule
// (GEM, CLAMP0, kappa_eff = 1, post-commit pull) with per-worker or shared
// first moments; General takes every mode as uniform runtime flags.
enum class Variant { General = 0, Fast = 1, FastGlobal = 2 };

// Launchers (defined in gem_kernels.hip).
// depth: kPrefetchShallow, or kPrefetchDeep for (Generated, Fast, no
// diagnostics), or kPrefetchNone for a pass of one commit (a.K == 1, no
// diagnostics, no recording); the routes in a must be planned for the same
// depth (a single commit's route is the same for every depth).
// stream_rows: non-temporal row and vector accesses (the diagnostic variant
// ignores it).  deep_lds: dynamic LDS bytes reserved per block of the
// deep-ring pass (deep_lds_bytes), 0 for none.
// rec: the fast recording pass (Generated, Fast, no diagnostics; one
// histogram per commit in a.pi_hist).
hipError_t launch_pass(const PassArgs& a, Source src, Variant v, bool bf16_out, bool diag,
                       bool rec, int depth, bool stream_rows, uint32_t deep_lds,
                       hipStream_t stream);


// Infinity Cache of one MI355X: a state this small stays cached across passes.
constexpr int64_t kInfinityCacheBytes = int64_t{256} << 20;
// stream_rows as for launch_pass (the diagnostic variant ignores it).
hipError_t launch_seg_step(const SegArgs& a, Source src, bool bf16_out, bool stream_rows,
                           hipStream_t stream);
// What the last block of each segment needs to form the segment's factor.
struct SegFactors {
    float* pi_seg;        // [nseg] out
    float k_eff, eps;
    int32_t literal;      // LITERAL pi (no clamp at zero)
    int32_t hist_per_seg; // histogram rows: one per segment, or one per commit
    uint32_t* hist;       // this commit's histogram rows, or null
    double* diag;         // [4] accumulators, or null
};
// seg_done: [nseg] counters, zero between launches (each launch leaves them zero).
hipError_t launch_seg_blocks(const double* part, int64_t npart, const int64_t* part_off,
                             const int64_t* seg_off, const int32_t* pair_seg,
                             const int32_t* pair_blk, int64_t npairs, double* sup,
                             const int64_t* sup_off, uint32_t* seg_done, const SegFactors& f,
                             hipStream_t stream);
hipError_t launch_generate(const float* S, int64_t nw, int32_t w, const float* h,
                           const float* ts, void* out, bool bf16, int64_t P, uint32_t t,
                           uint32_t key0, uint32_t key1, float neg_lr, float sigma,
                           hipStream_t stream);
// Rows w0 .. w0 + rows - 1 of the table's snapshot (base = S) or moment
// (base = M) pieces over indices [0, Pp) set to row[0, Pp), or to zero when
// row is null.
hipError_t launch_fill_rows(float* base, int64_t nw, int32_t w0, int32_t rows, int64_t Pp,
                            const float* row, hipStream_t stream);
// out[0, P) = worker w's row of the table's pieces at base.
hipError_t launch_read_row(const float* base, int64_t nw, int32_t w, int64_t P, float* out,
                           hipStream_t stream);
// out[k] = src[idx[k]] (a contiguous vector).
hipError_t launch_gather(const float* src, const int64_t* idx, int64_t count, float* out,
                         hipStream_t stream);
// out[w * count + k] = worker w's element idx[k] of the table's pieces at base, for all nw workers.
hipError_t launch_gather_rows(const float* base, int64_t nw, const int64_t* idx, int64_t count,
                              float* out, hipStream_t stream);
hipError_t launch_loss(const float* theta, const float* h, const float* ts, int64_t P,
                       double* out, hipStream_t stream);
// Device address of the current GPU's copy of the library's static scratch
// (GEM_SCRATCH_BYTES, 256-byte aligned); device is the current device.  The
// address is looked up once per device and kept.
hipError_t scratch_address(int device, void** out);
hipError_t launch_copy(const float* src, float* dst, int64_t count, hipStream_t stream);

}  // namespace gemk
