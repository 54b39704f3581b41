// gem_kernels.hip -- HIP kernels of the GEM commit pipeline for gfx950.
//
// The hot kernel is one fused pass: every thread owns four consecutive
// parameters (one 16-byte chunk of every row) and applies the pass's K
// commits to them in clock order.  theta, h and theta* are read once per
// pass and theta written once; a worker's snapshot and moment chunks are
// read (prefetched two commits ahead) at its first commit in the pass and
// written at its last, held in registers in between.  Rows are read and
// written as 128-bit accesses, consecutive lanes on consecutive chunks, so
// every wavefront moves 1 KiB contiguous per row.  There is no contraction:
// the work is streaming elementwise arithmetic (Philox, Box-Muller, the GEM
// step), bounded by HBM bandwidth and VALU issue, so no MFMA is involved.
//
// Also here: the per-segment variant of the scale factor (a streaming step
// kernel plus two small tree reductions per commit), the stand-alone update
// generator, and small gather, fill, loss and copy kernels.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "gem_device.hpp"
#include "gem_internal.hpp"

// Device scratch of the allocation-free entry point (gem_gather_static): one
// copy per GPU, held until the process ends.  In host code this name is only a
// stand-in for the symbol; the device address of the current GPU's copy comes
// from hipGetSymbolAddress (scratch_address below), and only that address is
// ever passed to kernels or copies.
static __device__ __align__(256) unsigned char scratch[GEM_SCRATCH_BYTES];

namespace gemk {

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};
}  // namespace

hipError_t scratch_address(int device, void** out)
{
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[device]) {
        // once per device, with that device current (the caller's)
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_dev[device] = p;
    }
    *out = g_scratch_dev[device];
    return hipSuccess;
}

namespace {

constexpr int kBlock = 256;

// Segments a block keeps block-local histograms for (per-segment mode);
// elements of further segments count straight into memory.
constexpr int kHistLdsSegs = 8;

// Recording pass (REC): the block keeps one histogram per commit of the pass
// in LDS for the whole pass, two bins per 32-bit word (16-bit counts: a block
// counts at most 1024 elements per commit), cleared once before the pass and
// flushed once after it -- no barrier between commits.
constexpr int kRecWords = (GEM_PI_BINS + 1) / 2;

struct DiagAcc {
    double ek = 0.0, proxy = 0.0, clamped = 0.0, elems = 0.0;
    uint32_t* hist = nullptr;   // block-local histograms of the current commit (LDS)
    int32_t seg_first = 0;      // per-segment mode: the block's first segment
    int32_t lds_rows = 1;       // histograms held in LDS
};

// Histogram bin of an applied scale factor, from its binary32 bits: 0 for
// <= 0 or NaN, 1 below 2^-20, 16 bins per octave over [2^-20, 2^20), and the
// last bin from 2^20 up.
__device__ __forceinline__ int scale_bin(float x)
{
    if (!(x > 0.0f)) return 0;
    const uint32_t b = __float_as_uint(x);
    const int octave = static_cast<int>((b >> 23) & 0xFFu) - 107;
    if (octave < 0) return 1;
    if (octave >= 40) return GEM_PI_BINS - 1;
    return 2 + octave * 16 + static_cast<int>((b >> 19) & 0xFu);
}

// The default rule's step on a thread's four elements (Fast variants, no
// diagnostics): the same arithmetic as commit_element, with one range check
// for the four quotients.  When all eight operand magnitudes lie in
// [2^-60, 2^60], each quotient is div_rn_core -- what div_rn takes for each of
// them; otherwise each goes through div_rn.  fmaxf / fminf skip a NaN
// operand, which may then reach div_rn_core: its quotient is NaN there as in
// the general division, and the clamp makes either pi = 0.
__device__ __forceinline__ void commit4_fast(const PassArgs& a, const float4& d, const float4& s,
                                             float4& th, float4& m, float4& snap,
                                             float* pi_out = nullptr)
{
    const float dv[4] = {d.x, d.y, d.z, d.w};
    const float sv[4] = {s.x, s.y, s.z, s.w};
    float tv[4] = {th.x, th.y, th.z, th.w};
    float mv[4] = {m.x, m.y, m.z, m.w};
    float num[4], den[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        mv[k] = __builtin_fmaf(a.mu, mv[k], dv[k]);                 // Alg. 1: m <- mu m + dtheta
        const float drift = tv[k] - sv[k];                          // theta_t - s_t (eq. 16)
        num[k] = __builtin_fabsf(mv[k]) - __builtin_fabsf(drift);
        den[k] = __builtin_fabsf(dv[k]) + a.eps;
    }
    float hi = __builtin_fabsf(num[0]), lo = hi;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if (k > 0) {
            hi = __builtin_fmaxf(hi, __builtin_fabsf(num[k]));
            lo = __builtin_fminf(lo, __builtin_fabsf(num[k]));
        }
        hi = __builtin_fmaxf(hi, __builtin_fabsf(den[k]));
        lo = __builtin_fminf(lo, __builtin_fabsf(den[k]));
    }
    // eq. 18, clamped at +0 (pi = q > 0 ? q : +0).  In the core range every
    // quotient is finite, so the clamp is the signed-integer maximum of its
    // bits with 0 (negative values and -0 have the sign bit set): one
    // instruction, where the float form needs a canonicalisation as well.
    float pi[4];
    if (lo >= 0x1p-60f && hi <= 0x1p60f) {
#pragma unroll
        for (int k = 0; k < 4; ++k)
            pi[k] = __int_as_float(max(__float_as_int(div_rn_core(num[k], den[k])), 0));
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float q = div_rn(num[k], den[k]);
            pi[k] = (q > 0.0f) ? q : 0.0f;
        }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        tv[k] = __builtin_fmaf(pi[k], dv[k], tv[k]);                // eq. 3
        if (pi_out) pi_out[k] = pi[k];
    }
    th = make_float4(tv[0], tv[1], tv[2], tv[3]);
    snap = th;
    m = make_float4(mv[0], mv[1], mv[2], mv[3]);
}

// One element of one commit.  th and m are the element's central value and
// the committing worker's moment (in/out); s is its snapshot; d the update.
// snap receives the value the worker's snapshot takes after this commit.
// FAST: the default rule (GEM, CLAMP0, kappa_eff = 1, post-commit pull) with
// no runtime mode tests; otherwise every mode is read from a.mode.
// hist_row: the histogram row this element's factor counts in, or null.
template <bool FAST, bool DIAG>
__device__ __forceinline__ void commit_element(const PassArgs& a, int tau, float d, float s,
                                               float& th, float& m, float& snap, bool live,
                                               DiagAcc& acc, uint32_t* hist_row)
{
    const float mn = __builtin_fmaf(a.mu, m, d);        // Alg. 1: m <- mu m + dtheta
    const float drift = th - s;                         // theta_t - s_t (eq. 16)
    float th_new;
    float pi_raw = 0.0f;
    float scale;                                        // factor applied to dtheta
    bool gem_rule = true;
    if (FAST) {
        const float num = __builtin_fabsf(mn) - __builtin_fabsf(drift);
        const float den = __builtin_fabsf(d) + a.eps;
        pi_raw = div_rn(num, den);                      // eq. 18 / Alg. 1
        const float pi = (pi_raw > 0.0f) ? pi_raw : 0.0f;
        th_new = __builtin_fmaf(pi, d, th);             // eq. 3
        snap = th_new;
        scale = pi;
    } else {
        if (a.mode & kModeDownpour) {
            gem_rule = false;
            th_new = th + d;                            // eq. 1
            scale = 1.0f;
        } else if (a.mode & kModeAdaptive) {
            gem_rule = false;
            th_new = th + d / static_cast<float>(tau + 1);
            scale = 1.0f / static_cast<float>(tau + 1);
        } else {
            const float km = (a.mode & kModeKappaMul) ? a.k_eff * __builtin_fabsf(mn)
                                                      : __builtin_fabsf(mn);
            const float num = km - __builtin_fabsf(drift);
            const float den = __builtin_fabsf(d) + a.eps;
            pi_raw = div_rn(num, den);
            const float pi = (a.mode & kModeLiteralPi) ? pi_raw
                                                       : ((pi_raw > 0.0f) ? pi_raw : 0.0f);
            th_new = __builtin_fmaf(pi, d, th);
            scale = pi;
        }
        snap = (a.mode & kModePrePull) ? th : th_new;
    }
    if (DIAG && live && hist_row) atomicAdd(&hist_row[scale_bin(scale)], 1u);
    if (DIAG && live) {
        const double e = static_cast<double>(th_new) - static_cast<double>(s);
        const double kmd = static_cast<double>(FAST ? 1.0f : a.k_eff) * static_cast<double>(mn);
        acc.ek += 0.5 * e * e;
        acc.proxy += 0.5 * kmd * kmd;
        if (gem_rule && !(pi_raw >= 0.0f)) acc.clamped += 1.0;
        acc.elems += 1.0;
    }
    th = th_new;
    m = mn;
}

// The simulated worker's update at snapshot s (notation table: -eta grad L(s)).
template <bool BF16>
__device__ __forceinline__ float stale_update(float neg_lr, float sigma, float s, float h, float ts,
                                              float z)
{
    const float nz = sigma * z;
    const float g = __builtin_fmaf(h, s - ts, nz);
    float d = neg_lr * g;
    if (BF16) d = round_to_bf16(d);
    return d;
}

__device__ __forceinline__ float bf16_bits_to_float(uint32_t b16) { return __uint_as_float(b16 << 16); }

// A caller update for chunk c: four elements, masked past the true length.
template <Source SRC>
__device__ __forceinline__ float4 load_given(const void* base, int64_t c, int64_t P)
{
    const int64_t i0 = c * 4;
    if (SRC == Source::GivenF32) {
        const float* p = static_cast<const float*>(base);
        if (i0 + 4 <= P) return *reinterpret_cast<const float4*>(p + i0);
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (i0 + 0 < P) v.x = p[i0 + 0];
        if (i0 + 1 < P) v.y = p[i0 + 1];
        if (i0 + 2 < P) v.z = p[i0 + 2];
        if (i0 + 3 < P) v.w = p[i0 + 3];
        return v;
    } else {
        const uint16_t* p = static_cast<const uint16_t*>(base);
        if (i0 + 4 <= P) {
            const uint2 u = *reinterpret_cast<const uint2*>(p + i0);
            return make_float4(bf16_bits_to_float(u.x & 0xFFFFu), bf16_bits_to_float(u.x >> 16),
                               bf16_bits_to_float(u.y & 0xFFFFu), bf16_bits_to_float(u.y >> 16));
        }
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (i0 + 0 < P) v.x = bf16_bits_to_float(p[i0 + 0]);
        if (i0 + 1 < P) v.y = bf16_bits_to_float(p[i0 + 1]);
        if (i0 + 2 < P) v.z = bf16_bits_to_float(p[i0 + 2]);
        if (i0 + 3 < P) v.w = bf16_bits_to_float(p[i0 + 3]);
        return v;
    }
}

struct Rows {
    float4 s, m;
};

// 16-byte loads and stores of the fused pass.  NT marks them non-temporal
// (streaming): each row chunk a pass touches is read once and written once,
// and over a state far larger than the caches the hint lets HBM streams
// bypass the cache residency a reused line would get (measured 7-12% faster
// passes); a state that fits the 256 MiB Infinity Cache keeps the default
// policy, which serves it from there.
typedef float v4f __attribute__((ext_vector_type(4)));

template <bool NT>
__device__ __forceinline__ float4 load4(const float* p)
{
    if constexpr (NT) {
        const v4f v = __builtin_nontemporal_load(reinterpret_cast<const v4f*>(p));
        return make_float4(v.x, v.y, v.z, v.w);
    } else {
        return *reinterpret_cast<const float4*>(p);
    }
}

template <bool NT>
__device__ __forceinline__ void store4(float* p, float4 v)
{
    if constexpr (NT) {
        __builtin_nontemporal_store(v4f{v.x, v.y, v.z, v.w}, reinterpret_cast<v4f*>(p));
    } else {
        *reinterpret_cast<float4*>(p) = v;
    }
}

// The same at a (uniform) base plus a 32-bit byte offset, which the scalar
// base + vector offset addressing takes as is.  FRESH gives each use its own
// copy of the offset (an empty asm), so that the offset's widening to 64 bits
// is not hoisted out of the pass loop: a widened offset no longer fits that
// addressing.
__device__ __forceinline__ uint32_t fresh(uint32_t x)
{
    asm volatile("" : "+v"(x));
    return x;
}

template <bool NT, bool FRESH = false>
__device__ __forceinline__ float4 load4_at(const float* base, uint32_t byte_off)
{
    if constexpr (FRESH) byte_off = fresh(byte_off);
    return load4<NT>(reinterpret_cast<const float*>(reinterpret_cast<const char*>(base) + byte_off));
}

template <bool NT, bool FRESH = false>
__device__ __forceinline__ void store4_at(float* base, uint32_t byte_off, float4 v)
{
    if constexpr (FRESH) byte_off = fresh(byte_off);
    store4<NT>(reinterpret_cast<float*>(reinterpret_cast<char*>(base) + byte_off), v);
}


// Per-thread context of a fused pass: the chunk, its central values and the
// problem coefficients, kept in registers for the whole pass.
struct Chunk {
    int64_t c;       // chunk index (= Philox counter q of its four elements)
    int64_t off;     // element offset 4c
    // Addresses as a block-uniform part and a 32-bit lane part: worker w's
    // snapshot chunk is at S + tile + w * 2 * kTileElems plus io bytes (io =
    // 4 * tin + t16), its moment chunk at M + the same; its sink entries at
    // sink_S / sink_M plus so bytes (so = 4 * sink0 + t16); theta, h and
    // theta* at blk0 plus t16 bytes.
    int64_t tile;    // table index of worker 0's snapshot piece of the block's tile
    int64_t tin;     // the block's first element offset inside its tile
    int64_t blk0;    // first element of the block
    int64_t sink0;   // first element of the block's sink entries
    uint32_t io;     // byte offset of the chunk inside its tile's piece
    uint32_t so;     // byte offset of the chunk's entries in the sink buffers
    uint32_t t16;    // 16 * threadIdx.x
    uint32_t q_lo, q_hi;   // words of the chunk index c (the Philox counter)
    bool active;
    bool l0, l1, l2, l3;   // elements below the true length (diagnostics)
    int32_t sg[4];         // per-segment histograms: each element's segment
    float4 th, hh, tt;
    float4 mg;       // the shared moment (global proxy mode)
};

// Register slots holding the (snapshot, moment) chunks of workers that commit
// again later in the same pass.
struct Held {
    Rows h0, h1, h2, h3;
};

__device__ __forceinline__ Rows held_get(const Held& h, uint32_t slot)
{
    switch (slot) {
    case 0: return h.h0;
    case 1: return h.h1;
    case 2: return h.h2;
    default: return h.h3;
    }
}

__device__ __forceinline__ Held held_put(Held h, uint32_t slot, const Rows& r)
{
    switch (slot) {
    case 0: h.h0 = r; break;
    case 1: h.h1 = r; break;
    case 2: h.h2 = r; break;
    default: h.h3 = r; break;
    }
    return h;
}

// One step's row access: worker w's piece of `table` if mem, else the sink.
// The shared-moment variant (VALU-bound) keeps the base block-uniform and
// adds the lane's 16 * threadIdx.x bytes, which saves vector instructions and
// registers (3-4% faster); the per-worker variants (HBM-bound) select a
// per-lane element offset, measured 0.3-4% faster for them.
template <bool UNIFORM, bool NT>
__device__ __forceinline__ float4 row_load(const float* table, const float* sink, bool mem,
                                           int32_t w, const Chunk& ch)
{
    const int64_t wrow = ch.tile + (static_cast<int64_t>(w) << (kTileShift + 1));
    if constexpr (UNIFORM)
        return load4_at<NT, true>(mem ? table + wrow + ch.tin : sink + ch.sink0, ch.t16);
    else
        return load4_at<NT>(mem ? table + wrow : sink, mem ? ch.io : ch.so);
}

template <bool UNIFORM, bool NT>
__device__ __forceinline__ void row_store(float* table, float* sink, bool mem, int32_t w,
                                          const Chunk& ch, float4 v)
{
    const int64_t wrow = ch.tile + (static_cast<int64_t>(w) << (kTileShift + 1));
    if constexpr (UNIFORM)
        store4_at<NT, true>(mem ? table + wrow + ch.tin : sink + ch.sink0, ch.t16, v);
    else
        store4_at<NT>(mem ? table + wrow : sink, mem ? ch.io : ch.so, v);
}

struct StepOut {
    Rows out;    // the worker's (snapshot, moment) chunk after commit j
    Rows next;   // ring entry for commit j + DEPTH
    Held held;
};


// Commit j of a pass.  The committing worker's (snapshot, moment) chunk comes
// from the prefetch ring (loaded DEPTH commits earlier: a first commit in the
// pass, or a worker whose earlier commit in the pass, at least DEPTH commits
// back, wrote its rows back) or from a register slot.  After the commit the
// chunk is written back (the worker's last commit in the pass, or no slot was
// free) or held in a slot; then the rows of commit j + DEPTH are prefetched
// into the ring entry just consumed, if that
// commit reads them from memory.  Every step issues one row-pair store and one
// row-pair load unconditionally -- those a step does not need go to the small
// sink buffer, which stays in cache -- so the wait for a step's rows never
// covers the loads issued after them.
template <Source SRC, Variant V, bool BF16, bool DIAG, int DEPTH, bool NT, bool REC>
__device__ __forceinline__ StepOut pass_step(const PassArgs& a, int j, Chunk& ch, Rows ring,
                                             Held held, DiagAcc& acc, uint32_t* rec_lds)
{
    const uint32_t route = a.routes[j];
    const uint32_t src = route & kRouteSlotMask;
    const uint32_t dst = (route >> kRouteDstShift) & kRouteSlotMask;
    const int w = a.worker[j];
    // (a single-commit pass reads its one commit's rows through the ring)
    Rows rows = (DEPTH == 1 || src == kFromRing) ? ring : held_get(held, src);
    constexpr bool FAST = V != Variant::General;
    const bool global_m = V == Variant::FastGlobal ||
                          (V == Variant::General && (a.mode & kModeGlobalProxy));
    if (global_m) rows.m = ch.mg;   // the shared moment, carried like theta

    float4 d;
    if (SRC == Source::Generated) {
        // The chunk index's high word is the block's (uniform): blocks start at
        // multiples of kBlock chunks, so adding the lane never carries into it.
        const uint64_t q = (static_cast<uint64_t>(ch.q_hi) << 32) | ch.q_lo;
        const float4 z = normals4(q, a.t0 + static_cast<uint32_t>(j),
                                  a.key0, a.key1);
        d.x = stale_update<BF16>(a.neg_lr, a.sigma, rows.s.x, ch.hh.x, ch.tt.x, z.x);
        d.y = stale_update<BF16>(a.neg_lr, a.sigma, rows.s.y, ch.hh.y, ch.tt.y, z.y);
        d.z = stale_update<BF16>(a.neg_lr, a.sigma, rows.s.z, ch.hh.z, ch.tt.z, z.z);
        d.w = stale_update<BF16>(a.neg_lr, a.sigma, rows.s.w, ch.hh.w, ch.tt.w, z.w);
    } else {
        d = ch.active ? load_given<SRC>(a.upd[j], ch.c, a.P) : make_float4(0.f, 0.f, 0.f, 0.f);
    }

    const int tau = a.tau[j];
    // Diagnostic histogram of this commit's scale factors: every thread of
    // the block is at commit j here (the loop is uniform), so the block-local
    // histogram is cleared, filled and flushed between barriers.
    const bool record = DIAG && acc.hist != nullptr && a.hist_first + j < a.hist_cap;
    const int lds_bins = acc.lds_rows * GEM_PI_BINS;
    if (DIAG && acc.hist != nullptr) {
        for (int b = threadIdx.x; b < lds_bins; b += kBlock) acc.hist[b] = 0u;
        __syncthreads();
    }
    // Each element's histogram row: the block-local one of its segment, or
    // (a segment beyond the block's LDS rows) its row of this commit in memory.
    uint32_t* hrow[4] = {nullptr, nullptr, nullptr, nullptr};
    if (DIAG && record) {
        uint32_t* commit_rows = a.pi_hist + (a.hist_first + j) * a.hist_rows * GEM_PI_BINS;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int ls = ch.sg[k] - acc.seg_first;
            hrow[k] = ls < acc.lds_rows ? acc.hist + ls * GEM_PI_BINS
                                        : commit_rows + static_cast<int64_t>(ch.sg[k]) * GEM_PI_BINS;
        }
    }
    StepOut r;
    r.out.m = rows.m;
    if constexpr (FAST && !DIAG) {
        float pis[4];
        commit4_fast(a, d, rows.s, ch.th, r.out.m, r.out.s, REC ? pis : nullptr);
        if constexpr (REC) {
            // this commit's factors into the block's LDS histogram (uniform
            // test: recording stops at the capacity)
            if (ch.active && a.hist_first + j < a.hist_cap) {
                uint32_t* row = rec_lds + j * kRecWords;
                uint32_t* spare = rec_lds + a.K * kRecWords + threadIdx.x;   // this lane's own word
                const bool live[4] = {ch.l0, ch.l1, ch.l2, ch.l3};
                // Clamped factors (+0, bin 0) are often most of a commit's:
                // the wave counts them with ballots and adds them once, while
                // their lanes (and padding elements) add to a word of their
                // own, so no add waits behind one address and no lane
                // branches.  A positive factor's bin is scale_bin's, in
                // integer steps: (bits >> 19) - 1710 clamped to [1, 642].
                uint32_t clamped = 0;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const uint32_t bits = __float_as_uint(pis[k]);   // +0 or positive
                    const bool counted = live[k] && bits != 0u;
                    clamped += static_cast<uint32_t>(__popcll(__ballot(live[k] && bits == 0u)));
                    const int bin = min(max(static_cast<int>(bits >> 19) - 1710, 1), GEM_PI_BINS - 1);
                    uint32_t* word = counted ? row + (bin >> 1) : spare;
                    atomicAdd(word, 1u << ((bin & 1) << 4));
                }
                const uint64_t lanes = __ballot(1);
                if (clamped != 0u && (threadIdx.x & 63u) == static_cast<uint32_t>(__builtin_ctzll(lanes)))
                    atomicAdd(&row[0], clamped);   // bin 0: the low half of word 0
            }
        }
    } else {
        commit_element<FAST, DIAG>(a, tau, d.x, rows.s.x, ch.th.x, r.out.m.x, r.out.s.x, ch.active && ch.l0, acc, hrow[0]);
        commit_element<FAST, DIAG>(a, tau, d.y, rows.s.y, ch.th.y, r.out.m.y, r.out.s.y, ch.active && ch.l1, acc, hrow[1]);
        commit_element<FAST, DIAG>(a, tau, d.z, rows.s.z, ch.th.z, r.out.m.z, r.out.s.z, ch.active && ch.l2, acc, hrow[2]);
        commit_element<FAST, DIAG>(a, tau, d.w, rows.s.w, ch.th.w, r.out.m.w, r.out.s.w, ch.active && ch.l3, acc, hrow[3]);
    }

    if (DIAG && acc.hist != nullptr) {
        __syncthreads();
        if (record) {
            uint32_t* dst = a.pi_hist +
                            ((a.hist_first + j) * a.hist_rows + acc.seg_first) * GEM_PI_BINS;
            for (int b = threadIdx.x; b < lds_bins; b += kBlock)
                if (acc.hist[b]) atomicAdd(&dst[b], acc.hist[b]);
        }
        __syncthreads();
    }
    if (global_m) ch.mg = r.out.m;
    if (DEPTH > 1 && dst != kToMemory) {
        // The shared-moment variant carries the moment in ch.mg: a held
        // slot keeps only the snapshot (no registers for a moment copy).
        Rows keep = r.out;
        if (V == Variant::FastGlobal) keep.m = make_float4(0.f, 0.f, 0.f, 0.f);
        held = held_put(held, dst, keep);
    }
    r.held = held;
    r.next = ring;
    if (ch.active) {
        // With the shared moment, only snapshot rows move; moment traffic goes
        // to the sink.
        constexpr bool U = V == Variant::FastGlobal;
        const bool st = DEPTH == 1 || dst == kToMemory;
        const bool st_m = st && !global_m;
        row_store<U, NT>(a.S, a.sink_S, st, w, ch, r.out.s);
        row_store<U, NT>(a.M, a.sink_M, st_m, w, ch, r.out.m);
        if constexpr (DEPTH > 1) {
            const bool pf = (route & kRoutePrefetch) != 0;
            const int jn = j + DEPTH < a.K ? j + DEPTH : j;
            const bool pf_m = pf && !global_m;
            r.next.s = row_load<U, NT>(a.S, a.sink_S, pf, a.worker[jn], ch);
            r.next.m = row_load<U, NT>(a.M, a.sink_M, pf_m, a.worker[jn], ch);
        }
    }
    return r;
}

// One pass over the 1024 elements of group grp (the block's 256 chunks).
template <Source SRC, Variant V, bool BF16, bool DIAG, int DEPTH, bool NT, bool REC>
__device__ __forceinline__ void pass_group(const PassArgs& a, int64_t grp, uint32_t* rec_lds)
{
    static_assert(!(REC && DIAG), "recording passes take the fast commit");
    const int64_t nchunk = a.Pp >> 2;
    const int64_t c = grp * kBlock + threadIdx.x;
    Chunk ch;
    ch.active = c < nchunk;
    if (!DIAG && !ch.active) return;   // (the diagnostic variant's barriers need every thread)
    ch.c = ch.active ? c : 0;   // inactive lanes (diagnostic variant) do no memory work
    ch.off = ch.c * 4;
    static_assert((kBlock & (kBlock - 1)) == 0, "block size a power of two");
    ch.q_hi = static_cast<uint32_t>((grp * kBlock) >> 32);
    ch.q_lo = static_cast<uint32_t>(ch.c);
    ch.l0 = ch.off + 0 < a.P;
    ch.l1 = ch.off + 1 < a.P;
    ch.l2 = ch.off + 2 < a.P;
    ch.l3 = ch.off + 3 < a.P;
    ch.th = make_float4(0.f, 0.f, 0.f, 0.f);
    ch.hh = ch.th;
    ch.tt = ch.th;
    ch.mg = ch.th;
    const bool global_m = V == Variant::FastGlobal ||
                          (V == Variant::General && (a.mode & kModeGlobalProxy));
    static_assert(kTileElems % (kBlock * 4) == 0, "a block's chunks lie in one tile");
    static_assert(kSinkChunks % kBlock == 0, "a block's sink entries are contiguous");
    ch.blk0 = grp * (kBlock * 4);
    ch.t16 = threadIdx.x * 16u;
    ch.tile = tile_index(a.nw, 0, ch.blk0 & ~(kTileElems - 1));
    ch.tin = ch.blk0 & (kTileElems - 1);
    ch.sink0 = ((ch.blk0 >> 2) & a.sink_mask) * 4;
    ch.io = static_cast<uint32_t>(ch.tin) * 4u + ch.t16;
    ch.so = static_cast<uint32_t>(ch.c & a.sink_mask) * 16u;   // = 4 * sink0 + t16
    // The shared moment is worker 0's.
    if (global_m && ch.active) ch.mg = load4_at<NT>(a.M + ch.tile, ch.io);
    // A depth-1 kernel runs single-commit passes only (the launch checks it).
    const int K = DEPTH == 1 ? 1 : a.K;
    // Ring of prefetched rows, unrolled DEPTH ways so that every entry
    // is a fixed set of registers: commit j reads ring[j mod depth] and refills
    // it for commit j + depth -- no register copy of an in-flight load.
    Rows ring[DEPTH];
    Held held{};
    if (ch.active) {
        ch.th = a.keep_theta ? load4_at<false>(a.theta + ch.blk0, ch.t16)
                             : load4_at<NT>(a.theta + ch.blk0, ch.t16);
        if (SRC == Source::Generated) {
            if (a.keep_problem) {
                ch.hh = load4_at<false>(a.h + ch.blk0, ch.t16);
                ch.tt = load4_at<false>(a.ts + ch.blk0, ch.t16);
            } else {
                ch.hh = load4_at<NT>(a.h + ch.blk0, ch.t16);
                ch.tt = load4_at<NT>(a.ts + ch.blk0, ch.t16);
            }
        }
#pragma unroll
        for (int u = 0; u < DEPTH; ++u) {
            // Commit u reads memory iff it is the first commit of its worker
            // (u < depth); the others prefetch from the sink.
            // With the shared moment only the snapshot row is read.
            const bool mem = u < K && (a.routes[u] & kRouteSlotMask) == kFromRing;
            const bool mem_m = mem && !global_m;
            constexpr bool U = V == Variant::FastGlobal;
            ring[u].s = row_load<U, NT>(a.S, a.sink_S, mem, a.worker[u], ch);
            ring[u].m = row_load<U, NT>(a.M, a.sink_M, mem_m, a.worker[u], ch);
        }
    } else {
#pragma unroll
        for (int u = 0; u < DEPTH; ++u) ring[u] = Rows{};
    }

    DiagAcc acc;
    ch.sg[0] = ch.sg[1] = ch.sg[2] = ch.sg[3] = 0;
    if constexpr (DIAG) {
        __shared__ uint32_t hist_lds[kHistLdsSegs * GEM_PI_BINS];
        if (a.pi_hist) {
            acc.hist = hist_lds;
            if (a.hist_rows > 1) {
                // The block's segments (uniform) and each element's segment.
                const int64_t g_lo = grp * kBlock * 4;
                const int64_t g_last = (g_lo + kBlock * 4 < a.P ? g_lo + kBlock * 4 : a.P) - 1;
                acc.seg_first = a.hseg_grp[grp];
                int32_t seg_last = acc.seg_first;
                while (a.hseg_off[seg_last + 1] <= g_last) ++seg_last;
                const int32_t rows = seg_last - acc.seg_first + 1;
                acc.lds_rows = rows < kHistLdsSegs ? rows : kHistLdsSegs;
                int32_t sg = acc.seg_first;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const int64_t i = ch.off + k;
                    if (ch.active && i < a.P)
                        while (a.hseg_off[sg + 1] <= i) ++sg;
                    ch.sg[k] = sg;
                }
            }
        }
    }
    int j = 0;
    for (; j + DEPTH <= K; j += DEPTH) {
#pragma unroll
        for (int u = 0; u < DEPTH; ++u) {
            const StepOut so = pass_step<SRC, V, BF16, DIAG, DEPTH, NT, REC>(a, j + u, ch, ring[u], held,
                                                                            acc, rec_lds);
            ring[u] = so.next;
            held = so.held;
        }
    }
    // At most DEPTH - 1 commits remain.
#pragma unroll
    for (int u = 0; u + 1 < DEPTH; ++u) {
        if (j + u < K) {
            const StepOut so = pass_step<SRC, V, BF16, DIAG, DEPTH, NT, REC>(a, j + u, ch, ring[u], held,
                                                                            acc, rec_lds);
            ring[u] = so.next;
            held = so.held;
        }
    }
    if (ch.active) {
        if (a.keep_theta) store4_at<false>(a.theta + ch.blk0, ch.t16, ch.th);
        else store4_at<NT>(a.theta + ch.blk0, ch.t16, ch.th);
    }
    if (global_m && ch.active) store4_at<NT>(a.M + ch.tile, ch.io, ch.mg);

    if (DIAG && a.diag) {
        __shared__ double red[4][kBlock];
        red[0][threadIdx.x] = acc.ek;
        red[1][threadIdx.x] = acc.proxy;
        red[2][threadIdx.x] = acc.clamped;
        red[3][threadIdx.x] = acc.elems;
        __syncthreads();
        for (int step = kBlock / 2; step > 0; step >>= 1) {
            if (static_cast<int>(threadIdx.x) < step) {
#pragma unroll
                for (int q = 0; q < 4; ++q) red[q][threadIdx.x] += red[q][threadIdx.x + step];
            }
            __syncthreads();
        }
        if (threadIdx.x < 4) atomicAdd(&a.diag[threadIdx.x], red[threadIdx.x][0]);
    }
}

// The fused pass: one group per block; the recording variant (REC) loops its
// blocks over the groups (a grid of a.rec_grid blocks, 0 for one per group)
// so that each block's per-pass LDS histograms gather many groups before
// their single flush -- one global atomic per nonzero bin and block.
template <Source SRC, Variant V, bool BF16, bool DIAG, int DEPTH, bool NT, bool REC>
__global__ __launch_bounds__(kBlock) void pass_kernel(const PassArgs a)
{
    extern __shared__ uint32_t dyn_lds[];   // REC: K rows of kRecWords, then a word per thread
    if constexpr (REC) {
        for (int w = threadIdx.x; w < a.K * kRecWords; w += kBlock) dyn_lds[w] = 0u;
        __syncthreads();
        const int64_t ngroups = ((a.Pp >> 2) + kBlock - 1) / kBlock;
        for (int64_t grp = blockIdx.x; grp < ngroups; grp += gridDim.x)
            pass_group<SRC, V, BF16, DIAG, DEPTH, NT, REC>(a, grp, dyn_lds);
        // the histograms into the recording, one atomic per nonzero bin
        __syncthreads();
        for (int w = threadIdx.x; w < a.K * kRecWords; w += kBlock) {
            const uint32_t v = dyn_lds[w];
            const int j = w / kRecWords;
            if (v == 0u || a.hist_first + j >= a.hist_cap) continue;
            uint32_t* row = a.pi_hist + (a.hist_first + j) * GEM_PI_BINS;
            const int b = 2 * (w - j * kRecWords);
            if (v & 0xFFFFu) atomicAdd(&row[b], v & 0xFFFFu);
            if (v >> 16) atomicAdd(&row[b + 1], v >> 16);
        }
    } else {
        pass_group<SRC, V, BF16, DIAG, DEPTH, NT, REC>(a, blockIdx.x, dyn_lds);
    }
}

// ---------------------------------------------------------------------------
// Segment-norm scale factors (one pi per segment of the parameter vector).
// A commit's pi needs sums of squares over whole segments, so each commit is
// split in two launches: the step kernel starts commit t (forms d, m and the
// drift, stores m, writes each 1024-index group's tree sums of squares), and
// seg_blocks_kernel adds the group sums of each 2^18-index block by the same
// tree, after which the last block of each segment adds the block sums in
// order and forms the segment's pi.  The next step kernel applies those
// factors (and the pull) before starting the next commit, generating the
// pending update again.
// ---------------------------------------------------------------------------

__device__ __forceinline__ float4 f4(const float* p) { return *reinterpret_cast<const float4*>(p); }
// c ? x : y on values (a conditional on two float4 objects selects between
// their addresses, which keeps them out of registers).
__device__ __forceinline__ float4 pick(bool c, float4 x, float4 y)
{
    return make_float4(c ? x.x : y.x, c ? x.y : y.y, c ? x.z : y.z, c ? x.w : y.w);
}
__device__ __forceinline__ float lane(const float4& v, int k)
{
    return k == 0 ? v.x : k == 1 ? v.y : k == 2 ? v.z : v.w;
}

// Sum of the block's 256 per-thread values by the adjacent-pairs tree: lane
// butterflies (which add pairs 2k, 2k+1, then pairs of pairs, ...) within
// each wave, then (wave 0 + wave 1) + (wave 2 + wave 3).  Thread 0 gets the
// result.  Every thread of the block must call it.
__device__ __forceinline__ double block_tree_sum(double v, double* lds)
{
#pragma unroll
    for (int mask = 1; mask < 64; mask <<= 1) v = v + __shfl_xor(v, mask);
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) lds[wave] = v;
    __syncthreads();
    const double r = (lds[0] + lds[1]) + (lds[2] + lds[3]);
    __syncthreads();
    return r;
}

// Three such sums at once, each in the same order as block_tree_sum, with one
// pair of barriers for the three.
__device__ __forceinline__ void block_tree_sum3(double& x, double& y, double& z, double (*lds)[4])
{
#pragma unroll
    for (int mask = 1; mask < 64; mask <<= 1) {
        x = x + __shfl_xor(x, mask);
        y = y + __shfl_xor(y, mask);
        z = z + __shfl_xor(z, mask);
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        lds[0][wave] = x;
        lds[1][wave] = y;
        lds[2][wave] = z;
    }
    __syncthreads();
    x = (lds[0][0] + lds[0][1]) + (lds[0][2] + lds[0][3]);
    y = (lds[1][0] + lds[1][1]) + (lds[1][2] + lds[1][3]);
    z = (lds[2][0] + lds[2][1]) + (lds[2][2] + lds[2][3]);
    __syncthreads();
}

// No occupancy hint: with no barrier in the kernel, the compiler's own
// register budget runs 2.5% faster than a 7-waves-per-SIMD cap.
template <Source SRC, bool BF16, bool DIAG, bool NT>
__global__ __launch_bounds__(kBlock)
void seg_step_kernel(const SegArgs a)
{
    static_assert(kBlock * 4 == kSegGroup, "one block per group of sums");
    __shared__ double lds[3][4];
    const int64_t grp = blockIdx.x;
    const int64_t c = grp * kBlock + threadIdx.x;
    const bool active = c < (a.Pp >> 2);   // the last group may hold fewer chunks
    const int64_t off = c * 4;
    // The block's segments: its first, and whether the whole block lies in it
    // (all but the blocks that hold a segment boundary), in which case every
    // element takes that segment's factor and the block forms one set of
    // sums.  The lookups are issued before the streaming loads, so their
    // latency hides behind those instead of delaying the update.
    const int32_t s_first = a.gseg[grp];
    const int64_t g_lo = grp * kSegGroup;
    const int64_t g_hi = (g_lo + kSegGroup < a.P) ? g_lo + kSegGroup : a.P;
    const int64_t s_lo = a.seg_off[s_first], s_hi = a.seg_off[s_first + 1];
    const bool one_seg = s_hi >= g_hi;
    const float pi_one = a.apply ? a.pi_seg[s_first] : 0.0f;

    const float* th_src = a.theta_row < 0 ? a.theta + off
                                          : a.S + tile_index(a.nw, a.theta_row, off);
    float4 th = active ? load4<NT>(th_src) : make_float4(0.f, 0.f, 0.f, 0.f);
    const float4 th_old = th;
    float4 hv = make_float4(0.f, 0.f, 0.f, 0.f), tv = hv;
    // h and theta* keep the default cache policy even when everything else
    // streams: every commit reads them, and with the other streams marked
    // non-temporal the Infinity Cache holds them from one launch to the next
    // (measured 10% faster at 25M parameters).
    if (SRC == Source::Generated && active) {
        hv = load4<false>(a.h + off);
        tv = load4<false>(a.ts + off);
    }
    // The rows this commit starts from, loaded with the others so that the
    // thread waits for memory once: the committing worker's snapshot (unused
    // when it is the pending worker, whose pull is stored below) and its
    // moment (no earlier store of this launch touches it).
    // A row that holds theta_t is not read again: the committing worker's
    // snapshot when it is the pending worker (it pulls below) or the worker
    // whose row held theta_t.
    const bool cur_pulls_now = a.apply && a.w_cur == a.w_prev;
    float4 s_cur = make_float4(0.f, 0.f, 0.f, 0.f), m_cur = s_cur;
    if (a.start && active) {
        if (!cur_pulls_now && a.w_cur != a.theta_row)
            s_cur = load4<NT>(a.S + tile_index(a.nw, a.w_cur, off));
        m_cur = load4<NT>(a.M + tile_index(a.nw, a.m_row, off));
    }
    // The pending worker's snapshot, to generate its update again (and for
    // the diagnostics' kinetic energy).
    float* srow = a.S + tile_index(a.nw, a.w_prev, off);
    float4 sp = make_float4(0.f, 0.f, 0.f, 0.f);
    if ((SRC == Source::Generated || DIAG) && a.apply && active)
        sp = a.w_prev == a.theta_row ? th_old : load4<NT>(srow);
    double ek = 0.0, proxy = 0.0;   // diagnostic variant: energies of the pending commit
    if (a.apply && active) {
        // The pending commit's update: the caller's, or generated again at
        // the worker's snapshot, which its pull below replaces.
        float4 d;
        if (SRC == Source::Generated) {
            const float4 z = normals4(static_cast<uint64_t>(c), a.t - 1u, a.key0, a.key1);
            d.x = stale_update<BF16>(a.neg_lr, a.sigma, sp.x, hv.x, tv.x, z.x);
            d.y = stale_update<BF16>(a.neg_lr, a.sigma, sp.y, hv.y, tv.y, z.y);
            d.z = stale_update<BF16>(a.neg_lr, a.sigma, sp.z, hv.z, tv.z, z.z);
            d.w = stale_update<BF16>(a.neg_lr, a.sigma, sp.w, hv.w, tv.w, z.w);
        } else {
            d = load_given<SRC>(a.upd_prev, c, a.P);
        }
        // eq. 3 with the factor of each element's segment (padding stays put)
        if (one_seg) {
            if (off + 0 < a.P) th.x = __builtin_fmaf(pi_one, d.x, th.x);
            if (off + 1 < a.P) th.y = __builtin_fmaf(pi_one, d.y, th.y);
            if (off + 2 < a.P) th.z = __builtin_fmaf(pi_one, d.z, th.z);
            if (off + 3 < a.P) th.w = __builtin_fmaf(pi_one, d.w, th.w);
        } else {
            int32_t seg = s_first;
            auto factor = [&](int64_t i) {
                while (a.seg_off[seg + 1] <= i) ++seg;
                return a.pi_seg[seg];
            };
            if (off + 0 < a.P) th.x = __builtin_fmaf(factor(off + 0), d.x, th.x);
            if (off + 1 < a.P) th.y = __builtin_fmaf(factor(off + 1), d.y, th.y);
            if (off + 2 < a.P) th.z = __builtin_fmaf(factor(off + 2), d.z, th.z);
            if (off + 3 < a.P) th.w = __builtin_fmaf(factor(off + 3), d.w, th.w);
        }
        store4<NT>(srow, pick(a.pre_pull, th_old, th));
        if (DIAG) {
            // E_k against the worker's snapshot (eq. 11) and the proxy energy
            // (eq. 22) of the pending commit, whose moment is already stored.
            const float4 mp = f4(a.M + tile_index(a.nw, a.m_row_prev, off));
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                if (off + k < a.P) {
                    const double e = static_cast<double>(lane(th, k)) - static_cast<double>(lane(sp, k));
                    const double km = static_cast<double>(a.k_eff) * static_cast<double>(lane(mp, k));
                    ek += 0.5 * e * e;
                    proxy += 0.5 * km * km;
                }
            }
        }
    }
    if (DIAG && a.apply) {   // uniform: every thread of the block takes part
        const double bek = block_tree_sum(ek, lds[0]);
        const double bpr = block_tree_sum(proxy, lds[1]);
        if (threadIdx.x == 0) {
            atomicAdd(&a.diag[0], bek);
            atomicAdd(&a.diag[1], bpr);
        }
    }
    if (!a.start) {
        if (active && a.store_theta) store4<NT>(a.theta + off, th);
        return;
    }

    float4 s, d, mo;
    mo = make_float4(0.f, 0.f, 0.f, 0.f);
    s = mo;
    d = mo;
    if (active) {
        if (cur_pulls_now) s = pick(a.pre_pull, th_old, th);   // just pulled
        else if (a.w_cur == a.theta_row) s = th_old;
        else s = s_cur;
        if (SRC == Source::Generated) {
            const float4 z = normals4(static_cast<uint64_t>(c), a.t, a.key0, a.key1);
            d.x = stale_update<BF16>(a.neg_lr, a.sigma, s.x, hv.x, tv.x, z.x);
            d.y = stale_update<BF16>(a.neg_lr, a.sigma, s.y, hv.y, tv.y, z.y);
            d.z = stale_update<BF16>(a.neg_lr, a.sigma, s.z, hv.z, tv.z, z.z);
            d.w = stale_update<BF16>(a.neg_lr, a.sigma, s.w, hv.w, tv.w, z.w);
        } else {
            d = load_given<SRC>(a.upd_cur, c, a.P);
        }
        float* mrow = a.M + tile_index(a.nw, a.m_row, off);
        mo = m_cur;
        float4 m;
        m.x = __builtin_fmaf(a.mu, mo.x, d.x);     // Alg. 1: m <- mu m + dtheta
        m.y = __builtin_fmaf(a.mu, mo.y, d.y);
        m.z = __builtin_fmaf(a.mu, mo.z, d.z);
        m.w = __builtin_fmaf(a.mu, mo.w, d.w);
        store4<NT>(mrow, m);
        if (a.store_theta) store4<NT>(a.theta + off, th);
        mo = m;
    }
    // Terms of the sums of squares: drift theta_t - s_t (eq. 16), m and d.
    double ta[4], tm[4], td[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const double dr = static_cast<double>(lane(th, k) - lane(s, k));
        const double mk = static_cast<double>(lane(mo, k));
        const double dk = static_cast<double>(lane(d, k));
        ta[k] = dr * dr;
        tm[k] = mk * mk;
        td[k] = dk * dk;
    }
    // One set of group sums per segment the group touches (terms outside the
    // segment count as zero); the loop is uniform across the block.
    for (int32_t seg = s_first; seg == s_first || a.seg_off[seg] < g_hi; ++seg) {
        const int64_t lo = seg == s_first ? s_lo : a.seg_off[seg];
        const int64_t hi = seg == s_first ? s_hi : a.seg_off[seg + 1];
        double ca = 0.0, cm = 0.0, cd = 0.0;
        if (one_seg && g_lo + kSegGroup <= a.P) {
            // the whole group inside one segment and below P: no masks
            ca = (ta[0] + ta[1]) + (ta[2] + ta[3]);
            cm = (tm[0] + tm[1]) + (tm[2] + tm[3]);
            cd = (td[0] + td[1]) + (td[2] + td[3]);
        } else if (active) {
            double xa[4], xm[4], xd[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const bool in = off + k >= lo && off + k < hi;
                xa[k] = in ? ta[k] : 0.0;
                xm[k] = in ? tm[k] : 0.0;
                xd[k] = in ? td[k] : 0.0;
            }
            ca = (xa[0] + xa[1]) + (xa[2] + xa[3]);
            cm = (xm[0] + xm[1]) + (xm[2] + xm[3]);
            cd = (xd[0] + xd[1]) + (xd[2] + xd[3]);
        }
        // The wave's 256-index subtree (lane butterflies add pairs 2k, 2k+1,
        // then pairs of pairs, ...); seg_blocks_kernel adds the group's four
        // wave sums as (w0 + w1) + (w2 + w3), the next level of the same
        // tree.  No barrier: each wave writes its own slot.
#pragma unroll
        for (int mask = 1; mask < 64; mask <<= 1) {
            ca = ca + __shfl_xor(ca, mask);
            cm = cm + __shfl_xor(cm, mask);
            cd = cd + __shfl_xor(cd, mask);
        }
        if ((threadIdx.x & 63) == 0) {
            const int64_t q = (a.part_off[seg] + (grp - (lo / kSegGroup))) * kWavesPerGroup +
                              (threadIdx.x >> 6);
            const int64_t stride = a.npart * kWavesPerGroup;
            a.part[q] = ca;
            a.part[stride + q] = cm;
            a.part[2 * stride + q] = cd;
        }
        if (one_seg) break;
    }
}

// The lanes of one wave see each other's LDS writes made before this point.
__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One wave (threadIdx.x < 64): add segment seg's index-block sums in
// increasing order (the lanes load 64 at a time into LDS; lane 0 adds them
// in order), take the norms (binary64 square root,
// rounded to binary32) and form pi as in the element step (eq. 18 with norms).
__device__ void reduce_segment(int32_t seg, const double* sup, int64_t nsup,
                               const int64_t* __restrict__ sup_off, float* __restrict__ pi_seg,
                               float k_eff, float eps, int32_t literal,
                               const int64_t* __restrict__ seg_off, uint32_t* hist,
                               int32_t hist_per_seg, double* diag, double (*tail)[64])
{
    const int64_t q0 = sup_off[seg], q1 = sup_off[seg + 1];
    double sa = 0.0, sm = 0.0, sd = 0.0;
    for (int64_t base = q0; base < q1; base += 64) {
        // the lanes load 64 block sums of each kind at once into LDS; lane 0
        // then adds them in order (one wave: its LDS accesses stay in order)
        const int64_t q = base + threadIdx.x;
        if (q < q1) {
            tail[0][threadIdx.x] = sup[q];
            tail[1][threadIdx.x] = sup[nsup + q];
            tail[2][threadIdx.x] = sup[2 * nsup + q];
        }
        wave_sync();
        if (threadIdx.x == 0) {
            const int cnt = (q1 - base < 64) ? static_cast<int>(q1 - base) : 64;
            for (int k = 0; k < cnt; ++k) {
                sa = sa + tail[0][k];
                sm = sm + tail[1][k];
                sd = sd + tail[2][k];
            }
        }
        wave_sync();
    }
    if (threadIdx.x != 0) return;
    const float na = static_cast<float>(sqrt(sa));
    const float nm = static_cast<float>(sqrt(sm));
    const float nd = static_cast<float>(sqrt(sd));
    const float num = k_eff * nm - na;
    const float den = nd + eps;
    const float pi_raw = num / den;
    const float pi = (literal || pi_raw > 0.0f) ? pi_raw : 0.0f;
    pi_seg[seg] = pi;
    if (diag) {   // clamped elements (raw pi negative or NaN) and elements
        const double size = static_cast<double>(seg_off[seg + 1] - seg_off[seg]);
        if (!(pi_raw >= 0.0f)) atomicAdd(&diag[2], size);
        atomicAdd(&diag[3], size);
    }
    // Recording: every element of the segment takes this factor, so its
    // histogram entry is one bin holding the segment's size.
    if (hist) {
        uint32_t* row = hist + (hist_per_seg ? static_cast<int64_t>(seg) * GEM_PI_BINS : 0);
        atomicAdd(&row[scale_bin(pi)], static_cast<uint32_t>(seg_off[seg + 1] - seg_off[seg]));
    }
}

// The tree's upper levels and the factors: one block per (segment, aligned
// block of kSegBlock indices) pair adds the 256 group sums of that index
// block -- zero for groups outside the segment -- by the same adjacent-pairs
// tree.  The last of a segment's pair blocks to finish (a device-scope
// counter per segment, its sums released and acquired by device fences)
// then reduces the segment's index-block sums and forms its factor; it also
// resets the counter for the next launch.  Which block is last does not
// change any sum: each is taken in one fixed order.
__global__ __launch_bounds__(kBlock) void seg_blocks_kernel(const double* __restrict__ part,
                                                            int64_t npart,
                                                            const int64_t* __restrict__ part_off,
                                                            const int64_t* __restrict__ seg_off,
                                                            const int32_t* __restrict__ pair_seg,
                                                            const int32_t* __restrict__ pair_blk,
                                                            double* sup, int64_t nsup,
                                                            const int64_t* __restrict__ sup_off,
                                                            uint32_t* seg_done, SegFactors f)
{
    static_assert(kBlock * kSegGroup == kSegBlock, "one thread per group of an index block");
    __shared__ double lds[3][4];
    __shared__ double tail[3][64];
    __shared__ int last;
    const int32_t seg = pair_seg[blockIdx.x];
    const int64_t blk = pair_blk[blockIdx.x];
    const int64_t g_lo = seg_off[seg] / kSegGroup;
    const int64_t g_hi = (seg_off[seg + 1] - 1) / kSegGroup;
    const int64_t grp = blk * kBlock + threadIdx.x;
    double va = 0.0, vm = 0.0, vd = 0.0;
    if (grp >= g_lo && grp <= g_hi) {
        // the group's four wave sums, (w0 + w1) + (w2 + w3)
        static_assert(kWavesPerGroup == 4, "four waves per group");
        const int64_t q = (part_off[seg] + (grp - g_lo)) * kWavesPerGroup;
        const int64_t stride = npart * kWavesPerGroup;
        const double* pa = part + q;
        const double* pm = part + stride + q;
        const double* pd = part + 2 * stride + q;
        va = (pa[0] + pa[1]) + (pa[2] + pa[3]);
        vm = (pm[0] + pm[1]) + (pm[2] + pm[3]);
        vd = (pd[0] + pd[1]) + (pd[2] + pd[3]);
    }
    double sa = va, sm = vm, sd = vd;
    block_tree_sum3(sa, sm, sd, lds);
    if (threadIdx.x == 0) {
        const int64_t q = sup_off[seg] + (blk - seg_off[seg] / kSegBlock);
        sup[q] = sa;
        sup[nsup + q] = sm;
        sup[2 * nsup + q] = sd;
        __threadfence();   // release this block's sums to every XCD
        const uint32_t pairs = static_cast<uint32_t>(sup_off[seg + 1] - sup_off[seg]);
        const uint32_t done = atomicAdd(&seg_done[seg], 1u) + 1u;
        last = done == pairs;
        if (done == pairs) atomicExch(&seg_done[seg], 0u);
    }
    __syncthreads();
    if (!last) return;
    __threadfence();       // acquire the other blocks' sums
    if (threadIdx.x < 64)
        reduce_segment(seg, sup, nsup, sup_off, f.pi_seg, f.k_eff, f.eps, f.literal, seg_off,
                       f.hist, f.hist_per_seg, f.diag, tail);
}

template <bool BF16>
__global__ __launch_bounds__(kBlock) void generate_kernel(const float* __restrict__ S, int64_t nw,
                                                         int32_t w, const float* __restrict__ h,
                                                         const float* __restrict__ ts, void* out,
                                                         int64_t P, uint32_t t, uint32_t key0,
                                                         uint32_t key1, float neg_lr, float sigma)
{
    const int64_t c = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const int64_t i0 = c * 4;
    if (i0 >= P) return;
    const float4 s = *reinterpret_cast<const float4*>(S + tile_index(nw, w, i0));
    const float4 hv = *reinterpret_cast<const float4*>(h + i0);
    const float4 tv = *reinterpret_cast<const float4*>(ts + i0);
    const float4 z = normals4(static_cast<uint64_t>(c), t, key0, key1);
    float d[4];
    d[0] = stale_update<BF16>(neg_lr, sigma, s.x, hv.x, tv.x, z.x);
    d[1] = stale_update<BF16>(neg_lr, sigma, s.y, hv.y, tv.y, z.y);
    d[2] = stale_update<BF16>(neg_lr, sigma, s.z, hv.z, tv.z, z.z);
    d[3] = stale_update<BF16>(neg_lr, sigma, s.w, hv.w, tv.w, z.w);
    if (BF16) {
        uint16_t* o = static_cast<uint16_t*>(out);
        if (i0 + 4 <= P) {
            uint2 u;
            u.x = (__float_as_uint(d[0]) >> 16) | (__float_as_uint(d[1]) & 0xFFFF0000u);
            u.y = (__float_as_uint(d[2]) >> 16) | (__float_as_uint(d[3]) & 0xFFFF0000u);
            *reinterpret_cast<uint2*>(o + i0) = u;
        } else {
            for (int k = 0; k < 4; ++k)
                if (i0 + k < P) o[i0 + k] = static_cast<uint16_t>(__float_as_uint(d[k]) >> 16);
        }
    } else {
        float* o = static_cast<float*>(out);
        if (i0 + 4 <= P) {
            *reinterpret_cast<float4*>(o + i0) = make_float4(d[0], d[1], d[2], d[3]);
        } else {
            for (int k = 0; k < 4; ++k)
                if (i0 + k < P) o[i0 + k] = d[k];
        }
    }
}

// Rows w0 .. w0 + rows - 1 of the table pieces at base, over [0, Pp): set to
// row (16-byte aligned), or to zero when row is null.
__global__ __launch_bounds__(kBlock) void fill_rows_kernel(float* base, int64_t nw, int32_t w0,
                                                           int32_t rows, int64_t Pp,
                                                           const float* row)
{
    const int64_t nchunk = Pp >> 2;
    const int64_t c = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (c >= nchunk) return;
    const float4 v = row ? reinterpret_cast<const float4*>(row)[c] : make_float4(0.f, 0.f, 0.f, 0.f);
    for (int32_t r = 0; r < rows; ++r)
        *reinterpret_cast<float4*>(base + tile_index(nw, w0 + r, c * 4)) = v;
}

// out[i] = worker w's element i of the table pieces at base, i < P (out of
// any alignment).
__global__ __launch_bounds__(kBlock) void read_row_kernel(const float* __restrict__ base,
                                                          int64_t nw, int32_t w, int64_t P,
                                                          float* __restrict__ out)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (i < P) out[i] = base[tile_index(nw, w, i)];
}

__global__ __launch_bounds__(kBlock) void gather_kernel(const float* __restrict__ src,
                                                        const int64_t* __restrict__ idx,
                                                        int64_t count, float* __restrict__ out)
{
    const int64_t k = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (k < count) out[k] = src[idx[k]];
}

// out[w * count + k] = worker w's element idx[k] of the table pieces at base,
// for workers w = w0 + blockIdx.y.
__global__ __launch_bounds__(kBlock) void gather_rows_kernel(const float* __restrict__ base,
                                                             int64_t nw, int64_t w0,
                                                             const int64_t* __restrict__ idx,
                                                             int64_t count, float* __restrict__ out)
{
    const int64_t k = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const int64_t w = w0 + blockIdx.y;
    if (k < count) out[w * count + k] = base[tile_index(nw, w, idx[k])];
}

__global__ __launch_bounds__(kBlock) void loss_kernel(const float* __restrict__ theta,
                                                      const float* __restrict__ h,
                                                      const float* __restrict__ ts, int64_t P,
                                                      double* out)
{
    __shared__ double red[kBlock];
    double acc = 0.0;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < P;
         i += static_cast<int64_t>(gridDim.x) * kBlock) {
        const double e = static_cast<double>(theta[i]) - static_cast<double>(ts[i]);
        acc += 0.5 * static_cast<double>(h[i]) * e * e;
    }
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int step = kBlock / 2; step > 0; step >>= 1) {
        if (static_cast<int>(threadIdx.x) < step) red[threadIdx.x] += red[threadIdx.x + step];
        __syncthreads();
    }
    if (threadIdx.x == 0) atomicAdd(out, red[0]);
}

// Plain copy, the bandwidth reference: one 16-byte chunk per thread and
// trip of a grid-stride loop whose grid covers the whole copy up to 4 GiB
// (2^20 blocks), with non-temporal loads and stores.  On MI355X this moves
// 6.5-6.6 TB/s of reads plus writes; default-policy accesses reach 6.2 TB/s,
// and tiles of four chunks per thread 5.6 TB/s.
__global__ __launch_bounds__(kBlock) void copy_kernel(const float* __restrict__ src,
                                                      float* __restrict__ dst, int64_t count)
{
    const int64_t n4 = count / 4;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    const int64_t first = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    for (int64_t k = first; k < n4; k += stride) store4<true>(dst + 4 * k, load4<true>(src + 4 * k));
    if (first < count - n4 * 4) dst[n4 * 4 + first] = src[n4 * 4 + first];
}

inline unsigned blocks_for(int64_t items) {
    return static_cast<unsigned>((items + kBlock - 1) / kBlock);
}

// lds: bytes of dynamic LDS reserved per block (unused by the kernel), which
// caps the blocks a CU holds at once.
template <Source SRC, Variant V, bool BF16, bool DIAG, int DEPTH, bool NT, bool REC = false>
hipError_t launch_one(const PassArgs& a, hipStream_t st, uint32_t lds = 0)
{
    if (REC) {
        // K histograms, then one spare word per thread
        const uint32_t need = (static_cast<uint32_t>(a.K) * kRecWords + kBlock) * 4u;
        lds = lds > need ? lds : need;
    }
    static_assert(DEPTH > 1 || (!REC && !DIAG), "depth 1: the plain single-commit pass");
    if (DEPTH == 1 && a.K != 1) return hipErrorInvalidValue;
    unsigned grid = blocks_for(a.Pp >> 2);
    if (REC && a.rec_grid > 0 && static_cast<unsigned>(a.rec_grid) < grid)
        grid = static_cast<unsigned>(a.rec_grid);
    hipLaunchKernelGGL((pass_kernel<SRC, V, BF16, DIAG, DEPTH, NT, REC>), dim3(grid), dim3(kBlock),
                       lds, st, a);
    return hipGetLastError();
}

// Recording passes of the default rule with per-worker moments on generated
// updates (one histogram per commit).
template <bool BF16>
hipError_t launch_rec(const PassArgs& a, int depth, bool stream, uint32_t deep_lds, hipStream_t st)
{
    constexpr Source G = Source::Generated;
    constexpr Variant F = Variant::Fast;
    if (depth == kPrefetchDeep)
        return stream ? launch_one<G, F, BF16, false, kPrefetchDeep, true, true>(a, st, deep_lds)
                      : launch_one<G, F, BF16, false, kPrefetchDeep, false, true>(a, st, deep_lds);
    if (depth != kPrefetchShallow) return hipErrorInvalidValue;
    return stream ? launch_one<G, F, BF16, false, kPrefetchShallow, true, true>(a, st)
                  : launch_one<G, F, BF16, false, kPrefetchShallow, false, true>(a, st);
}

// The diagnostic variant keeps the default cache policy.
template <Source SRC, Variant V, bool BF16>
hipError_t launch_d(const PassArgs& a, bool diag, bool stream, hipStream_t st)
{
    if (diag) return launch_one<SRC, V, BF16, true, kPrefetchShallow, false>(a, st);
    return stream ? launch_one<SRC, V, BF16, false, kPrefetchShallow, true>(a, st)
                  : launch_one<SRC, V, BF16, false, kPrefetchShallow, false>(a, st);
}

template <Source SRC, bool BF16>
hipError_t launch_fd(const PassArgs& a, Variant v, bool diag, int depth, bool stream,
                     uint32_t deep_lds, hipStream_t st)
{
    if (depth == kPrefetchDeep) {
        if constexpr (SRC == Source::Generated) {
            if (v == Variant::Fast && !diag)
                return stream ? launch_one<SRC, Variant::Fast, BF16, false, kPrefetchDeep, true>(
                                    a, st, deep_lds)
                              : launch_one<SRC, Variant::Fast, BF16, false, kPrefetchDeep, false>(
                                    a, st, deep_lds);
        }
        return hipErrorInvalidValue;
    }
    if (depth == kPrefetchNone && !diag) {
        switch (v) {
        case Variant::Fast:
            return stream ? launch_one<SRC, Variant::Fast, BF16, false, kPrefetchNone, true>(a, st)
                          : launch_one<SRC, Variant::Fast, BF16, false, kPrefetchNone, false>(a, st);
        case Variant::FastGlobal:
            return stream
                       ? launch_one<SRC, Variant::FastGlobal, BF16, false, kPrefetchNone, true>(a, st)
                       : launch_one<SRC, Variant::FastGlobal, BF16, false, kPrefetchNone, false>(a, st);
        case Variant::General: break;
        }
        return stream ? launch_one<SRC, Variant::General, BF16, false, kPrefetchNone, true>(a, st)
                      : launch_one<SRC, Variant::General, BF16, false, kPrefetchNone, false>(a, st);
    }
    if (depth != kPrefetchShallow && depth != kPrefetchNone) return hipErrorInvalidValue;
    switch (v) {
    case Variant::Fast: return launch_d<SRC, Variant::Fast, BF16>(a, diag, stream, st);
    case Variant::FastGlobal: return launch_d<SRC, Variant::FastGlobal, BF16>(a, diag, stream, st);
    case Variant::General: break;
    }
    return launch_d<SRC, Variant::General, BF16>(a, diag, stream, st);
}

}  // namespace

hipError_t launch_pass(const PassArgs& a, Source src, Variant v, bool bf16_out, bool diag,
                       bool rec, int depth, bool stream_rows, uint32_t deep_lds,
                       hipStream_t stream)
{
    if (rec) {
        if (src != Source::Generated || v != Variant::Fast || diag) return hipErrorInvalidValue;
        return bf16_out ? launch_rec<true>(a, depth, stream_rows, deep_lds, stream)
                        : launch_rec<false>(a, depth, stream_rows, deep_lds, stream);
    }
    switch (src) {
    case Source::Generated:
        return bf16_out ? launch_fd<Source::Generated, true>(a, v, diag, depth, stream_rows,
                                                             deep_lds, stream)
                        : launch_fd<Source::Generated, false>(a, v, diag, depth, stream_rows,
                                                              deep_lds, stream);
    case Source::GivenF32:
        return launch_fd<Source::GivenF32, false>(a, v, diag, depth, stream_rows, deep_lds, stream);
    case Source::GivenBF16:
        return launch_fd<Source::GivenBF16, false>(a, v, diag, depth, stream_rows, deep_lds,
                                                   stream);
    }
    return hipErrorInvalidValue;
}

template <bool DIAG, bool NT>
void launch_seg_step_d(const SegArgs& a, Source src, bool bf16_out, hipStream_t stream)
{
    const unsigned grid = blocks_for(a.Pp >> 2);
    switch (src) {
    case Source::Generated:
        if (bf16_out)
            hipLaunchKernelGGL((seg_step_kernel<Source::Generated, true, DIAG, NT>), dim3(grid),
                               dim3(kBlock), 0, stream, a);
        else
            hipLaunchKernelGGL((seg_step_kernel<Source::Generated, false, DIAG, NT>), dim3(grid),
                               dim3(kBlock), 0, stream, a);
        break;
    case Source::GivenF32:
        hipLaunchKernelGGL((seg_step_kernel<Source::GivenF32, false, DIAG, NT>), dim3(grid),
                           dim3(kBlock), 0, stream, a);
        break;
    case Source::GivenBF16:
        hipLaunchKernelGGL((seg_step_kernel<Source::GivenBF16, false, DIAG, NT>), dim3(grid),
                           dim3(kBlock), 0, stream, a);
        break;
    }
}

hipError_t launch_seg_step(const SegArgs& a, Source src, bool bf16_out, bool stream_rows,
                           hipStream_t stream)
{
    // The diagnostic variant keeps the default cache policy (one instance).
    if (a.diag) launch_seg_step_d<true, false>(a, src, bf16_out, stream);
    else if (stream_rows) launch_seg_step_d<false, true>(a, src, bf16_out, stream);
    else launch_seg_step_d<false, false>(a, src, bf16_out, stream);
    return hipGetLastError();
}

hipError_t launch_seg_blocks(const double* part, int64_t npart, const int64_t* part_off,
                             const int64_t* seg_off, const int32_t* pair_seg,
                             const int32_t* pair_blk, int64_t npairs, double* sup,
                             const int64_t* sup_off, uint32_t* seg_done, const SegFactors& f,
                             hipStream_t stream)
{
    if (npairs <= 0) return hipSuccess;
    hipLaunchKernelGGL(seg_blocks_kernel, dim3(static_cast<unsigned>(npairs)), dim3(kBlock), 0,
                       stream, part, npart, part_off, seg_off, pair_seg, pair_blk, sup, npairs,
                       sup_off, seg_done, f);
    return hipGetLastError();
}

hipError_t launch_generate(const float* S, int64_t nw, int32_t w, const float* h,
                           const float* ts, void* out, bool bf16, int64_t P, uint32_t t,
                           uint32_t key0, uint32_t key1, float neg_lr, float sigma,
                           hipStream_t stream)
{
    const unsigned grid = blocks_for((P + 3) / 4);
    if (bf16)
        hipLaunchKernelGGL(generate_kernel<true>, dim3(grid), dim3(kBlock), 0, stream, S, nw, w, h,
                           ts, out, P, t, key0, key1, neg_lr, sigma);
    else
        hipLaunchKernelGGL(generate_kernel<false>, dim3(grid), dim3(kBlock), 0, stream, S, nw, w, h,
                           ts, out, P, t, key0, key1, neg_lr, sigma);
    return hipGetLastError();
}

hipError_t launch_fill_rows(float* base, int64_t nw, int32_t w0, int32_t rows, int64_t Pp,
                            const float* row, hipStream_t stream)
{
    if (rows <= 0 || Pp <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_rows_kernel, dim3(blocks_for(Pp >> 2)), dim3(kBlock), 0, stream, base,
                       nw, w0, rows, Pp, row);
    return hipGetLastError();
}

hipError_t launch_read_row(const float* base, int64_t nw, int32_t w, int64_t P, float* out,
                           hipStream_t stream)
{
    if (P <= 0) return hipSuccess;
    hipLaunchKernelGGL(read_row_kernel, dim3(blocks_for(P)), dim3(kBlock), 0, stream, base, nw, w,
                       P, out);
    return hipGetLastError();
}

hipError_t launch_gather(const float* src, const int64_t* idx, int64_t count, float* out,
                         hipStream_t stream)
{
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(gather_kernel, dim3(blocks_for(count)), dim3(kBlock), 0, stream, src, idx,
                       count, out);
    return hipGetLastError();
}

hipError_t launch_gather_rows(const float* base, int64_t nw, const int64_t* idx, int64_t count,
                              float* out, hipStream_t stream)
{
    if (count <= 0 || nw <= 0) return hipSuccess;
    constexpr int64_t kMaxY = 65535;   // grid y limit
    for (int64_t w0 = 0; w0 < nw; w0 += kMaxY) {
        const int64_t rows = nw - w0 < kMaxY ? nw - w0 : kMaxY;
        hipLaunchKernelGGL(gather_rows_kernel, dim3(blocks_for(count), static_cast<unsigned>(rows)),
                           dim3(kBlock), 0, stream, base, nw, w0, idx, count, out);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_loss(const float* theta, const float* h, const float* ts, int64_t P, double* out,
                       hipStream_t stream)
{
    const int64_t want = blocks_for(P);
    const unsigned grid = static_cast<unsigned>(want < 4096 ? (want > 0 ? want : 1) : 4096);
    hipLaunchKernelGGL(loss_kernel, dim3(grid), dim3(kBlock), 0, stream, theta, h, ts, P, out);
    return hipGetLastError();
}

hipError_t launch_copy(const float* src, float* dst, int64_t count, hipStream_t stream)
{
    if (count <= 0) return hipSuccess;
    const int64_t want = (count / 4 + kBlock - 1) / kBlock;
    const int64_t cap = int64_t{1} << 20;
    const unsigned grid = static_cast<unsigned>(want < 1 ? 1 : want < cap ? want : cap);
    hipLaunchKernelGGL(copy_kernel, dim3(grid), dim3(kBlock), 0, stream, src, dst, count);
    return hipGetLastError();
}

}  // namespace gemk
