// gem_plan.hpp -- routes of the fused pass: where each commit's (snapshot,
// moment) chunk comes from and goes to.  Host code only, no HIP dependency
// (the host-logic tests compile it on the CPU).
#pragma once

#include <stdint.h>

namespace gemk {

// Per-commit route of a fused pass (host-planned, uniform across the grid).
// Bits 0-3: where the committing worker's (snapshot, moment) chunk comes from:
// a register slot 0..kHeldSlots-1 or the prefetch ring (memory).  Bits 4-7:
// where it goes: a register slot or memory.  Bit 8: prefetch the rows of
// commit j + depth, which reads them from memory.
constexpr int kHeldSlots = 4;
// How many commits ahead a step prefetches rows: the ring depth.  The deep
// ring is used by the default rule with per-worker moments on generated
// updates, in passes of at least kDeepMinK commits and without diagnostics;
// measured on MI355X it is 2-3% faster there, and 2-3% slower for the
// VALU-bound variants and for short passes, whose occupancy it lowers.
constexpr int kPrefetchShallow = 2;
constexpr int kPrefetchDeep = 4;
constexpr int kDeepMinK = 16;
// A pass of one commit needs no ring beyond that commit's own rows and no
// register slots: its kernel is compiled for exactly one commit (depth 1),
// which needs fewer registers, so more blocks fit a CU at once -- all of a
// 1.2M-parameter vector's blocks, instead of a full round and a tail.
constexpr int kPrefetchNone = 1;
// Blocks (of 256 threads, one wave per SIMD each) a CU holds at once in the
// deep-ring pass: measured on MI355X, its row streams run best with 3 waves
// per SIMD (4 are 1.8% slower, 2 are 7% slower).  The kernel needs few enough
// registers for 4, so an unused LDS reservation sets the cap: with L bytes of
// LDS per CU, a reservation just above L / (kDeepBlocksPerCU + 1) keeps the
// next block out, and stays far enough below L / kDeepBlocksPerCU that the
// allocation granularity does not push out one of the three.
constexpr int kDeepBlocksPerCU = 3;
inline uint32_t deep_lds_bytes(int64_t lds_per_cu)
{
    const int64_t b = (lds_per_cu / (kDeepBlocksPerCU + 1) / 1024 + 1) * 1024;
    const int64_t slack = 4096;   // per block, above any allocation granule
    return (b + slack) * kDeepBlocksPerCU <= lds_per_cu ? static_cast<uint32_t>(b) : 0u;
}

constexpr uint32_t kRouteSlotMask = 0xFu;
constexpr uint32_t kRouteDstShift = 4;
constexpr uint32_t kFromRing = 0xFu;
constexpr uint32_t kToMemory = 0xFu;
constexpr uint32_t kRoutePrefetch = 1u << 8;
// Longest pass the planner handles (GEM_K_MAX in gem.h).
constexpr int kPlanMaxK = 32;

inline uint32_t make_route(uint32_t src, uint32_t dst, bool prefetch)
{
    return src | (dst << kRouteDstShift) | (prefetch ? kRoutePrefetch : 0u);
}

// Routes of one pass of k <= kPlanMaxK commits for a kernel whose ring
// prefetches depth commits ahead.  A worker's chunk is read from memory at
// its first commit in the pass and written back at its last; in between it
// waits in one of kHeldSlots register slots.  When no slot is free the chunk
// is written back and re-read, which is only valid if the re-read is at least
// depth commits later: the prefetch for commit j + depth is issued right after
// commit j's store.  A nearer repeat that finds no free slot takes the slot of
// the held chunk whose next use is furthest away (Belady's rule), if that
// chunk can go back to memory instead (its re-read at least depth commits
// after its commit).  If none can, the pass has to end after commit j: the
// function then returns j + 1 and the routes are not valid; otherwise it
// returns k.  reads and writes count the row pairs that reach memory.
inline int plan_routes(const int32_t* worker, int k, int depth, uint32_t* routes, int* reads,
                       int* writes)
{
    int next[kPlanMaxK];
    for (int j = 0; j < k; ++j) {
        next[j] = -1;
        for (int q = j + 1; q < k; ++q)
            if (worker[q] == worker[j]) { next[j] = q; break; }
    }
    int held_by[kPlanMaxK];         // slot holding commit j's chunk, or -1
    int holder[kHeldSlots];         // commit whose chunk a slot holds, or -1
    for (int q = 0; q < kHeldSlots; ++q) holder[q] = -1;
    uint32_t src[kPlanMaxK], dst[kPlanMaxK];
    *reads = *writes = 0;
    for (int j = 0; j < k; ++j) {
        held_by[j] = -1;
        int prev = -1;
        for (int q = j - 1; q >= 0 && prev < 0; --q)
            if (worker[q] == worker[j]) prev = q;
        if (prev >= 0 && held_by[prev] >= 0) {
            src[j] = static_cast<uint32_t>(held_by[prev]);
            holder[held_by[prev]] = -1;
        } else {
            src[j] = kFromRing;
            *reads += 1;
        }
        dst[j] = kToMemory;
        if (next[j] >= 0) {
            int slot = -1;
            for (int q = 0; q < kHeldSlots && slot < 0; ++q)
                if (holder[q] < 0) slot = q;
            if (slot < 0 && next[j] - j < depth) {
                // Evict: the held chunk used furthest ahead goes back to memory
                // at its own commit and is read again through the ring.
                for (int q = 0; q < kHeldSlots; ++q) {
                    const int p = holder[q];
                    if (next[p] - p >= depth && (slot < 0 || next[p] > next[holder[slot]]))
                        slot = q;
                }
                if (slot < 0) return j + 1;
                const int p = holder[slot];
                dst[p] = kToMemory;
                held_by[p] = -1;
                *writes += 1;
            }
            if (slot >= 0) {
                holder[slot] = j;
                held_by[j] = slot;
                dst[j] = static_cast<uint32_t>(slot);
            }
        }
        if (dst[j] == kToMemory) *writes += 1;
    }
    for (int j = 0; j < k; ++j) {
        const int jn = j + depth;
        const bool pf = jn < k && src[jn] == kFromRing;
        routes[j] = make_route(src[j], dst[j], pf);
    }
    return k;
}

// The longest prefix of worker[0 .. k) (k <= kPlanMaxK) that plan_routes
// can route, with its routes: a shorter pass holds fewer workers at once, so
// this settles quickly.
inline int plan_pass(const int32_t* worker, int k, int depth, uint32_t* routes, int* reads,
                     int* writes)
{
    for (int fit; (fit = plan_routes(worker, k, depth, routes, reads, writes)) < k;) k = fit;
    return k;
}

}  // namespace gemk
