// Host-logic check of the fused pass's routes (gem_plan.hpp), on the CPU.
//
// Plans many commit sequences into passes the way the library does, then
// replays every pass the way the pass kernel moves one thread's (snapshot,
// moment) chunks: the prefetch ring filled depth commits ahead, the register
// slots, and each step's store before its prefetch load.  A chunk is tracked
// as (worker, version), the version counting the worker's commits applied to
// it.  Every commit must see its worker's latest version; after each pass
// memory must hold every worker's latest version and no slot may stay full;
// the planner's read and write counts must equal the replay's.
//
// Usage: plan_driver [seed] -- prints one summary line and "ok", or a
// failure description and exit status 1.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "../paper_1805_08469_amd/csrc/gem_plan.hpp"

namespace {

struct Chunk {
    int worker = -1;   // -1: the sink (no chunk)
    int version = 0;
};

int g_fail = 0;

void fail(const char* what, int pass_start, int j)
{
    if (g_fail++ < 10) std::printf("FAIL: %s (pass at %d, commit %d)\n", what, pass_start, j);
}

// Replays one planned pass; mem[w] and cur[w] hold the versions in memory and
// the latest version of each worker.
void replay(const int32_t* w, int k, int depth, const uint32_t* routes, int reads, int writes,
            std::vector<int>& mem, std::vector<int>& cur, int start)
{
    using namespace gemk;
    Chunk ring[8];
    Chunk slot[kHeldSlots];
    bool full[kHeldSlots] = {};
    int n_reads = 0, n_writes = 0;
    for (int u = 0; u < depth; ++u) {
        if (u < k && (routes[u] & kRouteSlotMask) == kFromRing) {
            ring[u] = Chunk{w[u], mem[w[u]]};
            ++n_reads;
        }
    }
    for (int j = 0; j < k; ++j) {
        const uint32_t src = routes[j] & kRouteSlotMask;
        const uint32_t dst = (routes[j] >> kRouteDstShift) & kRouteSlotMask;
        Chunk c;
        if (src == kFromRing) {
            c = ring[j % depth];
        } else if (src < static_cast<uint32_t>(kHeldSlots) && full[src]) {
            c = slot[src];
            full[src] = false;
        } else {
            fail("source slot is empty or out of range", start, j);
            return;
        }
        if (c.worker != w[j]) fail("commit reads another worker's chunk", start, j);
        if (c.version != cur[w[j]]) fail("commit reads a stale chunk", start, j);
        c.version = ++cur[w[j]];
        if (dst == kToMemory) {
            mem[w[j]] = c.version;
            ++n_writes;
        } else if (dst < static_cast<uint32_t>(kHeldSlots) && !full[dst]) {
            slot[dst] = c;
            full[dst] = true;
        } else {
            fail("destination slot is busy or out of range", start, j);
            return;
        }
        // The step's store (above) precedes its prefetch for commit j + depth.
        const int jn = j + depth;
        const bool needs = jn < k && (routes[jn] & kRouteSlotMask) == kFromRing;
        const bool pf = (routes[j] & kRoutePrefetch) != 0;
        if (pf != needs) fail("prefetch flag disagrees with the later commit's source", start, j);
        if (pf && jn < k) {
            ring[j % depth] = Chunk{w[jn], mem[w[jn]]};
            ++n_reads;
        } else {
            ring[j % depth] = Chunk{};
        }
    }
    for (int q = 0; q < kHeldSlots; ++q)
        if (full[q]) fail("a chunk is left in a register slot", start, k);
    for (int j = 0; j < k; ++j)
        if (mem[w[j]] != cur[w[j]]) fail("memory misses a worker's last version", start, j);
    if (n_reads != reads || n_writes != writes) fail("read / write counts differ", start, -1);
}

struct Totals {
    long passes = 0, commits = 0, lower_bound = 0, reads = 0, writes = 0, distinct = 0;
};

// Plans worker[0 .. T) into passes of at most kmax commits and replays them.
void run(const std::vector<int32_t>& worker, int n, int kmax, int depth, Totals& tot)
{
    std::vector<int> mem(n, 0), cur(n, 0);
    const int T = static_cast<int>(worker.size());
    int j0 = 0;
    uint32_t routes[gemk::kPlanMaxK];
    while (j0 < T) {
        int k = kmax < T - j0 ? kmax : T - j0;
        int reads = 0, writes = 0;
        k = gemk::plan_pass(worker.data() + j0, k, depth, routes, &reads, &writes);
        if (k < 1) {
            fail("empty pass", j0, 0);
            return;
        }
        replay(worker.data() + j0, k, depth, routes, reads, writes, mem, cur, j0);
        std::vector<bool> seen(n, false);
        for (int j = 0; j < k; ++j)
            if (!seen[worker[j0 + j]]) { seen[worker[j0 + j]] = true; ++tot.distinct; }
        tot.reads += reads;
        tot.writes += writes;
        ++tot.passes;
        j0 += k;
    }
    tot.commits += T;
    tot.lower_bound += (T + kmax - 1) / kmax;
    for (int w = 0; w < n; ++w)
        if (mem[w] != cur[w]) fail("final memory misses a version", T, w);
}

}  // namespace

int main(int argc, char** argv)
{
    const unsigned seed = argc > 1 ? static_cast<unsigned>(std::atoi(argv[1])) : 1u;
    std::mt19937 rng(seed);
    Totals tot;
    const int ks[] = {1, 2, 3, 4, 5, 7, 8, 16, 17, 31, 32};
    const int ns[] = {1, 2, 3, 4, 5, 6, 8, 12, 33, 100};
    for (int depth : {gemk::kPrefetchShallow, 3, gemk::kPrefetchDeep, 6}) {
        for (int kmax : ks) {
            for (int n : ns) {
                // uniform workers
                std::vector<int32_t> w(400);
                std::uniform_int_distribution<int> uni(0, n - 1);
                for (auto& x : w) x = uni(rng);
                run(w, n, kmax, depth, tot);
                // skewed workers (a few fast ones commit most often)
                std::geometric_distribution<int> geo(0.35);
                for (auto& x : w) x = geo(rng) % n;
                run(w, n, kmax, depth, tot);
                // runs of repeats
                for (size_t j = 0; j < w.size(); ++j) w[j] = static_cast<int32_t>((j / 3 + j % 2) % n);
                run(w, n, kmax, depth, tot);
            }
        }
        // Four workers held for a far repeat, then near repeats: eviction
        // keeps every pass whole.
        std::vector<int32_t> w;
        const int32_t block[] = {0, 1, 2, 3, 4, 4, 5, 5, 6, 6, 7, 7, 0, 1, 2, 3};
        for (int r = 0; r < 8; ++r) w.insert(w.end(), block, block + 16);
        Totals t2;
        run(w, 8, 32, depth, t2);
        if (t2.passes != 4) fail("eviction pattern cut a pass", 0, static_cast<int>(t2.passes));
        // A held chunk that cannot be evicted committed within the last
        // depth - 2 commits, so with kHeldSlots = 4 no pass is ever cut at
        // depth <= 5.  Five workers in turn at depth 6 keep four held chunks
        // due back within 5 commits: passes are cut, and stay correct.
        std::vector<int32_t> rr(320);
        for (size_t j = 0; j < rr.size(); ++j) rr[j] = static_cast<int32_t>(j % 5);
        Totals t3;
        run(rr, 5, 32, depth, t3);
        const bool cut = t3.passes > t3.lower_bound;
        if (cut != (depth > 5)) fail("round robin of five: cuts where none are possible, or none", 0, depth);
    }
    // The deep pass's LDS reservation admits kDeepBlocksPerCU blocks per CU
    // and not one more, whatever the CU's LDS size; no reservation where that
    // cannot be had.
    for (int64_t lds : {int64_t{160} << 10, int64_t{64} << 10, int64_t{96} << 10}) {
        const int64_t b = gemk::deep_lds_bytes(lds);
        if (!(b > 0 && (b + 4096) * gemk::kDeepBlocksPerCU <= lds &&
              b * (gemk::kDeepBlocksPerCU + 1) > lds))
            fail("LDS reservation does not cap the deep pass", 0, static_cast<int>(lds >> 10));
    }
    if (gemk::deep_lds_bytes(0) != 0 || gemk::deep_lds_bytes(2048) != 0)
        fail("LDS reservation on a CU without room for it", 0, 0);
    std::printf("passes %ld (lower bound %ld) commits %ld row reads %ld writes %ld distinct %ld\n",
                tot.passes, tot.lower_bound, tot.commits, tot.reads, tot.writes, tot.distinct);
    if (g_fail) {
        std::printf("%d failures\n", g_fail);
        return 1;
    }
    std::printf("ok\n");
    return 0;
}
