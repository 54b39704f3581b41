// Host-logic check of the snapshot and moment table layout (gem_layout.hpp),
// on the CPU: for n workers over P indices (padded to P' = ceil(P/64)*64),
// every snapshot and moment element of every worker has its own table index,
// all indices lie inside the table, and each worker's piece of a tile is
// contiguous, its moment piece directly after its snapshot piece.
//
// Usage: layout_driver -- prints "ok", or a failure and exit status 1.
#include <cstdint>
#include <cstdio>
#include <vector>

#include "../paper_1805_08469_amd/csrc/gem_layout.hpp"

namespace {

int g_fail = 0;

void fail(const char* what, int64_t n, int64_t P, int64_t w, int64_t i)
{
    if (g_fail++ < 10)
        std::printf("FAIL: %s (n %lld, P %lld, w %lld, i %lld)\n", what, static_cast<long long>(n),
                    static_cast<long long>(P), static_cast<long long>(w), static_cast<long long>(i));
}

// Every (worker, index, snapshot or moment) visited; small tables only.
void check_all(int64_t n, int64_t P)
{
    using namespace gemk;
    const int64_t Pp = (P + 63) / 64 * 64;
    const int64_t size = table_elems(n, Pp);
    std::vector<uint8_t> hit(static_cast<size_t>(size), 0);
    for (int64_t w = 0; w < n; ++w) {
        for (int64_t i = 0; i < Pp; ++i) {
            const int64_t s = tile_index(n, w, i);
            const int64_t m = s + kTileElems;
            if (s < 0 || m >= size) {
                fail("index outside the table", n, P, w, i);
                return;
            }
            if (hit[static_cast<size_t>(s)]++ || hit[static_cast<size_t>(m)]++)
                fail("two elements share a table index", n, P, w, i);
            if ((i + 1) % kTileElems != 0 && i + 1 < Pp && tile_index(n, w, i + 1) != s + 1)
                fail("a worker's piece of a tile is not contiguous", n, P, w, i);
        }
    }
    // The table holds nothing but whole tiles of n workers' two pieces.
    if (size != ((Pp + kTileElems - 1) / kTileElems) * n * 2 * kTileElems)
        fail("table size", n, P, -1, -1);
}

// Extremes and strides of a large table.
void check_large(int64_t n, int64_t P)
{
    using namespace gemk;
    const int64_t Pp = (P + 63) / 64 * 64;
    const int64_t size = table_elems(n, Pp);
    const int64_t last = tile_index(n, n - 1, Pp - 1) + kTileElems;
    if (last != size - 1 - (kTileElems - 1 - (Pp - 1) % kTileElems))
        fail("last moment element is not at the end of the last tile", n, P, n - 1, Pp - 1);
    if (last >= size) fail("index outside the table", n, P, n - 1, Pp - 1);
    for (int64_t w = 0; w + 1 < n; ++w)
        if (tile_index(n, w + 1, 0) - tile_index(n, w, 0) != 2 * kTileElems)
            fail("workers of a tile are not 64 KiB apart", n, P, w, 0);
    if (tile_index(n, 0, kTileElems) - tile_index(n, 0, 0) != n * 2 * kTileElems)
        fail("tiles are not n * 64 KiB apart", n, P, 0, kTileElems);
}

}  // namespace

int main()
{
    static_assert(gemk::tile_index(3, 2, 8192 + 5) == (1 * 3 + 2) * 16384 + 5, "index formula");
    for (int64_t n : {1, 2, 3, 7})
        for (int64_t P : {1, 63, 64, 65, 4096, 8191, 8192, 8193, 3 * 8192 + 5})
            check_all(n, P);
    check_all(100, 8192 + 64);
    for (int64_t n : {1, 50, 100, 1000})
        for (int64_t P : {1200000, 11700000, 25000000, 124000000}) check_large(n, P);
    if (g_fail) {
        std::printf("%d failures\n", g_fail);
        return 1;
    }
    std::printf("ok\n");
    return 0;
}
