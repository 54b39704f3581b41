// gem_layout.hpp -- layout of the snapshot and moment table in device memory.
// No HIP dependency: the host-logic tests compile it on the CPU; hipcc treats
// the constexpr functions as host and device functions.
#pragma once

#include <stdint.h>

namespace gemk {

// Layout of the snapshot and moment table.  The index range is cut into tiles
// of kTileElems elements; tile by tile, and within a tile worker by worker,
// the table holds the worker's snapshot piece of the tile followed by its
// moment piece:
//   S_w[i] = table[tile_index(n, w, i)],  M_w[i] = table[tile_index(n, w, i) + kTileElems].
// A committing worker's two pieces of a tile are one 64 KiB span, and every
// row a tile can need lies in one n * 64 KiB span.  Measured on MI355X, the
// fused pass streams its rows 6-11% faster this way than from separate
// row-major snapshot and moment tables.  Tiles of 2^13 and 2^14 elements
// measure best; 2^11, 2^12 and 2^15 are no faster than row-major rows.
constexpr int kTileShift = 13;
constexpr int64_t kTileElems = int64_t{1} << kTileShift;

constexpr int64_t tile_index(int64_t n, int64_t w, int64_t i)
{
    return (((i >> kTileShift) * n + w) << (kTileShift + 1)) + (i & (kTileElems - 1));
}

// Elements of the table for n workers over Pp indices (whole tiles).
constexpr int64_t table_elems(int64_t n, int64_t Pp)
{
    return ((Pp + kTileElems - 1) >> kTileShift) * n * 2 * kTileElems;
}

}  // namespace gemk
