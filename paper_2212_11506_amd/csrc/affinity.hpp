// Workspace layout and limits of the input-similarity call (bhtsne_affinities).
#pragma once
#include "common.hpp"

namespace bht {

constexpr int kAffMaxK = 256;      // neighbours per point, at most
constexpr int kAffLongCap = 4096;  // entries of one row of the symmetric P, at most
constexpr int kAffScanTileRows = 1024;
constexpr int kAffLaneMaxK = 128;  // up to this many neighbours, one point per lane in the search

struct AffLayout {
    int64_t n, k, scan_tiles;
    size_t header, sp, scol, indeg, cursor, ib, in_col, in_p, inonly, part, longrows, counters, dT, total;
};

inline AffLayout make_aff_layout(int64_t n, int64_t k)
{
    AffLayout A{};
    A.n = n;
    A.k = k;
    A.scan_tiles = (n + kAffScanTileRows - 1) / kAffScanTileRows;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off = align_up(off + bytes, 256);
        return o;
    };
    A.header = take(sizeof(Header));
    A.sp = take(8 * size_t(n) * size_t(k));      // p_{j|i}, then in column order
    A.scol = take(4 * size_t(n) * size_t(k));    // neighbours in column order
    A.indeg = take(4 * size_t(n));               // entries of each point's inbox
    A.cursor = take(4 * size_t(n));
    A.ib = take(8 * size_t(n + 1));              // inbox offsets
    A.in_col = take(4 * size_t(n) * size_t(k));  // inboxes: listing point, p
    A.in_p = take(8 * size_t(n) * size_t(k));
    A.inonly = take(4 * size_t(n));              // inbox entries not in the own list
    A.part = take(8 * size_t(A.scan_tiles + 1));
    A.longrows = take(4 * size_t(n));
    A.counters = take(16);
    A.dT = take(k <= kAffLaneMaxK ? 4 * size_t(n) * size_t(k) : 0); // distances by neighbour, then point
    A.total = off;
    return A;
}

} // namespace bht
