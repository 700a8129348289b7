// Workspace layout and limits of the input-similarity call (bhtsne_affinities).
#pragma once
#include "common.hpp"

namespace bht {

constexpr int kAffMaxK = 256;      // neighbours per point, at most
constexpr int kAffLongCap = 4096;  // entries of one row of the symmetric P, at most
constexpr int kAffScanTileRows = 1024;
constexpr int kAffLaneMaxK = 128;  // up to this many neighbours, one point per lane in the search

constexpr int kAffSortItems = 16;                          // pair keys per thread in a sort pass
constexpr int kAffSortTile = kSortBlock * kAffSortItems;   // pair keys per tile
constexpr int kAffMaxPasses = 3;                           // 8-bit digits of a point index (n < 2^24)
constexpr int kAffHistWords = kAffMaxPasses * kRadix;

// 8-bit passes that hold every pair key 0..n (a key n marks an invalid column)
inline int aff_passes(int64_t n) { return n < 256 ? 1 : n < 65536 ? 2 : 3; }

struct AffLayout {
    int64_t n, k, m, scan_tiles, sort_tiles;
    int passes;
    size_t header, p, scol, sorig, key[2], val[2], ib, inonly, part, longrows, counters, hist, status, total;
};

inline AffLayout make_aff_layout(int64_t n, int64_t k)
{
    AffLayout A{};
    A.n = n;
    A.k = k;
    A.m = n * k;
    A.scan_tiles = (n + kAffScanTileRows - 1) / kAffScanTileRows;
    A.sort_tiles = (A.m + kAffSortTile - 1) / kAffSortTile;
    A.passes = aff_passes(n);
    const size_t m = size_t(A.m);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off = align_up(off + bytes, 256);
        return o;
    };
    A.header = take(sizeof(Header));
    A.p = take(8 * m);                 // p_{j|i} in neighbour order
    A.scol = take(4 * m);              // each row's neighbours in column order
    A.sorig = take(m);                 // neighbour position of each sorted entry
    for (int b = 0; b < 2; ++b) {      // (column, entry) pairs, ping-pong buffers of the sort
        A.key[b] = take(4 * m);
        A.val[b] = take(4 * m);
    }
    A.ib = take(8 * size_t(n + 1));    // inbox offsets into the sorted pairs
    A.inonly = take(4 * size_t(n));    // inbox entries not in the own list
    A.part = take(8 * size_t(A.scan_tiles + 1));
    A.longrows = take(4 * size_t(n));
    A.counters = take(16);
    A.hist = take(4 * size_t(kHistCopies) * kAffHistWords);
    A.status = take(8 * size_t(A.passes) * size_t(A.sort_tiles) * kRadix);
    A.total = off;
    return A;
}

} // namespace bht
