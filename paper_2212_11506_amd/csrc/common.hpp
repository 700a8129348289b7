// Shared device-side definitions of the BH t-SNE gradient library (gfx950).
//
// Workspace layout, node record format and small wave64 helpers used by the
// kernels in this directory.  Nothing here is visible through the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace bht {

constexpr int kWave = 64;
constexpr int kRadixBits = 8;
constexpr int kRadix = 1 << kRadixBits;
constexpr int kSortPasses = 64 / kRadixBits;
constexpr int kSortBlock = 256;                    // 4 waves
constexpr int kSortItems = 8;                      // keys per thread
constexpr int kSortTile = kSortBlock * kSortItems; // keys per tile
// digit histograms of the sort: one copy per XCD (tile % 8), summed by the
// readers, so that the tiles' atomic adds spread over eight sets of addresses
constexpr int kHistCopies = 8;
constexpr int kHistWords = kSortPasses * (1 << kRadixBits);
constexpr int kScanBlock = 256;
constexpr int kScanItems = 4;
constexpr int kScanTile = kScanBlock * kScanItems;
constexpr int kBBoxBlocks = 512;
// evaluation kernels: the exact Z takes blocks of kZEvalPoints points, the KL
// at most kEvalMaxBlocks blocks striding over the rows
constexpr int kZEvalPoints = 2048;
constexpr int kEvalMaxBlocks = 2048;
// repulsive walk: 16 waves of consecutive points per block share one CU, so
// their walks, which overlap in most nodes, share the scalar cache's lines
constexpr int kRepBlock = 1024;
// A node of the pre-order tree: one 24-byte record
//   {com.x, com.y, count, thr, next, self}
// thr: the acceptance threshold as float bits (a cell of level L is summarised
//      for a point at squared distance d2 > thr = side(L)^2 / theta^2, +inf
//      when theta == 0; -1 for a single point, which is always taken);
// next: byte offset of the first record after the node's subtree;
// self: the sorted position of a single point, kNodeCell for a cell.
constexpr int kNodeBytes = 24;
// The fp64 variant's record: {com.x, com.y, thr (fp64), count (fp32), next,
// self, padding}, 40 bytes.
constexpr int kNodeBytes64 = 40;
// A 3-D embedding's record: {com.x, com.y, com.z, count, thr, next, self,
// padding}, 32 bytes: one scalar load of eight dwords.
constexpr int kNodeBytes3 = 32;
template <int D, typename T> constexpr int node_bytes() { return D == 3 ? kNodeBytes3 : (sizeof(T) == 8 ? kNodeBytes64 : kNodeBytes); }
constexpr uint32_t kNodeCell = 0xFFFFFFFFu;
// the 2n - 1 records end below 2^32 bytes
constexpr int64_t kMaxPoints = (int64_t(1) << 24) - 1;
constexpr int64_t kYPad = 16384 + 2;                   // padding points after the private copy of Y
// tiled attractive step: rows in blocks of kTileRows, columns in segments of
// kTileSeg points; row blocks spanning more than max_tiles_per_block segments
// keep the row-block kernel
constexpr int kTileRows = 1024;
constexpr int kTileSeg = 16384; // 128 KB of Y in LDS
constexpr int kTileMaxSeg = 16;
// Column windows of a sliced copy (points of Y held in LDS) and the tiles a
// row block may span: 16384 fp32 2-D points (128 KB), 8192 fp64 2-D points
// (128 KB) or 8192 3-D points (96 KB); the narrower windows take twice as many
// tiles, so every form covers the same column span of 2^18 points.
constexpr int window_points_of(int vbytes, int dim) { return vbytes == 4 && dim == 2 ? kTileSeg : kTileSeg / 2; }
constexpr int narrow_tiles_per_block(int vbytes, int dim = 2)
{
    return kTileMaxSeg * (kTileSeg / window_points_of(vbytes, dim));
}
// fp32 2-D row blocks may also span up to kTileWideSeg windows (2^21 points, a
// large cluster's rows) when the layout's tiles hold at least
// kTileWideEntries entries on average (four per row): sparser tiles cost more
// in partials and padding than another order or the windowed segments
constexpr int kTileWideSeg = 128;
constexpr int64_t kTileWideEntries = 4096;
constexpr int max_tiles_per_block(int vbytes, int dim = 2)
{
    return vbytes == 4 && dim == 2 ? kTileWideSeg : narrow_tiles_per_block(vbytes, dim);
}
// partial sums: kTileSlots per row, so a layout has at most kTileSlots tiles
// per row block on average
constexpr int kTileSlots = 32;
constexpr int kItemMaxTiles = 128; // tiles of one segment handled by one block
// sliced copy of a tile: 64 rows per slice (one per lane), chunks of 4 entries per lane
constexpr int kSellSlice = 64;
constexpr int kSellChunk = 4 * kSellSlice;
constexpr int kSlicesPerTile = kTileRows / kSellSlice;
// windowed segments: column windows of 2^18 points (2 MB of Y, resident in
// one XCD's 4 MB L2 beside the stream of P); n < 2^24 gives at most 64
constexpr int kWinShift = 18;
constexpr int kMaxWindows = 64;

// Status words of the decoupled look-back: 2 flag bits + 30-bit count.
constexpr uint32_t kFlagAggregate = 1u << 30;
constexpr uint32_t kFlagInclusive = 2u << 30;
constexpr uint32_t kValueMask = (1u << 30) - 1;
constexpr uint32_t kSpinLimit = 1u << 22;

// Device-side error flags (Header::flags).
constexpr uint32_t kErrNonFinite = 1u;
constexpr uint32_t kErrLookback = 2u;
constexpr uint32_t kErrRange = 4u;

// Per-call scalars, written by the kernels, read back by the host on demand.
struct Header {
    float bmin[3], bmax[3];   // bounding box (exact fp32 min/max; z only for 3-D embeddings)
    double cent[3];           // box centre
    double rspan;             // half of the widest extent
    double yroot[3];          // lower corner of the square (cube) domain
    double scale;             // 2^31 / r_span (2-D) or 2^20 / r_span (3-D); 0 when r_span == 0
    double Z;                 // normaliser of the last call
    unsigned long long interactions;
    uint32_t nodes;           // node count of the last tree
    uint32_t flags;           // kErr* bits, sticky until the host clears them
    uint32_t tile_counter[kSortPasses];
    uint32_t ticket_bbox;
    uint32_t ticket_rep;
    uint32_t attract_next; // next item of the persistent attractive kernel
    uint32_t ticket_eval;  // blocks done of an evaluation kernel (exact Z, KL)
    uint32_t max_depth;    // deepest leaf level of the last tree (32: a bucket of identical codes)
    uint32_t unsorted;     // layout build: some row's columns are not in window order
    uint32_t bfs_count[2]; // layout build: frontier sizes of the breadth-first search
    double eval;           // result of the last evaluation call
};

struct Layout {
    int64_t n, nnz, sort_tiles, scan_tiles, rep_blocks;
    size_t header, hist, bbox_part, codes0, codes1, idx0, idx1, status, ycopy, ys, levelmask,
        split_b, split_e, base, psum, scan_cnt, scan_sum, nodes, frep, fattr, partial, zpart, ipart, eval_part, total;
};

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

inline int64_t rep_blocks_for(int64_t n)
{
    int64_t b = (n + kRepBlock - 1) / kRepBlock;
    return (b + 7) / 8 * 8; // multiple of 8 for the XCD-contiguous remap
}

// `fbytes` is the size of a coordinate: 4 (fp32 path) or 8 (fp64 variant,
// which sizes the copies of Y, the node records and F_rep for fp64); `dim`
// the embedding's dimension (2, or 3 for the 3-D calls, fp32 only)
inline Layout make_layout(int64_t n, int64_t nnz, int fbytes = 4, int dim = 2)
{
    Layout L{};
    L.n = n;
    L.nnz = nnz;
    L.sort_tiles = (n + kSortTile - 1) / kSortTile;
    L.scan_tiles = (n + 1 + kScanTile - 1) / kScanTile;
    L.rep_blocks = rep_blocks_for(n);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off = align_up(off + bytes, 256);
        return o;
    };
    L.header = take(sizeof(Header));
    L.hist = take(sizeof(uint32_t) * kHistCopies * kHistWords);
    L.bbox_part = take(64 * kBBoxBlocks); // {min x, max x, min y, max y, non-finite flag}, fp32 or fp64
    L.codes0 = take(8 * size_t(n));
    L.codes1 = take(8 * size_t(n));
    L.idx0 = take(4 * size_t(n));
    L.idx1 = take(4 * size_t(n));
    L.status = take(4 * size_t(kSortPasses) * kRadix * size_t(L.sort_tiles));
    // + one LDS segment of padding: segment loads past the last point stay inside the buffer
    L.ycopy = take(size_t(dim) * size_t(fbytes) * size_t(n + kYPad));
    L.ys = take(size_t(dim) * size_t(fbytes) * size_t(n));
    L.levelmask = take(4 * size_t(n));
    L.split_b = take(4 * size_t(n));
    L.split_e = take(4 * size_t(n));
    L.base = take(4 * size_t(n + 1));
    L.psum = take(8 * size_t(dim) * size_t(n + 1));
    L.scan_cnt = take(4 * size_t(L.scan_tiles + 1));
    L.scan_sum = take(8 * size_t(dim) * size_t(L.scan_tiles + 1));
    // + 8 bytes: the 2-D walk loads 32 bytes at a record's offset
    L.nodes = take((dim == 3 ? kNodeBytes3 : (fbytes == 8 ? kNodeBytes64 : kNodeBytes)) * size_t(2 * n) + 8);
    L.frep = take(size_t(dim) * size_t(fbytes) * size_t(n));
    L.fattr = take(size_t(dim) * size_t(fbytes) * size_t(n));
    // partial attractive sums, one per (tile, sorted row slot): kTileSlots
    // tiles of kTileRows rows per row block
    L.partial = take(size_t(dim) * size_t(fbytes) * size_t((n + kTileRows - 1) / kTileRows) * kTileRows *
                     size_t(kTileSlots));
    L.zpart = take(8 * size_t(L.rep_blocks));
    const int64_t zb = (n + kZEvalPoints - 1) / kZEvalPoints;
    L.eval_part = take(8 * size_t(zb > kEvalMaxBlocks ? zb : kEvalMaxBlocks));
    L.ipart = take(8 * size_t(L.rep_blocks));
    L.total = off;
    return L;
}

template <typename T> __host__ __device__ inline T *at(void *ws, size_t off)
{
    return reinterpret_cast<T *>(static_cast<char *>(ws) + off);
}

// ---------------------------------------------------------------- wave64 helpers
__device__ inline int lane_id() { return __lane_id(); }

__device__ inline unsigned long long ballot(bool p) { return __ballot(p); }

__device__ inline uint32_t uniform(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }

template <typename T> __device__ inline T wave_sum(T v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ inline float wave_min(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o, kWave));
    return v;
}

__device__ inline float wave_max(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

__device__ inline double wave_min(double v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmin(v, __shfl_xor(v, o, kWave));
    return v;
}

__device__ inline double wave_max(double v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, kWave));
    return v;
}

__device__ inline float vmin(float a, float b) { return fminf(a, b); }
__device__ inline float vmax(float a, float b) { return fmaxf(a, b); }
__device__ inline double vmin(double a, double b) { return fmin(a, b); }
__device__ inline double vmax(double a, double b) { return fmax(a, b); }

// Geometry of the Morton tree of a D-dimensional embedding: a cell at level L
// holds the codes that share their top bits above cell_shift(L); its 2^D
// children are told apart by the D-bit digit of level L + 1.  2-D: 32 bits
// per axis interleaved into 64-bit codes, 32 levels.  3-D: 21 bits per axis
// interleaved into the low 63 bits (the top bit stays 0), 21 levels.
template <int D> struct Geom;
template <> struct Geom<2> {
    static constexpr int kBucketLevel = 32; // identical codes: a bucket cell at the last level
    __device__ static int split_level(uint64_t a, uint64_t b) { return __clzll((long long)(a ^ b)) >> 1; }
    __device__ static uint32_t digit(uint64_t code, int L) { return uint32_t(code >> (62 - 2 * L)) & 3u; }
    __device__ static int cell_shift(int L) { return 64 - 2 * L; }
};
template <> struct Geom<3> {
    static constexpr int kBucketLevel = 21;
    __device__ static int split_level(uint64_t a, uint64_t b) { return (__clzll((long long)(a ^ b)) - 1) / 3; }
    __device__ static uint32_t digit(uint64_t code, int L) { return uint32_t(code >> (60 - 3 * L)) & 7u; }
    __device__ static int cell_shift(int L) { return 63 - 3 * L; }
};

// two coordinates of the fp32 path or of the fp64 variant
template <typename T> struct Vec2;
template <> struct Vec2<float> { using type = float2; };
template <> struct Vec2<double> { using type = double2; };
template <typename T> using vec2_t = typename Vec2<T>::type;
__host__ __device__ inline float2 make_vec2(float x, float y) { return make_float2(x, y); }
__host__ __device__ inline double2 make_vec2(double x, double y) { return make_double2(x, y); }

// a point of a D-dimensional embedding with coordinates of type T
template <int D, typename T> struct PointOf;
template <> struct PointOf<2, float> { using type = float2; };
template <> struct PointOf<2, double> { using type = double2; };
template <> struct PointOf<3, float> { using type = float3; };
template <int D, typename T> using point_t = typename PointOf<D, T>::type;
__host__ __device__ inline float coord(const float2 &v, int k) { return k == 0 ? v.x : v.y; }
__host__ __device__ inline double coord(const double2 &v, int k) { return k == 0 ? v.x : v.y; }
__host__ __device__ inline float coord(const float3 &v, int k) { return k == 0 ? v.x : (k == 1 ? v.y : v.z); }
__host__ __device__ inline float2 make_point(const float *c, float2 *) { return make_float2(c[0], c[1]); }
__host__ __device__ inline double2 make_point(const double *c, double2 *) { return make_double2(c[0], c[1]); }
__host__ __device__ inline float3 make_point(const float *c, float3 *) { return make_float3(c[0], c[1], c[2]); }

// Logical block index such that each of the 8 XCDs (blocks are dealt to XCDs
// round-robin) receives one contiguous range of logical blocks.  `nblocks`
// must be a multiple of 8.
__device__ inline uint32_t xcd_contiguous(uint32_t b, uint32_t nblocks)
{
    uint32_t per = nblocks >> 3;
    return (b & 7u) * per + (b >> 3);
}

} // namespace bht
