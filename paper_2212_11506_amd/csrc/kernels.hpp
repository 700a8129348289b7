// Host-side launchers of the device kernels (internal to the library).
#pragma once

#include "common.hpp"
#include "affinity.hpp"

namespace bht {

template <typename T> struct StepArgsT {
    T alpha;         // exaggeration of the attractive term
    T learning_rate; // eta
    T momentum;      // mu
    T min_gain;
    int update;      // 0: gradient only
};
using StepArgs = StepArgsT<float>;

// Optional per-node exports of the tree (device arrays of at least 2n entries).
struct TreeDebug {
    uint8_t *level = nullptr;
    uint8_t *kind = nullptr; // 0 internal, 1 bucket, 2 single point
    uint32_t *begin = nullptr;
    uint32_t *end = nullptr;
};

// Device arrays of a locality layout (relabelled copy of P) inside caller memory.
struct LayoutView {
    uint32_t *perm = nullptr; // new position -> original index
    uint32_t *rank = nullptr; // original index -> new position
    int64_t *row_ptr = nullptr;
    int32_t *col = nullptr;
    float *val = nullptr;           // fp32 values (fp32 layouts)
    double *val64 = nullptr;        // the same region as fp64 values (the fp64 variant's layouts)
    // tiled copy: rows in blocks of kTileRows, columns in segments of 128 KB of
    // Y (kTileSeg fp32 points, kTileSeg / 2 fp64 points); one tile = (row
    // block, segment), sliced into units of 64 rows
    int32_t *blk_seg_lo = nullptr;  // [blocks] first segment of a row block
    int32_t *blk_nseg = nullptr;    // [blocks] segments of a row block (0: none)
    int32_t *blk_tiles = nullptr;   // [blocks * max_tiles_per_block] tile of (row block, k-th segment)
    int32_t *tile_blk = nullptr;    // [max tiles] row block of a tile; tiles are segment-major
    int32_t *tile_seg = nullptr;    // [max tiles] segment of a tile
    int32_t *tile_k = nullptr;      // [max tiles] segment of a tile counted from its block's first
    int2 *item_tiles = nullptr;     // [items] tiles [x, y) of an item (one segment), largest item first
    int32_t *run_len = nullptr;     // [max tiles * kTileRows] entries of a row in a tile's segment
    uint16_t *tperm = nullptr;      // [max tiles * kTileRows] sorted position -> row in the block
    uint16_t *tpos = nullptr;       // [max tiles * kTileRows] row in the block -> sorted position
    int32_t *unit_of = nullptr;     // [max units] unit (tile * 16 + slice) -> stored unit
    int32_t *unit_chunks = nullptr; // [max units] chunks of a stored unit
    int32_t *unit_tj = nullptr;     // [max units] tile * 16 + slice of a stored unit
    int32_t *unit_chunk0 = nullptr; // [max units] first chunk of a stored unit
    int4 *item_units = nullptr;     // [items] stored units [x, z) of an item, those from y on empty
    int4 *wave_units = nullptr;     // [items * 16] units [x, y) and chunks [z, z + w) of a wave
    uint16_t *tcol = nullptr;       // [max entries] column offset in the segment
    float *tval = nullptr;          // [max entries]
    double *tval64 = nullptr;       // the same region as fp64 values (the fp64 variant's layouts)
    int64_t max_tiles = 0, max_entries = 0;
    // windowed row segments (built instead of the sliced copy when rows have
    // no tile locality), carved from the sliced copy's memory: per column
    // window w, the segments [wstart[w], wstart[w + 1]) of the rows that have
    // entries in it, each {row, first entry, entry count} of the relabelled CSR
    int64_t *wstart = nullptr;      // [kMaxWindows + 1]
    uint32_t *seg_row = nullptr, *seg_start = nullptr, *seg_len = nullptr;
    int64_t max_segments = 0;
    size_t bytes = 0;
};

// Host copy of the small tile tables, filled when a layout is built.
struct TilePlan {
    bool tiled = false;
    int32_t blocks = 0, tiles = 0, items = 0;
    int64_t entries = 0;
    int32_t windows = 0;   // column windows of the windowed segments (0: none)
    int64_t segments = 0;
    int32_t order = 0;     // point order of the copy: kOrderMorton or kOrderBfs
};

// point orders of a layout (within each connected component of P's graph)
constexpr int kOrderMorton = 0; // Morton code of Y (index order without Y)
constexpr int kOrderBfs = 1;    // breadth-first level from the component's root, then index
constexpr int kOrderAuto = 2;   // Morton; BFS levels when Morton gives no tiles and BFS does

template <typename T> void launch_bbox(const T *Y, int64_t n, void *ws, const Layout &L, hipStream_t st);
// perm (nullable; a layout's position -> caller's index): the private copy of
// Y in the layout's order, ycopy[i] = Y[perm[i]], instead of the caller's
template <typename T>
void launch_morton(const T *Y, int64_t n, const uint32_t *perm, void *ws, const Layout &L, hipStream_t st);
// 3-D embeddings (Y n x 3 fp32): box, cube, 63-bit codes, digit histograms and
// the private copy of Y in the caller's order, or in perm's (nullable) order
void launch_bbox_morton3(const float *Y, int64_t n, const uint32_t *perm, void *ws, const Layout &L,
                         hipStream_t st);
// ysrc: Y in the original order, gathered into Morton order by the last pass
template <typename T> void launch_sort(int64_t n, const T *ysrc, void *ws, const Layout &L, hipStream_t st);
// the same with the points' type given (float3: 3-D embeddings)
template <typename V> void launch_sort_points(int64_t n, const V *ysrc, void *ws, const Layout &L, hipStream_t st);
// theta2 = theta^2 in fp64; D = 2 with T = float (the path) or double (the
// fp64 variant), or D = 3 with T = float (3-D embeddings)
template <int D, typename T>
void launch_tree(int64_t n, double theta2, void *ws, const Layout &L, const TreeDebug &dbg, hipStream_t st);
// evaluation: exact Z and KL, results in the header's eval field
void launch_z_exact(const float *Y, int64_t n, void *ws, const Layout &L, hipStream_t st);
void launch_kl(const float *Y, const int64_t *row_ptr, const int32_t *col, const float *val, int64_t n,
               int64_t nnz, double log_z, void *ws, const Layout &L, hipStream_t st);
// the tree's records as {com, count, threshold} and documented meta words (both nullable)
void launch_tree_unpack(int64_t n, void *ws, const Layout &L, float *summary, uint32_t *meta, hipStream_t st);
void launch_tree_unpack3(int64_t n, void *ws, const Layout &L, float *summary, float *thr, uint32_t *meta,
                         hipStream_t st);
// theta^2 <= 0.49: no point accepts a cell containing it, so the walk needs no
// comparison with the lane's own leaf
inline bool repulsive_self_test(float theta) { return double(theta) * double(theta) > 0.49; }
inline bool repulsive_self_test(double theta) { return theta * theta > 0.49; }
// the same in 3-D: a cube's centre of mass lies within sqrt(3) sides of any of its points
inline bool repulsive_self_test3(float theta) { return double(theta) * double(theta) > 0.33; }
template <int D, typename T>
void launch_repulsive(int64_t n, bool self_test, void *ws, const Layout &L, hipStream_t st);
template <int D, typename T>
void launch_attract(const int64_t *row_ptr, const int32_t *col, const T *val, int64_t n, int64_t nnz,
                    const StepArgsT<T> &a, T *Y, T *upd, T *gains, T *grad, void *ws, const Layout &L, hipStream_t st);

// vbytes: 4 (fp32 values) or 8 (the fp64 variant's layouts); dim: 2, or 3
// for 3-D embeddings (fp32)
LayoutView layout_view(void *mem, int64_t n, int64_t nnz, int vbytes = 4, int dim = 2);
// Builds the layout in the point order `order` (kOrder*; synchronises the
// stream); fills *plan with the tile tables' sizes and the order taken.
// Returns 0, 1 when P's row pointers are malformed (nothing else was read), or -1 on a HIP error.
// V = double: fp64 values, the sliced copy over 8192-point windows (up to 32 per row block).
// D = 3 (V = float, Y n x 3): the same over 8192-point windows of 3-D points;
// no windowed segments (plan->windows stays 0).
template <typename V, int D = 2>
int launch_layout_build(const int64_t *row_ptr, const int32_t *col, const V *val, int64_t n, int64_t nnz,
                        const V *Y, int order, const LayoutView &lv, TilePlan *plan, void *ws, const Layout &L,
                        hipStream_t st);
// attraction through windowed segments: F_attr in layout order (ws fattr)
template <typename T>
void launch_attract_windows(const LayoutView &lv, int64_t n, int blocks, int windows, void *ws, const Layout &L,
                            hipStream_t st);
// Attractive forces through a layout: the streaming tile kernel when the
// layout has tiles (tiles > 0, items > 0), else the row-block kernel.
// `blocks`: grid of the persistent sliced kernel (items are taken from a counter)
template <typename T>
void launch_attract_layout(const LayoutView &lv, int64_t n, int64_t nnz, int tiles, int items, int blocks,
                           int max_segs, int windows, void *ws, const Layout &L, hipStream_t st);
template <typename T>
void launch_update(const LayoutView &lv, int64_t n, bool layout_order, const StepArgsT<T> &a, T *Y, T *upd, T *gains,
                   T *grad, void *ws, const Layout &L, hipStream_t st);
// 3-D layouts: the sliced tile kernel and the row sums (F_attr in the
// caller's order), then the gradient and update from F_attr and F_rep
void launch_attract_layout3(const LayoutView &lv, int64_t n, int tiles, int items, int blocks, void *ws,
                            const Layout &L, hipStream_t st);
void launch_update3(int64_t n, const StepArgsT<float> &a, float *Y, float *upd, float *gains, float *grad, void *ws,
                    const Layout &L, hipStream_t st);

// input similarities from neighbour lists: clear, the index work (own-row
// order, pair sort, inbox offsets, union counts, row pointers with row_ptr[n]
// = nnz) and the search; then, once the caller's arrays are known to hold nnz
// entries, the rows of P
void launch_aff_clear(void *ws, const AffLayout &A, hipStream_t st);
void launch_aff_search(const float *dist, int64_t n, int k, double perplexity, double *sigma2, void *ws,
                       const AffLayout &A, hipStream_t st);
void launch_aff_index(const int32_t *idx, int64_t n, int k, int64_t *row_ptr, void *ws, const AffLayout &A,
                      hipStream_t st);
void launch_aff_back(int64_t n, int k, const int64_t *row_ptr, int32_t *col, float *val, void *ws,
                     const AffLayout &A, hipStream_t st);

} // namespace bht
