// Locality layout of P and the LDS-staged attractive kernel (gfx950).
//
// Attractive Force Computation (Algorithm 2) reads, for every stored p_ij, the
// embedding point y_j of a column that P's sparsity scatters over the whole
// index range.  Those random 8-byte reads, not the stream of P itself, bound
// the row-by-row kernel.  This file renumbers the points once per matrix so
// that the columns of neighbouring rows fall into compact index windows, and
// then serves the reads from LDS:
//
//   layout build (once per P; optionally refreshed as Y evolves)
//     1. connected components of P by hooking and pointer jumping; the final
//        label of a component is its smallest vertex;
//     2. sort key = (component, Morton code of Y) -> new order `perm`;
//     3. a relabelled copy of P: rows in the new order, columns renumbered
//        and sorted within each row.
//   per iteration
//     - the Morton kernel writes Y in the new order;
//     - attract_staged_kernel: a block owns 128 consecutive rows; each 16-lane
//       group keeps up to 256 entries of a row in registers as 16-byte
//       vectors (all loads issued up front), then the block walks its column
//       span in 16384-point LDS segments (filled by direct global->LDS loads)
//       and gathers y_j from LDS;
//     - update_kernel combines F_attr, F_rep and Z in the caller's order.
//
// When the rows of a block reach too many column windows for the sliced
// copy (no tile locality: a row's neighbours spread over a large component),
// the build makes windowed row segments instead: for each column window of
// 2^18 points (2 MB of Y, held in an XCD's L2), the list of (row, entry range)
// of the rows with entries there.  The attraction then takes one launch per
// window; the y_j it gathers stay in L2 while P streams through once.
//
// The order affects only speed: any permutation gives the same sums.
#include "common.hpp"
#include "kernels.hpp"

#include <algorithm>
#include <utility>
#include <vector>

namespace bht {

// ------------------------------------------------------------------ components
__global__ __launch_bounds__(256) void cc_init_kernel(uint32_t *__restrict__ parent, int64_t n)
{
    int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) parent[i] = uint32_t(i);
}

// One wave per row: hook the larger of two different roots under the smaller.
__global__ __launch_bounds__(256) void cc_hook_kernel(const int64_t *__restrict__ row_ptr,
                                                      const int32_t *__restrict__ col, int64_t n, int64_t nnz,
                                                      uint32_t *__restrict__ parent, uint32_t *__restrict__ changed)
{
    const int lane = lane_id();
    bool hooked = false;
    for (int64_t i = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / kWave; i < n;
         i += int64_t(gridDim.x) * (blockDim.x / kWave)) {
        int64_t s = row_ptr[i], e = row_ptr[i + 1];
        s = s < 0 ? 0 : s;
        e = e > nnz ? nnz : e;
        const uint32_t pi = parent[i];
        for (int64_t k = s + lane; k < e; k += kWave) {
            const int32_t j = col[k];
            if (uint32_t(j) >= uint32_t(n)) continue;
            const uint32_t pj = parent[j];
            if (pj != pi) {
                const uint32_t hi = pi > pj ? pi : pj, lo = pi > pj ? pj : pi;
                atomicMin(&parent[hi], lo);
                hooked = true;
            }
        }
    }
    if (ballot(hooked) && lane_id() == 0) atomicOr(changed, 1u);
}

// Pointer jumping to the root; parents always point to smaller ids, so every
// chain ends.
__global__ __launch_bounds__(256) void cc_compress_kernel(uint32_t *__restrict__ parent, int64_t n)
{
    int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n) return;
    uint32_t p = parent[i];
    for (;;) {
        const uint32_t pp = parent[p];
        if (pp >= p) break;
        p = pp;
    }
    parent[i] = p;
}

__global__ void flag_clear_kernel(uint32_t *__restrict__ flag) { *flag = 0u; }

// The row pointers alone, before any column or value is read: row_ptr[0] = 0,
// non-decreasing, row_ptr[n] = nnz.  A violation latches kErrRange, and the
// build stops before it reads P's entries.
__global__ __launch_bounds__(256) void csr_check_kernel(const int64_t *__restrict__ row_ptr, int64_t n, int64_t nnz,
                                                        Header *__restrict__ hdr)
{
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i > n) return;
    const int64_t a = row_ptr[i];
    bool bad = a < 0 || a > nnz;
    if (i == 0) bad |= a != 0;
    if (i == n) bad |= a != nnz;
    else bad |= row_ptr[i + 1] < a;
    if (bad) atomicOr(&hdr->flags, kErrRange);
}

// ------------------------------------------------------------------ sort keys
// key = component (26 bits) | top 38 bits of the Morton code (or the index).
__global__ __launch_bounds__(256) void layout_keys_kernel(uint64_t *__restrict__ keys, const uint32_t *__restrict__ comp,
                                                          int64_t n, int with_morton)
{
    int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const uint64_t low = with_morton ? (keys[i] >> 26) : uint64_t(i);
    keys[i] = (uint64_t(comp[i]) << 38) | low;
}

// Breadth-first levels from every component's root (the point whose label
// is itself), all components at once: dist[v] is the number of edges on a
// shortest path from v's root along P's rows.  The frontier of a level is a
// list built by appending; its order varies between runs, the levels do not.
constexpr uint32_t kBfsUnseen = 0xffffffffu;
constexpr int kBfsMaxLevels = 16383; // the level field of the key holds 14 bits

__global__ __launch_bounds__(256) void bfs_init_kernel(const uint32_t *__restrict__ comp, int64_t n,
                                                       uint32_t *__restrict__ dist, uint32_t *__restrict__ frontier,
                                                       uint32_t *__restrict__ count)
{
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const bool root = comp[i] == uint32_t(i);
    dist[i] = root ? 0u : kBfsUnseen;
    if (root) frontier[atomicAdd(count, 1u)] = uint32_t(i);
}

// one level: a wave per frontier point labels its unseen neighbours `level +
// 1` (the compare-and-swap lets exactly one finder append each of them)
__global__ __launch_bounds__(256) void bfs_expand_kernel(const int64_t *__restrict__ row_ptr,
                                                         const int32_t *__restrict__ col, int64_t n, int64_t nnz,
                                                         const uint32_t *__restrict__ frontier, uint32_t size,
                                                         uint32_t level, uint32_t *__restrict__ dist,
                                                         uint32_t *__restrict__ next, uint32_t *__restrict__ count)
{
    const int lane = lane_id();
    for (int64_t f = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / kWave; f < int64_t(size);
         f += int64_t(gridDim.x) * (blockDim.x / kWave)) {
        const uint32_t u = frontier[f];
        int64_t s = row_ptr[u], e = row_ptr[u + 1];
        s = s < 0 ? 0 : s;
        e = e > nnz ? nnz : e;
        for (int64_t k = s + lane; k < e; k += kWave) {
            const uint32_t w = uint32_t(col[k]);
            if (w >= uint32_t(n) || dist[w] != kBfsUnseen) continue;
            if (atomicCAS(&dist[w], kBfsUnseen, level + 1) == kBfsUnseen) next[atomicAdd(count, 1u)] = w;
        }
    }
}

// key = component (26 bits) | BFS level (14 bits; unreached points last) | index (24 bits)
__global__ __launch_bounds__(256) void layout_keys_bfs_kernel(uint64_t *__restrict__ keys,
                                                              const uint32_t *__restrict__ comp,
                                                              const uint32_t *__restrict__ dist, int64_t n)
{
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const uint64_t lev = dist[i] < uint32_t(kBfsMaxLevels) ? dist[i] : uint32_t(kBfsMaxLevels);
    keys[i] = (uint64_t(comp[i]) << 38) | (lev << 24) | uint64_t(i);
}

// Global digit histograms of existing keys and the clearing of the look-back
// words (the Morton kernel does both for the codes it makes).
__global__ __launch_bounds__(kSortBlock) void keys_hist_kernel(const uint64_t *__restrict__ keys, int64_t n,
                                                               uint32_t *__restrict__ hist, uint32_t *__restrict__ status,
                                                               int64_t tiles)
{
    __shared__ uint32_t sh[kSortPasses * kRadix];
    for (int k = threadIdx.x; k < kSortPasses * kRadix; k += kSortBlock) {
        sh[k] = 0;
        status[(int64_t(k / kRadix) * tiles + blockIdx.x) * kRadix + k % kRadix] = 0;
    }
    __syncthreads();
    const int64_t base = int64_t(blockIdx.x) * kSortTile;
    for (int r = 0; r < kSortItems; ++r) {
        int64_t i = base + r * kSortBlock + threadIdx.x;
        if (i < n) {
            const uint64_t code = keys[i];
#pragma unroll
            for (int p = 0; p < kSortPasses; ++p)
                atomicAdd(&sh[p * kRadix + int((code >> (p * kRadixBits)) & (kRadix - 1))], 1u);
        }
    }
    __syncthreads();
    uint32_t *hc = hist + (blockIdx.x % kHistCopies) * kHistWords;
    for (int k = threadIdx.x; k < kSortPasses * kRadix; k += kSortBlock)
        if (sh[k]) atomicAdd(&hc[k], sh[k]);
}

__global__ void sort_reset_kernel(Header *__restrict__ hdr, uint32_t *__restrict__ hist)
{
    for (int k = threadIdx.x; k < kHistCopies * kHistWords; k += blockDim.x) hist[k] = 0;
    if (threadIdx.x == 0) {
        for (int k = 0; k < kSortPasses; ++k) hdr->tile_counter[k] = 0;
        hdr->flags = 0;
    }
}

// ------------------------------------------------------------------ relabelled P
__global__ __launch_bounds__(256) void layout_rank_kernel(const uint32_t *__restrict__ perm, uint32_t *__restrict__ rank,
                                                          const int64_t *__restrict__ row_ptr, int64_t *__restrict__ len,
                                                          int64_t n)
{
    int64_t r = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (r >= n) return;
    const uint32_t old = perm[r];
    rank[old] = uint32_t(r);
    len[r] = (row_ptr[old + 1] - row_ptr[old] + 3) & ~int64_t(3); // padded to 16 bytes
}

// exclusive scan of int64 values: per-tile sums, one-block scan of those, tile scan
constexpr int kI64Items = 16;
constexpr int kI64Tile = 256 * kI64Items;

__device__ inline int64_t block_excl_i64(int64_t v, int64_t *s_wave, int64_t *total)
{
    const int lane = lane_id(), w = threadIdx.x / kWave;
    int64_t x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        int64_t y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) s_wave[w] = x;
    __syncthreads();
    int64_t off = 0, tot = 0;
    for (int k = 0; k < 4; ++k) {
        off += (k < w) ? s_wave[k] : 0;
        tot += s_wave[k];
    }
    *total = tot;
    return off + x - v;
}

__global__ __launch_bounds__(256) void i64_reduce_kernel(const int64_t *__restrict__ in, int64_t n,
                                                         int64_t *__restrict__ tile_sum)
{
    __shared__ int64_t s_wave[4];
    const int64_t first = int64_t(blockIdx.x) * kI64Tile + int64_t(threadIdx.x) * kI64Items;
    int64_t acc = 0;
    for (int k = 0; k < kI64Items; ++k)
        if (first + k < n) acc += in[first + k];
    int64_t tot;
    block_excl_i64(acc, s_wave, &tot);
    if (threadIdx.x == 0) tile_sum[blockIdx.x] = tot;
}

__global__ __launch_bounds__(256) void i64_top_kernel(int64_t *__restrict__ tile_sum, int64_t tiles,
                                                      int64_t *__restrict__ out_total)
{
    __shared__ int64_t s_wave[4];
    const int64_t per = (tiles + 255) / 256, first = int64_t(threadIdx.x) * per;
    int64_t acc = 0;
    for (int64_t k = 0; k < per; ++k)
        if (first + k < tiles) acc += tile_sum[first + k];
    int64_t tot;
    int64_t run = block_excl_i64(acc, s_wave, &tot);
    for (int64_t k = 0; k < per; ++k)
        if (first + k < tiles) {
            const int64_t v = tile_sum[first + k];
            tile_sum[first + k] = run;
            run += v;
        }
    if (threadIdx.x == 0) *out_total = tot;
}

__global__ __launch_bounds__(256) void i64_down_kernel(const int64_t *__restrict__ in, int64_t n,
                                                       const int64_t *__restrict__ tile_off, int64_t *__restrict__ out)
{
    __shared__ int64_t s_wave[4];
    const int64_t first = int64_t(blockIdx.x) * kI64Tile + int64_t(threadIdx.x) * kI64Items;
    int64_t loc[kI64Items], acc = 0;
#pragma unroll
    for (int k = 0; k < kI64Items; ++k) {
        loc[k] = (first + k < n) ? in[first + k] : 0;
        acc += loc[k];
    }
    int64_t tot;
    int64_t run = block_excl_i64(acc, s_wave, &tot) + tile_off[blockIdx.x];
#pragma unroll
    for (int k = 0; k < kI64Items; ++k) {
        if (first + k < n) out[first + k] = run;
        run += loc[k];
    }
}

// Column of padding and sentinel entries: larger than every real column.
constexpr int32_t kNoColumn = 0x7fffffff;

// One wave per new row: copy the old row with renumbered columns, padded to a
// multiple of 4 entries.
// V: the value type of P (float; double for the fp64 variant's layouts)
template <typename V>
__global__ __launch_bounds__(256) void layout_copy_kernel(const int64_t *__restrict__ row_ptr,
                                                          const int32_t *__restrict__ col, const V *__restrict__ val,
                                                          const uint32_t *__restrict__ perm,
                                                          const uint32_t *__restrict__ rank,
                                                          const int64_t *__restrict__ new_ptr, int64_t n, int64_t cap,
                                                          int32_t *__restrict__ new_col, V *__restrict__ new_val)
{
    const int lane = lane_id();
    for (int64_t r = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / kWave; r < n;
         r += int64_t(gridDim.x) * (blockDim.x / kWave)) {
        const uint32_t old = perm[r];
        const int64_t s = row_ptr[old], e = row_ptr[old + 1], d = new_ptr[r];
        const int64_t len = e - s, padded = (len + 3) & ~int64_t(3);
        for (int64_t t = lane; t < padded; t += kWave) {
            const int64_t o = d + t;
            if (o < 0 || o >= cap) continue;
            if (t < len) {
                const int32_t j = col[s + t];
                new_col[o] = uint32_t(j) < uint32_t(n) ? int32_t(rank[j]) : kNoColumn;
                new_val[o] = val[s + t];
            } else { // padding entries sort to the end and contribute nothing
                new_col[o] = kNoColumn;
                new_val[o] = V(0);
            }
        }
    }
}

template <typename V>
__global__ void layout_sentinel_kernel(const int64_t *__restrict__ new_ptr, int64_t n, int32_t *__restrict__ col,
                                       V *__restrict__ val)
{
    const int64_t e = new_ptr[n];
    for (int t = 0; t < 4; ++t) {
        col[e + t] = kNoColumn;
        val[e + t] = V(0);
    }
}

// One block per row: bitonic sort of the row's entries by (renumbered) column
// in LDS.  Sorted rows let the staged kernel skip, wave by wave, the register
// slots whose columns lie outside the LDS segment in hand, and give each
// column window one contiguous range of the row (windowed segments).  Rows
// longer than kSortRowMax keep their order: the staged kernel is as correct
// on them, and the segment build then falls back to it.  With fp32 values,
// 8192 covers every row the input-similarity step can produce (k + 4096);
// fp64 values fit 4096 in the same 64 KB of LDS.
template <typename V> constexpr int sort_row_max() { return sizeof(V) == 4 ? 8192 : 4096; }

template <typename V>
__global__ __launch_bounds__(256) void layout_sort_rows_kernel(const int64_t *__restrict__ row_ptr,
                                                               int32_t *__restrict__ col, V *__restrict__ val,
                                                               int64_t n)
{
    constexpr int kSortRowMax = sort_row_max<V>();
    __shared__ int32_t sk[kSortRowMax];
    __shared__ V sv[kSortRowMax];
    for (int64_t r = blockIdx.x; r < n; r += gridDim.x) {
        const int64_t s = row_ptr[r], len = row_ptr[r + 1] - s;
        if (len < 2 || len > kSortRowMax) continue; // block-uniform
        int size = 64;
        while (size < len) size <<= 1;
        __syncthreads();
        for (int t = threadIdx.x; t < size; t += blockDim.x) {
            sk[t] = t < len ? col[s + t] : 0x7fffffff;
            sv[t] = t < len ? val[s + t] : V(0);
        }
        __syncthreads();
        for (int k = 2; k <= size; k <<= 1)
            for (int j = k >> 1; j > 0; j >>= 1) {
                for (int t = threadIdx.x; t < size; t += blockDim.x) {
                    const int u = t ^ j;
                    if (u > t) {
                        const bool up = (t & k) == 0;
                        const int32_t a = sk[t], b = sk[u];
                        if ((a > b) == up) {
                            sk[t] = b;
                            sk[u] = a;
                            const V x = sv[t];
                            sv[t] = sv[u];
                            sv[u] = x;
                        }
                    }
                }
                __syncthreads();
            }
        for (int t = threadIdx.x; t < len; t += blockDim.x) {
            col[s + t] = sk[t];
            val[s + t] = sv[t];
        }
    }
}

// ------------------------------------------------------------------ tiled copy
// Column windows of the sliced copy: 16384 fp32 or 8192 fp64 2-D points
// (128 KB of LDS), or 8192 3-D points (96 KB).
template <typename T, int D> constexpr int window_points() { return window_points_of(sizeof(T), D); }

// Rows longer than the in-LDS row sort stay unsorted; the sliced copy finds a
// row's runs by binary search, so one such row rules it out.
__global__ __launch_bounds__(256) void long_rows_kernel(const int64_t *__restrict__ row_ptr, int64_t n,
                                                        int64_t max_len, uint32_t *__restrict__ flag)
{
    const int64_t r = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (r < n && row_ptr[r + 1] - row_ptr[r] > max_len) *flag = 1u;
}

// Segment range of each row block (its real entries' smallest and largest column).
template <int kSeg>
__global__ __launch_bounds__(256) void tile_block_range_kernel(const int64_t *__restrict__ row_ptr,
                                                               const int32_t *__restrict__ col, int64_t n,
                                                               int32_t *__restrict__ seg_lo, int32_t *__restrict__ nseg)
{
    __shared__ int s_lo[4], s_hi[4];
    const int64_t b = blockIdx.x;
    const int64_t r0 = b * kTileRows, r1 = (b + 1) * kTileRows < n ? (b + 1) * kTileRows : n;
    int lo = 0x7fffffff, hi = -1;
    for (int64_t k = row_ptr[r0] + threadIdx.x; k < row_ptr[r1]; k += blockDim.x) {
        const int32_t c = col[k];
        if (c != kNoColumn) {
            lo = min(lo, c);
            hi = max(hi, c);
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        lo = min(lo, __shfl_xor(lo, o, kWave));
        hi = max(hi, __shfl_xor(hi, o, kWave));
    }
    if (lane_id() == 0) {
        s_lo[threadIdx.x / kWave] = lo;
        s_hi[threadIdx.x / kWave] = hi;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < 4; ++w) {
            lo = min(lo, s_lo[w]);
            hi = max(hi, s_hi[w]);
        }
        lo = min(lo, s_lo[0]);
        hi = max(hi, s_hi[0]);
        seg_lo[b] = hi >= 0 ? lo / kSeg : 0;
        nseg[b] = hi >= 0 ? hi / kSeg - lo / kSeg + 1 : 0;
    }
}

// first position in the sorted row [a, e) whose column is >= key
__device__ inline int64_t row_lower_bound(const int32_t *__restrict__ col, int64_t a, int64_t e, int32_t key)
{
    while (a < e) {
        const int64_t m = a + (e - a) / 2;
        if (col[m] < key)
            a = m + 1;
        else
            e = m;
    }
    return a;
}

// Run length (entries in the tile's segment) of every (row, tile) of the tiled
// row blocks; one wave per row, one lane per segment of the row's block (a
// lane takes segments 64 apart in a block that spans more).
// Rows past n get empty runs.
template <int kSeg, int kMaxSeg>
__global__ __launch_bounds__(256) void tile_run_len_kernel(const int64_t *__restrict__ row_ptr,
                                                           const int32_t *__restrict__ col, int64_t n, int64_t rows,
                                                           const int32_t *__restrict__ seg_lo,
                                                           const int32_t *__restrict__ nseg,
                                                           const int32_t *__restrict__ blk_tiles,
                                                           int32_t *__restrict__ run_len)
{
    const int lane = lane_id();
    for (int64_t r = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / kWave; r < rows;
         r += int64_t(gridDim.x) * (blockDim.x / kWave)) {
        const int64_t b = r / kTileRows, rl = r % kTileRows;
        const int ns = nseg[b];
        for (int k = lane; k < ns; k += kWave) {
            int32_t len = 0;
            if (r < n) {
                const int64_t a = row_ptr[r], e = row_ptr[r + 1];
                const int32_t s0 = (seg_lo[b] + k) * kSeg;
                len = int32_t(row_lower_bound(col, a, e, s0 + kSeg) - row_lower_bound(col, a, e, s0));
            }
            run_len[int64_t(blk_tiles[b * kMaxSeg + k]) * kTileRows + rl] = len;
        }
    }
}

// Rows of each tile in order of decreasing run length (ties by row): slice j
// of a tile is the rows at sorted positions 64 j .. 64 j + 63, and needs
// ceil(longest run / 4) chunks.  One block of kTileRows threads per tile,
// bitonic sort of the unique keys (16384 - length, row) in LDS.
__global__ __launch_bounds__(kTileRows) void tile_sort_kernel(const int32_t *__restrict__ run_len,
                                                              uint16_t *__restrict__ tperm,
                                                              uint16_t *__restrict__ tpos,
                                                              int32_t *__restrict__ slice_chunks)
{
    static_assert(kTileSeg <= 16384 && kTileRows <= 1024, "sort key packs (16384 - length) and the row in 25 bits");
    __shared__ uint32_t key[kTileRows];
    const int64_t t = blockIdx.x;
    const int i = threadIdx.x;
    const int32_t len = run_len[t * kTileRows + i];
    key[i] = (uint32_t(kTileSeg - len) << 10) | uint32_t(i);
    __syncthreads();
    for (int k = 2; k <= kTileRows; k <<= 1)
        for (int j = k >> 1; j > 0; j >>= 1) {
            const int o = i ^ j;
            if (o > i) {
                const uint32_t a = key[i], b = key[o];
                const bool up = (i & k) == 0;
                if ((a > b) == up) {
                    key[i] = b;
                    key[o] = a;
                }
            }
            __syncthreads();
        }
    const uint32_t rl = key[i] & 1023u;
    tperm[t * kTileRows + i] = uint16_t(rl);
    tpos[t * kTileRows + rl] = uint16_t(i);
    if (i % kSellSlice == 0) {
        const int32_t longest = kTileSeg - int32_t(key[i] >> 10);
        slice_chunks[t * kSlicesPerTile + i / kSellSlice] = (longest + 3) / 4;
    }
}

template <typename T>
__global__ __launch_bounds__(256) void fill_zero_kernel(uint16_t *__restrict__ tcol, T *__restrict__ tval, int64_t m)
{
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < m; i += int64_t(gridDim.x) * blockDim.x) {
        tcol[i] = 0;
        tval[i] = T(0);
    }
}

// Copy every real entry of a row into the sliced copy: the row sits in lane
// (sorted position % 64) of unit (tile, sorted position / 64); its e-th entry
// in the segment goes to chunk e / 4, element e % 4 of that lane.  Everything
// else was zeroed (padding carries p = 0).
template <typename T, int D>
__global__ __launch_bounds__(256) void sell_copy_kernel(const int64_t *__restrict__ row_ptr,
                                                        const int32_t *__restrict__ col, const T *__restrict__ val,
                                                        int64_t n, const int32_t *__restrict__ seg_lo,
                                                        const int32_t *__restrict__ nseg,
                                                        const int32_t *__restrict__ blk_tiles,
                                                        const uint16_t *__restrict__ tpos,
                                                        const int32_t *__restrict__ unit_of,
                                                        const int32_t *__restrict__ unit_chunk0, int64_t max_entries,
                                                        uint16_t *__restrict__ tcol, T *__restrict__ tval)
{
    constexpr int kSeg = window_points<T, D>();
    constexpr int kMaxSeg = max_tiles_per_block(sizeof(T), D);
    const int lane = lane_id();
    for (int64_t r = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / kWave; r < n;
         r += int64_t(gridDim.x) * (blockDim.x / kWave)) {
        const int64_t b = r / kTileRows, rl = r % kTileRows;
        const int64_t a = row_ptr[r], e = row_ptr[r + 1];
        const int32_t lo = seg_lo[b];
        const int ns = nseg[b];
        for (int64_t j = a + lane; j < e; j += kWave) {
            const int32_t c = col[j];
            if (c == kNoColumn) continue;
            const int32_t sg = c / kSeg, k = sg - lo;
            if (k < 0 || k >= ns) continue;
            const int64_t t = blk_tiles[b * kMaxSeg + k];
            const int32_t pos = tpos[t * kTileRows + rl];
            const int32_t u = unit_of[t * kSlicesPerTile + pos / kSellSlice];
            const int64_t ei = j - row_lower_bound(col, a, e, sg * kSeg);
            const int64_t d = (int64_t(unit_chunk0[u]) + ei / 4) * kSellChunk + (pos % kSellSlice) * 4 + ei % 4;
            if (d < 0 || d >= max_entries) continue;
            tcol[d] = uint16_t(c - sg * kSeg);
            tval[d] = val[j];
        }
    }
}

// ------------------------------------------------------------------ windowed row segments
constexpr int kSegBlock = 256; // rows per block of the segment build

// Windows touched by each row (bit w: some real entry has its column in
// window w), and per (window, row block) the number of rows touching it,
// stored window-major: cnt[w * nblk + block].
// A row whose real entries are not in window order (longer than the row
// sort takes) sets *unsorted: its windows would not be contiguous ranges.
__global__ __launch_bounds__(kSegBlock) void seg_mask_kernel(const int64_t *__restrict__ row_ptr,
                                                             const int32_t *__restrict__ col, int64_t n, int nw,
                                                             int64_t nblk, uint64_t *__restrict__ mask,
                                                             int64_t *__restrict__ cnt, uint32_t *__restrict__ unsorted)
{
    __shared__ uint32_t s_cnt[kSegBlock / kWave][kMaxWindows];
    const int64_t r = int64_t(blockIdx.x) * kSegBlock + threadIdx.x;
    uint64_t m = 0;
    bool ordered = true;
    if (r < n) {
        uint32_t last = 0;
        for (int64_t k = row_ptr[r]; k < row_ptr[r + 1]; ++k) {
            const int32_t c = col[k];
            if (c != kNoColumn && uint32_t(c) < uint32_t(n)) {
                const uint32_t win = uint32_t(c) >> kWinShift;
                ordered &= win >= last;
                last = win;
                m |= 1ull << win;
            }
        }
        mask[r] = m;
    }
    if (ballot(!ordered) && lane_id() == 0) atomicOr(unsorted, 1u);
    const int w = threadIdx.x / kWave;
    for (int k = 0; k < nw; ++k) {
        const uint32_t c = uint32_t(__builtin_popcountll(ballot((m >> k) & 1u)));
        if (lane_id() == 0) s_cnt[w][k] = c;
    }
    __syncthreads();
    for (int k = threadIdx.x; k < nw; k += kSegBlock) {
        uint32_t t = 0;
        for (int q = 0; q < kSegBlock / kWave; ++q) t += s_cnt[q][k];
        cnt[int64_t(k) * nblk + blockIdx.x] = t;
    }
}

// Each row writes its segments at their window-major positions: the block's
// offset for the window plus the row's rank among the block's rows that touch
// it, so every window's segments are in row order.  The entry range of a
// window within the (column-sorted) row is found by walking the row once.
__global__ __launch_bounds__(kSegBlock) void seg_fill_kernel(const int64_t *__restrict__ row_ptr,
                                                             const int32_t *__restrict__ col, int64_t n, int nw,
                                                             int64_t nblk, const uint64_t *__restrict__ mask,
                                                             const int64_t *__restrict__ off, int64_t cap,
                                                             uint32_t *__restrict__ seg_row,
                                                             uint32_t *__restrict__ seg_start,
                                                             uint32_t *__restrict__ seg_len)
{
    __shared__ uint32_t s_cnt[kSegBlock / kWave][kMaxWindows];
    const int64_t r = int64_t(blockIdx.x) * kSegBlock + threadIdx.x;
    const uint64_t m = r < n ? mask[r] : 0ull;
    const int w = threadIdx.x / kWave;
    const uint64_t lt = (lane_id() == 0) ? 0ull : (~0ull >> (kWave - lane_id()));
    for (int k = 0; k < nw; ++k) {
        const uint32_t c = uint32_t(__builtin_popcountll(ballot((m >> k) & 1u)));
        if (lane_id() == 0) s_cnt[w][k] = c;
    }
    __syncthreads();
    int64_t e = 0, stop = 0;
    if (r < n) {
        e = row_ptr[r];
        stop = row_ptr[r + 1];
    }
    for (int k = 0; k < nw; ++k) {
        const bool has = (m >> k) & 1u;
        const uint64_t b = ballot(has);
        if (!has) continue;
        uint32_t rank = uint32_t(__builtin_popcountll(b & lt));
        for (int q = 0; q < w; ++q) rank += s_cnt[q][k];
        // the row's entries in window k: skip those below it, take those in it
        while (e < stop && (col[e] == kNoColumn || (uint32_t(col[e]) >> kWinShift) < uint32_t(k))) ++e;
        const int64_t first = e;
        while (e < stop && col[e] != kNoColumn && (uint32_t(col[e]) >> kWinShift) == uint32_t(k)) ++e;
        const int64_t pos = off[int64_t(k) * nblk + blockIdx.x] + rank;
        if (pos < cap) {
            seg_row[pos] = uint32_t(r);
            seg_start[pos] = uint32_t(first);
            seg_len[pos] = uint32_t(e - first);
        }
    }
}

// window starts: wstart[w] = offset of (window w, block 0); wstart[nw] = total
__global__ void seg_windows_kernel(const int64_t *__restrict__ off, int nw, int64_t nblk, const int64_t *__restrict__ total,
                                   int64_t *__restrict__ wstart)
{
    const int k = threadIdx.x;
    if (k < nw) wstart[k] = off[int64_t(k) * nblk];
    if (k == nw) wstart[k] = *total;
}

__global__ __launch_bounds__(256) void fill_zero_f32_kernel(float *__restrict__ f, int64_t m)
{
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < m; i += int64_t(gridDim.x) * blockDim.x)
        f[i] = 0.0f;
}

template <typename T> __global__ __launch_bounds__(256) void zero_vec2_kernel(vec2_t<T> *__restrict__ f, int64_t n)
{
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x)
        f[i] = make_vec2(T(0), T(0));
}

__device__ inline float wrecip(float x) { return __builtin_amdgcn_rcpf(x); }
// 1/x in fp64 for x >= 1: the approximate reciprocal and two Newton-Raphson
// steps, within about an ulp of the quotient
__device__ inline double wrecip(double x)
{
    double r = __builtin_amdgcn_rcp(x);
    r = fma(r, fma(-x, r, 1.0), r);
    r = fma(r, fma(-x, r, 1.0), r);
    return x != __builtin_huge_val() ? r : 0.0;
}

// One window: kWinG lanes per segment sum p_ij w_ij (y_i - y_j) over the
// segment's entries (strided, then a fixed butterfly) and add it to F_attr of
// the row.  Segments of one window belong to distinct rows, so the add needs
// no atomic; windows run in order, one launch each.
constexpr int kWinG = 16;
constexpr int kWinB = 4;

template <typename T>
__global__ __launch_bounds__(256) void attract_window_kernel(
    const int64_t *__restrict__ wstart, int w, const uint32_t *__restrict__ seg_row,
    const uint32_t *__restrict__ seg_start, const uint32_t *__restrict__ seg_len, const int32_t *__restrict__ col,
    const T *__restrict__ val, const vec2_t<T> *__restrict__ ycopy, int64_t n, vec2_t<T> *__restrict__ fattr)
{
    const int64_t s0 = wstart[w], s1 = wstart[w + 1];
    const int sub = lane_id() % kWinG;
    const int64_t per = int64_t(gridDim.x) * (256 / kWinG);
    for (int64_t s = s0 + (int64_t(blockIdx.x) * 256 + threadIdx.x) / kWinG; s < s1; s += per) {
        const uint32_t r = seg_row[s];
        const int64_t a = seg_start[s], e = a + seg_len[s];
        const vec2_t<T> yi = ycopy[r < uint32_t(n) ? r : 0];
        T fx = T(0), fy = T(0);
        // kWinB entries per lane at a time: their loads, then their gathers, are
        // in flight together (a segment's entries are few per lane, so one at a
        // time would leave the lane waiting out every latency in turn)
        for (int64_t k0 = a + sub; k0 < e; k0 += kWinB * kWinG) {
            int32_t j[kWinB];
            T p[kWinB];
#pragma unroll
            for (int u = 0; u < kWinB; ++u) {
                const int64_t k = k0 + u * kWinG;
                j[u] = k < e ? __builtin_nontemporal_load(col + k) : 0;
                p[u] = k < e ? __builtin_nontemporal_load(val + k) : T(0);
            }
            vec2_t<T> yj[kWinB];
#pragma unroll
            for (int u = 0; u < kWinB; ++u) yj[u] = ycopy[uint32_t(j[u]) < uint32_t(n) ? j[u] : 0];
#pragma unroll
            for (int u = 0; u < kWinB; ++u) {
                const T dx = yi.x - yj[u].x, dy = yi.y - yj[u].y;
                const T pw = p[u] * wrecip(T(1) + fma(dx, dx, dy * dy));
                fx = fma(pw, dx, fx);
                fy = fma(pw, dy, fy);
            }
        }
#pragma unroll
        for (int o = kWinG / 2; o > 0; o >>= 1) {
            fx += __shfl_xor(fx, o, kWinG);
            fy += __shfl_xor(fy, o, kWinG);
        }
        if (sub == 0 && r < uint32_t(n)) {
            vec2_t<T> f = fattr[r];
            f.x += fx;
            f.y += fy;
            fattr[r] = f;
        }
    }
}

// ------------------------------------------------------------------ staged attraction
constexpr int kAttG = 16; // lanes per row
constexpr int kAttV = 4;  // entries per 16-byte vector slot
constexpr int kAttU = 4;  // vector slots per lane and row: 16 * 4 * 4 = 256 entries

typedef int32_t v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

__device__ inline void attract_add(float2 yi, float2 yj, float p, float &fx, float &fy)
{
    const float dx = yi.x - yj.x, dy = yi.y - yj.y;
    const float pw = p * __builtin_amdgcn_rcpf(1.0f + fmaf(dx, dx, dy * dy));
    fx = fmaf(pw, dx, fx);
    fy = fmaf(pw, dy, fy);
}
__device__ inline void attract_add(double2 yi, double2 yj, double p, double &fx, double &fy)
{
    const double dx = yi.x - yj.x, dy = yi.y - yj.y;
    const double pw = p * wrecip(1.0 + fma(dx, dx, dy * dy));
    fx = fma(pw, dx, fx);
    fy = fma(pw, dy, fy);
}

__device__ inline void attract_add(float3 yi, float3 yj, float p, float &fx, float &fy, float &fz)
{
    const float dx = yi.x - yj.x, dy = yi.y - yj.y, dz = yi.z - yj.z;
    const float pw = p * __builtin_amdgcn_rcpf(1.0f + fmaf(dx, dx, fmaf(dy, dy, dz * dz)));
    fx = fmaf(pw, dx, fx);
    fy = fmaf(pw, dy, fy);
    fz = fmaf(pw, dz, fz);
}

// the same on whole points: f += p_ij w_ij (y_i - y_j)
__device__ inline void attract_acc(float2 yi, float2 yj, float p, float2 &f) { attract_add(yi, yj, p, f.x, f.y); }
__device__ inline void attract_acc(double2 yi, double2 yj, double p, double2 &f) { attract_add(yi, yj, p, f.x, f.y); }
__device__ inline void attract_acc(float3 yi, float3 yj, float p, float3 &f)
{
    attract_add(yi, yj, p, f.x, f.y, f.z);
}
// f += c where `live`, component by component
template <typename P> __device__ inline void point_add(P &f, const P &c, bool live = true)
{
    using T = decltype(c.x);
    f.x += live ? c.x : T(0);
    f.y += live ? c.y : T(0);
    if constexpr (sizeof(P) == 3 * sizeof(T)) f.z += live ? c.z : T(0);
}
static_assert(sizeof(float3) == 12, "3-D points are packed");

// kAttBlock threads, kAttSeg points of Y per LDS segment, kAttRG rows per lane group.
// Rows of the layout are sorted, padded to whole vectors and 16-byte aligned;
// lane `sub` of a row's group holds the vectors sub, sub + 16, sub + 32, ...
template <int kAttBlock, int kAttSeg, int kAttRG>
__global__ __launch_bounds__(kAttBlock) void attract_staged_kernel(
    const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col, const float *__restrict__ val,
    const float2 *__restrict__ ylay, const uint32_t *__restrict__ perm, int64_t n, int max_segs,
    float2 *__restrict__ fattr)
{
    constexpr int kAttGroups = kAttBlock / kAttG;
    constexpr int kAttRows = kAttGroups * kAttRG;
    constexpr int kSpan = kAttG * kAttV * kAttU; // entries held in registers per row
    __shared__ float4 sy4[kAttSeg / 2];         // one segment of Y: kAttSeg points
    __shared__ int s_lo, s_hi;
    const float2 *sy = reinterpret_cast<const float2 *>(sy4);
    const int lane = lane_id(), sub = lane % kAttG, grp = threadIdx.x / kAttG, wave = threadIdx.x / kWave;
    const uint32_t nb = gridDim.x;
    const int64_t row0 = int64_t(xcd_contiguous(blockIdx.x, nb)) * kAttRows;
    if (threadIdx.x == 0) {
        s_lo = 0x7fffffff;
        s_hi = -1;
    }
    const int32_t sentinel = int32_t(row_ptr[n]); // a vector of padding entries past the last row

    // row extents and y_i first, then all vector slots: one memory latency per block
    int32_t rs[kAttRG], re[kAttRG];
    float2 yi[kAttRG];
#pragma unroll
    for (int r = 0; r < kAttRG; ++r) {
        const int64_t i = row0 + int64_t(r) * kAttGroups + grp;
        rs[r] = re[r] = 0;
        yi[r] = make_float2(0.0f, 0.0f);
        if (i < n) {
            rs[r] = int32_t(row_ptr[i]);
            re[r] = int32_t(row_ptr[i + 1]);
            yi[r] = ylay[i];
        }
    }
    // rows too long for the in-LDS sort are unsorted: they skip the vector slots
    // (whose one-compare segment test needs sorted columns) and go direct
    int32_t ve[kAttRG], ov[kAttRG];
#pragma unroll
    for (int r = 0; r < kAttRG; ++r) {
        const bool sorted = re[r] - rs[r] <= sort_row_max<float>();
        ve[r] = sorted ? re[r] : rs[r];
        ov[r] = sorted ? rs[r] + kSpan : rs[r];
    }
    v4i c[kAttRG][kAttU];
    v4f p[kAttRG][kAttU];
    float fx[kAttRG], fy[kAttRG];
#pragma unroll
    for (int r = 0; r < kAttRG; ++r) {
        fx[r] = fy[r] = 0.0f;
#pragma unroll
        for (int u = 0; u < kAttU; ++u) {
            const int32_t k = rs[r] + (u * kAttG + sub) * kAttV;
            const int32_t kk = k < ve[r] ? k : sentinel;
            c[r][u] = __builtin_nontemporal_load(reinterpret_cast<const v4i *>(col + kk));
            p[r][u] = __builtin_nontemporal_load(reinterpret_cast<const v4f *>(val + kk));
        }
    }
    // the block's column span (entries ascend within a vector; padding is kNoColumn)
    int lo = 0x7fffffff, hi = -1;
#pragma unroll
    for (int r = 0; r < kAttRG; ++r)
#pragma unroll
        for (int u = 0; u < kAttU; ++u) {
            lo = min(lo, c[r][u].x);
#pragma unroll
            for (int v = 0; v < kAttV; ++v)
                if (c[r][u][v] != kNoColumn) hi = max(hi, c[r][u][v]);
        }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        lo = min(lo, __shfl_xor(lo, o, kWave));
        hi = max(hi, __shfl_xor(hi, o, kWave));
    }
    __syncthreads();
    if (lane == 0) {
        atomicMin(&s_lo, lo);
        atomicMax(&s_hi, hi);
    }
    __syncthreads();
    const int blo = s_lo & ~1, bhi = s_hi; // even start: segments move as 16-byte pairs
    const bool staged = bhi >= blo && (int64_t(bhi) - blo) / kAttSeg < max_segs;
    if (staged) {
        // the private copy of Y carries a segment of padding, so a segment that
        // runs past the last point still reads inside the buffer (unused values)
        static_assert(kYPad >= kAttSeg + 2, "padding must cover one segment");
        const float4 *y4 = reinterpret_cast<const float4 *>(ylay);
        for (int seg = blo; seg <= bhi; seg += kAttSeg) {
            __syncthreads(); // everyone is done with the previous segment
            // DMA the segment straight into LDS: each lane moves 16 bytes, a wave 1 KB
            const float4 *src = y4 + seg / 2 + threadIdx.x;
#pragma unroll
            for (int q = 0; q < kAttSeg / 2 / kAttBlock; ++q)
                __builtin_amdgcn_global_load_lds(static_cast<const void *>(src + q * kAttBlock),
                                                 (lds_void *)(sy4 + q * kAttBlock + wave * kWave), 16, 0, 0);
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            const int seg_end = seg + kAttSeg;
#pragma unroll
            for (int r = 0; r < kAttRG; ++r)
#pragma unroll
                for (int u = 0; u < kAttU; ++u) {
                    // one test per sorted vector: skip it unless it meets [seg, seg_end)
                    if (c[r][u].x < seg_end && c[r][u].w >= seg) {
#pragma unroll
                        for (int v = 0; v < kAttV; ++v) {
                            const uint32_t d = uint32_t(c[r][u][v] - seg);
                            if (d < uint32_t(kAttSeg)) attract_add(yi[r], sy[d], p[r][u][v], fx[r], fy[r]);
                        }
                    }
                    __builtin_amdgcn_sched_barrier(0); // bounded live ranges per slot
                }
        }
    } else {
#pragma unroll
        for (int r = 0; r < kAttRG; ++r)
#pragma unroll
            for (int u = 0; u < kAttU; ++u) {
#pragma unroll
                for (int v = 0; v < kAttV; ++v)
                    if (uint32_t(c[r][u][v]) < uint32_t(n)) attract_add(yi[r], ylay[c[r][u][v]], p[r][u][v], fx[r], fy[r]);
                __builtin_amdgcn_sched_barrier(0);
            }
    }
    // rows longer than the register slots: the rest straight from memory
#pragma unroll
    for (int r = 0; r < kAttRG; ++r) {
        const int64_t i = row0 + int64_t(r) * kAttGroups + grp;
        for (int32_t k = ov[r] + sub; k < re[r]; k += kAttG) {
            const int32_t j = col[k];
            if (uint32_t(j) < uint32_t(n)) attract_add(yi[r], ylay[j], val[k], fx[r], fy[r]);
        }
        float ax = fx[r], ay = fy[r];
#pragma unroll
        for (int o = kAttG / 2; o > 0; o >>= 1) {
            ax += __shfl_xor(ax, o, kWave);
            ay += __shfl_xor(ay, o, kWave);
        }
        if (i < n && sub == 0) fattr[perm[i]] = make_float2(ax, ay);
    }
}

// ------------------------------------------------------------------ tiled attraction
// The tiled copy is sliced: a unit is 64 rows of one tile (a slice, one row
// per lane, rows sorted by run length so that a slice's runs are alike) and
// holds ceil(longest run / 4) chunks; chunk k stores entries 4k .. 4k + 3 of
// every lane's row, so a wave reads each chunk as one contiguous 512-byte
// column block and one 1-KB value block.  Tiles are stored segment-major and
// handed out in items (up to kItemMaxTiles tiles of one segment).  One block
// per item puts the segment's 16384 points of Y in LDS once; each of its 16
// waves then streams its own units, whose chunks the layout stores back to
// back (units are dealt to waves longest first).  Chunk loads run
// kSellRing ahead of the sums in a ring of registers, across unit
// boundaries; a unit's row numbers and y_i are fetched two and one units
// ahead.  Each lane sums its own row, so the partial of a (row, tile) is
// formed in a fixed order; it goes to the row's sorted slot of the tile,
// partial[tile * kTileRows + position], so a unit's 64 lanes store one
// contiguous 512-byte block and every tile fills its 8 KB of partials
// (scattered 8-byte stores, one per row, cost a third of the kernel's time).
// attract_rows_kernel then adds each row's partials in tile order.
constexpr int kTileBlock = 1024;
// two chunks in flight per wave (16 waves per CU) measured fastest at 1.3M
// points: deeper rings (3, 4, 6, 8) streamed slower
constexpr int kSellRing = 2;
constexpr int kSellWaves = kTileBlock / kWave;
constexpr int kItemMaxUnits = kItemMaxTiles * kSlicesPerTile;

typedef uint16_t v4u16 __attribute__((ext_vector_type(4)));
typedef double v4d __attribute__((ext_vector_type(4)));
template <typename T> struct Vec4Of;
template <> struct Vec4Of<float> { using type = v4f; };
template <> struct Vec4Of<double> { using type = v4d; };

// (T, D) = (float, 2): fp32 values and centres, 16384-point windows; (double,
// 2): the fp64 variant, 8192-point windows (either is 128 KB of LDS); (float,
// 3): 3-D embeddings, 8192-point windows (96 KB).
template <typename T, int D>
__global__ __launch_bounds__(kTileBlock) void attract_sell_kernel(
    const int2 *__restrict__ item_tiles, const int4 *__restrict__ item_units, const int4 *__restrict__ wave_units,
    const int32_t *__restrict__ tile_blk, const int32_t *__restrict__ tile_seg,
    const int32_t *__restrict__ unit_chunks, const int32_t *__restrict__ unit_tj, const uint16_t *__restrict__ tperm,
    const uint16_t *__restrict__ tcol, const T *__restrict__ tval, const point_t<D, T> *__restrict__ ylay,
    int32_t nitems, Header *__restrict__ hdr, point_t<D, T> *__restrict__ partial)
{
    using V = point_t<D, T>;
    using V4 = typename Vec4Of<T>::type;
    constexpr int kSeg = window_points<T, D>();
    // a window of Y in 16-byte vectors, staged by every thread in equal shares
    constexpr int kSegVec = int(kSeg * sizeof(V) / 16);
    static_assert(kSegVec * 16 == int(kSeg * sizeof(V)) && kSegVec % kTileBlock == 0 &&
                      kSegVec * 16 <= kTileSeg * int(sizeof(float2)),
                  "a window is whole 16-byte vectors per thread, at most 128 KB of LDS");
    __shared__ v4f sy4[kSegVec];
    __shared__ int32_t s_row0[kItemMaxTiles];
    // per stored unit of the item: chunks (a run holds at most kTileSeg entries)
    // and (tile - t0) * 16 + slice, both below 2^16
    static_assert(kTileSeg / 4 < 65536 && kItemMaxUnits <= 65536, "unit tables are 16-bit");
    __shared__ uint16_t s_K[kItemMaxUnits], s_tj[kItemMaxUnits];
    __shared__ uint32_t s_item;
    const V *sy = reinterpret_cast<const V *>(sy4);
    // a fixed grid takes the items (stored largest first) from a counter; the
    // barrier at the top also keeps the LDS of one item until every wave is done
    for (;;) {
        if (threadIdx.x == 0) s_item = atomicAdd(&hdr->attract_next, 1u);
        __syncthreads();
        const uint32_t it = s_item;
        if (it >= uint32_t(nitems)) break; // block-uniform
        const int2 itr = item_tiles[it];
        const int32_t t0 = itr.x, t1 = itr.y;
        const int32_t sg = tile_seg[t0];
        const int4 iu = item_units[it]; // units [x, z) of the item; those from y on have no entries
        const int w = __builtin_amdgcn_readfirstlane(int(threadIdx.x) / kWave), lane = lane_id();
        const int4 wu = wave_units[int64_t(it) * kSellWaves + w]; // units [x, y), chunks [z, z + w)
        const int32_t G = wu.w;

        // this wave's chunk g (clamped: loads past the end are issued and unused)
        const uint16_t *tc = tcol + int64_t(wu.z) * kSellChunk + 4 * lane;
        const T *tv = tval + int64_t(wu.z) * kSellChunk + 4 * lane;
        v4u16 c[kSellRing];
        V4 p[kSellRing];
        auto issue = [&](int x, int32_t g) {
            const int64_t at = int64_t(g < G ? g : (G > 0 ? G - 1 : 0)) * kSellChunk;
            // read once per iteration: streamed past the caches' retained lines, which
            // the sort and tree running beside this kernel keep using
            c[x] = __builtin_nontemporal_load(reinterpret_cast<const v4u16 *>(tc + at));
            p[x] = __builtin_nontemporal_load(reinterpret_cast<const V4 *>(tv + at));
        };
        // the segment of Y (8 independent 16-byte loads per thread) and the first
        // chunks are in flight together
        static_assert(kYPad >= kSeg + 2 && kYPad >= kTileRows, "padding must cover one segment and one block");
        constexpr int kStage = kSegVec / kTileBlock;
        v4f stage[kStage];
        {
            const v4f *src = reinterpret_cast<const v4f *>(ylay) + int64_t(sg) * kSegVec + threadIdx.x;
#pragma unroll
            for (int q = 0; q < kStage; ++q) stage[q] = src[q * kTileBlock];
        }
#pragma unroll
        for (int x = 0; x < kSellRing; ++x) issue(x, x);
        v4f *sv = reinterpret_cast<v4f *>(sy4);
#pragma unroll
        for (int q = 0; q < kStage; ++q) sv[q * kTileBlock + threadIdx.x] = stage[q];
        for (int32_t j = threadIdx.x; j < t1 - t0; j += kTileBlock) s_row0[j] = tile_blk[t0 + j] * kTileRows;
        for (int32_t j = threadIdx.x; j < iu.z - iu.x; j += kTileBlock) {
            s_K[j] = uint16_t(unit_chunks[iu.x + j]);
            s_tj[j] = uint16_t(unit_tj[iu.x + j] - t0 * kSlicesPerTile);
        }
        __syncthreads();

        // LDS values that are the same in every lane, as scalars
        auto uni = [](int32_t v) { return __builtin_amdgcn_readfirstlane(v); };
        // this lane's sorted slot of unit u in the whole copy (where its partial
        // goes), its row in the block (a load), and the first row of the unit's block
        auto unit_at = [&](int32_t u) {
            const int32_t tj = uni(s_tj[u - iu.x]), t = t0 + tj / kSlicesPerTile, j = tj % kSlicesPerTile;
            return int64_t(t) * kTileRows + j * kSellSlice + lane;
        };
        auto unit_rl = [&](int32_t u) { return int32_t(tperm[unit_at(u)]); };
        auto unit_row0 = [&](int32_t u) { return uni(s_row0[uni(s_tj[u - iu.x]) / kSlicesPerTile]); };

        // units without entries in their tile's segment: their rows' partials are 0
        for (int32_t u = iu.y + w; u < iu.z; u += kSellWaves) partial[unit_at(u)] = V{};
        if (wu.x < wu.y) { // this wave has units
        const int32_t ulast = wu.y - 1;
        int32_t u = wu.x;             // unit being summed (wave-uniform)
        int32_t uend = uni(s_K[u - iu.x]); // its chunks end at this wave step
        // rows (layout order) of the current and the next unit, the next-but-one
        // unit's row in its block (added to its block's first row when it moves up)
        auto clampu = [&](int32_t x) { return x <= ulast ? x : ulast; };
        int32_t rowA = unit_row0(u) + unit_rl(u);
        int32_t rowB = unit_row0(clampu(u + 1)) + unit_rl(clampu(u + 1));
        int32_t rlC = unit_rl(clampu(u + 2));
        V yA = ylay[rowA], yB = ylay[rowB];
        // Wait here once for y of the first two units (the last loads issued):
        // otherwise the loop head, where this entry path meets the back edge,
        // would wait for them on every trip.  The empty statement only uses the
        // registers, which makes the compiler complete their loads before it.
        if constexpr (D == 3)
            asm volatile("" ::"v"(yA.x), "v"(yA.y), "v"(yA.z), "v"(yB.x), "v"(yB.y), "v"(yB.z));
        else
            asm volatile("" ::"v"(yA.x), "v"(yA.y), "v"(yB.x), "v"(yB.y));
        V f{};

        // one wave step: sum chunk g from ring slot x, refill the slot with chunk
        // g + kSellRing, and close the unit when g was its last chunk
        auto step = [&](int x, int32_t g) {
            const bool live = g < G; // wave-uniform; dead steps only occur after the last chunk
            V cs{};
#pragma unroll
            for (int v = 0; v < 4; ++v) attract_acc(yA, sy[c[x][v] & (kSeg - 1)], T(p[x][v]), cs);
            point_add(f, cs, live);
            issue(x, g + kSellRing);
            if (live && g + 1 == uend) {
                partial[unit_at(u)] = f;
                f = V{};
                ++u;
                if (u <= ulast) uend += uni(s_K[u - iu.x]);
                rowA = rowB;
                yA = yB;
                rowB = unit_row0(clampu(u + 1)) + rlC;
                yB = ylay[rowB];
                rlC = unit_rl(clampu(u + 2));
            }
        };
        for (int32_t g = 0; g < G; g += kSellRing) {
#pragma unroll
            for (int x = 0; x < kSellRing; ++x) step(x, g + x);
        }
        } // this wave has units
    }     // items
}

// ------------------------------------------------------------------ attractive row sums
// F_attr of each row: its partials of the block's tiles, k = 0, 1, ... in
// segment order, each at the row's sorted position in that tile, stored at the
// row's original index (perm), so that the update reads it in the caller's
// order without a gather.  Consecutive rows read one tile's 8 KB of partials
// at a time.
template <typename T, int D>
__global__ __launch_bounds__(256) void attract_rows_kernel(const point_t<D, T> *__restrict__ partial,
                                                           const int32_t *__restrict__ blk_nseg,
                                                           const int32_t *__restrict__ blk_tiles,
                                                           const uint16_t *__restrict__ tpos,
                                                           const uint32_t *__restrict__ perm, int64_t n,
                                                           point_t<D, T> *__restrict__ fattr)
{
    const int64_t r = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (r >= n) return;
    const int64_t b = r / kTileRows;
    const int rr = int(r % kTileRows);
    const int ns = blk_nseg[b];
    point_t<D, T> fa{};
    for (int k = 0; k < ns; ++k) {
        const int64_t t = blk_tiles[b * max_tiles_per_block(sizeof(T), D) + k];
        point_add(fa, partial[t * kTileRows + tpos[t * kTileRows + rr]]);
    }
    fattr[perm[r]] = fa;
}

// ------------------------------------------------------------------ gradient + update
// In the caller's order: g = 4 (alpha F_attr - F_rep / Z), then the gains /
// momentum update of the optimiser (when a.update).  F_attr is in the
// caller's order (rank == nullptr: the sliced and row-block kernels store it
// there) or in layout order, read at rank[i] (the windowed segments, which
// accumulate over launches).
template <typename T>
__global__ __launch_bounds__(256) void update_kernel(const vec2_t<T> *__restrict__ fattr_lay,
                                                     const uint32_t *__restrict__ rank,
                                                     const vec2_t<T> *__restrict__ frep, const Header *__restrict__ hdr,
                                                     int64_t n, StepArgsT<T> a, vec2_t<T> *__restrict__ Y,
                                                     vec2_t<T> *__restrict__ upd, vec2_t<T> *__restrict__ gains,
                                                     vec2_t<T> *__restrict__ grad)
{
    using V = vec2_t<T>;
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const T inv_z = T(1.0 / hdr->Z);
    const uint32_t r = rank ? rank[i] : uint32_t(i);
    const V fa = r < uint32_t(n) ? fattr_lay[r] : make_vec2(T(0), T(0));
    const V fr = frep[i];
    const T gx = T(4) * (a.alpha * fa.x - fr.x * inv_z);
    const T gy = T(4) * (a.alpha * fa.y - fr.y * inv_z);
    if (grad) grad[i] = make_vec2(gx, gy);
    if (a.update) {
        V u = upd[i], gn = gains[i];
        const V y = Y[i];
        gn.x = (u.x * gx < T(0)) ? gn.x + T(0.2) : gn.x * T(0.8);
        gn.y = (u.y * gy < T(0)) ? gn.y + T(0.2) : gn.y * T(0.8);
        gn.x = gn.x > a.min_gain ? gn.x : a.min_gain;
        gn.y = gn.y > a.min_gain ? gn.y : a.min_gain;
        u.x = a.momentum * u.x - a.learning_rate * gn.x * gx;
        u.y = a.momentum * u.y - a.learning_rate * gn.y * gy;
        Y[i] = make_vec2(y.x + u.x, y.y + u.y);
        upd[i] = u;
        gains[i] = gn;
    }
}

// 3-D embeddings: the same gradient and update on three components, with
// F_attr in the caller's order.
__global__ __launch_bounds__(256) void update3_kernel(const float3 *__restrict__ fattr,
                                                      const float3 *__restrict__ frep, const Header *__restrict__ hdr,
                                                      int64_t n, StepArgsT<float> a, float3 *__restrict__ Y,
                                                      float3 *__restrict__ upd, float3 *__restrict__ gains,
                                                      float3 *__restrict__ grad)
{
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float inv_z = float(1.0 / hdr->Z);
    const float3 fa = fattr[i], fr = frep[i];
    float g[3];
#pragma unroll
    for (int d = 0; d < 3; ++d) g[d] = 4.0f * (a.alpha * coord(fa, d) - coord(fr, d) * inv_z);
    if (grad) grad[i] = make_float3(g[0], g[1], g[2]);
    if (a.update) {
        const float3 u0 = upd[i], g0 = gains[i], y0 = Y[i];
        float u[3], gn[3], y[3];
#pragma unroll
        for (int d = 0; d < 3; ++d) {
            const float ud = coord(u0, d);
            float gd = (ud * g[d] < 0.0f) ? coord(g0, d) + 0.2f : coord(g0, d) * 0.8f;
            gd = gd > a.min_gain ? gd : a.min_gain;
            u[d] = a.momentum * ud - a.learning_rate * gd * g[d];
            gn[d] = gd;
            y[d] = coord(y0, d) + u[d];
        }
        Y[i] = make_float3(y[0], y[1], y[2]);
        upd[i] = make_float3(u[0], u[1], u[2]);
        gains[i] = make_float3(gn[0], gn[1], gn[2]);
    }
}

// ------------------------------------------------------------------ launchers
LayoutView layout_view(void *mem, int64_t n, int64_t nnz, int vbytes, int dim)
{
    LayoutView v;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off = align_up(off + bytes, 256);
        return o;
    };
    size_t o_perm = take(4 * size_t(n)), o_rank = take(4 * size_t(n)), o_ptr = take(8 * size_t(n + 1));
    // rows are padded to multiples of 4 entries, plus one 4-entry sentinel vector at the end
    const size_t cap = size_t(nnz) + 3 * size_t(n) + 4;
    size_t o_col = take(4 * cap), o_val = take(size_t(vbytes) * cap);
    // tiled copy: at most max_tiles_per_block tiles per row block and
    // kTileSlots per row block in all (the partial sums' slots), sliced
    const int64_t blocks = (n + kTileRows - 1) / kTileRows;
    const int max_seg = max_tiles_per_block(vbytes, dim);
    v.max_tiles = blocks * kTileSlots;
    // the sliced copy pads every run to its slice's longest run, rounded up to
    // whole chunks; it is built only when that fits in a quarter of nnz plus
    // one chunk per slice of the narrow span's tiles (else another kernel is used)
    v.max_entries = nnz + nnz / 4 +
                    int64_t(kSellChunk) * kSlicesPerTile * blocks * narrow_tiles_per_block(vbytes, dim) + kSellChunk;
    const int64_t max_units = v.max_tiles * kSlicesPerTile;
    size_t o_lo = take(4 * size_t(blocks)), o_ns = take(4 * size_t(blocks)),
           o_bt = take(4 * size_t(blocks) * max_seg), o_tb = take(4 * size_t(v.max_tiles)),
           o_ts = take(4 * size_t(v.max_tiles)), o_tk = take(4 * size_t(v.max_tiles)),
           o_it = take(8 * size_t(v.max_tiles)), o_rl = take(4 * size_t(v.max_tiles) * kTileRows),
           o_tp = take(2 * size_t(v.max_tiles) * kTileRows), o_tq = take(2 * size_t(v.max_tiles) * kTileRows),
           o_uo = take(4 * size_t(max_units)), o_uk = take(4 * size_t(max_units)), o_uj = take(4 * size_t(max_units)),
           o_uc = take(4 * size_t(max_units)), o_iu = take(16 * size_t(v.max_tiles)),
           o_wu = take(16 * size_t(v.max_tiles) * (kTileRows / kWave)), o_tc = take(2 * size_t(v.max_entries)),
           o_tv = take(size_t(vbytes) * size_t(v.max_entries));
    v.bytes = off;
    // windowed segments reuse the sliced copy's memory (tcol, then tval)
    const size_t seg_bytes = v.bytes - o_tc;
    v.max_segments = int64_t((seg_bytes - 8 * (kMaxWindows + 1) - 4 * 256) / 12);
    if (mem) {
        v.perm = at<uint32_t>(mem, o_perm);
        v.rank = at<uint32_t>(mem, o_rank);
        v.row_ptr = at<int64_t>(mem, o_ptr);
        v.col = at<int32_t>(mem, o_col);
        v.val = at<float>(mem, o_val);
        v.val64 = at<double>(mem, o_val);
        v.blk_seg_lo = at<int32_t>(mem, o_lo);
        v.blk_nseg = at<int32_t>(mem, o_ns);
        v.blk_tiles = at<int32_t>(mem, o_bt);
        v.tile_blk = at<int32_t>(mem, o_tb);
        v.tile_seg = at<int32_t>(mem, o_ts);
        v.tile_k = at<int32_t>(mem, o_tk);
        v.item_tiles = at<int2>(mem, o_it);
        v.run_len = at<int32_t>(mem, o_rl);
        v.tperm = at<uint16_t>(mem, o_tp);
        v.tpos = at<uint16_t>(mem, o_tq);
        v.unit_of = at<int32_t>(mem, o_uo);
        v.unit_chunks = at<int32_t>(mem, o_uk);
        v.unit_tj = at<int32_t>(mem, o_uj);
        v.unit_chunk0 = at<int32_t>(mem, o_uc);
        v.item_units = at<int4>(mem, o_iu);
        v.wave_units = at<int4>(mem, o_wu);
        v.tcol = at<uint16_t>(mem, o_tc);
        v.tval = at<float>(mem, o_tv);
        v.tval64 = at<double>(mem, o_tv);
        size_t o = o_tc;
        v.wstart = at<int64_t>(mem, o);
        o = align_up(o + 8 * (kMaxWindows + 1), 256);
        v.seg_row = at<uint32_t>(mem, o);
        o = align_up(o + 4 * size_t(v.max_segments), 256);
        v.seg_start = at<uint32_t>(mem, o);
        o = align_up(o + 4 * size_t(v.max_segments), 256);
        v.seg_len = at<uint32_t>(mem, o);
    }
    return v;
}

// The tiled copy of a built (sorted, padded) layout; plan->tiled stays false when
// some row block spans more than max_tiles_per_block segments, when the tiles
// outnumber the partial slots (kTileSlots per row block), when a row block
// spans more than the narrow limit while the tiles hold fewer than
// kTileWideEntries entries on average, or when the padding is too large.
template <typename T, int D>
static int build_tiles(const LayoutView &lv, int64_t n, int64_t nnz, TilePlan *plan, void *ws, const Layout &L,
                       hipStream_t st)
{
    constexpr int kSeg = window_points<T, D>();
    constexpr int kMaxSeg = max_tiles_per_block(sizeof(T), D);
    constexpr int kNarrow = narrow_tiles_per_block(sizeof(T), D);
    T *tval = sizeof(T) == 4 ? reinterpret_cast<T *>(lv.tval) : reinterpret_cast<T *>(lv.tval64);
    const T *val = sizeof(T) == 4 ? reinterpret_cast<const T *>(lv.val) : reinterpret_cast<const T *>(lv.val64);
    *plan = TilePlan{};
    const int64_t blocks = (n + kTileRows - 1) / kTileRows;
    plan->blocks = int32_t(blocks);
    Header *hdr = at<Header>(ws, L.header);
    flag_clear_kernel<<<1, 1, 0, st>>>(&hdr->unsorted);
    long_rows_kernel<<<unsigned((n + 255) / 256), 256, 0, st>>>(lv.row_ptr, n, sort_row_max<T>(), &hdr->unsorted);
    uint32_t unsorted = 0;
    if (hipMemcpyAsync(&unsorted, &hdr->unsorted, 4, hipMemcpyDeviceToHost, st) != hipSuccess) return -1;
    tile_block_range_kernel<kSeg><<<unsigned(blocks), 256, 0, st>>>(lv.row_ptr, lv.col, n, lv.blk_seg_lo, lv.blk_nseg);
    std::vector<int32_t> lo(blocks), ns(blocks);
    if (hipMemcpyAsync(lo.data(), lv.blk_seg_lo, 4 * blocks, hipMemcpyDeviceToHost, st) != hipSuccess) return -1;
    if (hipMemcpyAsync(ns.data(), lv.blk_nseg, 4 * blocks, hipMemcpyDeviceToHost, st) != hipSuccess) return -1;
    if (hipStreamSynchronize(st) != hipSuccess) return -1;
    if (unsorted) return 0; // a row too long to sort: keep the row-block kernel
    // tiles in segment-major order, (block, k) -> tile, then items of up to
    // `per` tiles that never straddle a segment (a few items per CU)
    std::vector<std::pair<int32_t, int32_t>> order; // (segment, block)
    bool wide = false;
    for (int64_t b = 0; b < blocks; ++b) {
        if (ns[b] > kMaxSeg) return 0; // too wide: keep the row-block kernel
        wide |= ns[b] > kNarrow;
        for (int k = 0; k < ns[b]; ++k) order.emplace_back(lo[b] + k, int32_t(b));
    }
    const int64_t tiles = int64_t(order.size());
    if (tiles == 0 || tiles > lv.max_tiles) return 0;
    if (wide && nnz < tiles * kTileWideEntries) return 0; // wide and sparse
    std::sort(order.begin(), order.end());
    std::vector<int32_t> bt(size_t(blocks) * kMaxSeg, -1), tb(tiles), ts(tiles), tk(tiles);
    for (int64_t t = 0; t < tiles; ++t) {
        ts[t] = order[t].first;
        tb[t] = order[t].second;
        tk[t] = ts[t] - lo[tb[t]];
        bt[size_t(tb[t]) * kMaxSeg + tk[t]] = int32_t(t);
    }
    if (hipMemcpyAsync(lv.blk_tiles, bt.data(), 4 * bt.size(), hipMemcpyHostToDevice, st) != hipSuccess) return -1;
    if (hipMemcpyAsync(lv.tile_blk, tb.data(), 4 * tiles, hipMemcpyHostToDevice, st) != hipSuccess) return -1;
    if (hipMemcpyAsync(lv.tile_seg, ts.data(), 4 * tiles, hipMemcpyHostToDevice, st) != hipSuccess) return -1;
    if (hipMemcpyAsync(lv.tile_k, tk.data(), 4 * tiles, hipMemcpyHostToDevice, st) != hipSuccess) return -1;
    // run lengths, rows sorted by run length in every tile, chunks per slice
    const int64_t rows = blocks * kTileRows;
    const unsigned gw = unsigned((rows + 3) / 4 < 65535 * 4 ? (rows + 3) / 4 : 65535 * 4);
    tile_run_len_kernel<kSeg, kMaxSeg><<<gw, 256, 0, st>>>(lv.row_ptr, lv.col, n, rows, lv.blk_seg_lo, lv.blk_nseg, lv.blk_tiles,
                                            lv.run_len);
    tile_sort_kernel<<<unsigned(tiles), kTileRows, 0, st>>>(lv.run_len, lv.tperm, lv.tpos, lv.unit_chunks);
    const int64_t units = tiles * kSlicesPerTile;
    std::vector<int32_t> sk(units); // chunks of slice (tile, j), indexed tile * 16 + j
    if (hipMemcpyAsync(sk.data(), lv.unit_chunks, 4 * units, hipMemcpyDeviceToHost, st) != hipSuccess) return -1;
    if (hipStreamSynchronize(st) != hipSuccess) return -1;
    // Items: runs of tiles of one segment holding about a quarter of a CU's
    // share of the chunks (at most kItemMaxTiles tiles), launched largest
    // first so that blocks handed to whichever CU frees up first balance out.
    // Each item stages its segment of Y once: coarser items stage less (a
    // sixteenth of a share per item measured 7% slower at 1.3M points).
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess)
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    std::vector<int64_t> tcost(tiles, 0);
    int64_t total = 0;
    for (int64_t t = 0; t < tiles; ++t) {
        for (int j = 0; j < kSlicesPerTile; ++j) tcost[t] += sk[t * kSlicesPerTile + j];
        total += tcost[t];
    }
    const int64_t target = std::max<int64_t>(1, total / (4 * int64_t(cus)));
    std::vector<int2> ranges;
    std::vector<int64_t> rcost;
    for (int64_t t = 0; t < tiles; ++t) {
        const bool fresh = ranges.empty() || ts[t] != ts[ranges.back().x] || t - ranges.back().x >= kItemMaxTiles ||
                           (rcost.back() > 0 && rcost.back() + tcost[t] > target);
        if (fresh) {
            ranges.push_back(make_int2(int32_t(t), int32_t(t)));
            rcost.push_back(0);
        }
        ranges.back().y = int32_t(t + 1);
        rcost.back() += tcost[t];
    }
    const int64_t nitems = int64_t(ranges.size());
    std::vector<int32_t> iorder(nitems);
    for (int64_t i = 0; i < nitems; ++i) iorder[i] = int32_t(i);
    std::stable_sort(iorder.begin(), iorder.end(), [&](int32_t a, int32_t b) { return rcost[a] > rcost[b]; });
    std::vector<int2> items(nitems);
    for (int64_t i = 0; i < nitems; ++i) items[i] = ranges[iorder[i]];
    if (hipMemcpyAsync(lv.item_tiles, items.data(), 8 * items.size(), hipMemcpyHostToDevice, st) != hipSuccess)
        return -1;
    // Units of every item: the ones with chunks are dealt to the block's waves
    // longest first, each to the wave with the least work so far (cost: chunks
    // plus one for the unit's bookkeeping); a wave's units and their chunks
    // are stored back to back.  Units without chunks come last.
    constexpr int W = kTileRows / kWave;
    std::vector<int32_t> uo(units), uk(units), uj(units), uc(units);
    std::vector<int4> iu(nitems), wu(size_t(nitems) * W);
    int64_t d = 0, chunk = 0;
    std::vector<int32_t> order_u;
    std::vector<std::vector<int32_t>> lists(W);
    for (int64_t i = 0; i < nitems; ++i) {
        order_u.clear();
        for (int64_t t = items[i].x; t < items[i].y; ++t)
            for (int j = 0; j < kSlicesPerTile; ++j)
                if (sk[t * kSlicesPerTile + j] > 0) order_u.push_back(int32_t(t * kSlicesPerTile + j));
        std::stable_sort(order_u.begin(), order_u.end(), [&](int32_t a, int32_t b) { return sk[a] > sk[b]; });
        int64_t load[W] = {};
        for (auto &l : lists) l.clear();
        for (int32_t tj : order_u) {
            const int wmin = int(std::min_element(load, load + W) - load);
            lists[wmin].push_back(tj);
            load[wmin] += sk[tj] + 1;
        }
        iu[i].x = int32_t(d);
        for (int w = 0; w < W; ++w) {
            int4 &q = wu[size_t(i) * W + w];
            q.x = int32_t(d);
            q.z = lists[w].empty() ? 0 : int32_t(chunk);
            for (int32_t tj : lists[w]) {
                uo[tj] = int32_t(d);
                uk[d] = sk[tj];
                uj[d] = tj;
                uc[d] = int32_t(chunk);
                chunk += sk[tj];
                ++d;
            }
            q.y = int32_t(d);
            q.w = lists[w].empty() ? 0 : int32_t(chunk - q.z);
        }
        iu[i].y = int32_t(d);
        for (int64_t t = items[i].x; t < items[i].y; ++t)
            for (int j = 0; j < kSlicesPerTile; ++j)
                if (sk[t * kSlicesPerTile + j] == 0) {
                    const int32_t tj = int32_t(t * kSlicesPerTile + j);
                    uo[tj] = int32_t(d);
                    uk[d] = 0;
                    uj[d] = tj;
                    uc[d] = int32_t(chunk);
                    ++d;
                }
        iu[i].z = int32_t(d);
        iu[i].w = 0;
        if (chunk * kSellChunk > lv.max_entries - kSellChunk) return 0; // too much padding: row-block kernel
    }
    const int64_t entries = chunk * kSellChunk;
    if (hipMemcpyAsync(lv.unit_of, uo.data(), 4 * units, hipMemcpyHostToDevice, st) != hipSuccess) return -1;
    if (hipMemcpyAsync(lv.unit_chunks, uk.data(), 4 * units, hipMemcpyHostToDevice, st) != hipSuccess) return -1;
    if (hipMemcpyAsync(lv.unit_tj, uj.data(), 4 * units, hipMemcpyHostToDevice, st) != hipSuccess) return -1;
    if (hipMemcpyAsync(lv.unit_chunk0, uc.data(), 4 * units, hipMemcpyHostToDevice, st) != hipSuccess) return -1;
    if (hipMemcpyAsync(lv.item_units, iu.data(), 16 * iu.size(), hipMemcpyHostToDevice, st) != hipSuccess) return -1;
    if (hipMemcpyAsync(lv.wave_units, wu.data(), 16 * wu.size(), hipMemcpyHostToDevice, st) != hipSuccess) return -1;
    // zeros everywhere (chunk 0 included, which lanes without work read), then the entries
    const int64_t zero = entries > kSellChunk ? entries : kSellChunk;
    fill_zero_kernel<T><<<unsigned(std::min<int64_t>((zero + 255) / 256, 65535 * 4)), 256, 0, st>>>(lv.tcol, tval,
                                                                                                    zero);
    sell_copy_kernel<T, D><<<unsigned(n < 65535 * 4 ? (n + 3) / 4 : 65535 * 4), 256, 0, st>>>(
        lv.row_ptr, lv.col, val, n, lv.blk_seg_lo, lv.blk_nseg, lv.blk_tiles, lv.tpos, lv.unit_of, lv.unit_chunk0,
        lv.max_entries, lv.tcol, tval);
    // the tables above must stay alive until the copies have been read
    if (hipStreamSynchronize(st) != hipSuccess) return -1;
    if (hipGetLastError() != hipSuccess) return -1;
    plan->tiled = true;
    plan->tiles = int32_t(tiles);
    plan->items = int32_t(nitems);
    plan->entries = entries;
    return 0;
}

// Windowed row segments of a built (sorted, padded) layout, for rows without
// tile locality; plan->windows stays 0 when they do not fit the memory.
static int build_windows(const LayoutView &lv, int64_t n, TilePlan *plan, void *ws, const Layout &L, hipStream_t st)
{
    plan->windows = 0;
    plan->segments = 0;
    const int nw = int((n + (int64_t(1) << kWinShift) - 1) >> kWinShift);
    if (nw < 1 || nw > kMaxWindows) return 0;
    const int64_t nblk = (n + kSegBlock - 1) / kSegBlock;
    uint64_t *mask = at<uint64_t>(ws, L.codes0);   // n words
    int64_t *cnt = at<int64_t>(ws, L.codes1);      // nw * nblk <= n / 4 words
    int64_t *off = reinterpret_cast<int64_t *>(at<double>(ws, L.psum)); // nw * nblk + 1 words
    int64_t *tsum = at<int64_t>(ws, L.scan_sum);
    const int64_t m = int64_t(nw) * nblk;
    Header *hdr = at<Header>(ws, L.header);
    flag_clear_kernel<<<1, 1, 0, st>>>(&hdr->unsorted);
    seg_mask_kernel<<<unsigned(nblk), kSegBlock, 0, st>>>(lv.row_ptr, lv.col, n, nw, nblk, mask, cnt, &hdr->unsorted);
    const int64_t tiles = (m + kI64Tile - 1) / kI64Tile;
    i64_reduce_kernel<<<unsigned(tiles), 256, 0, st>>>(cnt, m, tsum);
    i64_top_kernel<<<1, 256, 0, st>>>(tsum, tiles, off + m);
    i64_down_kernel<<<unsigned(tiles), 256, 0, st>>>(cnt, m, tsum, off);
    int64_t total = 0;
    uint32_t unsorted = 0;
    if (hipMemcpyAsync(&total, off + m, 8, hipMemcpyDeviceToHost, st) != hipSuccess) return -1;
    if (hipMemcpyAsync(&unsorted, &hdr->unsorted, 4, hipMemcpyDeviceToHost, st) != hipSuccess) return -1;
    if (hipStreamSynchronize(st) != hipSuccess) return -1;
    // rows out of window order, or more segments than the memory holds: keep the row-block kernel
    if (unsorted || total > lv.max_segments || total >= (int64_t(1) << 32)) return 0;
    seg_fill_kernel<<<unsigned(nblk), kSegBlock, 0, st>>>(lv.row_ptr, lv.col, n, nw, nblk, mask, off, lv.max_segments,
                                                          lv.seg_row, lv.seg_start, lv.seg_len);
    seg_windows_kernel<<<1, kMaxWindows + 1, 0, st>>>(off, nw, nblk, off + m, lv.wstart);
    if (hipStreamSynchronize(st) != hipSuccess) return -1;
    if (hipGetLastError() != hipSuccess) return -1;
    plan->windows = nw;
    plan->segments = total;
    return 0;
}

// Breadth-first levels into dist.  Returns 1 when every point was reached
// within kBfsMaxLevels levels and no level (past the roots) held more than
// kBfsMaxFront points, 0 when abandoned (the order would not bring columns
// together), -1 on a HIP error.  One host synchronisation per level.
constexpr uint32_t kBfsMaxFront = 4 * kTileSeg;

static int bfs_levels(const int64_t *row_ptr, const int32_t *col, int64_t n, int64_t nnz, const uint32_t *comp,
                      uint32_t *dist, void *ws, const Layout &L, hipStream_t st)
{
    Header *hdr = at<Header>(ws, L.header);
    uint32_t *fr[2] = {at<uint32_t>(ws, L.idx0), at<uint32_t>(ws, L.idx1)};
    uint32_t *cnt = hdr->bfs_count;
    flag_clear_kernel<<<1, 1, 0, st>>>(&cnt[0]);
    bfs_init_kernel<<<unsigned((n + 255) / 256), 256, 0, st>>>(comp, n, dist, fr[0], &cnt[0]);
    uint32_t size = 0, reached = 0;
    if (hipMemcpyAsync(&size, &cnt[0], 4, hipMemcpyDeviceToHost, st) != hipSuccess) return -1;
    if (hipStreamSynchronize(st) != hipSuccess) return -1;
    for (int level = 0; size > 0; ++level) {
        reached += size;
        if (level >= kBfsMaxLevels) return 0;
        uint32_t *next_cnt = &cnt[(level + 1) & 1];
        flag_clear_kernel<<<1, 1, 0, st>>>(next_cnt);
        const int64_t blocks = std::min<int64_t>((int64_t(size) + 3) / 4, 65535 * 4); // a wave per point
        bfs_expand_kernel<<<unsigned(blocks), 256, 0, st>>>(row_ptr, col, n, nnz, fr[level & 1], size,
                                                             uint32_t(level), dist, fr[(level + 1) & 1], next_cnt);
        if (hipMemcpyAsync(&size, next_cnt, 4, hipMemcpyDeviceToHost, st) != hipSuccess) return -1;
        if (hipStreamSynchronize(st) != hipSuccess) return -1;
        if (size > kBfsMaxFront) return 0;
    }
    return reached == uint32_t(n) ? 1 : 0;
}

// Renumbers the points by the keys of `order` and writes the relabelled rows:
// perm, rank, row pointers, columns and values, each row sorted.
template <typename V, int D>
static int relabel(const int64_t *row_ptr, const int32_t *col, const V *val, int64_t n, int64_t nnz, const V *Y,
                   int order, const LayoutView &lv, void *ws, const Layout &L, hipStream_t st)
{
    V *lval = sizeof(V) == 4 ? reinterpret_cast<V *>(lv.val) : reinterpret_cast<V *>(lv.val64);
    Header *hdr = at<Header>(ws, L.header);
    const uint32_t *comp = at<uint32_t>(ws, L.split_b);
    const unsigned gn = unsigned((n + 255) / 256);
    const unsigned gw = unsigned((n + 3) / 4 < 65535 * 4 ? (n + 3) / 4 : 65535 * 4);
    uint64_t *keys = at<uint64_t>(ws, L.codes0);
    if (order == kOrderBfs) {
        layout_keys_bfs_kernel<<<gn, 256, 0, st>>>(keys, comp, at<uint32_t>(ws, L.base), n);
    } else {
        // keys: component, then Morton order of Y when given
        if (Y) {
            if constexpr (D == 3) {
                launch_bbox_morton3(Y, n, nullptr, ws, L, st);
            } else {
                launch_bbox(Y, n, ws, L, st);
                launch_morton(Y, n, nullptr, ws, L, st);
            }
        } else {
            sort_reset_kernel<<<1, 256, 0, st>>>(hdr, at<uint32_t>(ws, L.hist));
        }
        layout_keys_kernel<<<gn, 256, 0, st>>>(keys, comp, n, Y ? 1 : 0);
    }
    sort_reset_kernel<<<1, 256, 0, st>>>(hdr, at<uint32_t>(ws, L.hist));
    keys_hist_kernel<<<unsigned(L.sort_tiles), kSortBlock, 0, st>>>(keys, n, at<uint32_t>(ws, L.hist),
                                                                    at<uint32_t>(ws, L.status), L.sort_tiles);
    // (the sorted copy of the points this also makes is not used)
    const V *ysrc = Y ? Y : reinterpret_cast<const V *>(at<char>(ws, L.ycopy));
    if constexpr (D == 3)
        launch_sort_points(n, reinterpret_cast<const float3 *>(ysrc), ws, L, st);
    else
        launch_sort(n, ysrc, ws, L, st);
    // new order -> rank, row lengths, row pointers, relabelled rows
    const uint32_t *perm_ws = at<uint32_t>(ws, L.idx0);
    if (hipMemcpyAsync(lv.perm, perm_ws, 4 * size_t(n), hipMemcpyDeviceToDevice, st) != hipSuccess) return -1;
    int64_t *len = at<int64_t>(ws, L.codes1); // scratch, n entries
    layout_rank_kernel<<<gn, 256, 0, st>>>(lv.perm, lv.rank, row_ptr, len, n);
    const int64_t tiles = (n + kI64Tile - 1) / kI64Tile;
    int64_t *tsum = at<int64_t>(ws, L.scan_sum); // >= tiles + 1 entries of 16 bytes
    i64_reduce_kernel<<<unsigned(tiles), 256, 0, st>>>(len, n, tsum);
    i64_top_kernel<<<1, 256, 0, st>>>(tsum, tiles, lv.row_ptr + n);
    i64_down_kernel<<<unsigned(tiles), 256, 0, st>>>(len, n, tsum, lv.row_ptr);
    const int64_t cap = nnz + 3 * n + 4;
    layout_copy_kernel<V><<<gw, 256, 0, st>>>(row_ptr, col, val, lv.perm, lv.rank, lv.row_ptr, n, cap, lv.col, lval);
    layout_sentinel_kernel<V><<<1, 1, 0, st>>>(lv.row_ptr, n, lv.col, lval);
    layout_sort_rows_kernel<V><<<unsigned(n < 65535 * 16 ? n : 65535 * 16), 256, 0, st>>>(lv.row_ptr, lv.col, lval, n);
    return hipGetLastError() != hipSuccess ? -1 : 0;
}

template <typename V, int D>
int launch_layout_build(const int64_t *row_ptr, const int32_t *col, const V *val, int64_t n, int64_t nnz,
                        const V *Y, int order, const LayoutView &lv, TilePlan *plan, void *ws, const Layout &L,
                        hipStream_t st)
{
    Header *hdr = at<Header>(ws, L.header);
    uint32_t *parent = at<uint32_t>(ws, L.split_b);
    uint32_t *changed = at<uint32_t>(ws, L.split_e);
    uint32_t *dist = at<uint32_t>(ws, L.base);
    const unsigned gn = unsigned((n + 255) / 256);
    const unsigned gw = unsigned((n + 3) / 4 < 65535 * 4 ? (n + 3) / 4 : 65535 * 4);
    // validate the row pointers first: every later kernel indexes P's entries by them
    flag_clear_kernel<<<1, 1, 0, st>>>(&hdr->flags);
    csr_check_kernel<<<unsigned((n + 1 + 255) / 256), 256, 0, st>>>(row_ptr, n, nnz, hdr);
    uint32_t flags = 0;
    if (hipMemcpyAsync(&flags, &hdr->flags, 4, hipMemcpyDeviceToHost, st) != hipSuccess) return -1;
    if (hipStreamSynchronize(st) != hipSuccess) return -1;
    if (flags & kErrRange) return 1;
    cc_init_kernel<<<gn, 256, 0, st>>>(parent, n);
    for (int it = 0; it < 64; ++it) {
        flag_clear_kernel<<<1, 1, 0, st>>>(changed);
        cc_hook_kernel<<<gw, 256, 0, st>>>(row_ptr, col, n, nnz, parent, changed);
        cc_compress_kernel<<<gn, 256, 0, st>>>(parent, n);
        uint32_t h = 0;
        if (hipMemcpyAsync(&h, changed, 4, hipMemcpyDeviceToHost, st) != hipSuccess) return -1;
        if (hipStreamSynchronize(st) != hipSuccess) return -1;
        if (h == 0) break;
    }
    // the first order: BFS levels when asked for (Morton if the search gives
    // up), else Morton
    int chosen = kOrderMorton;
    if (order == kOrderBfs) {
        const int rc = bfs_levels(row_ptr, col, n, nnz, parent, dist, ws, L, st);
        if (rc < 0) return -1;
        if (rc == 1) chosen = kOrderBfs;
    }
    if (relabel<V, D>(row_ptr, col, val, n, nnz, Y, chosen, lv, ws, L, st) != 0) return -1;
    *plan = TilePlan{};
    {
        int rc = build_tiles<V, D>(lv, n, nnz, plan, ws, L, st);
        if (rc != 0) return rc;
        if (plan->tiled) {
            plan->order = chosen;
            return 0;
        }
        if (order == kOrderAuto) {
            // Morton order gave no tiles: try the BFS levels, which bring a
            // row's columns together when P itself has locality (a kNN graph
            // of points on a low-dimensional set) whatever Y looks like
            rc = bfs_levels(row_ptr, col, n, nnz, parent, dist, ws, L, st);
            if (rc < 0) return -1;
            if (rc == 1) {
                if (relabel<V, D>(row_ptr, col, val, n, nnz, Y, kOrderBfs, lv, ws, L, st) != 0) return -1;
                rc = build_tiles<V, D>(lv, n, nnz, plan, ws, L, st);
                if (rc != 0) return rc;
                if (plan->tiled) {
                    plan->order = kOrderBfs;
                    return 0;
                }
                if (relabel<V, D>(row_ptr, col, val, n, nnz, Y, kOrderMorton, lv, ws, L, st) != 0) return -1;
            }
            *plan = TilePlan{};
        }
    }
    plan->order = chosen;
    // 3-D layouts have the sliced copy only
    if constexpr (D == 3) return 0;
    return build_windows(lv, n, plan, ws, L, st);
}
template int launch_layout_build<float, 2>(const int64_t *, const int32_t *, const float *, int64_t, int64_t,
                                           const float *, int, const LayoutView &, TilePlan *, void *,
                                           const Layout &, hipStream_t);
template int launch_layout_build<double, 2>(const int64_t *, const int32_t *, const double *, int64_t, int64_t,
                                            const double *, int, const LayoutView &, TilePlan *, void *,
                                            const Layout &, hipStream_t);
template int launch_layout_build<float, 3>(const int64_t *, const int32_t *, const float *, int64_t, int64_t,
                                           const float *, int, const LayoutView &, TilePlan *, void *,
                                           const Layout &, hipStream_t);

// One launch per column window, after F_attr is cleared (layout order).
template <typename T>
void launch_attract_windows(const LayoutView &lv, int64_t n, int blocks, int windows, void *ws, const Layout &L,
                            hipStream_t st)
{
    vec2_t<T> *fattr = at<vec2_t<T>>(ws, L.fattr);
    const T *val = sizeof(T) == 4 ? reinterpret_cast<const T *>(lv.val) : reinterpret_cast<const T *>(lv.val64);
    zero_vec2_kernel<T><<<unsigned(std::min<int64_t>((n + 255) / 256, 4096)), 256, 0, st>>>(fattr, n);
    // a grid that fills the chip; blocks stride over the window's segments
    const unsigned grid = unsigned(std::max(1, blocks) * 8);
    for (int w = 0; w < windows; ++w)
        attract_window_kernel<T><<<grid, 256, 0, st>>>(lv.wstart, w, lv.seg_row, lv.seg_start, lv.seg_len, lv.col, val,
                                                       at<vec2_t<T>>(ws, L.ycopy), n, fattr);
}
template void launch_attract_windows<float>(const LayoutView &, int64_t, int, int, void *, const Layout &,
                                            hipStream_t);
template void launch_attract_windows<double>(const LayoutView &, int64_t, int, int, void *, const Layout &,
                                             hipStream_t);

template <int B, int S, int RG>
static void launch_staged(const LayoutView &lv, int64_t n, int64_t nnz, int max_segs, void *ws, const Layout &L,
                          hipStream_t st)
{
    constexpr int rows = (B / kAttG) * RG;
    const int64_t blocks = ((n + rows - 1) / rows + 7) / 8 * 8; // multiple of 8 for the XCD remap
    attract_staged_kernel<B, S, RG><<<unsigned(blocks), B, 0, st>>>(lv.row_ptr, lv.col, lv.val, at<float2>(ws, L.ycopy),
                                                                   lv.perm, n, max_segs, at<float2>(ws, L.fattr));
}

template <typename T>
void launch_attract_layout(const LayoutView &lv, int64_t n, int64_t nnz, int tiles, int items, int blocks,
                           int max_segs, int windows, void *ws, const Layout &L, hipStream_t st)
{
    using V = vec2_t<T>;
    if (tiles == 0 && windows > 0) {
        launch_attract_windows<T>(lv, n, blocks, windows, ws, L, st);
        return;
    }
    if (tiles > 0) {
        const T *tval = sizeof(T) == 4 ? reinterpret_cast<const T *>(lv.tval) : reinterpret_cast<const T *>(lv.tval64);
        const unsigned grid = unsigned(blocks < items ? blocks : items);
        attract_sell_kernel<T, 2><<<grid, kTileBlock, 0, st>>>(lv.item_tiles, lv.item_units, lv.wave_units, lv.tile_blk,
                                                            lv.tile_seg, lv.unit_chunks, lv.unit_tj, lv.tperm, lv.tcol,
                                                            tval, at<V>(ws, L.ycopy), items, at<Header>(ws, L.header),
                                                            at<V>(ws, L.partial));
        attract_rows_kernel<T, 2><<<unsigned((n + 255) / 256), 256, 0, st>>>(at<V>(ws, L.partial), lv.blk_nseg,
                                                                         lv.blk_tiles, lv.tpos, lv.perm, n,
                                                                         at<V>(ws, L.fattr));
        return;
    }
    // 1024 threads (one block per CU: the segment fills 128 KB of LDS), 2 rows per lane group
    if constexpr (sizeof(T) == 4) launch_staged<1024, 16384, 2>(lv, n, nnz, max_segs, ws, L, st);
}
template void launch_attract_layout<float>(const LayoutView &, int64_t, int64_t, int, int, int, int, int, void *,
                                           const Layout &, hipStream_t);
template void launch_attract_layout<double>(const LayoutView &, int64_t, int64_t, int, int, int, int, int, void *,
                                            const Layout &, hipStream_t);

template <typename T>
void launch_update(const LayoutView &lv, int64_t n, bool layout_order, const StepArgsT<T> &a, T *Y, T *upd, T *gains,
                   T *grad, void *ws, const Layout &L, hipStream_t st)
{
    using V = vec2_t<T>;
    update_kernel<T><<<unsigned((n + 255) / 256), 256, 0, st>>>(
        at<V>(ws, L.fattr), layout_order ? lv.rank : nullptr, at<V>(ws, L.frep), at<Header>(ws, L.header), n, a, reinterpret_cast<V *>(Y),
        reinterpret_cast<V *>(upd), reinterpret_cast<V *>(gains), reinterpret_cast<V *>(grad));
}
template void launch_update<float>(const LayoutView &, int64_t, bool, const StepArgsT<float> &, float *, float *,
                                   float *, float *, void *, const Layout &, hipStream_t);
template void launch_update<double>(const LayoutView &, int64_t, bool, const StepArgsT<double> &, double *, double *,
                                    double *, double *, void *, const Layout &, hipStream_t);

void launch_attract_layout3(const LayoutView &lv, int64_t n, int tiles, int items, int blocks, void *ws,
                            const Layout &L, hipStream_t st)
{
    if (tiles <= 0 || items <= 0) { // a P with no entries: F_attr = 0
        fill_zero_f32_kernel<<<unsigned(std::min<int64_t>((3 * n + 255) / 256, 4096)), 256, 0, st>>>(
            at<float>(ws, L.fattr), 3 * n);
        return;
    }
    const unsigned grid = unsigned(blocks < items ? blocks : items);
    attract_sell_kernel<float, 3><<<grid, kTileBlock, 0, st>>>(
        lv.item_tiles, lv.item_units, lv.wave_units, lv.tile_blk, lv.tile_seg, lv.unit_chunks, lv.unit_tj, lv.tperm,
        lv.tcol, lv.tval, at<float3>(ws, L.ycopy), items, at<Header>(ws, L.header), at<float3>(ws, L.partial));
    attract_rows_kernel<float, 3><<<unsigned((n + 255) / 256), 256, 0, st>>>(
        at<float3>(ws, L.partial), lv.blk_nseg, lv.blk_tiles, lv.tpos, lv.perm, n, at<float3>(ws, L.fattr));
}

void launch_update3(int64_t n, const StepArgsT<float> &a, float *Y, float *upd, float *gains, float *grad, void *ws,
                    const Layout &L, hipStream_t st)
{
    update3_kernel<<<unsigned((n + 255) / 256), 256, 0, st>>>(
        at<float3>(ws, L.fattr), at<float3>(ws, L.frep), at<Header>(ws, L.header), n, a, reinterpret_cast<float3 *>(Y),
        reinterpret_cast<float3 *>(upd), reinterpret_cast<float3 *>(gains), reinterpret_cast<float3 *>(grad));
}

} // namespace bht
