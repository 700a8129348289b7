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
    for (int k = threadIdx.x; k < kSortPasses * kRadix; k += kSortBlock)
        if (sh[k]) atomicAdd(&hist[k], sh[k]);
}

__global__ void sort_reset_kernel(Header *__restrict__ hdr, uint32_t *__restrict__ hist)
{
    for (int k = threadIdx.x; k < kSortPasses * kRadix; k += blockDim.x) hist[k] = 0;
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
__global__ __launch_bounds__(256) void layout_copy_kernel(const int64_t *__restrict__ row_ptr,
                                                          const int32_t *__restrict__ col, const float *__restrict__ val,
                                                          const uint32_t *__restrict__ perm,
                                                          const uint32_t *__restrict__ rank,
                                                          const int64_t *__restrict__ new_ptr, int64_t n, int64_t cap,
                                                          int32_t *__restrict__ new_col, float *__restrict__ new_val)
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
                new_val[o] = 0.0f;
            }
        }
    }
}

__global__ void layout_sentinel_kernel(const int64_t *__restrict__ new_ptr, int64_t n, int32_t *__restrict__ col,
                                       float *__restrict__ val)
{
    const int64_t e = new_ptr[n];
    for (int t = 0; t < 4; ++t) {
        col[e + t] = kNoColumn;
        val[e + t] = 0.0f;
    }
}

// One block per row: bitonic sort of the row's entries by (renumbered) column
// in LDS.  Sorted rows let the staged kernel skip, wave by wave, the register
// slots whose columns lie outside the LDS segment in hand.  Rows longer than
// kSortRowMax keep their order (only speed depends on it).
constexpr int kSortRowMax = 4096;

__global__ __launch_bounds__(256) void layout_sort_rows_kernel(const int64_t *__restrict__ row_ptr,
                                                               int32_t *__restrict__ col, float *__restrict__ val,
                                                               int64_t n)
{
    __shared__ int32_t sk[kSortRowMax];
    __shared__ float sv[kSortRowMax];
    for (int64_t r = blockIdx.x; r < n; r += gridDim.x) {
        const int64_t s = row_ptr[r], len = row_ptr[r + 1] - s;
        if (len < 2 || len > kSortRowMax) continue; // block-uniform
        int size = 64;
        while (size < len) size <<= 1;
        __syncthreads();
        for (int t = threadIdx.x; t < size; t += blockDim.x) {
            sk[t] = t < len ? col[s + t] : 0x7fffffff;
            sv[t] = t < len ? val[s + t] : 0.0f;
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
                            const float x = sv[t];
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
// Segment range of each row block (its real entries' smallest and largest column).
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
        seg_lo[b] = hi >= 0 ? lo / kTileSeg : 0;
        nseg[b] = hi >= 0 ? hi / kTileSeg - lo / kTileSeg + 1 : 0;
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

// Padded run length of every (row, tile) of the tiled row blocks; one wave per
// row, one lane per segment of the row's block.  Rows past n get empty runs.
__global__ __launch_bounds__(256) void tile_run_len_kernel(const int64_t *__restrict__ row_ptr,
                                                           const int32_t *__restrict__ col, int64_t n, int64_t rows,
                                                           const int32_t *__restrict__ seg_lo,
                                                           const int32_t *__restrict__ nseg,
                                                           const int32_t *__restrict__ blk_tiles, int32_t *__restrict__ run_len)
{
    const int lane = lane_id();
    for (int64_t r = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / kWave; r < rows;
         r += int64_t(gridDim.x) * (blockDim.x / kWave)) {
        const int64_t b = r / kTileRows, rl = r % kTileRows;
        const int ns = nseg[b];
        if (lane >= ns) continue;
        int32_t len = 0;
        if (r < n) {
            const int64_t a = row_ptr[r], e = row_ptr[r + 1];
            const int32_t s0 = (seg_lo[b] + lane) * kTileSeg;
            const int64_t x = row_lower_bound(col, a, e, s0), y = row_lower_bound(col, a, e, s0 + kTileSeg);
            len = int32_t((y - x + 3) & ~int64_t(3));
        }
        run_len[int64_t(blk_tiles[b * kTileMaxSeg + lane]) * kTileRows + rl] = len;
    }
}

// Copy every real entry of a row into its tile run (16-bit column offset within
// the segment), then pad each run with zero-valued entries.
__global__ __launch_bounds__(256) void tile_copy_kernel(const int64_t *__restrict__ row_ptr,
                                                        const int32_t *__restrict__ col, const float *__restrict__ val,
                                                        int64_t n, const int32_t *__restrict__ seg_lo,
                                                        const int32_t *__restrict__ nseg,
                                                        const int32_t *__restrict__ blk_tiles,
                                                        const int32_t *__restrict__ run_off, int64_t max_entries,
                                                        uint16_t *__restrict__ tcol, float *__restrict__ tval)
{
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
            const int32_t sg = c / kTileSeg, k = sg - lo;
            if (k < 0 || k >= ns) continue;
            const int64_t start = row_lower_bound(col, a, e, sg * kTileSeg);
            const int64_t d = int64_t(run_off[int64_t(blk_tiles[b * kTileMaxSeg + k]) * kTileRows + rl]) + (j - start);
            if (d < 0 || d >= max_entries) continue;
            tcol[d] = uint16_t(c - sg * kTileSeg);
            tval[d] = val[j];
        }
        if (lane < ns) { // zero padding at the end of this row's run in segment lo + lane
            const int64_t t = int64_t(blk_tiles[b * kTileMaxSeg + lane]) * kTileRows + rl;
            const int32_t s0 = (lo + lane) * kTileSeg;
            const int64_t len = row_lower_bound(col, a, e, s0 + kTileSeg) - row_lower_bound(col, a, e, s0);
            for (int64_t d = run_off[t] + len; d < run_off[t + 1]; ++d)
                if (d >= 0 && d < max_entries) {
                    tcol[d] = 0;
                    tval[d] = 0.0f;
                }
        }
    }
}

// in-place exclusive scan of int32 values (totals < 2^31): tile sums, one-block scan, tile scan
__global__ __launch_bounds__(256) void i32_reduce_kernel(const int32_t *__restrict__ in, int64_t m,
                                                         int64_t *__restrict__ tile_sum)
{
    __shared__ int64_t s_wave[4];
    const int64_t first = int64_t(blockIdx.x) * kI64Tile + int64_t(threadIdx.x) * kI64Items;
    int64_t acc = 0;
    for (int k = 0; k < kI64Items; ++k)
        if (first + k < m) acc += in[first + k];
    int64_t tot;
    block_excl_i64(acc, s_wave, &tot);
    if (threadIdx.x == 0) tile_sum[blockIdx.x] = tot;
}

__global__ __launch_bounds__(256) void i32_down_kernel(int32_t *__restrict__ io, int64_t m,
                                                       const int64_t *__restrict__ tile_off)
{
    __shared__ int64_t s_wave[4];
    const int64_t first = int64_t(blockIdx.x) * kI64Tile + int64_t(threadIdx.x) * kI64Items;
    int64_t loc[kI64Items], acc = 0;
#pragma unroll
    for (int k = 0; k < kI64Items; ++k) {
        loc[k] = (first + k < m) ? io[first + k] : 0;
        acc += loc[k];
    }
    int64_t tot;
    int64_t run = block_excl_i64(acc, s_wave, &tot) + tile_off[blockIdx.x];
#pragma unroll
    for (int k = 0; k < kI64Items; ++k) {
        if (first + k < m) io[first + k] = int32_t(run);
        run += loc[k];
    }
}

__global__ void i64_to_i32_kernel(const int64_t *__restrict__ x, int32_t *__restrict__ y) { *y = int32_t(*x); }

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

// kAttBlock threads, kAttSeg points of Y per LDS segment, kAttRG rows per lane group.
// Rows of the layout are sorted, padded to whole vectors and 16-byte aligned;
// lane `sub` of a row's group holds the vectors sub, sub + 16, sub + 32, ...
template <int kAttBlock, int kAttSeg, int kAttRG>
__global__ __launch_bounds__(kAttBlock) void attract_staged_kernel(
    const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col, const float *__restrict__ val,
    const float2 *__restrict__ ylay, int64_t n, int max_segs, float2 *__restrict__ fattr)
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
        const bool sorted = re[r] - rs[r] <= kSortRowMax;
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
        if (i < n && sub == 0) fattr[i] = make_float2(ax, ay);
    }
}

// ------------------------------------------------------------------ tiled attraction
// Tiles are stored segment-major and handed out in items: up to kItemMaxTiles
// consecutive tiles of one segment.  One block per item puts the segment's
// 16384 points of Y in LDS once, then each wave walks the item's tiles without
// further barriers.  In a tile, 4-lane group g owns the adjacent rows 4g..4g+3
// (their runs are bounded by 5 consecutive run offsets) and takes 4 entries
// per lane and row per step (an 8-byte column load and a 16-byte value load).
// The loads of the next step, or of the next tile's first step, are issued
// before the current entries are summed, into the other of two register
// buffers; run offsets and y_i are fetched one tile ahead.  Plain loads: with
// the non-temporal hint the half-used lines left the cache before the next
// step came back for their other half.  No load sits in
// divergent code (finished lanes load entry 0 and discard it), so each wait
// covers only loads issued a step earlier.  Padding entries carry p = 0.  The
// partial sum of row rl of block b for the k-th segment of the block goes to
// partial[(b * kTileRows + rl) * kTileMaxSeg + k]; rows add them up later in
// a fixed order, so the result does not depend on scheduling.
constexpr int kTileBlock = 1024;
constexpr int kTileG = 4;                                  // lanes per row group
constexpr int kTileRPT = kTileRows / (kTileBlock / kTileG); // rows per lane group
constexpr int kTileStep = 4 * kTileG;                       // entries per row and step
static_assert(kTileRPT == 4, "a group's rows are read as one 16-byte vector of run offsets");

typedef uint16_t v4u16 __attribute__((ext_vector_type(4)));
typedef int32_t v4i32 __attribute__((ext_vector_type(4)));

__device__ inline float quad_sum(float x)
{
    // sum over the 4 lanes of a group (DPP quad permutations); every lane of
    // the group gets the same bits since float addition commutes
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, false)); // [1,0,3,2]
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xF, 0xF, false)); // [2,3,0,1]
    return x;
}

__global__ __launch_bounds__(kTileBlock) void attract_stream_kernel(
    const int32_t *__restrict__ item_tile0, const int32_t *__restrict__ tile_blk,
    const int32_t *__restrict__ tile_seg, const int32_t *__restrict__ tile_k, const int32_t *__restrict__ run_off, const uint16_t *__restrict__ tcol, const float *__restrict__ tval,
    const float2 *__restrict__ ylay, int32_t nitems, float2 *__restrict__ partial)
{
    __shared__ float4 sy4[kTileSeg / 2];
    __shared__ int32_t s_blk[kItemMaxTiles], s_k[kItemMaxTiles];
    const float2 *sy = reinterpret_cast<const float2 *>(sy4);
    const uint32_t it = xcd_contiguous(blockIdx.x, gridDim.x);
    if (it >= uint32_t(nitems)) return; // block-uniform, before any barrier
    const int32_t t0 = item_tile0[it], t1 = item_tile0[it + 1];
    const int32_t sg = tile_seg[t0];
    const int sub = lane_id() % kTileG, grp = threadIdx.x / kTileG;

    // run offsets of rows 4 grp .. 4 grp + 4 and y_i of rows 4 grp + q in tile
    // t.  Past the item's last tile a real tile is read and never used, so no
    // load is guarded.
    auto fetch_rows = [&](int32_t t, int32_t blk, v4i32 &b, int32_t &b4, float2 *yi) {
        const int32_t *ro = run_off + int64_t(t) * kTileRows + 4 * grp;
        b = *reinterpret_cast<const v4i32 *>(ro);
        b4 = ro[4];
        // rows past n lie in the padding of the Y copy and have empty runs
        const float4 *y4 = reinterpret_cast<const float4 *>(ylay + int64_t(blk) * kTileRows + 4 * grp);
        const float4 u = y4[0], w = y4[1];
        yi[0] = make_float2(u.x, u.y);
        yi[1] = make_float2(u.z, u.w);
        yi[2] = make_float2(w.x, w.y);
        yi[3] = make_float2(w.z, w.w);
    };
    v4i32 rb, nrb; // run starts of the current and of the next tile
    int32_t rb4, nrb4; // end of the last run
    float2 yi[kTileRPT], nyi[kTileRPT];
    fetch_rows(t0, tile_blk[t0], rb, rb4, yi);
    {
        const int32_t tn = t0 + 1 < t1 ? t0 + 1 : t0;
        fetch_rows(tn, tile_blk[tn], nrb, nrb4, nyi);
    }
    static_assert(kYPad >= kTileSeg + 2 && kYPad >= kTileRows, "padding must cover one segment and one block");
    // the segment of Y, 8 independent 16-byte loads per thread, in flight
    // together with the first entries below
    constexpr int kStage = kTileSeg / 2 / kTileBlock;
    v4f stage[kStage];
    {
        const v4f *src = reinterpret_cast<const v4f *>(ylay) + int64_t(sg) * (kTileSeg / 2) + threadIdx.x;
#pragma unroll
        for (int q = 0; q < kStage; ++q) stage[q] = src[q * kTileBlock];
    }
    auto run_end = [](const v4i32 &b, int32_t b4, int q) { return q < 3 ? b[q + 1] : b4; };
    // entry index of this lane for row q at step offset `off` (0 once past the run)
    auto entry = [&](const v4i32 &b, int32_t b4, int q, int32_t off) {
        const int32_t at = b[q] + off + 4 * sub;
        return at < run_end(b, b4, q) ? at : 0;
    };
    // two buffers of entries, used in turn: a step sums one while the other
    // receives the next step's loads
    v4u16 ca[kTileRPT], cb[kTileRPT];
    v4f pa[kTileRPT], pb[kTileRPT];
#pragma unroll
    for (int q = 0; q < kTileRPT; ++q) {
        const int32_t ia = entry(rb, rb4, q, 0);
        ca[q] = *reinterpret_cast<const v4u16 *>(tcol + ia);
        pa[q] = *reinterpret_cast<const v4f *>(tval + ia);
    }
    v4f *sv = reinterpret_cast<v4f *>(sy4);
#pragma unroll
    for (int q = 0; q < kStage; ++q) sv[q * kTileBlock + threadIdx.x] = stage[q];
    for (int32_t j = threadIdx.x; j < t1 - t0; j += kTileBlock) {
        s_blk[j] = tile_blk[t0 + j];
        s_k[j] = tile_k[t0 + j];
    }
    __syncthreads();

    float fx[kTileRPT], fy[kTileRPT];
#pragma unroll
    for (int q = 0; q < kTileRPT; ++q) fx[q] = fy[q] = 0.0f;
    int32_t off = 0; // wave-uniform offset of the current step in the tile's runs
    // one step: loads for the next step (or the next tile's first entries)
    // into (cn, pn), then the sum over (cc, pc); returns whether this tile
    // has another step for any row of the wave
    auto step = [&](const v4u16(&cc)[kTileRPT], const v4f(&pc)[kTileRPT], v4u16(&cn)[kTileRPT],
                    v4f(&pn)[kTileRPT]) -> bool {
        bool mine = false;
#pragma unroll
        for (int q = 0; q < kTileRPT; ++q) mine |= rb[q] + off + kTileStep < run_end(rb, rb4, q);
        const bool more = __builtin_amdgcn_ballot_w64(mine) != 0; // wave-uniform
        if (more) {
#pragma unroll
            for (int q = 0; q < kTileRPT; ++q) {
                const int32_t ia = entry(rb, rb4, q, off + kTileStep);
                cn[q] = *reinterpret_cast<const v4u16 *>(tcol + ia);
                pn[q] = *reinterpret_cast<const v4f *>(tval + ia);
            }
        } else {
#pragma unroll
            for (int q = 0; q < kTileRPT; ++q) {
                const int32_t ia = entry(nrb, nrb4, q, 0);
                cn[q] = *reinterpret_cast<const v4u16 *>(tcol + ia);
                pn[q] = *reinterpret_cast<const v4f *>(tval + ia);
            }
        }
#pragma unroll
        for (int q = 0; q < kTileRPT; ++q) {
            float cx = 0.0f, cy = 0.0f;
#pragma unroll
            for (int v = 0; v < 4; ++v) attract_add(yi[q], sy[cc[q][v] & (kTileSeg - 1)], pc[q][v], cx, cy);
            const bool live = rb[q] + off + 4 * sub < run_end(rb, rb4, q);
            fx[q] += live ? cx : 0.0f;
            fy[q] += live ? cy : 0.0f;
        }
        off += kTileStep;
        return more;
    };
    // end of tile t: lane sub stores the partial of row 4 grp + sub, then the
    // rows move on to tile t + 1 and the offsets of tile t + 2 are fetched
    auto tile_end = [&](int32_t t) {
        const int32_t j = t - t0;
        float ax = 0.0f, ay = 0.0f;
#pragma unroll
        for (int q = 0; q < kTileRPT; ++q) {
            const float sx = quad_sum(fx[q]), sy_ = quad_sum(fy[q]);
            ax = sub == q ? sx : ax;
            ay = sub == q ? sy_ : ay;
            fx[q] = fy[q] = 0.0f;
            yi[q] = nyi[q];
        }
        partial[(int64_t(s_blk[j]) * kTileRows + 4 * grp + sub) * kTileMaxSeg + s_k[j]] = make_float2(ax, ay);
        rb = nrb;
        rb4 = nrb4;
        off = 0;
        const int32_t tn = t + 2 < t1 ? t + 2 : t;
        fetch_rows(tn, s_blk[tn - t0], nrb, nrb4, nyi);
    };

    // steps alternate between the buffers across tile boundaries (two per trip)
    int32_t t = t0;
    for (;;) {
        if (!step(ca, pa, cb, pb)) {
            tile_end(t);
            if (++t == t1) break;
        }
        if (!step(cb, pb, ca, pa)) {
            tile_end(t);
            if (++t == t1) break;
        }
    }
}

// ------------------------------------------------------------------ gradient + update
// In the caller's order: g = 4 (alpha F_attr - F_rep / Z), then the gains /
// momentum update of the optimiser (when a.update).
// F_attr of a row in layout order: either one value per row, or (tiled) the
// sum of the row's per-tile partials in tile order.
__global__ __launch_bounds__(256) void update_kernel(const float2 *__restrict__ fattr_lay,
                                                     const uint32_t *__restrict__ rank, int tiled,
                                                     const int32_t *__restrict__ blk_nseg,
                                                     const float2 *__restrict__ frep, const Header *__restrict__ hdr,
                                                     int64_t n, StepArgs a, float2 *__restrict__ Y,
                                                     float2 *__restrict__ upd, float2 *__restrict__ gains,
                                                     float2 *__restrict__ grad)
{
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float inv_z = float(1.0 / hdr->Z);
    const uint32_t r = rank[i];
    float2 fa = make_float2(0.0f, 0.0f);
    if (r < uint32_t(n)) {
        if (tiled) { // the row's partials are adjacent: [row][segment of its block]
            const int ns = blk_nseg[r / kTileRows];
            const float2 *q = fattr_lay + int64_t(r) * kTileMaxSeg;
            for (int k = 0; k < ns; ++k) {
                fa.x += q[k].x;
                fa.y += q[k].y;
            }
        } else {
            fa = fattr_lay[r];
        }
    }
    const float2 fr = frep[i];
    const float gx = 4.0f * (a.alpha * fa.x - fr.x * inv_z);
    const float gy = 4.0f * (a.alpha * fa.y - fr.y * inv_z);
    if (grad) grad[i] = make_float2(gx, gy);
    if (a.update) {
        float2 u = upd[i], gn = gains[i];
        const float2 y = Y[i];
        gn.x = (u.x * gx < 0.0f) ? gn.x + 0.2f : gn.x * 0.8f;
        gn.y = (u.y * gy < 0.0f) ? gn.y + 0.2f : gn.y * 0.8f;
        gn.x = fmaxf(gn.x, a.min_gain);
        gn.y = fmaxf(gn.y, a.min_gain);
        u.x = a.momentum * u.x - a.learning_rate * gn.x * gx;
        u.y = a.momentum * u.y - a.learning_rate * gn.y * gy;
        Y[i] = make_float2(y.x + u.x, y.y + u.y);
        upd[i] = u;
        gains[i] = gn;
    }
}

// ------------------------------------------------------------------ launchers
LayoutView layout_view(void *mem, int64_t n, int64_t nnz)
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
    size_t o_col = take(4 * cap), o_val = take(4 * cap);
    // tiled copy: at most kTileMaxSeg tiles per row block, runs padded to 4 entries
    const int64_t blocks = (n + kTileRows - 1) / kTileRows;
    v.max_tiles = blocks * kTileMaxSeg;
    v.max_entries = nnz + 3 * int64_t(kTileRows) * v.max_tiles + 8;
    size_t o_lo = take(4 * size_t(blocks)), o_ns = take(4 * size_t(blocks)),
           o_bt = take(4 * size_t(blocks) * kTileMaxSeg), o_tb = take(4 * size_t(v.max_tiles)),
           o_ts = take(4 * size_t(v.max_tiles)), o_tk = take(4 * size_t(v.max_tiles)),
           o_it = take(4 * size_t(v.max_tiles + 1)),
           o_ro = take(4 * size_t(v.max_tiles * kTileRows + 1)), o_tc = take(2 * size_t(v.max_entries)),
           o_tv = take(4 * size_t(v.max_entries));
    v.bytes = off;
    if (mem) {
        v.perm = at<uint32_t>(mem, o_perm);
        v.rank = at<uint32_t>(mem, o_rank);
        v.row_ptr = at<int64_t>(mem, o_ptr);
        v.col = at<int32_t>(mem, o_col);
        v.val = at<float>(mem, o_val);
        v.blk_seg_lo = at<int32_t>(mem, o_lo);
        v.blk_nseg = at<int32_t>(mem, o_ns);
        v.blk_tiles = at<int32_t>(mem, o_bt);
        v.tile_blk = at<int32_t>(mem, o_tb);
        v.tile_seg = at<int32_t>(mem, o_ts);
        v.tile_k = at<int32_t>(mem, o_tk);
        v.item_tile0 = at<int32_t>(mem, o_it);
        v.run_off = at<int32_t>(mem, o_ro);
        v.tcol = at<uint16_t>(mem, o_tc);
        v.tval = at<float>(mem, o_tv);
    }
    return v;
}

// The tiled copy of a built (sorted, padded) layout; plan->tiled stays false when
// some row block spans more than kTileMaxSeg segments.
static int build_tiles(const LayoutView &lv, int64_t n, TilePlan *plan, void *ws, const Layout &L, hipStream_t st)
{
    *plan = TilePlan{};
    const int64_t blocks = (n + kTileRows - 1) / kTileRows;
    plan->blocks = int32_t(blocks);
    tile_block_range_kernel<<<unsigned(blocks), 256, 0, st>>>(lv.row_ptr, lv.col, n, lv.blk_seg_lo, lv.blk_nseg);
    std::vector<int32_t> lo(blocks), ns(blocks);
    if (hipMemcpyAsync(lo.data(), lv.blk_seg_lo, 4 * blocks, hipMemcpyDeviceToHost, st) != hipSuccess) return -1;
    if (hipMemcpyAsync(ns.data(), lv.blk_nseg, 4 * blocks, hipMemcpyDeviceToHost, st) != hipSuccess) return -1;
    if (hipStreamSynchronize(st) != hipSuccess) return -1;
    // tiles in segment-major order, (block, k) -> tile, then items of up to
    // `per` tiles that never straddle a segment (a few items per CU)
    std::vector<std::pair<int32_t, int32_t>> order; // (segment, block)
    for (int64_t b = 0; b < blocks; ++b) {
        if (ns[b] > kTileMaxSeg) return 0; // too wide: keep the row-block kernel
        for (int k = 0; k < ns[b]; ++k) order.emplace_back(lo[b] + k, int32_t(b));
    }
    const int64_t tiles = int64_t(order.size());
    if (tiles == 0 || tiles > lv.max_tiles) return 0;
    std::sort(order.begin(), order.end());
    std::vector<int32_t> bt(size_t(blocks) * kTileMaxSeg, -1), tb(tiles), ts(tiles), tk(tiles), items;
    for (int64_t t = 0; t < tiles; ++t) {
        ts[t] = order[t].first;
        tb[t] = order[t].second;
        tk[t] = ts[t] - lo[tb[t]];
        bt[size_t(tb[t]) * kTileMaxSeg + tk[t]] = int32_t(t);
    }
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess)
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const int64_t per = std::min<int64_t>(kItemMaxTiles, std::max<int64_t>(1, (tiles + 4 * cus - 1) / (4 * cus)));
    for (int64_t t = 0; t < tiles; ++t)
        if (items.empty() || ts[t] != ts[items.back()] || t - items.back() >= per) items.push_back(int32_t(t));
    const int64_t nitems = int64_t(items.size());
    items.push_back(int32_t(tiles));
    if (hipMemcpyAsync(lv.blk_tiles, bt.data(), 4 * bt.size(), hipMemcpyHostToDevice, st) != hipSuccess) return -1;
    if (hipMemcpyAsync(lv.tile_blk, tb.data(), 4 * tiles, hipMemcpyHostToDevice, st) != hipSuccess) return -1;
    if (hipMemcpyAsync(lv.tile_seg, ts.data(), 4 * tiles, hipMemcpyHostToDevice, st) != hipSuccess) return -1;
    if (hipMemcpyAsync(lv.tile_k, tk.data(), 4 * tiles, hipMemcpyHostToDevice, st) != hipSuccess) return -1;
    if (hipMemcpyAsync(lv.item_tile0, items.data(), 4 * items.size(), hipMemcpyHostToDevice, st) != hipSuccess)
        return -1;
    const int64_t rows = blocks * kTileRows, m = tiles * kTileRows;
    const unsigned gw = unsigned((rows + 3) / 4 < 65535 * 4 ? (rows + 3) / 4 : 65535 * 4);
    tile_run_len_kernel<<<gw, 256, 0, st>>>(lv.row_ptr, lv.col, n, rows, lv.blk_seg_lo, lv.blk_nseg, lv.blk_tiles,
                                            lv.run_off);
    const int64_t st_tiles = (m + kI64Tile - 1) / kI64Tile;
    int64_t *tsum = at<int64_t>(ws, L.codes1); // scratch: m / 4096 + 1 entries << n
    int64_t *total = at<int64_t>(ws, L.codes1) + st_tiles + 1;
    i32_reduce_kernel<<<unsigned(st_tiles), 256, 0, st>>>(lv.run_off, m, tsum);
    i64_top_kernel<<<1, 256, 0, st>>>(tsum, st_tiles, total);
    i32_down_kernel<<<unsigned(st_tiles), 256, 0, st>>>(lv.run_off, m, tsum);
    i64_to_i32_kernel<<<1, 1, 0, st>>>(total, lv.run_off + m);
    int64_t entries = 0;
    if (hipMemcpyAsync(&entries, total, 8, hipMemcpyDeviceToHost, st) != hipSuccess) return -1;
    if (hipStreamSynchronize(st) != hipSuccess) return -1;
    if (entries > lv.max_entries) return 0;
    tile_copy_kernel<<<unsigned(n < 65535 * 4 ? (n + 3) / 4 : 65535 * 4), 256, 0, st>>>(
        lv.row_ptr, lv.col, lv.val, n, lv.blk_seg_lo, lv.blk_nseg, lv.blk_tiles, lv.run_off, lv.max_entries, lv.tcol,
        lv.tval);
    if (hipGetLastError() != hipSuccess) return -1;
    plan->tiled = true;
    plan->tiles = int32_t(tiles);
    plan->items = int32_t(nitems);
    plan->entries = entries;
    return 0;
}

int launch_layout_build(const int64_t *row_ptr, const int32_t *col, const float *val, int64_t n, int64_t nnz,
                        const float *Y, const LayoutView &lv, TilePlan *plan, void *ws, const Layout &L,
                        hipStream_t st)
{
    Header *hdr = at<Header>(ws, L.header);
    uint32_t *parent = at<uint32_t>(ws, L.split_b);
    uint32_t *changed = at<uint32_t>(ws, L.split_e);
    const unsigned gn = unsigned((n + 255) / 256);
    const unsigned gw = unsigned((n + 3) / 4 < 65535 * 4 ? (n + 3) / 4 : 65535 * 4);
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
    // keys: component, then Morton order of Y when given
    if (Y) {
        launch_bbox(Y, n, ws, L, st);
        launch_morton(Y, n, nullptr, ws, L, st);
    } else {
        sort_reset_kernel<<<1, 256, 0, st>>>(hdr, at<uint32_t>(ws, L.hist));
    }
    uint64_t *keys = at<uint64_t>(ws, L.codes0);
    layout_keys_kernel<<<gn, 256, 0, st>>>(keys, parent, n, Y ? 1 : 0);
    sort_reset_kernel<<<1, 256, 0, st>>>(hdr, at<uint32_t>(ws, L.hist));
    keys_hist_kernel<<<unsigned(L.sort_tiles), kSortBlock, 0, st>>>(keys, n, at<uint32_t>(ws, L.hist),
                                                                    at<uint32_t>(ws, L.status), L.sort_tiles);
    launch_sort(n, Y ? Y : reinterpret_cast<const float *>(at<float2>(ws, L.ycopy)), ws, L, st);
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
    layout_copy_kernel<<<gw, 256, 0, st>>>(row_ptr, col, val, lv.perm, lv.rank, lv.row_ptr, n, cap, lv.col, lv.val);
    layout_sentinel_kernel<<<1, 1, 0, st>>>(lv.row_ptr, n, lv.col, lv.val);
    layout_sort_rows_kernel<<<unsigned(n < 65535 * 16 ? n : 65535 * 16), 256, 0, st>>>(lv.row_ptr, lv.col, lv.val, n);
    if (hipGetLastError() != hipSuccess) return -1;
    return build_tiles(lv, n, plan, ws, L, st);
}

template <int B, int S, int RG>
static void launch_staged(const LayoutView &lv, int64_t n, int64_t nnz, int max_segs, void *ws, const Layout &L,
                          hipStream_t st)
{
    constexpr int rows = (B / kAttG) * RG;
    const int64_t blocks = ((n + rows - 1) / rows + 7) / 8 * 8; // multiple of 8 for the XCD remap
    attract_staged_kernel<B, S, RG><<<unsigned(blocks), B, 0, st>>>(lv.row_ptr, lv.col, lv.val, at<float2>(ws, L.ycopy),
                                                                   n, max_segs, at<float2>(ws, L.fattr));
}

void launch_attract_layout(const LayoutView &lv, int64_t n, int64_t nnz, int tiles, int items, int max_segs, void *ws,
                           const Layout &L, hipStream_t st)
{
    if (tiles > 0) {
        const unsigned grid = unsigned((items + 7) / 8 * 8); // multiple of 8 for the XCD remap
        attract_stream_kernel<<<grid, kTileBlock, 0, st>>>(lv.item_tile0, lv.tile_blk, lv.tile_seg, lv.tile_k,
                                                           lv.run_off, lv.tcol, lv.tval, at<float2>(ws, L.ycopy),
                                                           items, at<float2>(ws, L.partial));
        return;
    }
    // 1024 threads (one block per CU: the segment fills 128 KB of LDS), 2 rows per lane group
    launch_staged<1024, 16384, 2>(lv, n, nnz, max_segs, ws, L, st);
}

void launch_update(const LayoutView &lv, int64_t n, int tiled, const StepArgs &a, float *Y, float *upd, float *gains,
                   float *grad, void *ws, const Layout &L, hipStream_t st)
{
    update_kernel<<<unsigned((n + 255) / 256), 256, 0, st>>>(
        at<float2>(ws, tiled ? L.partial : L.fattr), lv.rank, tiled, lv.blk_nseg, at<float2>(ws, L.frep),
        at<Header>(ws, L.header), n, a,
        reinterpret_cast<float2 *>(Y), reinterpret_cast<float2 *>(upd), reinterpret_cast<float2 *>(gains),
        reinterpret_cast<float2 *>(grad));
}

} // namespace bht
