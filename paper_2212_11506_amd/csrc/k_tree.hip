// Compressed quadtree over the sorted Morton codes, with cell summaries.
//
// Quadtree Building: a cell at level L is the set of codes that share their
// top 2L bits, so every cell is a contiguous range of the sorted codes.  A
// cell is a node of the compressed tree when its points fall into at least
// two quadrants (the root always is one); a run of identical codes forms a
// bucket cell at level 32, and every point is a single-point leaf (the
// members of a bucket are its children, so a walk treats a bucket like any
// other cell: its summary when far enough, else its points one by one).
//
// Parallel construction, one thread per sorted position:
//   1. For each adjacent pair (s, s+1) the split level is
//      lambda_s = floor(clz(M_s ^ M_s+1) / 2).  The cell at that level around
//      s is found by galloping searches; the first split of a cell owns it and
//      marks bit L of levelmask[begin].
//   2. Nodes are numbered in depth-first pre-order, which is the order of
//      (begin, level), bucket members sitting at level 33.  With cnt(x) = 1
//      (the point's leaf) + 1 if a bucket starts at x + popcount(levelmask[x])
//      and base = exclusive scan of cnt, node (L, [b,e)) sits at
//      base[b] + popcount(levelmask[b] & (2^L - 1)), and the first node after
//      its subtree is base[e].
//   3. Summaries (Parallel Summarization) come from fp64 prefix sums of the
//      sorted coordinates: com = (S[e] - S[b]) / (e - b), so no bottom-up
//      level sweep is needed (cells of up to 32 points sum their points
//      directly instead).
//
// The same kernels build the octree of a 3-D embedding: D = 3 reads 3-bit
// digits from 63-bit codes (Geom<3>), keeps three prefix sums and writes
// 32-byte records; D = 2 with T = double is the fp64 variant.
#include "common.hpp"
#include "kernels.hpp"

namespace bht {

// first index in [0, s] whose code shares the top (64 - sh) bits of key
__device__ inline int64_t gallop_left(const uint64_t *__restrict__ codes, int64_t s, uint64_t key, int sh)
{
    int64_t hi = s, lo = -1, step = 1;
    for (;;) {
        int64_t probe = s - step;
        if (probe < 0) break;
        if (((codes[probe] ^ key) >> sh) != 0) {
            lo = probe;
            break;
        }
        hi = probe;
        step <<= 1;
    }
    while (hi - lo > 1) {
        int64_t mid = lo + (hi - lo) / 2;
        if (((codes[mid] ^ key) >> sh) == 0)
            hi = mid;
        else
            lo = mid;
    }
    return hi;
}

// one past the last index >= s whose code shares the top (64 - sh) bits of key
__device__ inline int64_t gallop_right(const uint64_t *__restrict__ codes, int64_t s, int64_t n,
                                       uint64_t key, int sh)
{
    int64_t lo = s, hi = n, step = 1;
    for (;;) {
        int64_t probe = s + step;
        if (probe >= n) break;
        if (((codes[probe] ^ key) >> sh) != 0) {
            hi = probe;
            break;
        }
        lo = probe;
        step <<= 1;
    }
    while (hi - lo > 1) {
        int64_t mid = lo + (hi - lo) / 2;
        if (((codes[mid] ^ key) >> sh) == 0)
            lo = mid;
        else
            hi = mid;
    }
    return hi;
}

// equality run of identical codes starting at x
__device__ inline int64_t run_end(const uint64_t *__restrict__ codes, int64_t x, int64_t n)
{
    uint64_t k = codes[x];
    if (x + 1 >= n || codes[x + 1] != k) return x + 1;
    int64_t lo = x + 1, hi = n, step = 2;
    for (;;) {
        int64_t probe = x + step;
        if (probe >= n) break;
        if (codes[probe] != k) {
            hi = probe;
            break;
        }
        lo = probe;
        step <<= 1;
    }
    while (hi - lo > 1) {
        int64_t mid = lo + (hi - lo) / 2;
        if (codes[mid] == k)
            lo = mid;
        else
            hi = mid;
    }
    return hi;
}

// ------------------------------------------------------------------ 1. splits
// One block per kSplitBlock consecutive splits.  The sorted codes around the
// block, kSplitWin on either side, are staged in LDS and each split gallops
// there for the two ends of its cell.  An end beyond the window (a cell of
// more than kSplitWin points past the block) is found by one wave for the
// whole block: 64 probes per round narrow the range 65-fold, so four or five
// rounds of loads replace the twenty-odd dependent loads of a gallop through
// global memory, which the other lanes of its wave would have waited for.
constexpr int kSplitBlock = 512;
constexpr int kSplitWin = 1024;

__device__ inline bool same_cell(uint64_t c, uint64_t key, int sh) { return ((c ^ key) >> sh) == 0; }

// first index in (lo, hi] whose code shares the top (64 - sh) bits of key, where
// the codes sharing them are a suffix of (lo, hi] that includes hi (one wave)
__device__ inline int64_t wave_first_same(const uint64_t *__restrict__ codes, int64_t lo, int64_t hi,
                                          uint64_t key, int sh)
{
    const int lane = lane_id();
    while (hi - lo > 1) {
        const int64_t span = hi - lo - 1; // candidates lo + 1 .. hi - 1
        const int64_t step = span <= kWave ? 1 : (span + kWave) / (kWave + 1);
        const int64_t p = lo + (int64_t(lane) + 1) * step;
        const bool in = p < hi;
        const uint64_t yes = ballot(in && same_cell(codes[p], key, sh));
        const uint64_t inm = ballot(in);
        if (yes) {
            const int k = __ffsll((unsigned long long)yes) - 1;
            hi = lo + (int64_t(k) + 1) * step;
            lo = k > 0 ? lo + int64_t(k) * step : lo;
        } else {
            const int k = 63 - __clzll((long long)inm); // last probe in range
            lo = lo + (int64_t(k) + 1) * step;
        }
    }
    return hi;
}

// first index in [lo, hi) whose code does not share the top bits of key, where
// the codes sharing them are a prefix of [lo, hi) that includes lo (hi if none)
__device__ inline int64_t wave_first_other(const uint64_t *__restrict__ codes, int64_t lo, int64_t hi,
                                           uint64_t key, int sh)
{
    const int lane = lane_id();
    // invariant: codes[lo] shares, index hi differs (or is the end)
    while (hi - lo > 1) {
        const int64_t span = hi - lo - 1;
        const int64_t step = span <= kWave ? 1 : (span + kWave) / (kWave + 1);
        const int64_t p = lo + (int64_t(lane) + 1) * step;
        const bool in = p < hi;
        const uint64_t no = ballot(in && !same_cell(codes[p], key, sh));
        const uint64_t inm = ballot(in);
        if (no) {
            const int k = __ffsll((unsigned long long)no) - 1;
            hi = lo + (int64_t(k) + 1) * step;
            lo = k > 0 ? lo + int64_t(k) * step : lo;
        } else {
            const int k = 63 - __clzll((long long)inm);
            lo = lo + (int64_t(k) + 1) * step;
        }
    }
    return hi;
}

template <int D>
__global__ __launch_bounds__(kSplitBlock) void tree_splits_kernel(const uint64_t *__restrict__ codes, int64_t n,
                                                                  uint32_t *__restrict__ levelmask,
                                                                  uint32_t *__restrict__ split_b,
                                                                  uint32_t *__restrict__ split_e)
{
    using G = Geom<D>;
    __shared__ uint64_t s_c[kSplitBlock + 2 * kSplitWin + 1];
    __shared__ int64_t s_b[kSplitBlock], s_e[kSplitBlock];
    __shared__ uint16_t s_hard[2 * kSplitBlock];
    __shared__ uint32_t s_nhard;
    const int t = threadIdx.x;
    const int64_t base = int64_t(blockIdx.x) * kSplitBlock;
    const int64_t wlo = base > kSplitWin ? base - kSplitWin : 0;
    const int64_t whi = base + kSplitBlock + kSplitWin < n ? base + kSplitBlock + kSplitWin : n;
    for (int64_t i = t; i < whi - wlo; i += kSplitBlock) s_c[i] = codes[wlo + i];
    if (t == 0) s_nhard = 0;
    __syncthreads();

    const int64_t s = base + t;
    if (s == 0) atomicOr(&levelmask[0], 1u); // the root always exists
    bool split = false;
    int L = 0;
    uint64_t ms = 0;
    if (s < n - 1) {
        ms = s_c[s - wlo];
        const uint64_t mn = s_c[s + 1 - wlo];
        split = ms != mn;
        if (split) L = G::split_level(ms, mn);
    }
    int64_t b = 0, e = n;
    if (split && L > 0) {
        const int sh = G::cell_shift(L);
        // in window coordinates; the window holds s and s + 1
        const int64_t bl = gallop_left(s_c, s - wlo, ms, sh);
        const int64_t el = gallop_right(s_c, s + 1 - wlo, whi - wlo, ms, sh);
        b = wlo + bl;
        e = wlo + el;
        if (bl == 0 && wlo > 0) s_hard[atomicAdd(&s_nhard, 1u)] = uint16_t(2 * t);      // begin before the window
        if (el == whi - wlo && whi < n) s_hard[atomicAdd(&s_nhard, 1u)] = uint16_t(2 * t + 1); // end after it
    }
    s_b[t] = b;
    s_e[t] = e;
    __syncthreads();
    // cell ends past the window: one wave each
    const uint32_t nh = s_nhard;
    for (uint32_t h = uint32_t(t / kWave); h < nh; h += kSplitBlock / kWave) {
        const int owner = s_hard[h] >> 1, dir = s_hard[h] & 1;
        const uint64_t key = s_c[base + owner - wlo];
        const int sh = G::cell_shift(G::split_level(key, s_c[base + owner + 1 - wlo]));
        if (dir == 0) {
            // codes[wlo] shares the cell; find its first index in [0, wlo]
            const int64_t r = wave_first_same(codes, -1, wlo, key, sh);
            if (lane_id() == 0) s_b[owner] = r;
        } else {
            // codes[whi - 1] shares the cell; find the first index past it
            const int64_t r = wave_first_other(codes, whi - 1, n, key, sh);
            if (lane_id() == 0) s_e[owner] = r;
        }
    }
    __syncthreads();
    if (!split) {
        if (s < n - 1) split_e[s] = 0;
        return;
    }
    b = s_b[t];
    e = s_e[t];
    const uint64_t cb = b >= wlo ? s_c[b - wlo] : codes[b];
    const bool owner = G::digit(cb, L) == G::digit(ms, L);
    if (owner) {
        atomicOr(&levelmask[b], 1u << L);
        split_b[s] = uint32_t(b);
        split_e[s] = uint32_t(e);
    } else {
        split_e[s] = 0;
    }
}

// ------------------------------------------------------------------ 2. scans
// One element per sorted position: its node count and its coordinates
// relative to the box centre (D of them), scanned together.
template <int D> struct ScanVal {
    uint32_t c;
    double s[D];
};

template <int D> __device__ inline ScanVal<D> scan_add(const ScanVal<D> &a, const ScanVal<D> &b)
{
    ScanVal<D> r;
    r.c = a.c + b.c;
#pragma unroll
    for (int k = 0; k < D; ++k) r.s[k] = a.s[k] + b.s[k];
    return r;
}

template <int D> __device__ inline ScanVal<D> scan_zero()
{
    ScanVal<D> r;
    r.c = 0;
#pragma unroll
    for (int k = 0; k < D; ++k) r.s[k] = 0.0;
    return r;
}

template <int D> __device__ inline ScanVal<D> shfl_up(const ScanVal<D> &v, int o)
{
    ScanVal<D> r;
    r.c = __shfl_up(v.c, o, kWave);
#pragma unroll
    for (int k = 0; k < D; ++k) r.s[k] = __shfl_up(v.s[k], o, kWave);
    return r;
}

template <int D, typename T>
__device__ inline ScanVal<D> element(const uint64_t *__restrict__ codes, const uint32_t *__restrict__ levelmask,
                                     const point_t<D, T> *__restrict__ ys, int64_t x, int64_t n, const double *c)
{
    const uint64_t k = codes[x];
    const uint32_t bucket = (x == 0 || codes[x - 1] != k) && x + 1 < n && codes[x + 1] == k ? 1u : 0u;
    const point_t<D, T> y = ys[x];
    ScanVal<D> r;
    r.c = 1u + bucket + uint32_t(__popc(levelmask[x]));
#pragma unroll
    for (int d = 0; d < D; ++d) r.s[d] = double(coord(y, d)) - c[d];
    return r;
}

// exclusive block scan of one ScanVal per thread (256 threads); returns the block total
template <int D>
__device__ inline ScanVal<D> block_scan_excl(ScanVal<D> v, ScanVal<D> *s_wave /*[4]*/, ScanVal<D> *out_total)
{
    int lane = lane_id(), w = threadIdx.x / kWave;
    ScanVal<D> x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        ScanVal<D> y = shfl_up(x, o);
        if (lane >= o) x = scan_add(y, x);
    }
    if (lane == kWave - 1) s_wave[w] = x;
    __syncthreads();
    ScanVal<D> off = scan_zero<D>(), tot = scan_zero<D>();
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if (k < w) off = scan_add(off, s_wave[k]);
        tot = scan_add(tot, s_wave[k]);
    }
    *out_total = tot;
    // exclusive: total of earlier waves + inclusive-in-wave of the previous lane
    ScanVal<D> prev = shfl_up(x, 1);
    if (lane == 0) prev = scan_zero<D>();
    return scan_add(off, prev);
}

template <int D> __device__ inline void load_centre(const Header *hdr, double *c)
{
#pragma unroll
    for (int d = 0; d < D; ++d) c[d] = hdr->cent[d];
}

template <int D, typename T>
__global__ __launch_bounds__(kScanBlock) void scan_reduce_kernel(
    const uint64_t *__restrict__ codes, const uint32_t *__restrict__ levelmask,
    const point_t<D, T> *__restrict__ ys, const Header *__restrict__ hdr, int64_t n,
    uint32_t *__restrict__ tile_cnt, double *__restrict__ tile_sum)
{
    __shared__ ScanVal<D> s_wave[4];
    double c[D];
    load_centre<D>(hdr, c);
    int64_t first = int64_t(blockIdx.x) * kScanTile + int64_t(threadIdx.x) * kScanItems;
    ScanVal<D> acc = scan_zero<D>();
    for (int k = 0; k < kScanItems; ++k) {
        int64_t x = first + k;
        if (x < n) acc = scan_add(acc, element<D, T>(codes, levelmask, ys, x, n, c));
    }
    ScanVal<D> tot;
    block_scan_excl(acc, s_wave, &tot);
    if (threadIdx.x == 0) {
        tile_cnt[blockIdx.x] = tot.c;
#pragma unroll
        for (int d = 0; d < D; ++d) tile_sum[int64_t(blockIdx.x) * D + d] = tot.s[d];
    }
}

// one block: exclusive scan over the tile totals, in place; totals -> base[n], psum[n]
template <int D>
__global__ __launch_bounds__(kScanBlock) void scan_top_kernel(uint32_t *__restrict__ tile_cnt,
                                                              double *__restrict__ tile_sum, int64_t tiles,
                                                              int64_t n, uint32_t *__restrict__ base,
                                                              double *__restrict__ psum,
                                                              Header *__restrict__ hdr)
{
    __shared__ ScanVal<D> s_wave[4];
    int64_t per = (tiles + kScanBlock - 1) / kScanBlock;
    int64_t first = int64_t(threadIdx.x) * per;
    auto load = [&](int64_t t) {
        ScanVal<D> v;
        v.c = tile_cnt[t];
#pragma unroll
        for (int d = 0; d < D; ++d) v.s[d] = tile_sum[t * D + d];
        return v;
    };
    ScanVal<D> acc = scan_zero<D>();
    for (int64_t k = 0; k < per; ++k) {
        int64_t t = first + k;
        if (t < tiles) acc = scan_add(acc, load(t));
    }
    ScanVal<D> tot;
    ScanVal<D> run = block_scan_excl(acc, s_wave, &tot);
    for (int64_t k = 0; k < per; ++k) {
        int64_t t = first + k;
        if (t < tiles) {
            const ScanVal<D> v = load(t);
            tile_cnt[t] = run.c;
#pragma unroll
            for (int d = 0; d < D; ++d) tile_sum[t * D + d] = run.s[d];
            run = scan_add(run, v);
        }
    }
    if (threadIdx.x == 0) {
        base[n] = tot.c;
#pragma unroll
        for (int d = 0; d < D; ++d) psum[n * D + d] = tot.s[d];
        hdr->nodes = tot.c;
    }
}

template <int D, typename T>
__global__ __launch_bounds__(kScanBlock) void scan_down_kernel(
    const uint64_t *__restrict__ codes, const uint32_t *__restrict__ levelmask,
    const point_t<D, T> *__restrict__ ys, const Header *__restrict__ hdr, int64_t n,
    const uint32_t *__restrict__ tile_cnt, const double *__restrict__ tile_sum,
    uint32_t *__restrict__ base, double *__restrict__ psum)
{
    __shared__ ScanVal<D> s_wave[4];
    double c[D];
    load_centre<D>(hdr, c);
    int64_t first = int64_t(blockIdx.x) * kScanTile + int64_t(threadIdx.x) * kScanItems;
    ScanVal<D> loc[kScanItems];
    ScanVal<D> acc = scan_zero<D>();
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        int64_t x = first + k;
        loc[k] = (x < n) ? element<D, T>(codes, levelmask, ys, x, n, c) : scan_zero<D>();
        acc = scan_add(acc, loc[k]);
    }
    ScanVal<D> tot;
    ScanVal<D> run = block_scan_excl(acc, s_wave, &tot);
    ScanVal<D> tile_off;
    tile_off.c = tile_cnt[blockIdx.x];
#pragma unroll
    for (int d = 0; d < D; ++d) tile_off.s[d] = tile_sum[int64_t(blockIdx.x) * D + d];
    run = scan_add(tile_off, run);
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        int64_t x = first + k;
        if (x < n) {
            base[x] = run.c;
#pragma unroll
            for (int d = 0; d < D; ++d) psum[x * D + d] = run.s[d];
        }
        run = scan_add(run, loc[k]);
    }
}

// ------------------------------------------------------------------ 3. nodes
__device__ inline double accept_threshold(double rspan, int L, double theta2)
{
    if (!(theta2 > 0.0)) return INFINITY;
    double side = ldexp(2.0 * rspan, -L);
    return side * side / theta2;
}

// one node record, as three 8-byte stores (records are 8-byte aligned)
__device__ inline void store_node(char *__restrict__ nodes, int64_t pre, float2 com, float count, float thr,
                                  uint32_t next, uint32_t self)
{
    uint2 *r = reinterpret_cast<uint2 *>(nodes + pre * kNodeBytes);
    r[0] = make_uint2(__float_as_uint(com.x), __float_as_uint(com.y));
    r[1] = make_uint2(__float_as_uint(count), __float_as_uint(thr));
    r[2] = make_uint2(next, self);
}

// the fp64 variant's record: {com.x, com.y, thr, count, next, self}
__device__ inline void store_node(char *__restrict__ nodes, int64_t pre, double2 com, float count, double thr,
                                  uint32_t next, uint32_t self)
{
    double *d = reinterpret_cast<double *>(nodes + pre * kNodeBytes64);
    d[0] = com.x;
    d[1] = com.y;
    d[2] = thr;
    uint2 *r = reinterpret_cast<uint2 *>(d + 3);
    r[0] = make_uint2(__float_as_uint(count), next);
    r[1] = make_uint2(self, 0u);
}

// a 3-D record: {com.x, com.y, com.z, count, thr, next, self, 0}, two 16-byte stores
__device__ inline void store_node(char *__restrict__ nodes, int64_t pre, float3 com, float count, float thr,
                                  uint32_t next, uint32_t self)
{
    uint4 *r = reinterpret_cast<uint4 *>(nodes + pre * kNodeBytes3);
    r[0] = make_uint4(__float_as_uint(com.x), __float_as_uint(com.y), __float_as_uint(com.z), __float_as_uint(count));
    r[1] = make_uint4(__float_as_uint(thr), next, self, 0u);
}

// Centre of mass of the sorted points [b, e).  Small cells sum their points
// directly (fp64, relative to the first point, so nothing cancels); larger
// cells take the difference of the fp64 prefix sums, whose rounding error
// divided by the count stays far below fp32 resolution.
constexpr int64_t kDirectSum = 32;

template <int D, typename T>
__device__ inline point_t<D, T> centre_of_mass(const double *__restrict__ psum, const point_t<D, T> *__restrict__ ys,
                                               int64_t b, int64_t e, const double *c)
{
    const double inv = 1.0 / double(e - b);
    T out[D];
    if (e - b <= kDirectSum) {
        const point_t<D, T> y0 = ys[b];
        double acc[D];
#pragma unroll
        for (int d = 0; d < D; ++d) acc[d] = 0.0;
        for (int64_t s = b + 1; s < e; ++s) {
            const point_t<D, T> y = ys[s];
#pragma unroll
            for (int d = 0; d < D; ++d) acc[d] += double(coord(y, d)) - double(coord(y0, d));
        }
#pragma unroll
        for (int d = 0; d < D; ++d) out[d] = T(double(coord(y0, d)) + acc[d] * inv);
    } else {
#pragma unroll
        for (int d = 0; d < D; ++d) out[d] = T(c[d] + (psum[e * D + d] - psum[b * D + d]) * inv);
    }
    return make_point(out, static_cast<point_t<D, T> *>(nullptr));
}

// D = 2, T = float: 24-byte records with fp32 centres and thresholds; T =
// double (the fp64 variant): 40-byte records with fp64 centres and
// thresholds; D = 3: 32-byte records.  theta2 is theta^2 in fp64.
template <int D, typename T>
__global__ __launch_bounds__(256) void tree_nodes_kernel(
    const uint64_t *__restrict__ codes, int64_t n, const uint32_t *__restrict__ levelmask,
    const uint32_t *__restrict__ split_b, const uint32_t *__restrict__ split_e,
    const uint32_t *__restrict__ base, const double *__restrict__ psum, const point_t<D, T> *__restrict__ ys,
    Header *__restrict__ hdr, double theta2, char *__restrict__ nodes, TreeDebug dbg)
{
    using G = Geom<D>;
    constexpr int kBytes = node_bytes<D, T>();
    constexpr int kLast = G::kBucketLevel; // bucket cells; their points sit one level below
    int64_t x = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    double c[D];
    load_centre<D>(hdr, c);
    const double rspan = hdr->rspan;
    // acceptance thresholds of the cell levels 0..kLast
    __shared__ T s_thr[kLast + 1];
    // deepest leaf level of the block (a single point's level, kLast for a bucket)
    __shared__ uint32_t s_depth;
    if (threadIdx.x <= kLast) s_thr[threadIdx.x] = T(accept_threshold(rspan, int(threadIdx.x), theta2));
    if (threadIdx.x == 0) s_depth = 0;
    __syncthreads();
    uint32_t depth = 0;
    // A record's next offset must lie past the record itself: the repulsive
    // walk advances to it, so this is what makes every walk end.  Records
    // that break it (or fall outside the array) are only reachable from a
    // corrupted sort; they are not written and the call is flagged, and the
    // walk then does not start.
    auto emit = [&](int64_t pre, point_t<D, T> com, int64_t b, int64_t e, int L, int64_t next, int kind) {
        if (pre >= 2 * n || next > 2 * n || next <= pre) {
            atomicOr(&hdr->flags, kErrRange);
            return;
        }
        const bool single = kind == 2;
        store_node(nodes, pre, com, float(e - b), single ? T(-1) : s_thr[L], uint32_t(next * kBytes),
                   single ? uint32_t(b) : kNodeCell);
        if (dbg.level) {
            dbg.level[pre] = uint8_t(L);
            dbg.kind[pre] = uint8_t(kind);
            dbg.begin[pre] = uint32_t(b);
            dbg.end[pre] = uint32_t(e);
        }
    };
    if (x < n) {
        // (a) the internal node owned by split x
        if (x < n - 1 && split_e[x] != 0) {
            int64_t b = split_b[x], e = split_e[x];
            int L = G::split_level(codes[x], codes[x + 1]);
            int64_t pre = base[b] + __popc(levelmask[b] & ((1u << L) - 1u));
            emit(pre, centre_of_mass<D, T>(psum, ys, b, e, c), b, e, L, base[e], 0);
        }
        // (b) the root, when no split lies at level 0 (all points in one child cell)
        if (x == 0 && G::digit(codes[0], 0) == G::digit(codes[n - 1], 0))
            emit(0, centre_of_mass<D, T>(psum, ys, 0, n, c), 0, n, 0, base[n], 0);
        // (c) the leaf of point x, preceded by its bucket when a run of identical
        // codes starts at x (bucket members are leaves one level below the bucket)
        if (x == 0 || codes[x - 1] != codes[x]) {
            int64_t e = run_end(codes, x, n);
            int64_t pre = base[x] + __popc(levelmask[x]);
            if (e == x + 1) {
                int lv = -1;
                if (x > 0) lv = G::split_level(codes[x - 1], codes[x]);
                if (x + 1 < n) {
                    int r = G::split_level(codes[x], codes[x + 1]);
                    lv = r > lv ? r : lv;
                }
                emit(pre, ys[x], x, e, lv + 1, pre + 1, 2);
                depth = uint32_t(lv + 1);
            } else {
                emit(pre, centre_of_mass<D, T>(psum, ys, x, e, c), x, e, kLast, base[e], 1);
                emit(pre + 1, ys[x], x, x + 1, kLast + 1, pre + 2, 2);
                depth = kLast;
            }
        } else {
            emit(base[x], ys[x], x, x + 1, kLast + 1, int64_t(base[x]) + 1, 2); // a later member of a bucket
        }
    }
    // the block's deepest leaf; the global maximum only takes the atomic when
    // the block beats the value it reads (the value only grows, so a stale
    // read costs at most an extra atomic), which keeps thousands of blocks
    // from queueing on one address
    for (int o = kWave / 2; o > 0; o >>= 1) {
        const uint32_t v = uint32_t(__shfl_xor(int(depth), o, kWave));
        depth = v > depth ? v : depth;
    }
    if (lane_id() == 0 && depth) atomicMax(&s_depth, depth);
    __syncthreads();
    if (threadIdx.x == 0 && s_depth > __hip_atomic_load(&hdr->max_depth, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
        atomicMax(&hdr->max_depth, s_depth);
}

// ------------------------------------------------------------------ debug export
// Records in the documented form: {com, count, threshold} and the meta word as
// the skip index of a cell or begin | 0xC0000000 for a single point.
__global__ __launch_bounds__(256) void tree_unpack_kernel(const char *__restrict__ nodes,
                                                          const Header *__restrict__ hdr, int64_t cap,
                                                          float4 *__restrict__ summary, uint32_t *__restrict__ meta)
{
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    const int64_t count = hdr->nodes < cap ? int64_t(hdr->nodes) : cap;
    if (i >= count) return;
    const uint2 *r = reinterpret_cast<const uint2 *>(nodes + i * kNodeBytes);
    const uint2 a = r[0], b = r[1], c = r[2];
    if (summary)
        summary[i] = make_float4(__uint_as_float(a.x), __uint_as_float(a.y), __uint_as_float(b.x), __uint_as_float(b.y));
    if (meta) meta[i] = c.y != kNodeCell ? (c.y | 0xC0000000u) : c.x / uint32_t(kNodeBytes);
}

// The 3-D records in the same documented form: summary {com x, com y, com z,
// count} and threshold, meta as above.
__global__ __launch_bounds__(256) void tree_unpack3_kernel(const char *__restrict__ nodes,
                                                           const Header *__restrict__ hdr, int64_t cap,
                                                           float4 *__restrict__ summary, float *__restrict__ thr,
                                                           uint32_t *__restrict__ meta)
{
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    const int64_t count = hdr->nodes < cap ? int64_t(hdr->nodes) : cap;
    if (i >= count) return;
    const uint4 *r = reinterpret_cast<const uint4 *>(nodes + i * kNodeBytes3);
    const uint4 a = r[0], b = r[1];
    if (summary)
        summary[i] = make_float4(__uint_as_float(a.x), __uint_as_float(a.y), __uint_as_float(a.z), __uint_as_float(a.w));
    if (thr) thr[i] = __uint_as_float(b.x);
    if (meta) meta[i] = b.z != kNodeCell ? (b.z | 0xC0000000u) : b.y / uint32_t(kNodeBytes3);
}

// ------------------------------------------------------------------ launchers
template <int D, typename T>
void launch_tree(int64_t n, double theta2, void *ws, const Layout &L, const TreeDebug &dbg, hipStream_t st)
{
    const uint64_t *codes = at<uint64_t>(ws, L.codes0);
    uint32_t *lm = at<uint32_t>(ws, L.levelmask);
    uint32_t *sb = at<uint32_t>(ws, L.split_b), *se = at<uint32_t>(ws, L.split_e);
    const point_t<D, T> *ys = at<point_t<D, T>>(ws, L.ys);
    Header *hdr = at<Header>(ws, L.header);
    uint32_t *base = at<uint32_t>(ws, L.base);
    double *psum = at<double>(ws, L.psum);
    uint32_t *tc = at<uint32_t>(ws, L.scan_cnt);
    double *ts = at<double>(ws, L.scan_sum);
    unsigned gn = unsigned((n + 255) / 256);
    tree_splits_kernel<D><<<unsigned((n + kSplitBlock - 1) / kSplitBlock), kSplitBlock, 0, st>>>(codes, n, lm, sb, se);
    scan_reduce_kernel<D, T><<<unsigned(L.scan_tiles), kScanBlock, 0, st>>>(codes, lm, ys, hdr, n, tc, ts);
    scan_top_kernel<D><<<1, kScanBlock, 0, st>>>(tc, ts, L.scan_tiles, n, base, psum, hdr);
    scan_down_kernel<D, T><<<unsigned(L.scan_tiles), kScanBlock, 0, st>>>(codes, lm, ys, hdr, n, tc, ts, base, psum);
    tree_nodes_kernel<D, T><<<gn, 256, 0, st>>>(codes, n, lm, sb, se, base, psum, ys, hdr, theta2,
                                                at<char>(ws, L.nodes), dbg);
}
template void launch_tree<2, float>(int64_t, double, void *, const Layout &, const TreeDebug &, hipStream_t);
template void launch_tree<2, double>(int64_t, double, void *, const Layout &, const TreeDebug &, hipStream_t);
template void launch_tree<3, float>(int64_t, double, void *, const Layout &, const TreeDebug &, hipStream_t);

void launch_tree_unpack(int64_t n, void *ws, const Layout &L, float *summary, uint32_t *meta, hipStream_t st)
{
    tree_unpack_kernel<<<unsigned((2 * n + 255) / 256), 256, 0, st>>>(
        at<char>(ws, L.nodes), at<Header>(ws, L.header), 2 * n,
        reinterpret_cast<float4 *>(summary), meta);
}

void launch_tree_unpack3(int64_t n, void *ws, const Layout &L, float *summary, float *thr, uint32_t *meta,
                         hipStream_t st)
{
    tree_unpack3_kernel<<<unsigned((2 * n + 255) / 256), 256, 0, st>>>(
        at<char>(ws, L.nodes), at<Header>(ws, L.header), 2 * n, reinterpret_cast<float4 *>(summary), thr, meta);
}

} // namespace bht
