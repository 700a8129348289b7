// Input similarities from the k nearest neighbours of every point (gfx950).
//
// Background, "Input similarity computation": with N_i the k neighbours of
// point i at distances d_ij,
//     p_{j|i} = exp(-d_ij^2 / 2 sigma_i^2) / sum_{l in N_i} exp(-d_il^2 / 2 sigma_i^2),
// and p_ij = (p_{j|i} + p_{i|j}) / (2N) over the union of both patterns.
// Binary Search Perplexity: sigma_i^2 is bisected (the middle point of the
// current interval each step) until the perplexity exp(H) of p_{.|i} equals u.
//
// GPU design, one call:
//   1. search: one wave per row, the k squared distances spread over the
//      lanes in fp64; every step is two wave sums (sum w, sum a w).  The
//      search runs to machine precision: it stops when the midpoint equals an
//      end of the interval and keeps the upper end;
//   2. own rows: each row's neighbours sorted by column in LDS, carrying p;
//   3. pairs: for every entry (i, j) a binary search of i in row j marks the
//      pair mutual (both rows hold it) or counts a reverse entry for row j;
//   4. row pointers: an exclusive scan of k + reverse entries per row;
//   5. fill: each row's own entries first, in column order, with the mutual
//      partner's p added; the reverse entries go to slots taken with an
//      atomic counter per row;
//   6. a final sort of every output row by column makes the result canonical.
// Rows whose union holds more than kAffLongCap entries are rejected.
#include "common.hpp"
#include "kernels.hpp"

namespace bht {

constexpr int kAffSearchBlock = 256;      // four rows per block
constexpr int kAffMaxSteps = 2200;        // halvings across the whole fp64 range
constexpr int kAffShortCap = 256;         // row sorts by one wave
constexpr int kAffLongThreads = 256;

// every lane takes lane 0's value, so branches on it stay wave-uniform
__device__ inline double uniform_d(double v)
{
    const unsigned long long b = static_cast<unsigned long long>(__double_as_longlong(v));
    const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(b));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(b >> 32));
    return __longlong_as_double(static_cast<long long>((static_cast<unsigned long long>(hi) << 32) | lo));
}

__device__ inline double wave_min_d(double v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmin(v, __shfl_xor(v, o, kWave));
    return v;
}

__device__ inline double wave_max_d(double v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, kWave));
    return v;
}

__global__ void aff_clear_kernel(Header *__restrict__ hdr, uint32_t *__restrict__ extra, uint32_t *__restrict__ fill,
                                 uint32_t *__restrict__ counters, int64_t n)
{
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) {
        extra[i] = 0;
        fill[i] = 0;
    }
    if (i == 0) {
        hdr->flags = 0;
        counters[0] = 0;
    }
}

// a = d'^2 / (2 sigma^2) from the reciprocal of 2 sigma^2: a tie (d' = 0) gives
// 0 also where the reciprocal overflows (the smallest sigma^2)
__device__ inline double scaled(double dp, double inv) { return dp > 0.0 ? dp * inv : 0.0; }

// Entropy (nats) of the Gaussian weights at sigma^2 = s2 over this lane's
// shifted squared distances (an infinite s2 gives log k).  a e^-a is taken as
// 0 where the weight underflows.  The result is lane 0's, in every lane.
template <int kPer> __device__ inline double row_entropy(const double (&dp)[kPer], int k, double s2)
{
    const double inv = isinf(s2) ? 0.0 : 1.0 / (2.0 * s2);
    double s = 0.0, t = 0.0;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        if (q < kPer - 1 || (kPer - 1) * kWave + lane_id() < k) {
            const double a = scaled(dp[q], inv);
            const double w = exp(-a);
            s += w;
            t += w > 0.0 ? a * w : 0.0;
        }
    }
    s = uniform_d(wave_sum(s));
    t = uniform_d(wave_sum(t));
    return log(s) + t / s;
}

// 1. the search; writes p_{j|i} in the neighbour order and sigma_i^2.  kPer
// = ceil(k / 64) distances per lane.
template <int kPer>
__global__ __launch_bounds__(kAffSearchBlock) void aff_search_kernel(const float *__restrict__ dist, int64_t n, int k,
                                                                     double log_u, double *__restrict__ p,
                                                                     double *__restrict__ sigma2,
                                                                     Header *__restrict__ hdr)
{
    const int64_t i = int64_t(blockIdx.x) * (kAffSearchBlock / kWave) + threadIdx.x / kWave;
    if (i >= n) return; // whole waves
    const int lane = lane_id();
    double dp[kPer];
    double mn = INFINITY, mx = 0.0;
    bool bad = false;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int e = q * kWave + lane;
        dp[q] = 0.0;
        if (e < k) {
            const float d = dist[i * k + e];
            if (!(d >= 0.0f) || isinf(d)) bad = true; // NaN, negative or infinite
            const double dd = bad ? 0.0 : double(d) * double(d);
            dp[q] = dd;
            mn = fmin(mn, dd);
        }
    }
    if (ballot(bad) && lane == 0) atomicOr(&hdr->flags, kErrNonFinite);
    mn = uniform_d(wave_min_d(mn));
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        dp[q] = q * kWave + lane < k ? dp[q] - mn : 0.0;
        mx = fmax(mx, dp[q]);
    }
    mx = uniform_d(wave_max_d(mx));
    double lo = 0.0, hi = mx > 0.0 ? mx : 1.0;
    if (mx > 0.0) {
        // grow the top of the interval until the perplexity there reaches u
        while (!isinf(hi) && row_entropy<kPer>(dp, k, hi) < log_u) hi *= 2.0;
        if (!isinf(hi)) {
            for (int s = 0; s < kAffMaxSteps; ++s) {
                const double mid = 0.5 * (lo + hi);
                if (mid <= lo || mid >= hi) break;
                if (row_entropy<kPer>(dp, k, mid) < log_u)
                    lo = mid;
                else
                    hi = mid;
            }
        }
    }
    // p_{j|i} at sigma^2 = hi
    const double inv = isinf(hi) ? 0.0 : 1.0 / (2.0 * hi);
    double w[kPer], s = 0.0;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        w[q] = 0.0;
        if (q * kWave + lane < k) {
            w[q] = exp(-scaled(dp[q], inv));
            s += w[q];
        }
    }
    s = uniform_d(wave_sum(s));
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int e = q * kWave + lane;
        if (e < k) p[i * k + e] = w[q] / s;
    }
    if (sigma2 && lane == 0) sigma2[i] = hi;
}

// 1'. the search with one point per lane (k <= kAffLaneMaxK).  The distances
// are first transposed (dT[e n + i]) so that the lanes of a wave read
// neighbour e of their 64 points as one contiguous 256-byte load; each lane
// then runs its own bisection with sums over its own row and no cross-lane
// work.  Same steps and readings as the wave kernel; d^2 - min d^2 is one
// fp64 fma, exact up to its single rounding (the square of an fp32 value is
// exact in fp64).
constexpr int kAffTransRows = 64;

__global__ __launch_bounds__(256) void aff_transpose_kernel(const float *__restrict__ dist, int64_t n, int k,
                                                            float *__restrict__ dT)
{
    __shared__ float tile[kAffTransRows][kAffLaneMaxK + 1];
    const int64_t r0 = int64_t(blockIdx.x) * kAffTransRows;
    const int rows = int(n - r0 < kAffTransRows ? n - r0 : kAffTransRows);
    for (int x = threadIdx.x; x < rows * k; x += blockDim.x) tile[x / k][x % k] = dist[r0 * k + x];
    __syncthreads();
    for (int x = threadIdx.x; x < kAffTransRows * k; x += blockDim.x) {
        const int e = x / kAffTransRows, r = x % kAffTransRows;
        if (r < rows) dT[int64_t(e) * n + r0 + r] = tile[r][e];
    }
}

__global__ __launch_bounds__(256) void aff_search_lane_kernel(const float *__restrict__ dT, int64_t n, int k,
                                                              double log_u, double *__restrict__ p,
                                                              double *__restrict__ sigma2, Header *__restrict__ hdr)
{
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float *col = dT + i;
    double mn = INFINITY;
    bool bad = false;
    for (int e = 0; e < k; ++e) {
        const float x = col[int64_t(e) * n];
        if (!(x >= 0.0f) || isinf(x)) bad = true; // NaN, negative or infinite
        mn = fmin(mn, double(x) * double(x));
    }
    if (bad) {
        atomicOr(&hdr->flags, kErrNonFinite);
        return;
    }
    double mx = 0.0;
    for (int e = 0; e < k; ++e) {
        const double x = col[int64_t(e) * n];
        mx = fmax(mx, fma(x, x, -mn));
    }
    // entropy (nats) at sigma^2 = s2 over this lane's row
    auto entropy = [&](double s2) {
        const double inv = isinf(s2) ? 0.0 : 1.0 / (2.0 * s2);
        double sw = 0.0, tw = 0.0;
#pragma unroll 4
        for (int e = 0; e < k; ++e) {
            const double x = col[int64_t(e) * n];
            const double a = scaled(fma(x, x, -mn), inv);
            const double w = exp(-a);
            sw += w;
            tw += w > 0.0 ? a * w : 0.0;
        }
        return log(sw) + tw / sw;
    };
    double lo = 0.0, hi = mx > 0.0 ? mx : 1.0;
    if (mx > 0.0) {
        while (!isinf(hi) && entropy(hi) < log_u) hi *= 2.0;
        if (!isinf(hi)) {
            for (int s = 0; s < kAffMaxSteps; ++s) {
                const double mid = 0.5 * (lo + hi);
                if (mid <= lo || mid >= hi) break;
                if (entropy(mid) < log_u)
                    lo = mid;
                else
                    hi = mid;
            }
        }
    }
    const double inv = isinf(hi) ? 0.0 : 1.0 / (2.0 * hi);
    double sw = 0.0;
    for (int e = 0; e < k; ++e) {
        const double x = col[int64_t(e) * n];
        sw += exp(-scaled(fma(x, x, -mn), inv));
    }
    for (int e = 0; e < k; ++e) {
        const double x = col[int64_t(e) * n];
        p[i * k + e] = exp(-scaled(fma(x, x, -mn), inv)) / sw;
    }
    if (sigma2) sigma2[i] = hi;
}

// Ascending sort of len (key, value) pairs held in LDS by the block, padded
// with all-ones keys to the next power of two (the arrays hold that many).
__device__ inline void lds_bitonic(uint32_t *key, uint32_t *val, int len)
{
    int size = 1;
    while (size < len) size <<= 1;
    for (int t = len + threadIdx.x; t < size; t += blockDim.x) {
        key[t] = 0xffffffffu;
        val[t] = 0u;
    }
    for (int span = 2; span <= size; span <<= 1) {
        for (int stride = span >> 1; stride > 0; stride >>= 1) {
            __syncthreads();
            for (int t = threadIdx.x; t < size / 2; t += blockDim.x) {
                const int a = 2 * stride * (t / stride) + (t % stride), b = a + stride;
                const bool up = (a & span) == 0;
                const uint32_t ka = key[a], kb = key[b];
                if ((ka > kb) == up) {
                    key[a] = kb;
                    key[b] = ka;
                    const uint32_t v = val[a];
                    val[a] = val[b];
                    val[b] = v;
                }
            }
        }
    }
    __syncthreads();
}

// 2. own rows by column: (col, p) in place, one wave per row.  Flags columns
// outside [0, n), the row itself and repeated neighbours.
__global__ __launch_bounds__(kWave) void aff_own_sort_kernel(const int32_t *__restrict__ idx, int64_t n, int k,
                                                             int32_t *__restrict__ scol, double *__restrict__ sp,
                                                             Header *__restrict__ hdr)
{
    __shared__ uint32_t s_key[kAffMaxK];
    __shared__ uint32_t s_pos[kAffMaxK];
    __shared__ double s_p[kAffMaxK];
    const int64_t i = blockIdx.x;
    bool bad = false;
    for (int e = threadIdx.x; e < k; e += kWave) {
        const uint32_t c = uint32_t(idx[i * k + e]);
        if (c >= uint32_t(n) || int64_t(c) == i) bad = true;
        s_key[e] = c;
        s_pos[e] = uint32_t(e);
        s_p[e] = sp[i * k + e];
    }
    lds_bitonic(s_key, s_pos, k);
    for (int e = threadIdx.x; e < k; e += kWave) {
        if (e > 0 && s_key[e] == s_key[e - 1]) bad = true;
        scol[i * k + e] = int32_t(s_key[e]);
        sp[i * k + e] = s_p[s_pos[e]];
    }
    if (ballot(bad) && threadIdx.x == 0) atomicOr(&hdr->flags, kErrRange);
}

// 3. mutual pairs and reverse counts; mpos holds the partner's position in
// row j, or -1
__global__ __launch_bounds__(256) void aff_pairs_kernel(const int32_t *__restrict__ scol, int64_t n, int k,
                                                        int16_t *__restrict__ mpos, uint32_t *__restrict__ extra)
{
    const int64_t x = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (x >= n * k) return;
    const int64_t i = x / k;
    const uint32_t j = uint32_t(scol[x]);
    if (j >= uint32_t(n) || int64_t(j) == i) { // flagged by the sort
        mpos[x] = -1;
        return;
    }
    const int32_t *row = scol + int64_t(j) * k;
    int a = 0, b = k; // first position in row j whose column is >= i
    while (a < b) {
        const int m = (a + b) >> 1;
        if (int64_t(row[m]) < i)
            a = m + 1;
        else
            b = m;
    }
    if (a < k && int64_t(row[a]) == i) {
        mpos[x] = int16_t(a);
    } else {
        mpos[x] = -1;
        atomicAdd(&extra[j], 1u);
    }
}

// 4. row pointers: exclusive scan of k + extra over tiles of 1024 rows
constexpr int kAffScanBlock = 256, kAffScanItems = 4, kAffScanTile = kAffScanBlock * kAffScanItems;
static_assert(kAffScanTile == kAffScanTileRows, "one scan tile per partial");

__device__ inline unsigned long long block_scan_excl(unsigned long long v, unsigned long long *s_w,
                                                     unsigned long long *total)
{
    const int lane = lane_id(), w = threadIdx.x / kWave;
    unsigned long long x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const unsigned long long y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) s_w[w] = x;
    __syncthreads();
    unsigned long long off = 0, tot = 0;
#pragma unroll
    for (int q = 0; q < kAffScanBlock / kWave; ++q) {
        off += q < w ? s_w[q] : 0ull;
        tot += s_w[q];
    }
    __syncthreads();
    *total = tot;
    return off + x - v;
}

__global__ __launch_bounds__(kAffScanBlock) void aff_scan_part_kernel(const uint32_t *__restrict__ extra, int64_t n,
                                                                      int k, unsigned long long *__restrict__ part)
{
    __shared__ unsigned long long s_w[kAffScanBlock / kWave];
    const int64_t base = int64_t(blockIdx.x) * kAffScanTile + int64_t(threadIdx.x) * kAffScanItems;
    unsigned long long v = 0;
#pragma unroll
    for (int q = 0; q < kAffScanItems; ++q)
        if (base + q < n) v += uint64_t(k) + extra[base + q];
    unsigned long long tot;
    block_scan_excl(v, s_w, &tot);
    if (threadIdx.x == 0) part[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kAffScanBlock) void aff_scan_top_kernel(unsigned long long *__restrict__ part,
                                                                     int64_t tiles, int64_t *__restrict__ row_ptr,
                                                                     int64_t n)
{
    __shared__ unsigned long long s_w[kAffScanBlock / kWave];
    unsigned long long carry = 0;
    for (int64_t b = 0; b < tiles; b += kAffScanBlock) {
        const int64_t t = b + threadIdx.x;
        const unsigned long long v = t < tiles ? part[t] : 0ull;
        unsigned long long tot;
        const unsigned long long ex = block_scan_excl(v, s_w, &tot);
        if (t < tiles) part[t] = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) row_ptr[n] = int64_t(carry);
}

__global__ __launch_bounds__(kAffScanBlock) void aff_scan_down_kernel(const uint32_t *__restrict__ extra, int64_t n,
                                                                      int k,
                                                                      const unsigned long long *__restrict__ part,
                                                                      int64_t *__restrict__ row_ptr)
{
    __shared__ unsigned long long s_w[kAffScanBlock / kWave];
    const int64_t base = int64_t(blockIdx.x) * kAffScanTile + int64_t(threadIdx.x) * kAffScanItems;
    unsigned long long len[kAffScanItems], v = 0;
#pragma unroll
    for (int q = 0; q < kAffScanItems; ++q) {
        len[q] = base + q < n ? uint64_t(k) + extra[base + q] : 0ull;
        v += len[q];
    }
    unsigned long long tot;
    unsigned long long off = part[blockIdx.x] + block_scan_excl(v, s_w, &tot);
#pragma unroll
    for (int q = 0; q < kAffScanItems; ++q) {
        if (base + q < n) row_ptr[base + q] = int64_t(off);
        off += len[q];
    }
}

// 5. fill the output rows
__global__ __launch_bounds__(256) void aff_fill_kernel(const int32_t *__restrict__ scol,
                                                       const double *__restrict__ sp,
                                                       const int16_t *__restrict__ mpos, int64_t n, int k,
                                                       const int64_t *__restrict__ row_ptr,
                                                       uint32_t *__restrict__ fill, int32_t *__restrict__ col,
                                                       float *__restrict__ val)
{
    const int64_t x = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (x >= n * k) return;
    const int64_t i = x / k;
    const int e = int(x - i * k);
    const uint32_t j = uint32_t(scol[x]);
    if (j >= uint32_t(n) || int64_t(j) == i) return; // flagged
    const double pji = sp[x];
    const int m = mpos[x];
    const double inv2n = 1.0 / (2.0 * double(n));
    const double own = m >= 0 ? pji + sp[int64_t(j) * k + m] : pji;
    col[row_ptr[i] + e] = int32_t(j);
    val[row_ptr[i] + e] = float(own * inv2n);
    if (m < 0) {
        const int64_t slot = row_ptr[j] + k + atomicAdd(&fill[j], 1u);
        col[slot] = int32_t(i);
        val[slot] = float(pji * inv2n);
    }
}

// 6. output rows by column: rows of up to kAffShortCap entries by one wave
// each; longer rows are listed for the block kernel below
__global__ __launch_bounds__(kWave) void aff_row_sort_kernel(const int64_t *__restrict__ row_ptr, int64_t n,
                                                             int32_t *__restrict__ col, float *__restrict__ val,
                                                             uint32_t *__restrict__ longrows,
                                                             uint32_t *__restrict__ counters)
{
    __shared__ uint32_t s_key[kAffShortCap];
    __shared__ uint32_t s_val[kAffShortCap];
    const int64_t i = blockIdx.x;
    const int64_t b = row_ptr[i], len = row_ptr[i + 1] - b;
    if (len > kAffShortCap) {
        if (threadIdx.x == 0) longrows[atomicAdd(&counters[0], 1u)] = uint32_t(i);
        return;
    }
    for (int e = threadIdx.x; e < len; e += kWave) {
        s_key[e] = uint32_t(col[b + e]);
        s_val[e] = __float_as_uint(val[b + e]);
    }
    lds_bitonic(s_key, s_val, int(len));
    for (int e = threadIdx.x; e < len; e += kWave) {
        col[b + e] = int32_t(s_key[e]);
        val[b + e] = __uint_as_float(s_val[e]);
    }
}

__global__ __launch_bounds__(kAffLongThreads) void aff_long_sort_kernel(const int64_t *__restrict__ row_ptr,
                                                                        int32_t *__restrict__ col,
                                                                        float *__restrict__ val,
                                                                        const uint32_t *__restrict__ longrows,
                                                                        const uint32_t *__restrict__ counters,
                                                                        Header *__restrict__ hdr)
{
    __shared__ uint32_t s_key[kAffLongCap];
    __shared__ uint32_t s_val[kAffLongCap];
    const uint32_t count = counters[0];
    for (uint32_t r = blockIdx.x; r < count; r += gridDim.x) {
        const int64_t i = longrows[r];
        const int64_t b = row_ptr[i], len = row_ptr[i + 1] - b;
        if (len > kAffLongCap) { // over the documented limit: left unsorted
            if (threadIdx.x == 0) atomicOr(&hdr->flags, kErrRange);
            continue;
        }
        __syncthreads();
        for (int e = threadIdx.x; e < len; e += kAffLongThreads) {
            s_key[e] = uint32_t(col[b + e]);
            s_val[e] = __float_as_uint(val[b + e]);
        }
        lds_bitonic(s_key, s_val, int(len));
        for (int e = threadIdx.x; e < len; e += kAffLongThreads) {
            col[b + e] = int32_t(s_key[e]);
            val[b + e] = __uint_as_float(s_val[e]);
        }
    }
}

// ------------------------------------------------------------------ launchers
void launch_aff_front(const int32_t *idx, const float *dist, int64_t n, int k, double perplexity,
                      int64_t *row_ptr, double *sigma2, void *ws, const AffLayout &A, hipStream_t st)
{
    Header *hdr = at<Header>(ws, A.header);
    uint32_t *extra = at<uint32_t>(ws, A.extra), *fill = at<uint32_t>(ws, A.fill);
    uint32_t *counters = at<uint32_t>(ws, A.counters);
    double *sp = at<double>(ws, A.sp);
    int32_t *scol = at<int32_t>(ws, A.scol);
    aff_clear_kernel<<<unsigned((n + 255) / 256), 256, 0, st>>>(hdr, extra, fill, counters, n);
    const unsigned sb = unsigned((n + 3) / 4);
    const double lu = log(perplexity);
    if (k <= kAffLaneMaxK) {
        float *dT = at<float>(ws, A.dT);
        aff_transpose_kernel<<<unsigned((n + kAffTransRows - 1) / kAffTransRows), 256, 0, st>>>(dist, n, k, dT);
        aff_search_lane_kernel<<<unsigned((n + 255) / 256), 256, 0, st>>>(dT, n, k, lu, sp, sigma2, hdr);
    }
    else switch ((k + kWave - 1) / kWave) {
    case 1: aff_search_kernel<1><<<sb, kAffSearchBlock, 0, st>>>(dist, n, k, lu, sp, sigma2, hdr); break;
    case 2: aff_search_kernel<2><<<sb, kAffSearchBlock, 0, st>>>(dist, n, k, lu, sp, sigma2, hdr); break;
    case 3: aff_search_kernel<3><<<sb, kAffSearchBlock, 0, st>>>(dist, n, k, lu, sp, sigma2, hdr); break;
    default: aff_search_kernel<4><<<sb, kAffSearchBlock, 0, st>>>(dist, n, k, lu, sp, sigma2, hdr); break;
    }
    static_assert(kAffMaxK <= 4 * kWave, "four distances per lane at most");
    aff_own_sort_kernel<<<unsigned(n), kWave, 0, st>>>(idx, n, k, scol, sp, hdr);
    const int64_t entries = n * k;
    aff_pairs_kernel<<<unsigned((entries + 255) / 256), 256, 0, st>>>(scol, n, k, at<int16_t>(ws, A.mpos), extra);
    unsigned long long *part = at<unsigned long long>(ws, A.part);
    aff_scan_part_kernel<<<unsigned(A.scan_tiles), kAffScanBlock, 0, st>>>(extra, n, k, part);
    aff_scan_top_kernel<<<1, kAffScanBlock, 0, st>>>(part, A.scan_tiles, row_ptr, n);
    aff_scan_down_kernel<<<unsigned(A.scan_tiles), kAffScanBlock, 0, st>>>(extra, n, k, part, row_ptr);
}

void launch_aff_back(int64_t n, int k, const int64_t *row_ptr, int32_t *col, float *val, void *ws,
                     const AffLayout &A, hipStream_t st)
{
    const int64_t entries = n * k;
    uint32_t *counters = at<uint32_t>(ws, A.counters);
    aff_fill_kernel<<<unsigned((entries + 255) / 256), 256, 0, st>>>(
        at<int32_t>(ws, A.scol), at<double>(ws, A.sp), at<int16_t>(ws, A.mpos), n, k, row_ptr,
        at<uint32_t>(ws, A.fill), col, val);
    aff_row_sort_kernel<<<unsigned(n), kWave, 0, st>>>(row_ptr, n, col, val, at<uint32_t>(ws, A.longrows), counters);
    aff_long_sort_kernel<<<256, kAffLongThreads, 0, st>>>(row_ptr, col, val, at<uint32_t>(ws, A.longrows), counters,
                                                          at<Header>(ws, A.header));
}

} // namespace bht
