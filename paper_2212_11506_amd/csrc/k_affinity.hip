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
//   1. search: for k <= 128 one point per lane over a transposed copy of the
//      distances (one coalesced load per neighbour for the wave's 64 points);
//      for larger k one wave per point with two wave sums per step.  The
//      search runs to machine precision: it stops when the midpoint equals an
//      end of the interval and keeps the upper end;
//   2. own rows: each row's neighbours sorted by column in LDS, carrying p;
//   3. inboxes: every entry (i, j) is scattered into row j's inbox (column i,
//      p_{j|i}) at offsets from a scan of the in-degrees;
//   4. per row: the inbox sorted in LDS, the own entries found in it counted
//      (P's row holds k plus the inbox-only entries), row pointers scanned;
//   5. per row: the union of the own list and the inbox written in column
//      order, a pair in both lists once with the sum of its two p.
// At most kAffLongCap points may list the same point.
#include "common.hpp"
#include "kernels.hpp"

namespace bht {

constexpr int kAffSearchBlock = 256;      // four rows per block
constexpr int kAffMaxSteps = 2200;        // halvings across the whole fp64 range
constexpr int kAffShortCap = 256;         // inboxes handled by one wave
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

__global__ void aff_clear_kernel(Header *__restrict__ hdr, uint32_t *__restrict__ indeg,
                                 uint32_t *__restrict__ cursor, uint32_t *__restrict__ counters, int64_t n)
{
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) {
        indeg[i] = 0;
        cursor[i] = 0;
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

// 3. inboxes: an entry (i, j) of i's list is also an entry of row j of P;
// row j's inbox collects them (column i, value p_{j|i}).  Counts first.
__global__ __launch_bounds__(256) void aff_indeg_kernel(const int32_t *__restrict__ scol, int64_t n, int k,
                                                        uint32_t *__restrict__ indeg)
{
    const int64_t x = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (x >= n * k) return;
    const int64_t i = x / k;
    const uint32_t j = uint32_t(scol[x]);
    if (j < uint32_t(n) && int64_t(j) != i) atomicAdd(&indeg[j], 1u); // others are flagged
}

// exclusive scan of base + cnt[i] over tiles of 1024 rows, into out[0..n]
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

__global__ __launch_bounds__(kAffScanBlock) void aff_scan_part_kernel(const uint32_t *__restrict__ cnt, int64_t n,
                                                                      int base, unsigned long long *__restrict__ part)
{
    __shared__ unsigned long long s_w[kAffScanBlock / kWave];
    const int64_t b0 = int64_t(blockIdx.x) * kAffScanTile + int64_t(threadIdx.x) * kAffScanItems;
    unsigned long long v = 0;
#pragma unroll
    for (int q = 0; q < kAffScanItems; ++q)
        if (b0 + q < n) v += uint64_t(base) + cnt[b0 + q];
    unsigned long long tot;
    block_scan_excl(v, s_w, &tot);
    if (threadIdx.x == 0) part[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kAffScanBlock) void aff_scan_top_kernel(unsigned long long *__restrict__ part,
                                                                     int64_t tiles, int64_t *__restrict__ out,
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
    if (threadIdx.x == 0) out[n] = int64_t(carry);
}

__global__ __launch_bounds__(kAffScanBlock) void aff_scan_down_kernel(const uint32_t *__restrict__ cnt, int64_t n,
                                                                      int base,
                                                                      const unsigned long long *__restrict__ part,
                                                                      int64_t *__restrict__ out)
{
    __shared__ unsigned long long s_w[kAffScanBlock / kWave];
    const int64_t b0 = int64_t(blockIdx.x) * kAffScanTile + int64_t(threadIdx.x) * kAffScanItems;
    unsigned long long len[kAffScanItems], v = 0;
#pragma unroll
    for (int q = 0; q < kAffScanItems; ++q) {
        len[q] = b0 + q < n ? uint64_t(base) + cnt[b0 + q] : 0ull;
        v += len[q];
    }
    unsigned long long tot;
    unsigned long long off = part[blockIdx.x] + block_scan_excl(v, s_w, &tot);
#pragma unroll
    for (int q = 0; q < kAffScanItems; ++q) {
        if (b0 + q < n) out[b0 + q] = int64_t(off);
        off += len[q];
    }
}

// the entries into the inboxes, at slots taken with a counter per row (their
// order is sorted away below)
__global__ __launch_bounds__(256) void aff_scatter_kernel(const int32_t *__restrict__ scol,
                                                          const double *__restrict__ sp, int64_t n, int k,
                                                          const int64_t *__restrict__ ib,
                                                          uint32_t *__restrict__ cursor,
                                                          int32_t *__restrict__ in_col, double *__restrict__ in_p)
{
    const int64_t x = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (x >= n * k) return;
    const int64_t i = x / k;
    const uint32_t j = uint32_t(scol[x]);
    if (j >= uint32_t(n) || int64_t(j) == i) return;
    const int64_t slot = ib[j] + atomicAdd(&cursor[j], 1u);
    in_col[slot] = int32_t(i);
    in_p[slot] = sp[x];
}

// first position in the sorted a[0..len) whose value is >= key
__device__ inline int lower_bound_u32(const uint32_t *a, int len, uint32_t key)
{
    int lo = 0, hi = len;
    while (lo < hi) {
        const int m = (lo + hi) >> 1;
        if (a[m] < key)
            lo = m + 1;
        else
            hi = m;
    }
    return lo;
}

// Exclusive prefix counts MO[0..k] of the flags f[0..k) (k <= 256) into LDS,
// by the whole block; returns the total in every thread.
__device__ inline uint32_t block_flag_scan(const uint8_t *f, int k, uint32_t *MO, uint32_t *s_w)
{
    const int per = (k + int(blockDim.x) - 1) / int(blockDim.x);
    const int e0 = int(threadIdx.x) * per;
    uint32_t c = 0;
    for (int e = e0; e < e0 + per && e < k; ++e) c += f[e];
    const int lane = lane_id(), w = threadIdx.x / kWave;
    uint32_t x = c;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) s_w[w] = x;
    __syncthreads();
    uint32_t off = 0, tot = 0;
    for (int q = 0; q < int(blockDim.x) / kWave; ++q) {
        off += q < w ? s_w[q] : 0u;
        tot += s_w[q];
    }
    uint32_t run = off + x - c;
    for (int e = e0; e < e0 + per && e < k; ++e) {
        MO[e] = run;
        run += f[e];
    }
    if (threadIdx.x == 0) MO[k] = tot;
    __syncthreads();
    return tot;
}

// 4./5. one row j of P from its own list (k columns in order, with p_{c|j})
// and its inbox (m columns, with p_{j|c}).  kWrite = false: sort the inbox in
// place and count the inbox entries that are not in the own list (P's row
// has k plus that many entries); kWrite = true: write the row in column
// order.  With MO[e] the number of own entries before e that are also in the
// inbox, own entry e goes to e + t - MO[e] (t: inbox entries below its
// column) and an inbox-only entry at inbox position t to e' + t - MO[e'] (e':
// own entries below its column).  A pair in both lists is written once, with
// (p_{c|j} + p_{j|c}) / 2N: the same fp64 sum in both rows, so P is exactly
// symmetric.
template <int kCap, bool kWrite> struct AffRowLds {
    uint32_t own[kAffMaxK];
    double ownp[kAffMaxK];
    uint32_t in[kCap];
    uint32_t pos[kWrite ? 1 : kCap];
    double inp[kCap];
    uint8_t fl[kAffMaxK];
    uint32_t mo[kAffMaxK + 1];
    uint32_t w[kAffLongThreads / kWave];
};

template <int kCap, bool kWrite>
__device__ inline void aff_row(int64_t j, int k, int64_t n, const int32_t *__restrict__ scol,
                               const double *__restrict__ sp, const int64_t *__restrict__ ib,
                               int32_t *__restrict__ in_col, double *__restrict__ in_p,
                               uint32_t *__restrict__ inonly, const int64_t *__restrict__ row_ptr,
                               int32_t *__restrict__ col, float *__restrict__ val, AffRowLds<kCap, kWrite> &L)
{
    const int64_t b = ib[j];
    const int m = int(ib[j + 1] - b);
    for (int e = threadIdx.x; e < k; e += blockDim.x) {
        L.own[e] = uint32_t(scol[j * k + e]);
        L.ownp[e] = sp[j * k + e];
    }
    for (int t = threadIdx.x; t < m; t += blockDim.x) {
        L.in[t] = uint32_t(in_col[b + t]);
        L.inp[t] = in_p[b + t];
        if (!kWrite) L.pos[t] = uint32_t(t);
    }
    if (!kWrite) lds_bitonic(L.in, L.pos, m); // ends with a barrier
    __syncthreads();
    for (int e = threadIdx.x; e < k; e += blockDim.x) {
        const int t = lower_bound_u32(L.in, m, L.own[e]);
        L.fl[e] = t < m && L.in[t] == L.own[e];
    }
    __syncthreads();
    const uint32_t both = block_flag_scan(L.fl, k, L.mo, L.w);
    if (!kWrite) {
        for (int t = threadIdx.x; t < m; t += blockDim.x) {
            in_col[b + t] = int32_t(L.in[t]);
            in_p[b + t] = L.inp[L.pos[t]];
        }
        if (threadIdx.x == 0) inonly[j] = uint32_t(m) - both;
        return;
    }
    const int64_t o = row_ptr[j];
    const double inv2n = 1.0 / (2.0 * double(n));
    for (int e = threadIdx.x; e < k; e += blockDim.x) {
        const int t = lower_bound_u32(L.in, m, L.own[e]);
        const int64_t q = o + e + t - L.mo[e];
        col[q] = int32_t(L.own[e]);
        val[q] = float((L.fl[e] ? L.ownp[e] + L.inp[t] : L.ownp[e]) * inv2n);
    }
    for (int t = threadIdx.x; t < m; t += blockDim.x) {
        const int e = lower_bound_u32(L.own, k, L.in[t]);
        if (e < k && L.own[e] == L.in[t]) continue; // written with the own entry
        const int64_t q = o + e + t - L.mo[e];
        col[q] = int32_t(L.in[t]);
        val[q] = float(L.inp[t] * inv2n);
    }
}

// rows whose inbox fits kAffShortCap: one wave each; longer ones are listed
// (by the counting pass) for the block kernel
template <bool kWrite>
__global__ __launch_bounds__(kWave) void aff_row_kernel(int64_t n, int k, const int32_t *__restrict__ scol,
                                                        const double *__restrict__ sp,
                                                        const int64_t *__restrict__ ib, int32_t *__restrict__ in_col,
                                                        double *__restrict__ in_p, uint32_t *__restrict__ inonly,
                                                        const int64_t *__restrict__ row_ptr,
                                                        int32_t *__restrict__ col, float *__restrict__ val,
                                                        uint32_t *__restrict__ longrows,
                                                        uint32_t *__restrict__ counters)
{
    __shared__ AffRowLds<kAffShortCap, kWrite> L;
    const int64_t j = blockIdx.x;
    if (ib[j + 1] - ib[j] > kAffShortCap) {
        if (!kWrite && threadIdx.x == 0) longrows[atomicAdd(&counters[0], 1u)] = uint32_t(j);
        return;
    }
    aff_row<kAffShortCap, kWrite>(j, k, n, scol, sp, ib, in_col, in_p, inonly, row_ptr, col, val, L);
}

template <bool kWrite>
__global__ __launch_bounds__(kAffLongThreads) void aff_long_row_kernel(
    int64_t n, int k, const int32_t *__restrict__ scol, const double *__restrict__ sp,
    const int64_t *__restrict__ ib, int32_t *__restrict__ in_col, double *__restrict__ in_p,
    uint32_t *__restrict__ inonly, const int64_t *__restrict__ row_ptr, int32_t *__restrict__ col,
    float *__restrict__ val, const uint32_t *__restrict__ longrows, const uint32_t *__restrict__ counters,
    Header *__restrict__ hdr)
{
    __shared__ AffRowLds<kAffLongCap, kWrite> L;
    const uint32_t count = counters[0];
    for (uint32_t r = blockIdx.x; r < count; r += gridDim.x) {
        const int64_t j = longrows[r];
        if (ib[j + 1] - ib[j] > kAffLongCap) { // over the documented limit
            if (!kWrite && threadIdx.x == 0) {
                atomicOr(&hdr->flags, kErrRange);
                inonly[j] = 0;
            }
            continue;
        }
        __syncthreads();
        aff_row<kAffLongCap, kWrite>(j, k, n, scol, sp, ib, in_col, in_p, inonly, row_ptr, col, val, L);
    }
}

// ------------------------------------------------------------------ launchers
void launch_aff_front(const int32_t *idx, const float *dist, int64_t n, int k, double perplexity,
                      int64_t *row_ptr, double *sigma2, void *ws, const AffLayout &A, hipStream_t st)
{
    Header *hdr = at<Header>(ws, A.header);
    uint32_t *indeg = at<uint32_t>(ws, A.indeg), *cursor = at<uint32_t>(ws, A.cursor);
    uint32_t *inonly = at<uint32_t>(ws, A.inonly), *counters = at<uint32_t>(ws, A.counters);
    double *sp = at<double>(ws, A.sp);
    int32_t *scol = at<int32_t>(ws, A.scol);
    int64_t *ib = at<int64_t>(ws, A.ib);
    int32_t *in_col = at<int32_t>(ws, A.in_col);
    double *in_p = at<double>(ws, A.in_p);
    uint32_t *longrows = at<uint32_t>(ws, A.longrows);
    unsigned long long *part = at<unsigned long long>(ws, A.part);
    aff_clear_kernel<<<unsigned((n + 255) / 256), 256, 0, st>>>(hdr, indeg, cursor, counters, n);
    const double lu = log(perplexity);
    if (k <= kAffLaneMaxK) {
        float *dT = at<float>(ws, A.dT);
        aff_transpose_kernel<<<unsigned((n + kAffTransRows - 1) / kAffTransRows), 256, 0, st>>>(dist, n, k, dT);
        aff_search_lane_kernel<<<unsigned((n + 255) / 256), 256, 0, st>>>(dT, n, k, lu, sp, sigma2, hdr);
    } else {
        const unsigned sb = unsigned((n + 3) / 4);
        if ((k + kWave - 1) / kWave == 3)
            aff_search_kernel<3><<<sb, kAffSearchBlock, 0, st>>>(dist, n, k, lu, sp, sigma2, hdr);
        else
            aff_search_kernel<4><<<sb, kAffSearchBlock, 0, st>>>(dist, n, k, lu, sp, sigma2, hdr);
    }
    static_assert(kAffMaxK <= 4 * kWave && kAffLaneMaxK >= 2 * kWave, "three or four distances per lane");
    aff_own_sort_kernel<<<unsigned(n), kWave, 0, st>>>(idx, n, k, scol, sp, hdr);
    const unsigned eb = unsigned((n * k + 255) / 256);
    aff_indeg_kernel<<<eb, 256, 0, st>>>(scol, n, k, indeg);
    aff_scan_part_kernel<<<unsigned(A.scan_tiles), kAffScanBlock, 0, st>>>(indeg, n, 0, part);
    aff_scan_top_kernel<<<1, kAffScanBlock, 0, st>>>(part, A.scan_tiles, ib, n);
    aff_scan_down_kernel<<<unsigned(A.scan_tiles), kAffScanBlock, 0, st>>>(indeg, n, 0, part, ib);
    aff_scatter_kernel<<<eb, 256, 0, st>>>(scol, sp, n, k, ib, cursor, in_col, in_p);
    aff_row_kernel<false><<<unsigned(n), kWave, 0, st>>>(n, k, scol, sp, ib, in_col, in_p, inonly, nullptr,
                                                         nullptr, nullptr, longrows, counters);
    aff_long_row_kernel<false><<<256, kAffLongThreads, 0, st>>>(n, k, scol, sp, ib, in_col, in_p, inonly, nullptr,
                                                                nullptr, nullptr, longrows, counters, hdr);
    aff_scan_part_kernel<<<unsigned(A.scan_tiles), kAffScanBlock, 0, st>>>(inonly, n, k, part);
    aff_scan_top_kernel<<<1, kAffScanBlock, 0, st>>>(part, A.scan_tiles, row_ptr, n);
    aff_scan_down_kernel<<<unsigned(A.scan_tiles), kAffScanBlock, 0, st>>>(inonly, n, k, part, row_ptr);
}

void launch_aff_back(int64_t n, int k, const int64_t *row_ptr, int32_t *col, float *val, void *ws,
                     const AffLayout &A, hipStream_t st)
{
    const int32_t *scol = at<int32_t>(ws, A.scol);
    const double *sp = at<double>(ws, A.sp);
    const int64_t *ib = at<int64_t>(ws, A.ib);
    int32_t *in_col = at<int32_t>(ws, A.in_col);
    double *in_p = at<double>(ws, A.in_p);
    uint32_t *inonly = at<uint32_t>(ws, A.inonly), *counters = at<uint32_t>(ws, A.counters);
    uint32_t *longrows = at<uint32_t>(ws, A.longrows);
    aff_row_kernel<true><<<unsigned(n), kWave, 0, st>>>(n, k, scol, sp, ib, in_col, in_p, inonly, row_ptr, col, val,
                                                        longrows, counters);
    aff_long_row_kernel<true><<<256, kAffLongThreads, 0, st>>>(n, k, scol, sp, ib, in_col, in_p, inonly, row_ptr,
                                                               col, val, longrows, counters,
                                                               at<Header>(ws, A.header));
}

} // namespace bht
