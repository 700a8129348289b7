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
//   1. own rows: each row's (column, neighbour position) pairs sorted by a
//      bitonic network in registers, giving the row in column order and the
//      place of each entry's p;
//   2. inboxes: the pairs (column j, place of p_{j|i}) of all rows, in entry
//      order, sorted by j with a stable LSD radix sort (8-bit digits,
//      onesweep passes with decoupled look-back), so that row j's inbox (the
//      points that list j) comes out in increasing i with no atomics;
//   3. per row: the own entries found in the inbox counted (P's row holds k
//      plus the inbox-only entries), row pointers scanned;
//   4. search: for k <= 128 four lanes per point with the distances in
//      registers; for larger k one wave per point with two wave sums per
//      step.  The search runs to machine precision: it stops when the
//      midpoint equals an end of the interval and keeps the upper end.  It
//      writes p_{j|i} in the neighbour order;
//   5. per row: the union of the own list and the inbox written in column
//      order, a pair in both lists once with the sum of its two p.
// Steps 1-3 read only the neighbour indices.  On a second stream beside the
// search they slowed each other down as much as they overlapped (the search
// keeps the VALU busy and holds the wave slots the sort passes wait for), so
// the steps run in order.
// At most kAffLongCap points may list the same point.
#include "common.hpp"
#include "kernels.hpp"

#include <algorithm>
#include <type_traits>

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

// the flags, tile counters, histograms and look-back words of one call
__global__ __launch_bounds__(256) void aff_clear_kernel(Header *__restrict__ hdr, uint32_t *__restrict__ hist,
                                                        unsigned long long *__restrict__ status, int64_t status_words,
                                                        uint32_t *__restrict__ counters)
{
    const int64_t i0 = int64_t(blockIdx.x) * blockDim.x + threadIdx.x, stride = int64_t(gridDim.x) * blockDim.x;
    for (int64_t i = i0; i < status_words; i += stride) status[i] = 0ull;
    for (int64_t i = i0; i < int64_t(kHistCopies) * kAffHistWords; i += stride) hist[i] = 0u;
    if (i0 == 0) {
        hdr->flags = 0;
        for (int q = 0; q < kSortPasses; ++q) hdr->tile_counter[q] = 0;
        counters[0] = 0;
    }
}

// a = d'^2 / (2 sigma^2) from the reciprocal of 2 sigma^2: a tie (d' = 0) gives
// 0 also where the reciprocal overflows (the smallest sigma^2)
__device__ inline double scaled(double dp, double inv) { return dp > 0.0 ? dp * inv : 0.0; }

// Entropy (nats) of the Gaussian weights at sigma^2 = s2 over this lane's
// shifted squared distances (an infinite s2 gives log k).  a e^-a is taken as
// 0 where the weight underflows.  The result is lane 0's, in every lane.
// With kVar, also *var = the weights' variance of a (see search_sigma2).
template <int kPer, bool kVar = false>
__device__ inline double row_entropy(const double (&dp)[kPer], int k, double s2, double *var = nullptr)
{
    const double inv = isinf(s2) ? 0.0 : 1.0 / (2.0 * s2);
    double s = 0.0, t = 0.0, t2 = 0.0;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        if (q < kPer - 1 || (kPer - 1) * kWave + lane_id() < k) {
            const double a = scaled(dp[q], inv);
            const double w = exp(-a);
            s += w;
            t += w > 0.0 ? a * w : 0.0;
            if (kVar) t2 += w > 0.0 ? a * (a * w) : 0.0;
        }
    }
    s = uniform_d(wave_sum(s));
    t = uniform_d(wave_sum(t));
    if (kVar) {
        t2 = uniform_d(wave_sum(t2));
        const double m = t / s;
        *var = fmax(t2 / s - m * m, 0.0);
    }
    return log(s) + t / s;
}

// Margin of the entropy, in nats, beyond which a comparison with log u is
// taken as settled: the evaluation's rounding (up to 256 terms summed in
// fp64, each within a few ulps, then a log and a quotient of at most about
// ten) stays below 3e-13, so a point whose computed entropy is more than
// kAffMargin below log u has every smaller sigma^2 below it too (the entropy
// increases with sigma^2), and likewise above.
constexpr double kAffMargin = 1e-11;
constexpr int kAffNewtonMax = 12;

// sigma^2 of one row: the upper end of the bisection interval [0, hi], hi
// doubled from mx until the entropy there reaches log u, halved until the
// midpoint equals an end (each midpoint goes below when its entropy is under
// log u).  The decisions depend only on the sign of H(mid) - log u, and H
// increases with sigma^2; so first Newton's method on ln sigma^2 (dH / d ln
// sigma^2 = v, the weights' variance of a), kept inside the settled bounds,
// brings a settled bound A below the root and B above it close together,
// and the bisection then evaluates only the midpoints between them: the same
// decisions, hence the same result bit for bit, with about half the
// evaluations.  `entropy(s2)` and `entropy_var(s2, v)` give the row's
// entropy, equal in every lane of the row's group, so the group branches alike.
template <typename E, typename EV>
__device__ __forceinline__ double search_sigma2(double mx, double log_u, E &&entropy, EV &&entropy_var)
{
    double lo = 0.0, hi = mx > 0.0 ? mx : 1.0;
    if (!(mx > 0.0)) return hi;
    double A = 0.0, B = INFINITY, h = 0.0, v = 0.0;
    auto settle = [&](double s2, double hs) {
        if (hs < log_u - kAffMargin)
            A = fmax(A, s2);
        else if (hs > log_u + kAffMargin)
            B = fmin(B, s2);
    };
    // grow the top of the interval until the perplexity there reaches u
    for (;;) {
        if (isinf(hi)) return hi;
        h = entropy_var(hi, v);
        settle(hi, h);
        if (h >= log_u) break;
        hi *= 2.0;
    }
    // the bounds only spare evaluations below; from a point within the
    // margin, one probe on either side
    double s2 = hi;
    for (int it = 0; it < kAffNewtonMax && B > A; ++it) {
        if (fabs(h - log_u) <= kAffMargin) {
            const double d = v > 0.0 ? fmin(4.0 * kAffMargin / v, 0.25) : 0.25;
            const double sa = s2 * (1.0 - d), sb = s2 * (1.0 + d);
            settle(sa, entropy(sa));
            settle(sb, entropy(sb));
            break;
        }
        const double r = (h - log_u) / v;
        double sn = s2 * (1.0 - r);
        if (!(v > 0.0) || !(sn > A) || !(sn < B) || !(r < 1.0)) {
            // outside the bounds: halve them on the log scale (a far start,
            // where the entropy is flat, drops 64-fold)
            sn = isinf(B) ? 2.0 * fmax(A, s2) : (A > 0.0 ? sqrt(A * B) : B * (1.0 / 64.0));
        }
        if (sn == s2) break;
        s2 = sn;
        h = entropy_var(s2, v);
        settle(s2, h);
    }
    // the bisection, as if every midpoint were evaluated
    for (int s = 0; s < kAffMaxSteps; ++s) {
        const double mid = 0.5 * (lo + hi);
        if (mid <= lo || mid >= hi) break;
        const bool below = mid <= A ? true : (mid >= B ? false : entropy(mid) < log_u);
        if (below)
            lo = mid;
        else
            hi = mid;
    }
    return hi;
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
    const double hi = search_sigma2(
        mx, log_u, [&](double s2) { return row_entropy<kPer>(dp, k, s2); },
        [&](double s2, double &v) { return row_entropy<kPer, true>(dp, k, s2, &v); });
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

// 2^-x for 0 <= x <= kExp2Clamp: x = n + r with n = rint(x), so r = x - n,
// |r| <= 1/2, is exact (no reduction error), then 2^-r = exp(-r ln 2) from
// its Taylor series to degree 13 (coefficients (ln 2)^d / d!; the truncation
// is below 5e-18 relative for |r ln 2| <= 0.35) by Horner's rule, and the
// factor 2^-n as an exponent adjustment, which flushes to 0 beyond the
// subnormal range (x > 1074).  The arguments here are never negative, so the
// overflow branches of a general exponential are not needed.
constexpr double kLn2 = 0.6931471805599453;  // ln 2
constexpr double kLog2e = 1.4426950408889634; // 1 / ln 2
constexpr int kExpDegree = 13;
constexpr double kExp2Clamp = 1500.0; // 2^-1500 is 0 in fp64

constexpr double ln2_pow_over_factorial(int d)
{
    double c = 1.0;
    for (int q = 1; q <= d; ++q) c *= kLn2 / double(q);
    return c;
}

__device__ inline double exp2_neg(double x)
{
    const double nn = rint(x);
    const double s = nn - x; // -r, exact
    double q = ln2_pow_over_factorial(kExpDegree);
#pragma unroll
    for (int d = kExpDegree - 1; d >= 0; --d) q = fma(q, s, ln2_pow_over_factorial(d));
    return ldexp(q, -int(nn));
}

// sums over the four lanes of a row: butterflies, so all four get the same bits
__device__ inline double quad_sum(double v)
{
    v += __shfl_xor(v, 1, kWave);
    return v + __shfl_xor(v, 2, kWave);
}

__device__ inline double quad_min(double v)
{
    v = fmin(v, __shfl_xor(v, 1, kWave));
    return fmin(v, __shfl_xor(v, 2, kWave));
}

__device__ inline double quad_max(double v)
{
    v = fmax(v, __shfl_xor(v, 1, kWave));
    return fmax(v, __shfl_xor(v, 2, kWave));
}

__device__ inline bool quad_any(bool b)
{
    int x = b ? 1 : 0;
    x |= __shfl_xor(x, 1, kWave);
    x |= __shfl_xor(x, 2, kWave);
    return x != 0;
}

// 1'. the search with four lanes per row (k <= kAffLaneMaxK).  Lane g of a
// row holds the shifted squared distances of neighbours g, g + 4, g + 8, ...
// in registers (kPer slots; the unused ones hold NaN), so a bisection step
// reads no memory.  The row's sums are quad butterflies, equal to the bit in
// its four lanes, so the four take the same branches.  Same steps and
// readings as the wave kernel.  Per neighbour and step: x = a / ln 2 with a
// = d'^2 / 2 sigma^2 (the slots hold d'^2 / ln 2), clamped at kExp2Clamp
// (2^-x is 0 in fp64 from 1075 on; NaN slots clamp to it too), the weight
// 2^-x = exp(-a) by exp2_neg, and the entropy log S + ln 2 sum(x w) / S.  A
// step whose 1 / 2 sigma^2 is infinite (sigma^2 in the subnormal range) takes
// the limit: weight 1 at d' = 0, else 0.
constexpr int kAffG = 4;

// f(0), f(1), ..., f(N - 1) with compile-time arguments, so that arrays
// indexed by them stay in registers whatever the unroller decides
template <int Q, int N> struct StaticFor {
    template <typename F> __device__ __forceinline__ static void run(F &&f)
    {
        f(std::integral_constant<int, Q>{});
        StaticFor<Q + 1, N>::run(f);
    }
};
template <int N> struct StaticFor<N, N> {
    template <typename F> __device__ __forceinline__ static void run(F &&) {}
};

// entropy (nats) of the Gaussian weights at sigma^2 = s2 over a row held as
// in aff_search_quad_kernel; the same value in the row's four lanes.  With
// kVar, also *var = the weights' variance of a = d'^2 / 2 sigma^2, which is
// dH / d ln sigma^2 (the entropy's own sums are formed exactly as without it).
template <int kPer, bool kVar = false>
__device__ __forceinline__ double row_entropy_quad(const double (&dp)[kPer], double s2, double *var = nullptr)
{
    const double inv = isinf(s2) ? 0.0 : 1.0 / (2.0 * s2);
    double sw = 0.0, tw = 0.0, t2 = 0.0;
    if (!isinf(inv)) {
        StaticFor<0, kPer>::run([&](auto qc) {
            const double x = fmin(dp[decltype(qc)::value] * inv, kExp2Clamp); // a / ln 2
            const double w = exp2_neg(x);
            sw += w;
            tw = fma(x, w, tw);
            if (kVar) t2 = fma(x, x * w, t2);
        });
    } else {
        // a = 0 or +inf: a w = 0
        StaticFor<0, kPer>::run([&](auto qc) { sw += dp[decltype(qc)::value] == 0.0 ? 1.0 : 0.0; });
    }
    sw = quad_sum(sw);
    tw = quad_sum(tw);
    if (kVar) {
        t2 = quad_sum(t2);
        const double m = kLn2 * tw / sw;
        *var = fmax(kLn2 * kLn2 * t2 / sw - m * m, 0.0);
    }
    return log(sw) + kLn2 * tw / sw;
}


template <int kPer>
__device__ __forceinline__ void search_row_quad(const float *__restrict__ dist, int64_t i, int g, int k,
                                                double log_u, double *__restrict__ p, double *__restrict__ sigma2,
                                                Header *__restrict__ hdr)
{
    const float *row = dist + i * k;
    double dp[kPer];
    double mn = INFINITY;
    bool bad = false;
    StaticFor<0, kPer>::run([&](auto qc) {
        constexpr int q = decltype(qc)::value;
        const int e = g + kAffG * q;
        const float x = e < k ? row[e] : 0.0f;
        if (!(x >= 0.0f) || isinf(x)) bad = true; // NaN, negative or infinite
        dp[q] = double(x);
        if (e < k) mn = fmin(mn, dp[q] * dp[q]);
    });
    if (quad_any(bad)) {
        if (g == 0) atomicOr(&hdr->flags, kErrNonFinite);
        return;
    }
    mn = quad_min(mn);
    double mx = 0.0;
    StaticFor<0, kPer>::run([&](auto qc) {
        constexpr int q = decltype(qc)::value;
        const bool live = g + kAffG * q < k;
        dp[q] = live ? fma(dp[q], dp[q], -mn) : __builtin_nan("");
        if (live) mx = fmax(mx, dp[q]);
    });
    mx = quad_max(mx);
    // from here on the slots hold d'^2 / ln 2, so that a / ln 2 = slot / 2 sigma^2
    StaticFor<0, kPer>::run([&](auto qc) { dp[decltype(qc)::value] *= kLog2e; });
    const double hi = search_sigma2(
        mx, log_u, [&](double s2) { return row_entropy_quad<kPer>(dp, s2); },
        [&](double s2, double &v) { return row_entropy_quad<kPer, true>(dp, s2, &v); });
    // p_{j|i} at sigma^2 = hi
    const double inv = isinf(hi) ? 0.0 : 1.0 / (2.0 * hi);
    double sw = 0.0;
    auto weight = [&](double d) { return !isinf(inv) ? exp2_neg(fmin(d * inv, kExp2Clamp)) : (d == 0.0 ? 1.0 : 0.0); };
    StaticFor<0, kPer>::run([&](auto qc) { sw += weight(dp[decltype(qc)::value]); });
    sw = quad_sum(sw);
    StaticFor<0, kPer>::run([&](auto qc) {
        constexpr int q = decltype(qc)::value;
        const int e = g + kAffG * q;
        if (e < k) p[i * k + e] = weight(dp[q]) / sw;
    });
    if (sigma2 && g == 0) sigma2[i] = hi;
}

// rows i = blockIdx.x * 64 + threadIdx.x / 4, strided by the grid
template <int kPer>
__global__ __launch_bounds__(256) void aff_search_quad_kernel(const float *__restrict__ dist, int64_t n, int k,
                                                              double log_u, double *__restrict__ p,
                                                              double *__restrict__ sigma2, Header *__restrict__ hdr)
{
    const int g = int(threadIdx.x % kAffG);
    for (int64_t i = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) / kAffG; i < n;
         i += int64_t(gridDim.x) * (blockDim.x / kAffG))
        search_row_quad<kPer>(dist, i, g, k, log_u, p, sigma2, hdr); // whole quads take the same rows
}

// 2. own rows in column order, one wave per row (four rows per block).  The
// entries, packed as column * 256 + neighbour position (distinct, so the
// order is strict and ties keep the neighbour order) and padded with all-ones
// to 64 kS slots, are sorted by a bitonic network held in registers: slot x
// = 64 q + lane; partners fewer than 64 slots apart are exchanged by lane
// shuffles, farther ones within the lane.  Writes the row in column order
// (scol) and each entry's neighbour position (sorig), and flags columns
// outside [0, n), the row itself and repeated neighbours.  kS: 1, 2 or 4 (k
// <= 64 kS).
template <int kS>
__global__ __launch_bounds__(256) void aff_own_sort_kernel(const int32_t *__restrict__ idx, int64_t n, int k,
                                                           int32_t *__restrict__ scol, uint8_t *__restrict__ sorig,
                                                           Header *__restrict__ hdr)
{
    constexpr int kN = kS * kWave;
    const int w = threadIdx.x / kWave, lane = lane_id();
    const int64_t i = int64_t(blockIdx.x) * (256 / kWave) + w;
    if (i >= n) return; // whole waves
    uint32_t v[kS];
    bool bad = false;
#pragma unroll
    for (int q = 0; q < kS; ++q) {
        const int e = q * kWave + lane;
        v[q] = 0xffffffffu;
        if (e < k) {
            const uint32_t c = uint32_t(idx[i * k + e]);
            if (c >= uint32_t(n) || int64_t(c) == i) bad = true;
            v[q] = ((c < 0xffffffu ? c : 0xffffffu) << 8) | uint32_t(e);
        }
    }
#pragma unroll
    for (int size = 2; size <= kN; size <<= 1) {
#pragma unroll
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            if (stride >= kWave) {
                const int qs = stride / kWave;
#pragma unroll
                for (int q = 0; q < kS; ++q) {
                    if (q & qs) continue;
                    const bool up = ((q * kWave + lane) & size) == 0;
                    const uint32_t a = v[q], b = v[q | qs];
                    v[q] = up ? min(a, b) : max(a, b);
                    v[q | qs] = up ? max(a, b) : min(a, b);
                }
            } else {
#pragma unroll
                for (int q = 0; q < kS; ++q) {
                    const uint32_t o = uint32_t(__shfl_xor(int(v[q]), stride, kWave));
                    const bool up = ((q * kWave + lane) & size) == 0;
                    const bool low = (lane & stride) == 0;
                    v[q] = (low == up) ? min(v[q], o) : max(v[q], o);
                }
            }
        }
    }
#pragma unroll
    for (int q = 0; q < kS; ++q) {
        const int x = q * kWave + lane;
        // the slot before: the lane below, or the last lane of the slot row before
        uint32_t prev = uint32_t(__shfl_up(int(v[q]), 1, kWave));
        if (q > 0) {
            const uint32_t last = uint32_t(__shfl(int(v[q > 0 ? q - 1 : 0]), kWave - 1, kWave));
            if (lane == 0) prev = last;
        }
        if (x < k) {
            if (x > 0 && (prev >> 8) == (v[q] >> 8)) bad = true;
            const uint32_t e = v[q] & 0xffu;
            scol[i * k + x] = int32_t(v[q] >> 8);
            sorig[i * k + x] = uint8_t(e);
        }
    }
    if (ballot(bad) && lane == 0) atomicOr(&hdr->flags, kErrRange);
}

// 3. the pairs.  Key of an entry: its column, or n for a column outside
// [0, n) (the call fails on those, but the sort still sees keys in range).
__device__ inline uint32_t pair_key(int32_t c, int64_t n)
{
    return uint32_t(c) < uint32_t(n) ? uint32_t(c) : uint32_t(n);
}

// digit counts of every pass, per block in LDS, added into kHistCopies copies
__global__ __launch_bounds__(256) void aff_hist_kernel(const int32_t *__restrict__ scol, int64_t m, int64_t n,
                                                       int passes, uint32_t *__restrict__ hist)
{
    __shared__ uint32_t s_h[kAffHistWords];
    for (int q = threadIdx.x; q < kAffHistWords; q += blockDim.x) s_h[q] = 0u;
    __syncthreads();
    for (int64_t x = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; x < m; x += int64_t(gridDim.x) * blockDim.x) {
        const uint32_t key = pair_key(scol[x], n);
        for (int q = 0; q < passes; ++q) atomicAdd(&s_h[q * kRadix + ((key >> (q * kRadixBits)) & (kRadix - 1))], 1u);
    }
    __syncthreads();
    uint32_t *h = hist + (blockIdx.x % kHistCopies) * kAffHistWords;
    for (int q = threadIdx.x; q < passes * kRadix; q += blockDim.x)
        if (s_h[q]) atomicAdd(&h[q], s_h[q]);
}

// Block-wide exclusive scan of one value per thread (kSortBlock threads).
__device__ inline uint32_t aff_block_scan(uint32_t v, uint32_t *s_wave)
{
    const int lane = lane_id(), w = threadIdx.x / kWave;
    uint32_t x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) s_wave[w] = x;
    __syncthreads();
    uint32_t off = 0;
#pragma unroll
    for (int q = 0; q < kSortBlock / kWave; ++q) off += q < w ? s_wave[q] : 0u;
    __syncthreads();
    return off + x - v;
}

// look-back words: flag bits above a 32-bit count
constexpr unsigned long long kAffAggregate = 1ull << 32, kAffInclusive = 2ull << 32;

static_assert(kSortBlock == kRadix, "thread t owns digit t in the scans and the look-back");

// One stable pass over 8-bit digit `pass` of the keys, carrying a 32-bit
// value.  Tiles are numbered in start order by a counter, so a tile's
// predecessors have all started; the look-back adds their per-digit counts
// until one publishes its inclusive prefix.  The first pass reads the keys
// from the sorted own rows (columns, mapped by pair_key) in entry order and
// makes the values, the places of the entries' p in p: entry x of row i = x
// / k takes i k + sorig[x].  So each inbox comes out in increasing listing
// point.
template <bool kFirst>
__global__ __launch_bounds__(kSortBlock) void aff_pair_pass_kernel(
    const uint32_t *__restrict__ kin, const uint32_t *__restrict__ vin, const uint8_t *__restrict__ sorig,
    uint32_t *__restrict__ kout, uint32_t *__restrict__ vout, unsigned long long *__restrict__ status,
    const uint32_t *__restrict__ hist, Header *__restrict__ hdr, int pass, int64_t m, int64_t n, int k)
{
    constexpr int kWaves = kSortBlock / kWave;
    constexpr int kSeg = kWave * kAffSortItems; // keys per wave segment
    __shared__ uint32_t s_tile;
    __shared__ uint32_t s_wcnt[kWaves][kRadix];
    __shared__ uint32_t s_lstart[kRadix];
    __shared__ uint32_t s_gofs[kRadix];
    __shared__ uint32_t s_scan[kWaves];
    __shared__ uint32_t s_keys[kAffSortTile];
    __shared__ uint32_t s_vals[kAffSortTile];

    const int t = threadIdx.x, w = t / kWave, lane = lane_id();
    const int shift = pass * kRadixBits;
    if (t == 0) s_tile = atomicAdd(&hdr->tile_counter[pass], 1u);
    for (int q = t; q < kWaves * kRadix; q += kSortBlock) (&s_wcnt[0][0])[q] = 0;
    __syncthreads();
    const uint32_t tile = s_tile;
    const int64_t base = int64_t(tile) * kAffSortTile;
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));

    uint32_t key[kAffSortItems], vv[kAffSortItems], rank[kAffSortItems];
#pragma unroll
    for (int r = 0; r < kAffSortItems; ++r) {
        const int64_t p = base + w * kSeg + r * kWave + lane;
        const bool valid = p < m;
        key[r] = valid ? (kFirst ? pair_key(int32_t(kin[p]), n) : kin[p]) : 0u;
        if (kFirst) {
            const uint32_t x = uint32_t(p), row = x / uint32_t(k);
            vv[r] = valid ? row * uint32_t(k) + sorig[p] : 0u;
        } else {
            vv[r] = valid ? vin[p] : 0u;
        }
    }
#pragma unroll
    for (int r = 0; r < kAffSortItems; ++r) {
        const int64_t p = base + w * kSeg + r * kWave + lane;
        const bool valid = p < m;
        const uint32_t d = (key[r] >> shift) & (kRadix - 1);
        uint64_t peers = ballot(valid);
#pragma unroll
        for (int b = 0; b < kRadixBits; ++b) {
            const bool bit = (d >> b) & 1u;
            const uint64_t mk = ballot(bit);
            peers &= bit ? mk : ~mk;
        }
        const int leader = peers ? __ffsll((unsigned long long)peers) - 1 : lane;
        uint32_t old = 0;
        if (valid && lane == leader) {
            old = s_wcnt[w][d];
            s_wcnt[w][d] = old + uint32_t(__popcll(peers));
        }
        old = __shfl(old, leader, kWave);
        rank[r] = old + uint32_t(__popcll(peers & lt_mask));
    }
    __syncthreads();

    // thread t owns digit t: per-wave offsets, tile count, look-back
    const uint32_t d = t;
    uint32_t tot = 0;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) {
        const uint32_t c = s_wcnt[q][d];
        s_wcnt[q][d] = tot;
        tot += c;
    }
    unsigned long long *my = status + int64_t(tile) * kRadix + d;
    __hip_atomic_store(my, (tile == 0 ? kAffInclusive : kAffAggregate) | tot, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
    s_lstart[d] = aff_block_scan(tot, s_scan);
    uint32_t h = 0;
#pragma unroll
    for (int c = 0; c < kHistCopies; ++c) h += hist[c * kAffHistWords + pass * kRadix + d];
    const uint32_t dbase = aff_block_scan(h, s_scan);
    uint32_t excl = 0;
    if (tile > 0) {
        int64_t tt = int64_t(tile) - 1;
        uint32_t spins = 0;
        for (;;) {
            const unsigned long long sv =
                __hip_atomic_load(status + tt * kRadix + d, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if ((sv >> 32) == 0) { // not published yet
                if (++spins > kSpinLimit) {
                    atomicOr(&hdr->flags, kErrLookback);
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
                continue;
            }
            excl += uint32_t(sv);
            if (sv & kAffInclusive) break;
            if (--tt < 0) break; // cannot happen: tile 0 publishes an inclusive prefix
        }
        __hip_atomic_store(my, kAffInclusive | (excl + tot), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    s_gofs[d] = dbase + excl;
    __syncthreads();

    // rank -> position inside the tile, staged through LDS, then out in digit runs
#pragma unroll
    for (int r = 0; r < kAffSortItems; ++r) {
        const int64_t p = base + w * kSeg + r * kWave + lane;
        if (p < m) {
            const uint32_t dd = (key[r] >> shift) & (kRadix - 1);
            const uint32_t lp = s_lstart[dd] + s_wcnt[w][dd] + rank[r];
            s_keys[lp] = key[r];
            s_vals[lp] = vv[r];
        }
    }
    __syncthreads();
    const int tile_n = int(m - base < kAffSortTile ? m - base : kAffSortTile);
    for (int j = t; j < tile_n; j += kSortBlock) {
        const uint32_t k2 = s_keys[j];
        const uint32_t dd = (k2 >> shift) & (kRadix - 1);
        const uint64_t out = uint64_t(s_gofs[dd]) + (uint32_t(j) - s_lstart[dd]);
        if (out < uint64_t(m)) {
            kout[out] = k2;
            vout[out] = s_vals[j];
        } else {
            atomicOr(&hdr->flags, kErrRange);
        }
    }
}

// inbox offsets from the sorted keys (all in [0, n]): ib[j] = the first
// position whose key is >= j, for j = 0..n; every j is written by exactly one
// thread, the one at the end of the gap that contains it
__global__ __launch_bounds__(256) void aff_inbox_kernel(const uint32_t *__restrict__ keys, int64_t m, int64_t n,
                                                        int64_t *__restrict__ ib)
{
    const int64_t x = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (x > m) return;
    // clamped, so that even keys left unsorted by a failed look-back write in bounds
    const int64_t lo = x == 0 ? -1 : (keys[x - 1] < n ? int64_t(keys[x - 1]) : n);
    const int64_t hi = x == m ? n : (keys[x] < n ? int64_t(keys[x]) : n);
    for (int64_t j = lo + 1; j <= hi; ++j) ib[j] = x;
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
// and its inbox (m columns in order, with p_{j|c}): the sorted pairs
// [ib[j], ib[j + 1]), each holding c k + e for the neighbour e of row c that
// is j (the place of p_{j|c} in p).
// kWrite = false: count the inbox entries that are not in the own list (P's
// row has k plus that many entries); kWrite = true: write the row in column
// order.  With MO[e] the number of own entries before e that are also in the
// inbox, own entry e goes to e + t - MO[e] (t: inbox entries below its
// column) and an inbox-only entry at inbox position t to e' + t - MO[e'] (e':
// own entries below its column).  A pair in both lists is written once, with
// (p_{c|j} + p_{j|c}) / 2N: the same fp64 sum in both rows, so P is exactly
// symmetric.  p is in neighbour order: sorted entry e of row c sits at
// c k + sorig[c k + e].
template <int kCap, bool kWrite> struct AffRowLds {
    uint32_t own[kAffMaxK];
    double ownp[kWrite ? kAffMaxK : 1];
    uint32_t in[kCap];
    double inp[kWrite ? kCap : 1];
    uint8_t fl[kAffMaxK];
    uint32_t mo[kAffMaxK + 1];
    uint32_t w[kAffLongThreads / kWave];
};

struct AffRowArgs {
    int64_t n, m; // points, pairs
    int k;
    const int32_t *scol;
    const uint8_t *sorig;
    const double *p;
    const int64_t *ib;
    const uint32_t *pair; // values of the sorted pairs: places in p
    uint32_t *inonly;
    const int64_t *row_ptr;
    int32_t *col;
    float *val;
};

// a row's inbox range, clamped to the pairs (the offsets are sound unless the
// sort failed, which the call reports)
__device__ inline void inbox_range(const AffRowArgs &a, int64_t j, int64_t *b, int *len)
{
    int64_t lo = a.ib[j], hi = a.ib[j + 1];
    lo = lo < 0 ? 0 : lo > a.m ? a.m : lo;
    hi = hi < lo ? lo : hi > a.m ? a.m : hi;
    *b = lo;
    *len = int(hi - lo < int64_t(1) << 30 ? hi - lo : int64_t(1) << 30);
}

template <int kCap, bool kWrite>
__device__ inline void aff_row(int64_t j, const AffRowArgs &a, AffRowLds<kCap, kWrite> &L)
{
    const int k = a.k;
    int64_t b;
    int m;
    inbox_range(a, j, &b, &m);
    for (int e = threadIdx.x; e < k; e += blockDim.x) {
        L.own[e] = uint32_t(a.scol[j * k + e]);
        if (kWrite) L.ownp[e] = a.p[j * k + a.sorig[j * k + e]];
    }
    for (int t = threadIdx.x; t < m; t += blockDim.x) {
        uint32_t x = a.pair[b + t]; // c k + the neighbour position of j in row c
        x = x < uint64_t(a.m) ? x : 0u; // only a failed sort leaves other values
        L.in[t] = x / uint32_t(k);
        if (kWrite) L.inp[t] = a.p[x];
    }
    __syncthreads();
    for (int e = threadIdx.x; e < k; e += blockDim.x) {
        const int t = lower_bound_u32(L.in, m, L.own[e]);
        L.fl[e] = t < m && L.in[t] == L.own[e];
    }
    __syncthreads();
    const uint32_t both = block_flag_scan(L.fl, k, L.mo, L.w);
    if (!kWrite) {
        if (threadIdx.x == 0) a.inonly[j] = uint32_t(m) - both;
        return;
    }
    const int64_t o = a.row_ptr[j];
    const double inv2n = 1.0 / (2.0 * double(a.n));
    for (int e = threadIdx.x; e < k; e += blockDim.x) {
        const int t = lower_bound_u32(L.in, m, L.own[e]);
        const int64_t q = o + e + t - L.mo[e];
        a.col[q] = int32_t(L.own[e]);
        a.val[q] = float((L.fl[e] ? L.ownp[e] + L.inp[t] : L.ownp[e]) * inv2n);
    }
    for (int t = threadIdx.x; t < m; t += blockDim.x) {
        const int e = lower_bound_u32(L.own, k, L.in[t]);
        if (e < k && L.own[e] == L.in[t]) continue; // written with the own entry
        const int64_t q = o + e + t - L.mo[e];
        a.col[q] = int32_t(L.in[t]);
        a.val[q] = float(L.inp[t] * inv2n);
    }
}

// rows whose inbox fits kAffShortCap: one wave each; longer ones are listed
// (by the counting pass) for the block kernel
template <bool kWrite>
__global__ __launch_bounds__(kWave) void aff_row_kernel(AffRowArgs a, uint32_t *__restrict__ longrows,
                                                        uint32_t *__restrict__ counters)
{
    __shared__ AffRowLds<kAffShortCap, kWrite> L;
    const int64_t j = blockIdx.x;
    int64_t b;
    int m;
    inbox_range(a, j, &b, &m);
    if (m > kAffShortCap) {
        if (!kWrite && threadIdx.x == 0) longrows[atomicAdd(&counters[0], 1u)] = uint32_t(j);
        return;
    }
    aff_row<kAffShortCap, kWrite>(j, a, L);
}

template <bool kWrite>
__global__ __launch_bounds__(kAffLongThreads) void aff_long_row_kernel(AffRowArgs a,
                                                                       const uint32_t *__restrict__ longrows,
                                                                       const uint32_t *__restrict__ counters,
                                                                       Header *__restrict__ hdr)
{
    __shared__ AffRowLds<kAffLongCap, kWrite> L;
    const uint32_t count = counters[0];
    for (uint32_t r = blockIdx.x; r < count; r += gridDim.x) {
        const int64_t j = longrows[r];
        int64_t b;
        int m;
        inbox_range(a, j, &b, &m);
        if (m > kAffLongCap) { // over the documented limit
            if (!kWrite && threadIdx.x == 0) {
                atomicOr(&hdr->flags, kErrRange);
                a.inonly[j] = 0;
            }
            continue;
        }
        __syncthreads();
        aff_row<kAffLongCap, kWrite>(j, a, L);
    }
}

// ------------------------------------------------------------------ launchers
static AffRowArgs row_args(int64_t n, int k, void *ws, const AffLayout &A)
{
    AffRowArgs a{};
    a.n = n;
    a.m = A.m;
    a.k = k;
    a.scol = at<int32_t>(ws, A.scol);
    a.sorig = at<uint8_t>(ws, A.sorig);
    a.p = at<double>(ws, A.p);
    a.ib = at<int64_t>(ws, A.ib);
    a.pair = at<uint32_t>(ws, A.val[(A.passes - 1) & 1]); // the last pass's output
    a.inonly = at<uint32_t>(ws, A.inonly);
    return a;
}

void launch_aff_clear(void *ws, const AffLayout &A, hipStream_t st)
{
    const int64_t words = int64_t(A.passes) * A.sort_tiles * kRadix;
    const int64_t blocks = std::min<int64_t>(2048, std::max<int64_t>(1, (words + 255) / 256));
    aff_clear_kernel<<<unsigned(blocks), 256, 0, st>>>(at<Header>(ws, A.header), at<uint32_t>(ws, A.hist),
                                                       at<unsigned long long>(ws, A.status), words,
                                                       at<uint32_t>(ws, A.counters));
}

// step 1: p_{j|i} in neighbour order and sigma_i^2
void launch_aff_search(const float *dist, int64_t n, int k, double perplexity, double *sigma2, void *ws,
                       const AffLayout &A, hipStream_t st)
{
    Header *hdr = at<Header>(ws, A.header);
    double *p = at<double>(ws, A.p);
    const double lu = log(perplexity);
    if (k <= kAffLaneMaxK) {
        const unsigned qb = unsigned((n + 63) / 64); // blocks of 64 rows
        if (k <= 8 * kAffG)
            aff_search_quad_kernel<8><<<qb, 256, 0, st>>>(dist, n, k, lu, p, sigma2, hdr);
        else if (k <= 16 * kAffG)
            aff_search_quad_kernel<16><<<qb, 256, 0, st>>>(dist, n, k, lu, p, sigma2, hdr);
        else if (k <= 24 * kAffG)
            aff_search_quad_kernel<24><<<qb, 256, 0, st>>>(dist, n, k, lu, p, sigma2, hdr);
        else
            aff_search_quad_kernel<32><<<qb, 256, 0, st>>>(dist, n, k, lu, p, sigma2, hdr);
    } else {
        const unsigned sb = unsigned((n + 3) / 4);
        if ((k + kWave - 1) / kWave == 3)
            aff_search_kernel<3><<<sb, kAffSearchBlock, 0, st>>>(dist, n, k, lu, p, sigma2, hdr);
        else
            aff_search_kernel<4><<<sb, kAffSearchBlock, 0, st>>>(dist, n, k, lu, p, sigma2, hdr);
    }
    static_assert(kAffMaxK <= 4 * kWave && kAffLaneMaxK == 32 * kAffG && kAffLaneMaxK >= 2 * kWave,
                  "three or four distances per lane in the wave kernel, at most 32 per lane in the quad kernel");
}

// steps 2-4 (the neighbour indices only): sorted own rows, the pair sort,
// inbox offsets, the union counts and P's row pointers
void launch_aff_index(const int32_t *idx, int64_t n, int k, int64_t *row_ptr, void *ws, const AffLayout &A,
                      hipStream_t st)
{
    Header *hdr = at<Header>(ws, A.header);
    int32_t *scol = at<int32_t>(ws, A.scol);
    uint8_t *sorig = at<uint8_t>(ws, A.sorig);
    uint32_t *hist = at<uint32_t>(ws, A.hist), *counters = at<uint32_t>(ws, A.counters);
    uint32_t *inonly = at<uint32_t>(ws, A.inonly), *longrows = at<uint32_t>(ws, A.longrows);
    unsigned long long *part = at<unsigned long long>(ws, A.part);
    const unsigned rb = unsigned((n + 3) / 4);
    if (k <= kWave)
        aff_own_sort_kernel<1><<<rb, 256, 0, st>>>(idx, n, k, scol, sorig, hdr);
    else if (k <= 2 * kWave)
        aff_own_sort_kernel<2><<<rb, 256, 0, st>>>(idx, n, k, scol, sorig, hdr);
    else
        aff_own_sort_kernel<4><<<rb, 256, 0, st>>>(idx, n, k, scol, sorig, hdr);
    const int64_t m = A.m;
    aff_hist_kernel<<<unsigned(std::min<int64_t>(2048, (m + 255) / 256)), 256, 0, st>>>(scol, m, n, A.passes, hist);
    const uint32_t *kin = reinterpret_cast<const uint32_t *>(scol), *vin = nullptr;
    for (int q = 0; q < A.passes; ++q) {
        uint32_t *kout = at<uint32_t>(ws, A.key[q & 1]), *vout = at<uint32_t>(ws, A.val[q & 1]);
        unsigned long long *status = at<unsigned long long>(ws, A.status) + int64_t(q) * A.sort_tiles * kRadix;
        if (q == 0)
            aff_pair_pass_kernel<true><<<unsigned(A.sort_tiles), kSortBlock, 0, st>>>(
                kin, vin, sorig, kout, vout, status, hist, hdr, q, m, n, k);
        else
            aff_pair_pass_kernel<false><<<unsigned(A.sort_tiles), kSortBlock, 0, st>>>(
                kin, vin, sorig, kout, vout, status, hist, hdr, q, m, n, k);
        kin = kout;
        vin = vout;
    }
    int64_t *ib = at<int64_t>(ws, A.ib);
    aff_inbox_kernel<<<unsigned((m + 1 + 255) / 256), 256, 0, st>>>(kin, m, n, ib);
    const AffRowArgs a = row_args(n, k, ws, A);
    aff_row_kernel<false><<<unsigned(n), kWave, 0, st>>>(a, longrows, counters);
    aff_long_row_kernel<false><<<256, kAffLongThreads, 0, st>>>(a, longrows, counters, hdr);
    aff_scan_part_kernel<<<unsigned(A.scan_tiles), kAffScanBlock, 0, st>>>(inonly, n, k, part);
    aff_scan_top_kernel<<<1, kAffScanBlock, 0, st>>>(part, A.scan_tiles, row_ptr, n);
    aff_scan_down_kernel<<<unsigned(A.scan_tiles), kAffScanBlock, 0, st>>>(inonly, n, k, part, row_ptr);
}

// step 5: P's rows
void launch_aff_back(int64_t n, int k, const int64_t *row_ptr, int32_t *col, float *val, void *ws,
                     const AffLayout &A, hipStream_t st)
{
    AffRowArgs a = row_args(n, k, ws, A);
    a.row_ptr = row_ptr;
    a.col = col;
    a.val = val;
    uint32_t *counters = at<uint32_t>(ws, A.counters), *longrows = at<uint32_t>(ws, A.longrows);
    aff_row_kernel<true><<<unsigned(n), kWave, 0, st>>>(a, longrows, counters);
    aff_long_row_kernel<true><<<256, kAffLongThreads, 0, st>>>(a, longrows, counters, at<Header>(ws, A.header));
}

} // namespace bht
