// Bounding box, Morton codes and the radix sort of the codes (gfx950).
//
// Quadtree Building (Algorithm 1 and the paragraph on Morton codes): the
// square domain is centred on the bounding box with half-side r_span, each
// coordinate is quantised to 32 bits and the two are bit-interleaved with
// dimension 0 in the even bits.  Sorting the codes puts points of a cell next
// to each other, which is what the tree build and the repulsive traversal
// rely on.
//
// The sort is an LSD radix sort over 8-bit digits (8 passes).  The global
// digit histograms of all passes are accumulated while the codes are formed;
// each pass is then a single kernel that ranks a tile in LDS, finds the
// tile's global offsets with a decoupled look-back over the tiles before it,
// and writes the tile out digit by digit.
#include "common.hpp"
#include "kernels.hpp"

namespace bht {

// ------------------------------------------------------------------ bbox
// T: float (the path) or double (the fp64 variant); each block writes
// {min x, max x, min y, max y, non-finite flag} as 8 T.
template <typename T>
__global__ __launch_bounds__(256) void bbox_partial_kernel(const vec2_t<T> *__restrict__ Y, int64_t n,
                                                           T *__restrict__ part)
{
    T mnx = INFINITY, mny = INFINITY, mxx = -INFINITY, mxy = -INFINITY;
    uint32_t bad = 0;
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
         i += int64_t(gridDim.x) * blockDim.x) {
        const vec2_t<T> y = Y[i];
        bad |= !(isfinite(y.x) && isfinite(y.y));
        mnx = vmin(mnx, y.x);
        mxx = vmax(mxx, y.x);
        mny = vmin(mny, y.y);
        mxy = vmax(mxy, y.y);
    }
    mnx = wave_min(mnx);
    mny = wave_min(mny);
    mxx = wave_max(mxx);
    mxy = wave_max(mxy);
    bool anybad = ballot(bad != 0) != 0;
    __shared__ T s[4][4];
    __shared__ uint32_t sb[4];
    int w = threadIdx.x / kWave;
    if (lane_id() == 0) {
        s[w][0] = mnx;
        s[w][1] = mxx;
        s[w][2] = mny;
        s[w][3] = mxy;
        sb[w] = anybad;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        T r[4] = {s[0][0], s[0][1], s[0][2], s[0][3]};
        uint32_t b = sb[0];
        for (int k = 1; k < 4; ++k) {
            r[0] = vmin(r[0], s[k][0]);
            r[1] = vmax(r[1], s[k][1]);
            r[2] = vmin(r[2], s[k][2]);
            r[3] = vmax(r[3], s[k][3]);
            b |= sb[k];
        }
        T *o = part + 8 * blockIdx.x;
        o[0] = r[0];
        o[1] = r[1];
        o[2] = r[2];
        o[3] = r[3];
        reinterpret_cast<uint32_t *>(o + 4)[0] = b;
    }
}

// The per-call scalars and counters, reset by the box kernel that starts a call.
__device__ inline void reset_call_state(Header *hdr, uint32_t nonfinite)
{
    hdr->flags = nonfinite ? kErrNonFinite : 0u;
    hdr->Z = 0.0;
    hdr->interactions = 0;
    for (int k = 0; k < kSortPasses; ++k) hdr->tile_counter[k] = 0;
    hdr->ticket_bbox = 0;
    hdr->ticket_rep = 0;
    hdr->attract_next = 0;
    hdr->max_depth = 0;
}

// One block: finish the box, derive the quantisation parameters in fp64 and
// reset the per-call counters and histograms.
template <typename T>
__global__ __launch_bounds__(256) void bbox_final_kernel(const T *__restrict__ part, int nparts,
                                                         Header *__restrict__ hdr,
                                                         uint32_t *__restrict__ hist)
{
    T mnx = INFINITY, mny = INFINITY, mxx = -INFINITY, mxy = -INFINITY;
    uint32_t bad = 0;
    for (int k = threadIdx.x; k < nparts; k += blockDim.x) {
        const T *p = part + 8 * k;
        mnx = vmin(mnx, p[0]);
        mxx = vmax(mxx, p[1]);
        mny = vmin(mny, p[2]);
        mxy = vmax(mxy, p[3]);
        bad |= reinterpret_cast<const uint32_t *>(p + 4)[0];
    }
    mnx = wave_min(mnx);
    mny = wave_min(mny);
    mxx = wave_max(mxx);
    mxy = wave_max(mxy);
    bool anybad = ballot(bad != 0) != 0;
    __shared__ T s[4][4];
    __shared__ uint32_t sb[4];
    int w = threadIdx.x / kWave;
    if (lane_id() == 0) {
        s[w][0] = mnx;
        s[w][1] = mxx;
        s[w][2] = mny;
        s[w][3] = mxy;
        sb[w] = anybad;
    }
    for (int k = threadIdx.x; k < kHistCopies * kHistWords; k += blockDim.x) hist[k] = 0;
    __syncthreads();
    if (threadIdx.x == 0) {
        T r[4] = {s[0][0], s[0][1], s[0][2], s[0][3]};
        uint32_t b = sb[0];
        for (int k = 1; k < 4; ++k) {
            r[0] = vmin(r[0], s[k][0]);
            r[1] = vmax(r[1], s[k][1]);
            r[2] = vmin(r[2], s[k][2]);
            r[3] = vmax(r[3], s[k][3]);
            b |= sb[k];
        }
        hdr->bmin[0] = float(r[0]);
        hdr->bmax[0] = float(r[1]);
        hdr->bmin[1] = float(r[2]);
        hdr->bmax[1] = float(r[3]);
        // fp64, fixed operation order: the codes depend on these bits
        double c0 = (double(r[0]) + double(r[1])) * 0.5;
        double c1 = (double(r[2]) + double(r[3])) * 0.5;
        double e0 = double(r[1]) - double(r[0]);
        double e1 = double(r[3]) - double(r[2]);
        double rs = 0.5 * (e0 > e1 ? e0 : e1);
        hdr->cent[0] = c0;
        hdr->cent[1] = c1;
        hdr->rspan = rs;
        hdr->yroot[0] = c0 - rs;
        hdr->yroot[1] = c1 - rs;
        hdr->scale = rs > 0.0 ? 2147483648.0 / rs : 0.0;
        reset_call_state(hdr, b);
    }
}

// ------------------------------------------------------------------ Morton
template <typename T> __device__ inline uint32_t quantise(T y, double yroot, double scale)
{
    double q = (double(y) - yroot) * scale;
    if (!(q > 0.0)) return 0u; // also catches NaN
    if (q >= 4294967295.0) return 0xffffffffu;
    return uint32_t(q); // truncation toward zero
}

// Interleaving by its definition: bit k of a grid coordinate goes to bit 2k
// of its spread word, and dimension d is then shifted to bit 2k + d.  The
// spread is taken a byte at a time: entry b of a 256-entry table holds byte b
// with each bit k moved to bit 2k (built from that rule, one entry per
// thread), and byte j of the coordinate lands at bit 16 j of the word.
__device__ inline uint32_t spread_byte_rule(uint32_t b)
{
    uint32_t s = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) s |= ((b >> k) & 1u) << (2 * k);
    return s;
}

__device__ inline uint64_t spread_by_bytes(const uint16_t *__restrict__ tab, uint32_t v)
{
    return uint64_t(tab[v & 0xffu]) | (uint64_t(tab[(v >> 8) & 0xffu]) << 16) |
           (uint64_t(tab[(v >> 16) & 0xffu]) << 32) | (uint64_t(tab[v >> 24]) << 48);
}

// Codes of one tile of points, the private copy of Y (in the caller's order,
// or in a layout order when `perm` is given: position i holds the point
// perm[i], gathered, which costs less than scattering each point to its
// position), the 8 global digit histograms; also clears the per-position tree
// masks and this tile's look-back status words of every pass.
template <typename T>
__global__ __launch_bounds__(kSortBlock) void morton_kernel(
    const vec2_t<T> *__restrict__ Y, int64_t n, const Header *__restrict__ hdr,
    uint64_t *__restrict__ codes, vec2_t<T> *__restrict__ ycopy, const uint32_t *__restrict__ perm,
    uint32_t *__restrict__ hist, uint32_t *__restrict__ levelmask, uint32_t *__restrict__ status, int64_t tiles)
{
    __shared__ uint32_t sh[kSortPasses * kRadix];
    __shared__ uint16_t s_spread[256];
    static_assert(kSortBlock == 256, "one spread-table entry per thread");
    s_spread[threadIdx.x] = uint16_t(spread_byte_rule(threadIdx.x));
    for (int k = threadIdx.x; k < kSortPasses * kRadix; k += kSortBlock) sh[k] = 0;
    // clear this tile's look-back words of every pass
    for (int k = threadIdx.x; k < kSortPasses * kRadix; k += kSortBlock) {
        int pass = k / kRadix, d = k % kRadix;
        status[(int64_t(pass) * tiles + blockIdx.x) * kRadix + d] = 0;
    }
    __syncthreads();
    const double yr0 = hdr->yroot[0], yr1 = hdr->yroot[1], sc = hdr->scale;
    const int64_t base = int64_t(blockIdx.x) * kSortTile;
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        int64_t i = base + r * kSortBlock + threadIdx.x;
        if (i < n) {
            const vec2_t<T> y = Y[i];
            if (perm) {
                const uint32_t p = perm[i];
                if (p < uint32_t(n)) ycopy[i] = Y[p];
            } else {
                ycopy[i] = y;
            }
            uint64_t code = spread_by_bytes(s_spread, quantise(y.x, yr0, sc)) |
                            (spread_by_bytes(s_spread, quantise(y.y, yr1, sc)) << 1);
            codes[i] = code;
            levelmask[i] = 0;
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

// ------------------------------------------------------------------ 3-D box and codes
// A 3-D embedding: the domain is the cube centred on the box with half-side
// r_span (the widest half extent); each coordinate is quantised to 21 bits,
// trunc((y - y_root) * 2^20 / r_span) clamped to [0, 2^21 - 1], in fp64 in
// a fixed order, and bit k of dimension d goes to bit 3k + d of the code
// (63 bits; the top bit stays 0).
__global__ __launch_bounds__(256) void bbox3_partial_kernel(const float3 *__restrict__ Y, int64_t n,
                                                            float *__restrict__ part)
{
    float mn[3] = {INFINITY, INFINITY, INFINITY}, mx[3] = {-INFINITY, -INFINITY, -INFINITY};
    uint32_t bad = 0;
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x) {
        const float3 y = Y[i];
        bad |= !(isfinite(y.x) && isfinite(y.y) && isfinite(y.z));
#pragma unroll
        for (int d = 0; d < 3; ++d) {
            mn[d] = fminf(mn[d], coord(y, d));
            mx[d] = fmaxf(mx[d], coord(y, d));
        }
    }
#pragma unroll
    for (int d = 0; d < 3; ++d) {
        mn[d] = wave_min(mn[d]);
        mx[d] = wave_max(mx[d]);
    }
    const bool anybad = ballot(bad != 0) != 0;
    __shared__ float s[4][6];
    __shared__ uint32_t sb[4];
    const int w = threadIdx.x / kWave;
    if (lane_id() == 0) {
#pragma unroll
        for (int d = 0; d < 3; ++d) {
            s[w][2 * d] = mn[d];
            s[w][2 * d + 1] = mx[d];
        }
        sb[w] = anybad;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        float *o = part + 8 * blockIdx.x; // {min x, max x, min y, max y, min z, max z, flag}
        uint32_t b = 0;
        for (int d = 0; d < 3; ++d) {
            float lo = s[0][2 * d], hi = s[0][2 * d + 1];
            for (int k = 1; k < 4; ++k) {
                lo = fminf(lo, s[k][2 * d]);
                hi = fmaxf(hi, s[k][2 * d + 1]);
            }
            o[2 * d] = lo;
            o[2 * d + 1] = hi;
        }
        for (int k = 0; k < 4; ++k) b |= sb[k];
        reinterpret_cast<uint32_t *>(o + 6)[0] = b;
    }
}

__global__ __launch_bounds__(256) void bbox3_final_kernel(const float *__restrict__ part, int nparts,
                                                          Header *__restrict__ hdr, uint32_t *__restrict__ hist)
{
    float mn[3] = {INFINITY, INFINITY, INFINITY}, mx[3] = {-INFINITY, -INFINITY, -INFINITY};
    uint32_t bad = 0;
    for (int k = threadIdx.x; k < nparts; k += blockDim.x) {
        const float *p = part + 8 * k;
#pragma unroll
        for (int d = 0; d < 3; ++d) {
            mn[d] = fminf(mn[d], p[2 * d]);
            mx[d] = fmaxf(mx[d], p[2 * d + 1]);
        }
        bad |= reinterpret_cast<const uint32_t *>(p + 6)[0];
    }
#pragma unroll
    for (int d = 0; d < 3; ++d) {
        mn[d] = wave_min(mn[d]);
        mx[d] = wave_max(mx[d]);
    }
    const bool anybad = ballot(bad != 0) != 0;
    __shared__ float s[4][6];
    __shared__ uint32_t sb[4];
    const int w = threadIdx.x / kWave;
    if (lane_id() == 0) {
#pragma unroll
        for (int d = 0; d < 3; ++d) {
            s[w][2 * d] = mn[d];
            s[w][2 * d + 1] = mx[d];
        }
        sb[w] = anybad;
    }
    for (int k = threadIdx.x; k < kHistCopies * kHistWords; k += blockDim.x) hist[k] = 0;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t b = 0;
        for (int k = 0; k < 4; ++k) b |= sb[k];
        double c[3], widest = 0.0;
        for (int d = 0; d < 3; ++d) {
            float lo = s[0][2 * d], hi = s[0][2 * d + 1];
            for (int k = 1; k < 4; ++k) {
                lo = fminf(lo, s[k][2 * d]);
                hi = fmaxf(hi, s[k][2 * d + 1]);
            }
            hdr->bmin[d] = lo;
            hdr->bmax[d] = hi;
            // fp64, fixed operation order: the codes depend on these bits
            c[d] = (double(lo) + double(hi)) * 0.5;
            const double ext = double(hi) - double(lo);
            widest = ext > widest ? ext : widest;
        }
        const double rs = 0.5 * widest;
        for (int d = 0; d < 3; ++d) {
            hdr->cent[d] = c[d];
            hdr->yroot[d] = c[d] - rs;
        }
        hdr->rspan = rs;
        hdr->scale = rs > 0.0 ? 1048576.0 / rs : 0.0;
        reset_call_state(hdr, b);
    }
}

__device__ inline uint32_t quantise21(float y, double yroot, double scale)
{
    double q = (double(y) - yroot) * scale;
    if (!(q > 0.0)) return 0u; // also catches NaN
    if (q >= 2097151.0) return 2097151u;
    return uint32_t(q); // truncation toward zero
}

// Three-way spread by the interleaving rule: entry b of the table holds byte
// b with each bit k moved to bit 3k; byte j of a 21-bit coordinate lands at
// bit 24 j of the word.
__device__ inline uint32_t spread3_byte_rule(uint32_t b)
{
    uint32_t s = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) s |= ((b >> k) & 1u) << (3 * k);
    return s;
}

__device__ inline uint64_t spread3_by_bytes(const uint32_t *__restrict__ tab, uint32_t v)
{
    return uint64_t(tab[v & 0xffu]) | (uint64_t(tab[(v >> 8) & 0xffu]) << 24) | (uint64_t(tab[v >> 16]) << 48);
}

__global__ __launch_bounds__(kSortBlock) void morton3_kernel(
    const float3 *__restrict__ Y, int64_t n, const Header *__restrict__ hdr, uint64_t *__restrict__ codes,
    float3 *__restrict__ ycopy, const uint32_t *__restrict__ perm, uint32_t *__restrict__ hist,
    uint32_t *__restrict__ levelmask, uint32_t *__restrict__ status, int64_t tiles)
{
    __shared__ uint32_t sh[kSortPasses * kRadix];
    __shared__ uint32_t s_spread[256];
    static_assert(kSortBlock == 256, "one spread-table entry per thread");
    s_spread[threadIdx.x] = spread3_byte_rule(threadIdx.x);
    for (int k = threadIdx.x; k < kSortPasses * kRadix; k += kSortBlock) sh[k] = 0;
    for (int k = threadIdx.x; k < kSortPasses * kRadix; k += kSortBlock) {
        const int pass = k / kRadix, d = k % kRadix;
        status[(int64_t(pass) * tiles + blockIdx.x) * kRadix + d] = 0;
    }
    __syncthreads();
    const double yr0 = hdr->yroot[0], yr1 = hdr->yroot[1], yr2 = hdr->yroot[2], sc = hdr->scale;
    const int64_t base = int64_t(blockIdx.x) * kSortTile;
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        const int64_t i = base + r * kSortBlock + threadIdx.x;
        if (i < n) {
            const float3 y = Y[i];
            const uint32_t p = perm ? perm[i] : uint32_t(i); // a layout's order, or the caller's
            ycopy[i] = p == uint32_t(i) ? y : Y[p < uint32_t(n) ? p : uint32_t(i)];
            const uint64_t code = spread3_by_bytes(s_spread, quantise21(y.x, yr0, sc)) |
                                  (spread3_by_bytes(s_spread, quantise21(y.y, yr1, sc)) << 1) |
                                  (spread3_by_bytes(s_spread, quantise21(y.z, yr2, sc)) << 2);
            codes[i] = code;
            levelmask[i] = 0;
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

// ------------------------------------------------------------------ onesweep pass
// Block-wide exclusive scan of one value per thread (256 threads).
__device__ inline uint32_t block_exclusive_scan256(uint32_t v, uint32_t *s_wave /*[4]*/,
                                                   uint32_t *total)
{
    int lane = lane_id(), w = threadIdx.x / kWave;
    uint32_t x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        uint32_t y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) s_wave[w] = x;
    __syncthreads();
    uint32_t off = 0, tot = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        uint32_t t = s_wave[k];
        off += (k < w) ? t : 0u;
        tot += t;
    }
    if (total) *total = tot;
    return off + x - v;
}

__device__ inline void publish(uint32_t *p, uint32_t word)
{
    __hip_atomic_store(p, word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ inline uint32_t peek(const uint32_t *p)
{
    return __hip_atomic_load(const_cast<uint32_t *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

static_assert(kSortBlock == kRadix, "thread t owns digit t in the scans and the look-back");

// V: the point type gathered by the last pass (float2, double2 or float3)
template <bool kFirst, bool kLast, typename V = float2>
__global__ __launch_bounds__(kSortBlock) void onesweep_kernel(
    const uint64_t *__restrict__ keys_in, const uint32_t *__restrict__ idx_in,
    uint64_t *__restrict__ keys_out, uint32_t *__restrict__ idx_out,
    uint32_t *__restrict__ status, const uint32_t *__restrict__ hist, Header *__restrict__ hdr,
    int pass, int64_t n, const V *__restrict__ ysrc, V *__restrict__ ys)
{
    constexpr int kWaves = kSortBlock / kWave;
    constexpr int kSeg = kWave * kSortItems; // keys per wave segment
    __shared__ uint32_t s_tile;
    __shared__ uint32_t s_wcnt[kWaves][kRadix];
    __shared__ uint32_t s_lstart[kRadix];
    __shared__ uint32_t s_gofs[kRadix];
    __shared__ uint32_t s_scan[4];
    __shared__ uint64_t s_keys[kSortTile];
    __shared__ uint32_t s_idx[kSortTile];

    const int t = threadIdx.x, w = t / kWave, lane = lane_id();
    const int shift = pass * kRadixBits;
    if (t == 0) s_tile = atomicAdd(&hdr->tile_counter[pass], 1u);
    for (int k = t; k < kWaves * kRadix; k += kSortBlock) (&s_wcnt[0][0])[k] = 0;
    __syncthreads();
    const uint32_t tile = s_tile;
    const int64_t base = int64_t(tile) * kSortTile;
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));

    uint64_t key[kSortItems];
    uint32_t rank[kSortItems], ixv[kSortItems];
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        int64_t p = base + w * kSeg + r * kWave + lane;
        bool valid = p < n;
        key[r] = valid ? keys_in[p] : ~0ull;
        // the payload is loaded with the key, so its latency is not exposed after the look-back
        ixv[r] = kFirst ? uint32_t(p) : (valid ? idx_in[p] : 0u);
        uint32_t d = uint32_t(key[r] >> shift) & (kRadix - 1);
        uint64_t peers = ballot(valid);
#pragma unroll
        for (int b = 0; b < kRadixBits; ++b) {
            bool bit = (d >> b) & 1u;
            uint64_t m = ballot(bit);
            peers &= bit ? m : ~m;
        }
        int leader = peers ? __ffsll((unsigned long long)peers) - 1 : lane;
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
    uint32_t c[kWaves], tot = 0;
#pragma unroll
    for (int k = 0; k < kWaves; ++k) {
        c[k] = s_wcnt[k][d];
        s_wcnt[k][d] = tot;
        tot += c[k];
    }
    uint32_t *my = status + int64_t(tile) * kRadix + d;
    publish(my, (tile == 0 ? kFlagInclusive : kFlagAggregate) | tot);
    uint32_t lstart = block_exclusive_scan256(tot, s_scan, nullptr);
    s_lstart[d] = lstart;
    // global start of digit d: exclusive scan of the histogram
    uint32_t h = 0;
#pragma unroll
    for (int c = 0; c < kHistCopies; ++c) h += hist[c * kHistWords + pass * kRadix + d];
    __syncthreads();
    uint32_t dbase = block_exclusive_scan256(h, s_scan, nullptr);
    uint32_t excl = 0;
    if (tile > 0) {
        // look back kLook predecessors per round trip: add their aggregates
        // until an inclusive prefix; stop at a tile that has not published yet
        // and read again from there
        constexpr int kLook = 8;
        int64_t tt = int64_t(tile) - 1;
        uint32_t spins = 0;
        for (;;) {
            uint32_t sv[kLook];
#pragma unroll
            for (int k = 0; k < kLook; ++k) sv[k] = tt - k >= 0 ? peek(status + (tt - k) * kRadix + d) : 0u;
            int used = 0;
            bool found = false;
#pragma unroll
            for (int k = 0; k < kLook; ++k) {
                if (used != k || tt - k < 0 || (sv[k] & ~kValueMask) == 0) continue; // stopped earlier
                excl += sv[k] & kValueMask;
                used = k + 1;
                if (sv[k] & kFlagInclusive) {
                    found = true;
                    used = kLook + 1; // stop consuming
                }
            }
            if (found) break;
            tt -= used;
            if (tt < 0) break; // cannot happen: tile 0 publishes an inclusive prefix
            if (used < kLook) { // tile tt has not published yet
                if (++spins > kSpinLimit) { // a predecessor never published: give up loudly
                    atomicOr(&hdr->flags, kErrLookback);
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
        }
        publish(my, kFlagInclusive | (excl + tot));
    }
    s_gofs[d] = dbase + excl;
    __syncthreads();

    // rank -> position inside the tile, staged through LDS
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        int64_t p = base + w * kSeg + r * kWave + lane;
        if (p < n) {
            uint32_t dd = uint32_t(key[r] >> shift) & (kRadix - 1);
            uint32_t lp = s_lstart[dd] + s_wcnt[w][dd] + rank[r];
            s_keys[lp] = key[r];
            s_idx[lp] = ixv[r];
        }
    }
    __syncthreads();
    const int tile_n = int(n - base < kSortTile ? n - base : kSortTile);
    for (int j = t; j < tile_n; j += kSortBlock) {
        uint64_t k = s_keys[j];
        uint32_t dd = uint32_t(k >> shift) & (kRadix - 1);
        uint32_t out = s_gofs[dd] + (uint32_t(j) - s_lstart[dd]);
        if (out < uint32_t(n)) {
            keys_out[out] = k;
            uint32_t ix = s_idx[j];
            idx_out[out] = ix;
            if (kLast) ys[out] = ix < uint32_t(n) ? ysrc[ix] : V{};
        } else {
            atomicOr(&hdr->flags, kErrRange);
        }
    }
}

// ------------------------------------------------------------------ launchers
template <typename T> void launch_bbox(const T *Y, int64_t n, void *ws, const Layout &L, hipStream_t st)
{
    int blocks = int((n + 255) / 256);
    if (blocks > kBBoxBlocks) blocks = kBBoxBlocks;
    bbox_partial_kernel<T><<<blocks, 256, 0, st>>>(reinterpret_cast<const vec2_t<T> *>(Y), n,
                                                   at<T>(ws, L.bbox_part));
    bbox_final_kernel<T><<<1, 256, 0, st>>>(at<T>(ws, L.bbox_part), blocks, at<Header>(ws, L.header),
                                            at<uint32_t>(ws, L.hist));
}
template void launch_bbox<float>(const float *, int64_t, void *, const Layout &, hipStream_t);
template void launch_bbox<double>(const double *, int64_t, void *, const Layout &, hipStream_t);

void launch_bbox_morton3(const float *Y, int64_t n, const uint32_t *perm, void *ws, const Layout &L, hipStream_t st)
{
    int blocks = int((n + 255) / 256);
    if (blocks > kBBoxBlocks) blocks = kBBoxBlocks;
    const float3 *y3 = reinterpret_cast<const float3 *>(Y);
    bbox3_partial_kernel<<<blocks, 256, 0, st>>>(y3, n, at<float>(ws, L.bbox_part));
    bbox3_final_kernel<<<1, 256, 0, st>>>(at<float>(ws, L.bbox_part), blocks, at<Header>(ws, L.header),
                                          at<uint32_t>(ws, L.hist));
    morton3_kernel<<<unsigned(L.sort_tiles), kSortBlock, 0, st>>>(
        y3, n, at<Header>(ws, L.header), at<uint64_t>(ws, L.codes0), at<float3>(ws, L.ycopy), perm,
        at<uint32_t>(ws, L.hist), at<uint32_t>(ws, L.levelmask), at<uint32_t>(ws, L.status), L.sort_tiles);
}

template <typename T>
void launch_morton(const T *Y, int64_t n, const uint32_t *perm, void *ws, const Layout &L, hipStream_t st)
{
    morton_kernel<T><<<unsigned(L.sort_tiles), kSortBlock, 0, st>>>(
        reinterpret_cast<const vec2_t<T> *>(Y), n, at<Header>(ws, L.header), at<uint64_t>(ws, L.codes0),
        at<vec2_t<T>>(ws, L.ycopy), perm, at<uint32_t>(ws, L.hist), at<uint32_t>(ws, L.levelmask),
        at<uint32_t>(ws, L.status), L.sort_tiles);
}
template void launch_morton<float>(const float *, int64_t, const uint32_t *, void *, const Layout &, hipStream_t);
template void launch_morton<double>(const double *, int64_t, const uint32_t *, void *, const Layout &,
                                    hipStream_t);

// the last pass also gathers the points in sorted order (from `ysrc`, in the
// order the codes were made)
template <typename V> void launch_sort_points(int64_t n, const V *ysrc, void *ws, const Layout &L, hipStream_t st)
{
    uint64_t *k[2] = {at<uint64_t>(ws, L.codes0), at<uint64_t>(ws, L.codes1)};
    uint32_t *x[2] = {at<uint32_t>(ws, L.idx0), at<uint32_t>(ws, L.idx1)};
    Header *hdr = at<Header>(ws, L.header);
    const uint32_t *hist = at<uint32_t>(ws, L.hist);
    V *ys = at<V>(ws, L.ys);
    for (int p = 0; p < kSortPasses; ++p) {
        uint32_t *status = at<uint32_t>(ws, L.status) + int64_t(p) * L.sort_tiles * kRadix;
        int src = p & 1, dst = src ^ 1;
        dim3 g(unsigned(L.sort_tiles));
        if (p == 0)
            onesweep_kernel<true, false, V><<<g, kSortBlock, 0, st>>>(k[src], nullptr, k[dst], x[dst], status, hist,
                                                                     hdr, p, n, nullptr, nullptr);
        else if (p == kSortPasses - 1)
            onesweep_kernel<false, true, V><<<g, kSortBlock, 0, st>>>(k[src], x[src], k[dst], x[dst], status,
                                                                     hist, hdr, p, n, ysrc, ys);
        else
            onesweep_kernel<false, false, V><<<g, kSortBlock, 0, st>>>(k[src], x[src], k[dst], x[dst], status,
                                                                      hist, hdr, p, n, nullptr, nullptr);
    }
}
template void launch_sort_points<float3>(int64_t, const float3 *, void *, const Layout &, hipStream_t);

template <typename T> void launch_sort(int64_t n, const T *ysrc, void *ws, const Layout &L, hipStream_t st)
{
    launch_sort_points(n, reinterpret_cast<const vec2_t<T> *>(ysrc), ws, L, st);
}
template void launch_sort<float>(int64_t, const float *, void *, const Layout &, hipStream_t);
template void launch_sort<double>(int64_t, const double *, void *, const Layout &, hipStream_t);

} // namespace bht
