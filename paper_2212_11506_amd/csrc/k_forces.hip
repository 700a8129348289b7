// Repulsive (Barnes-Hut) and attractive forces, gradient and update (gfx950).
//
// Repulsive Force Computation: every point walks the tree depth first; a
// cell whose side is small against its distance (side^2 < theta^2 d^2) is
// replaced by its summary, otherwise its children are visited; leaves are
// taken point by point, excluding the point itself.  The normaliser Z (the
// q_ij definition) is the sum of all the kernel values used.
//
// GPU design: points are processed in Morton order, one lane per point, and a
// wavefront walks the pre-order node array together.  The current node index
// is wave-uniform (scalar loads of the 20-byte node record); a lane that
// summarises a cell parks itself until the walk reaches the cell's skip
// index, so its own interaction list is exactly the depth-first one, while the
// wave only descends where some lane needs it.  No stack is needed.
//
// Attractive Force Computation (Algorithm 2): a group of lanes per CSR row,
// coalesced column/value reads, fused with the gradient assembly
// g = 4 (alpha F_attr - F_rep / Z) and the gains/momentum update.
#include "common.hpp"
#include "kernels.hpp"

namespace bht {

__device__ inline float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// Lane masks straight from the vector compares (one instruction each, no
// conversion through a boolean per lane): predicates as in LLVM's icmp/fcmp.
constexpr int kCmpUge = 35, kCmpNe = 33, kCmpSgt = 38;
__device__ inline uint64_t mask_uge(uint32_t a, uint32_t b) { return __builtin_amdgcn_uicmp(a, b, kCmpUge); }
__device__ inline uint64_t mask_ne(uint32_t a, uint32_t b) { return __builtin_amdgcn_uicmp(a, b, kCmpNe); }
// the predicate, not the operand type, decides signedness
__device__ inline uint64_t mask_sgt(int32_t a, int32_t b)
{
    return __builtin_amdgcn_uicmp(uint32_t(a), uint32_t(b), kCmpSgt);
}
// x in the lanes whose bit of m is set, else 0 (one v_cndmask on the mask)
__device__ inline float keep_lanes(uint64_t m, float x)
{
    float r;
    asm("v_cndmask_b32_e64 %0, 0, %1, %2" : "=v"(r) : "v"(x), "s"(m));
    return r;
}
// x in the lanes whose bit of m is set, else y
__device__ inline uint32_t pick_lanes_u(uint64_t m, uint32_t x, uint32_t y)
{
    uint32_t r;
    asm("v_cndmask_b32_e64 %0, %1, %2, %3" : "=v"(r) : "v"(y), "v"(x), "s"(m));
    return r;
}

// One lane per point.  Every visit runs the same straight-line code: a single
// point is a cell that is always accepted (its threshold is -1) unless it is
// the lane's own point (its meta word then equals the lane's self code), and
// a bucket of identical points is a cell whose children are its points.  The
// acceptance test yields a lane mask, the weight is zeroed outside it, the
// interaction count is its population, and the next node is a scalar select
// (the skip index when no lane descends into the cell).  One 16-byte record per
// node (the meta word in its fourth component) is one scalar load per visit.
//
// The threshold of a cell of level L is side(L)^2 / theta^2 = thr(0) * 4^-L,
// so unless it leaves the normal range its float bits are those of thr(0)
// minus L << 24; the walk forms them from the meta word's level field in
// scalar code.  A single point's field is all ones, which takes the bits below
// zero as an integer, and for squared distances (never negative) the integer
// order of the bits is the float order, so one signed compare accepts every
// single point and tests every cell.  When the shortcut does not reproduce the
// thresholds (theta = 0, or a domain so small or large that thr leaves the
// normal range) the walk reads each threshold from the table instead.
template <bool kShift>
__device__ inline void repulsive_walk(const char *nbase, const uint32_t *__restrict__ thr_table, uint32_t thr0,
                                      uint32_t total, float2 yi, uint32_t self, uint32_t &resume, float &fx,
                                      float &fy, float &z, uint32_t &inter)
{
    uint32_t cur = 0;
    while (cur < total) {
        const float4 r = *reinterpret_cast<const float4 *>(nbase + (cur << 4));
        const uint32_t m = __float_as_uint(r.w);
        const uint32_t lv = m >> kMetaLevelShift;
        const uint32_t thr = kShift ? thr0 - (lv << 24) : thr_table[lv];
        const float dx = yi.x - r.x, dy = yi.y - r.y;
        const float d2 = fmaf(dx, dx, dy * dy);
        const uint64_t act = mask_uge(cur, resume);
        const uint64_t take = act & mask_sgt(__float_as_int(d2), int32_t(thr)) & mask_ne(m, self);
        const float wgt = fast_rcp(1.0f + d2);
        const float nw = keep_lanes(take, r.z * wgt);
        z += nw;
        const float nw2 = nw * wgt;
        fx = fmaf(nw2, dx, fx);
        fy = fmaf(nw2, dy, fy);
        inter += uint32_t(__builtin_popcountll(take));
        const uint64_t rej = act & ~take;
        // the skip index of a cell, 0 for a single point (negative meta word)
        const uint32_t skip = uint32_t(max(int32_t(m), 0)) & kMetaSkipMask;
        // accepting lanes park until the walk leaves a cell.  A lane that
        // takes a node is active, so its old resume index is at most cur and
        // the new one (skip, or 0 after a single point) keeps every later node
        // that the old one allowed: no max is needed
        resume = pick_lanes_u(take, skip, resume);
        // a skip index lies beyond its cell: skip when no lane descends
        cur = rej ? cur + 1 : max(cur + 1, skip);
    }
}

__global__ __launch_bounds__(kRepBlock) void repulsive_kernel(
    const float4 *__restrict__ nodes, const uint32_t *__restrict__ thr_table, const float2 *__restrict__ ys,
    const uint32_t *__restrict__ perm, Header *__restrict__ hdr, int64_t n, float2 *__restrict__ frep,
    double *__restrict__ zpart, unsigned long long *__restrict__ ipart)
{
    const uint32_t nb = gridDim.x;
    const uint32_t lb = xcd_contiguous(blockIdx.x, nb);
    const int w = threadIdx.x / kWave;
    const int64_t s64 = int64_t(lb) * kRepBlock + threadIdx.x;
    const bool valid = s64 < n;
    const uint32_t si = uint32_t(s64);
    const uint32_t self = kMetaSingle | si; // meta word of this lane's own single-point node
    const float2 yi = valid ? ys[s64] : make_float2(0.0f, 0.0f);
    uint32_t resume = valid ? 0u : 0xffffffffu;
    float fx = 0.0f, fy = 0.0f, z = 0.0f;
    uint32_t total = uniform(hdr->nodes);
    const uint32_t cap = uint32_t(2 * n);
    total = total < cap ? total : cap;
    // does thr(0) - (L << 24) reproduce the thresholds of levels 0..32, and
    // stay above the bits of every single point's field?
    const uint32_t thr0 = uniform(thr_table[0]);
    const int lane = lane_id();
    const uint32_t tl = thr_table[lane < 33 ? lane : 0];
    const bool shift_ok = lane >= 33 || tl == thr0 - (uint32_t(lane) << 24);
    const bool shift = ballot(shift_ok) == ~0ull && thr0 < 0x7F000000u;
    // node records by 32-bit byte offset (fewer than 2^27 nodes)
    const char *nbase = reinterpret_cast<const char *>(nodes);

    uint32_t inter = 0; // this wave's interactions (a launch has fewer than 2^32 per wave)
    if (shift)
        repulsive_walk<true>(nbase, thr_table, thr0, total, yi, self, resume, fx, fy, z, inter);
    else
        repulsive_walk<false>(nbase, thr_table, thr0, total, yi, self, resume, fx, fy, z, inter);

    if (valid) {
        const uint32_t p = perm[si];
        if (p < uint32_t(n)) frep[p] = make_float2(fx, fy);
    }
    // deterministic Z: wave -> block partial -> fixed-order sum in the last block
    double zw = wave_sum(double(z));
    __shared__ double s_z[kRepBlock / kWave];
    __shared__ unsigned long long s_i[kRepBlock / kWave];
    __shared__ bool s_last;
    if (lane_id() == 0) {
        s_z[w] = zw;
        s_i[w] = inter;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double zb = 0.0;
        unsigned long long ib = 0;
        for (int k = 0; k < kRepBlock / kWave; ++k) {
            zb += s_z[k];
            ib += s_i[k];
        }
        zpart[lb] = zb;
        ipart[lb] = ib;
        __threadfence();
        s_last = atomicAdd(&hdr->ticket_rep, 1u) == nb - 1;
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    // last block: each thread sums a fixed contiguous chunk, then a fixed tree
    const uint32_t per = (nb + kRepBlock - 1) / kRepBlock;
    double zs = 0.0;
    unsigned long long is = 0;
    for (uint32_t k = threadIdx.x * per; k < (threadIdx.x + 1) * per && k < nb; ++k) {
        zs += zpart[k];
        is += ipart[k];
    }
    zs = wave_sum(zs);
    is = wave_sum(is);
    __syncthreads();
    if (lane_id() == 0) {
        s_z[w] = zs;
        s_i[w] = is;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double Z = 0.0;
        unsigned long long I = 0;
        for (int k = 0; k < kRepBlock / kWave; ++k) {
            Z += s_z[k];
            I += s_i[k];
        }
        hdr->Z = Z;
        hdr->interactions = I;
    }
}

template <int G, bool kUpdate>
__global__ __launch_bounds__(256) void attract_kernel(
    const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col, const float *__restrict__ val,
    const float2 *__restrict__ ycopy, const float2 *__restrict__ frep, Header *__restrict__ hdr,
    int64_t n, int64_t nnz, StepArgs a, float2 *__restrict__ Y, float2 *__restrict__ upd, float2 *__restrict__ gains,
    float2 *__restrict__ grad)
{
    const int sub = lane_id() % G;
    constexpr int kRows = 256 / G;
    const float inv_z = float(1.0 / hdr->Z);
    for (int64_t row0 = int64_t(blockIdx.x) * kRows; row0 < n; row0 += int64_t(gridDim.x) * kRows) {
        const int64_t i = row0 + threadIdx.x / G;
        const bool valid = i < n;
        float fx = 0.0f, fy = 0.0f;
        float2 yi = make_float2(0.0f, 0.0f);
        if (valid) {
            yi = ycopy[i];
            int64_t s = row_ptr[i], e = row_ptr[i + 1];
            if (s < 0 || e > nnz) { // malformed row: skip what lies outside the arrays
                if (sub == 0) atomicOr(&hdr->flags, kErrRange);
                s = s < 0 ? 0 : s;
                e = e > nnz ? nnz : e;
            }
            for (int64_t k = s + sub; k < e; k += G) {
                // P is streamed once per call: keep it out of the caches that hold Y
                const int32_t j = __builtin_nontemporal_load(col + k);
                if (uint32_t(j) >= uint32_t(n)) {
                    atomicOr(&hdr->flags, kErrRange);
                    continue;
                }
                const float p = __builtin_nontemporal_load(val + k);
                const float2 yj = ycopy[j];
                const float dx = yi.x - yj.x, dy = yi.y - yj.y;
                const float pw = p * fast_rcp(1.0f + fmaf(dx, dx, dy * dy));
                fx = fmaf(pw, dx, fx);
                fy = fmaf(pw, dy, fy);
            }
        }
#pragma unroll
        for (int o = G / 2; o > 0; o >>= 1) {
            fx += __shfl_xor(fx, o, kWave);
            fy += __shfl_xor(fy, o, kWave);
        }
        if (valid && sub == 0) {
            const float2 fr = frep[i];
            const float gx = 4.0f * (a.alpha * fx - fr.x * inv_z);
            const float gy = 4.0f * (a.alpha * fy - fr.y * inv_z);
            if (grad) grad[i] = make_float2(gx, gy);
            if (kUpdate) {
                float2 u = upd[i], gn = gains[i];
                gn.x = (u.x * gx < 0.0f) ? gn.x + 0.2f : gn.x * 0.8f;
                gn.y = (u.y * gy < 0.0f) ? gn.y + 0.2f : gn.y * 0.8f;
                gn.x = fmaxf(gn.x, a.min_gain);
                gn.y = fmaxf(gn.y, a.min_gain);
                u.x = a.momentum * u.x - a.learning_rate * gn.x * gx;
                u.y = a.momentum * u.y - a.learning_rate * gn.y * gy;
                Y[i] = make_float2(yi.x + u.x, yi.y + u.y);
                upd[i] = u;
                gains[i] = gn;
            }
        }
    }
}

// ------------------------------------------------------------------ launchers
void launch_repulsive(int64_t n, void *ws, const Layout &L, hipStream_t st)
{
    repulsive_kernel<<<unsigned(L.rep_blocks), kRepBlock, 0, st>>>(
        at<float4>(ws, L.nodes), at<uint32_t>(ws, L.thr_table), at<float2>(ws, L.ys), at<uint32_t>(ws, L.idx0),
        at<Header>(ws, L.header), n, at<float2>(ws, L.frep), at<double>(ws, L.zpart),
        at<unsigned long long>(ws, L.ipart));
}

void launch_attract(const int64_t *row_ptr, const int32_t *col, const float *val, int64_t n, int64_t nnz,
                    const StepArgs &a, float *Y, float *upd, float *gains, float *grad, void *ws, const Layout &L,
                    hipStream_t st)
{
    constexpr int G = 64; // one wave per row: rows hold ~100-200 entries
    int64_t blocks = (n + (256 / G) - 1) / (256 / G);
    if (blocks > 65535 * 8) blocks = 65535 * 8;
    const float2 *yc = at<float2>(ws, L.ycopy);
    const float2 *fr = at<float2>(ws, L.frep);
    Header *hdr = at<Header>(ws, L.header);
    if (a.update)
        attract_kernel<G, true><<<unsigned(blocks), 256, 0, st>>>(
            row_ptr, col, val, yc, fr, hdr, n, nnz, a, reinterpret_cast<float2 *>(Y), reinterpret_cast<float2 *>(upd),
            reinterpret_cast<float2 *>(gains), reinterpret_cast<float2 *>(grad));
    else
        attract_kernel<G, false><<<unsigned(blocks), 256, 0, st>>>(row_ptr, col, val, yc, fr, hdr, n, nnz, a, nullptr,
                                                                 nullptr, nullptr,
                                                                 reinterpret_cast<float2 *>(grad));
}

} // namespace bht
