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
// is wave-uniform (scalar loads of the 24-byte node record); a lane that
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
constexpr int kCmpUge = 35, kCmpNe = 33, kCmpOgt = 2;
__device__ inline uint64_t mask_uge(uint32_t a, uint32_t b) { return __builtin_amdgcn_uicmp(a, b, kCmpUge); }
__device__ inline uint64_t mask_ne(uint32_t a, uint32_t b) { return __builtin_amdgcn_uicmp(a, b, kCmpNe); }
__device__ inline uint64_t mask_ogt(float a, float b) { return __builtin_amdgcn_fcmpf(a, b, kCmpOgt); }

// The interaction with one node in the lanes of `take` only: EXEC is narrowed
// to the mask for the block and restored after it, so lanes outside keep their
// sums and resume offsets and no per-lane select is needed.  The instruction
// between the reciprocal and its first use gives the one wait state that a
// transcendental result needs before another VALU reads it on gfx950.
__device__ inline void take_node(uint64_t take, float d2, float dx, float dy, float cnt, uint32_t next, float &z,
                                 float &fx, float &fy, uint32_t &resume)
{
    float w, t;
    uint64_t saved;
    asm volatile("s_and_saveexec_b64 %[sv], %[take]\n\t"
                 "v_add_f32 %[w], 1.0, %[d2]\n\t"
                 "v_rcp_f32 %[w], %[w]\n\t"
                 "v_mov_b32 %[res], %[next]\n\t"
                 "v_mul_f32 %[t], %[cnt], %[w]\n\t"
                 "v_fmac_f32 %[z], %[cnt], %[w]\n\t"
                 "v_mul_f32 %[t], %[t], %[w]\n\t"
                 "v_fmac_f32 %[fx], %[t], %[dx]\n\t"
                 "v_fmac_f32 %[fy], %[t], %[dy]\n\t"
                 "s_mov_b64 exec, %[sv]"
                 : [z] "+v"(z), [fx] "+v"(fx), [fy] "+v"(fy), [res] "+v"(resume), [w] "=&v"(w), [t] "=&v"(t),
                   [sv] "=&s"(saved)
                 : [take] "s"(take), [d2] "v"(d2), [cnt] "s"(cnt), [dx] "v"(dx), [dy] "v"(dy), [next] "s"(next)
                 : "scc");
}

// One lane per point.  Every visit runs the same code on a 24-byte record read
// with one scalar load: a single point is a node whose threshold (-1) every
// lane passes, and a bucket of identical points is a cell whose children are
// its points.  The acceptance test gives the lanes that take the node; the
// interaction terms are accumulated in those lanes only, which also park until
// the walk reaches the node's next offset.  The next node is the first child
// when some active lane descends, else the node's next offset.
//
// The lane's own point: with theta^2 <= 0.49 no point accepts a cell that
// contains it (the centre of mass lies in the cell's square, so the squared
// distance is at most 2 side^2, below side^2 / theta^2), so every lane reaches
// its own leaf and takes it once with d2 = 0: a weight of exactly 1 in z and
// nothing in the force, removed after the walk.  Larger theta compares the
// leaf's position with the lane's.
template <bool kSelf>
__device__ inline void repulsive_walk(const char *nbase, uint32_t end, float2 yi, uint32_t si, uint32_t &resume,
                                      float &fx, float &fy, float &z, uint32_t &inter)
{
    uint32_t cur = 0; // byte offset of the current record
    while (cur < end) {
        // the record and 8 bytes beyond it: one 32-byte scalar load
        typedef uint32_t u32x8 __attribute__((ext_vector_type(8)));
        const u32x8 r = *reinterpret_cast<const u32x8 *>(nbase + cur);
        const float cx = __uint_as_float(r[0]), cy = __uint_as_float(r[1]);
        const float cnt = __uint_as_float(r[2]), thr = __uint_as_float(r[3]);
        const uint32_t next = r[4];
        const float dx = yi.x - cx, dy = yi.y - cy;
        const float d2 = fmaf(dx, dx, dy * dy);
        const uint64_t act = mask_uge(cur, resume);
        uint64_t take = act & mask_ogt(d2, thr);
        if (kSelf) take &= mask_ne(r[5], si);
        const uint64_t rej = act & ~take;
        inter += uint32_t(__builtin_popcountll(take));
        take_node(take, d2, dx, dy, cnt, next, z, fx, fy, resume);
        // the first child follows its cell; no lane descends: jump past the subtree
        cur = rej ? cur + kNodeBytes : next;
    }
}

// The 3-D interaction with one node in the lanes of `take` (see take_node).
__device__ inline void take_node3(uint64_t take, float d2, float dx, float dy, float dz, float cnt, uint32_t next,
                                  float &z, float &fx, float &fy, float &fz, uint32_t &resume)
{
    float w, t;
    uint64_t saved;
    asm volatile("s_and_saveexec_b64 %[sv], %[take]\n\t"
                 "v_add_f32 %[w], 1.0, %[d2]\n\t"
                 "v_rcp_f32 %[w], %[w]\n\t"
                 "v_mov_b32 %[res], %[next]\n\t"
                 "v_mul_f32 %[t], %[cnt], %[w]\n\t"
                 "v_fmac_f32 %[z], %[cnt], %[w]\n\t"
                 "v_mul_f32 %[t], %[t], %[w]\n\t"
                 "v_fmac_f32 %[fx], %[t], %[dx]\n\t"
                 "v_fmac_f32 %[fy], %[t], %[dy]\n\t"
                 "v_fmac_f32 %[fz], %[t], %[dz]\n\t"
                 "s_mov_b64 exec, %[sv]"
                 : [z] "+v"(z), [fx] "+v"(fx), [fy] "+v"(fy), [fz] "+v"(fz), [res] "+v"(resume), [w] "=&v"(w),
                   [t] "=&v"(t), [sv] "=&s"(saved)
                 : [take] "s"(take), [d2] "v"(d2), [cnt] "s"(cnt), [dx] "v"(dx), [dy] "v"(dy), [dz] "v"(dz),
                   [next] "s"(next)
                 : "scc");
}

// The walk over a 3-D embedding's octree: the same visit order and lane
// masks on 32-byte records {com.x, com.y, com.z, count, thr, next, self, 0},
// each exactly one 32-byte scalar load.  With theta^2 <= 0.33 no point
// accepts a cell containing it (the centre of mass lies in the cell's cube,
// so the squared distance is at most 3 side^2, below side^2 / theta^2), and
// the lane's own leaf is taken once with weight 1 as in 2-D.
template <bool kSelf>
__device__ inline void repulsive_walk3(const char *nbase, uint32_t end, float3 yi, uint32_t si, uint32_t &resume,
                                       float &fx, float &fy, float &fz, float &z, uint32_t &inter)
{
    uint32_t cur = 0;
    while (cur < end) {
        typedef uint32_t u32x8 __attribute__((ext_vector_type(8)));
        const u32x8 r = *reinterpret_cast<const u32x8 *>(nbase + cur);
        const float dx = yi.x - __uint_as_float(r[0]), dy = yi.y - __uint_as_float(r[1]);
        const float dz = yi.z - __uint_as_float(r[2]);
        const float cnt = __uint_as_float(r[3]), thr = __uint_as_float(r[4]);
        const uint32_t next = r[5];
        const float d2 = fmaf(dx, dx, fmaf(dy, dy, dz * dz));
        const uint64_t act = mask_uge(cur, resume);
        uint64_t take = act & mask_ogt(d2, thr);
        if (kSelf) take &= mask_ne(r[6], si);
        const uint64_t rej = act & ~take;
        inter += uint32_t(__builtin_popcountll(take));
        take_node3(take, d2, dx, dy, dz, cnt, next, z, fx, fy, fz, resume);
        cur = rej ? cur + kNodeBytes3 : next;
    }
}

// 1/x in fp64 for x >= 1: the hardware's approximate reciprocal (measured on
// gfx950 within 2^-24.4 relative over x in [1, 1e8]) refined by one
// Newton-Raphson step r <- r + r (1 - x r), which squares the relative error:
// within 2^-48.7 (11 ulps) of the quotient, so a weight and its square carry
// below 5e-15 relative error, and Z, a sum of positive weights, no more (the
// IEEE division sequence costs three times the instructions); 1/inf stays 0.
__device__ inline double recip(double x)
{
    const double r = __builtin_amdgcn_rcp(x);
    return x != __builtin_huge_val() ? fma(r, fma(-x, r, 1.0), r) : 0.0;
}
__device__ inline float recip(float x) { return fast_rcp(x); }

// The fp64 variant of the walk: the same visit order and acceptance test on
// 40-byte records with fp64 centres and thresholds; the lanes that take a
// node accumulate under the compiler's own EXEC mask.
template <bool kSelf>
__device__ inline void repulsive_walk64(const char *nbase, uint32_t end, double2 yi, uint32_t si, uint32_t &resume,
                                        double &fx, double &fy, double &z, uint32_t &inter)
{
    uint32_t cur = 0; // byte offset of the current record
    while (cur < end) {
        const double *d = reinterpret_cast<const double *>(nbase + cur);
        const double cx = d[0], cy = d[1], thr = d[2];
        const uint32_t *u = reinterpret_cast<const uint32_t *>(d + 3);
        const double cnt = double(__uint_as_float(u[0]));
        const uint32_t next = u[1], self = u[2];
        const double dx = yi.x - cx, dy = yi.y - cy;
        const double d2 = fma(dx, dx, dy * dy);
        const bool act = cur >= resume;
        bool tk = act & (d2 > thr);
        if (kSelf) tk &= self != si;
        const uint64_t take = ballot(tk);
        const uint64_t rej = ballot(act & !tk);
        inter += uint32_t(__builtin_popcountll(take));
        if (tk) {
            const double wgt = recip(1.0 + d2);
            const double nw = cnt * wgt;
            z += nw;
            const double nw2 = nw * wgt;
            fx = fma(nw2, dx, fx);
            fy = fma(nw2, dy, fy);
            resume = next;
        }
        cur = rej ? cur + kNodeBytes64 : next;
    }
}

// D = 2, T = float: the path (24-byte records); T = double: the fp64
// variant; D = 3: 3-D embeddings (32-byte records).
template <int D, typename T>
__global__ __launch_bounds__(kRepBlock) void repulsive_kernel(
    const char *__restrict__ nodes, const point_t<D, T> *__restrict__ ys, const uint32_t *__restrict__ perm,
    Header *__restrict__ hdr, int64_t n, int self_test, point_t<D, T> *__restrict__ frep, double *__restrict__ zpart,
    unsigned long long *__restrict__ ipart)
{
    using V = point_t<D, T>;
    const uint32_t nb = gridDim.x;
    const uint32_t lb = xcd_contiguous(blockIdx.x, nb);
    const int w = threadIdx.x / kWave;
    const int64_t s64 = int64_t(lb) * kRepBlock + threadIdx.x;
    const bool valid = s64 < n;
    const uint32_t si = uint32_t(s64);
    const V yi = valid ? ys[s64] : V{};
    uint32_t resume = valid ? 0u : 0xffffffffu;
    T fx = 0, fy = 0, fz = 0, z = 0;
    uint32_t total = uniform(hdr->nodes);
    const uint32_t cap = uint32_t(2 * n - 1);
    total = total < cap ? total : cap;
    // Every record's next offset lies past the record (the tree kernel checks
    // it and flags the call otherwise), so each visit advances and the walk
    // ends after at most `total` visits.  A flagged tree is not walked.
    if (uniform(hdr->flags) & (kErrLookback | kErrRange)) total = 0;
    const uint32_t end = total * uint32_t(node_bytes<D, T>());

    uint32_t inter = 0; // this wave's interactions (a launch has fewer than 2^32 per wave)
    if constexpr (D == 3) {
        if (self_test)
            repulsive_walk3<true>(nodes, end, yi, si, resume, fx, fy, fz, z, inter);
        else
            repulsive_walk3<false>(nodes, end, yi, si, resume, fx, fy, fz, z, inter);
    } else if constexpr (sizeof(T) == 8) {
        if (self_test)
            repulsive_walk64<true>(nodes, end, yi, si, resume, fx, fy, z, inter);
        else
            repulsive_walk64<false>(nodes, end, yi, si, resume, fx, fy, z, inter);
    } else {
        if (self_test)
            repulsive_walk<true>(nodes, end, yi, si, resume, fx, fy, z, inter);
        else
            repulsive_walk<false>(nodes, end, yi, si, resume, fx, fy, z, inter);
    }
    if (!self_test) {
        // each valid lane took its own leaf once, with weight 1
        if (valid) z -= T(1);
        inter -= uint32_t(__builtin_popcountll(ballot(valid)));
    }

    if (valid) {
        const uint32_t p = perm[si];
        const T f[3] = {fx, fy, fz};
        if (p < uint32_t(n)) frep[p] = make_point(f, static_cast<V *>(nullptr));
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


constexpr int kAttB = 4;

// D = 2, T = float: the path's plain-CSR attraction; T = double: the fp64
// variant; D = 3: 3-D embeddings.  Coordinates are handled component by
// component (unrolled).
template <int G, bool kUpdate, int D, typename T>
__global__ __launch_bounds__(256) void attract_kernel(
    const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col, const T *__restrict__ val,
    const point_t<D, T> *__restrict__ ycopy, const point_t<D, T> *__restrict__ frep, Header *__restrict__ hdr,
    int64_t n, int64_t nnz, StepArgsT<T> a, point_t<D, T> *__restrict__ Y, point_t<D, T> *__restrict__ upd,
    point_t<D, T> *__restrict__ gains, point_t<D, T> *__restrict__ grad)
{
    using V = point_t<D, T>;
    const int sub = lane_id() % G;
    constexpr int kRows = 256 / G;
    const T inv_z = T(1.0 / hdr->Z);
    for (int64_t row0 = int64_t(blockIdx.x) * kRows; row0 < n; row0 += int64_t(gridDim.x) * kRows) {
        const int64_t i = row0 + threadIdx.x / G;
        const bool valid = i < n;
        T f[D];
#pragma unroll
        for (int d = 0; d < D; ++d) f[d] = T(0);
        V yi{};
        if (valid) {
            yi = ycopy[i];
            int64_t s = row_ptr[i], e = row_ptr[i + 1];
            if (s < 0 || e > nnz) { // malformed row: skip what lies outside the arrays
                if (sub == 0) atomicOr(&hdr->flags, kErrRange);
                s = s < 0 ? 0 : s;
                e = e > nnz ? nnz : e;
            }
            // kAttB entries per lane at a time: their loads, then their gathers,
            // are in flight together
            for (int64_t k0 = s + sub; k0 < e; k0 += kAttB * G) {
                int32_t j[kAttB];
                T p[kAttB];
#pragma unroll
                for (int u = 0; u < kAttB; ++u) {
                    const int64_t k = k0 + u * G;
                    // P is streamed once per call: keep it out of the caches that hold Y
                    j[u] = k < e ? __builtin_nontemporal_load(col + k) : 0;
                    p[u] = k < e ? __builtin_nontemporal_load(val + k) : T(0);
                    if (uint32_t(j[u]) >= uint32_t(n)) {
                        atomicOr(&hdr->flags, kErrRange);
                        j[u] = 0;
                        p[u] = T(0);
                    }
                }
                V yj[kAttB];
#pragma unroll
                for (int u = 0; u < kAttB; ++u) yj[u] = ycopy[j[u]];
#pragma unroll
                for (int u = 0; u < kAttB; ++u) {
                    T dv[D];
#pragma unroll
                    for (int d = 0; d < D; ++d) dv[d] = coord(yi, d) - coord(yj[u], d);
                    T d2 = dv[D - 1] * dv[D - 1];
#pragma unroll
                    for (int d = D - 2; d >= 0; --d) d2 = fma(dv[d], dv[d], d2);
                    const T pw = p[u] * recip(T(1) + d2);
#pragma unroll
                    for (int d = 0; d < D; ++d) f[d] = fma(pw, dv[d], f[d]);
                }
            }
        }
#pragma unroll
        for (int o = G / 2; o > 0; o >>= 1) {
#pragma unroll
            for (int d = 0; d < D; ++d) f[d] += __shfl_xor(f[d], o, kWave);
        }
        if (valid && sub == 0) {
            const V fr = frep[i];
            T g[D];
#pragma unroll
            for (int d = 0; d < D; ++d) g[d] = T(4) * (a.alpha * f[d] - coord(fr, d) * inv_z);
            if (grad) grad[i] = make_point(g, static_cast<V *>(nullptr));
            if (kUpdate) {
                const V u0 = upd[i], g0 = gains[i];
                T u[D], gn[D], y[D];
#pragma unroll
                for (int d = 0; d < D; ++d) {
                    const T ud = coord(u0, d);
                    T gd = (ud * g[d] < T(0)) ? coord(g0, d) + T(0.2) : coord(g0, d) * T(0.8);
                    gd = vmax(gd, a.min_gain);
                    u[d] = a.momentum * ud - a.learning_rate * gd * g[d];
                    gn[d] = gd;
                    y[d] = coord(yi, d) + u[d];
                }
                Y[i] = make_point(y, static_cast<V *>(nullptr));
                upd[i] = make_point(u, static_cast<V *>(nullptr));
                gains[i] = make_point(gn, static_cast<V *>(nullptr));
            }
        }
    }
}

// ------------------------------------------------------------------ launchers
template <int D, typename T>
void launch_repulsive(int64_t n, bool self_test, void *ws, const Layout &L, hipStream_t st)
{
    using V = point_t<D, T>;
    repulsive_kernel<D, T><<<unsigned(L.rep_blocks), kRepBlock, 0, st>>>(
        at<char>(ws, L.nodes), at<V>(ws, L.ys), at<uint32_t>(ws, L.idx0), at<Header>(ws, L.header), n,
        self_test ? 1 : 0, at<V>(ws, L.frep), at<double>(ws, L.zpart), at<unsigned long long>(ws, L.ipart));
}
template void launch_repulsive<2, float>(int64_t, bool, void *, const Layout &, hipStream_t);
template void launch_repulsive<2, double>(int64_t, bool, void *, const Layout &, hipStream_t);
template void launch_repulsive<3, float>(int64_t, bool, void *, const Layout &, hipStream_t);

template <int D, typename T>
void launch_attract(const int64_t *row_ptr, const int32_t *col, const T *val, int64_t n, int64_t nnz,
                    const StepArgsT<T> &a, T *Y, T *upd, T *gains, T *grad, void *ws, const Layout &L, hipStream_t st)
{
    constexpr int G = 64; // one wave per row: rows hold ~100-200 entries
    int64_t blocks = (n + (256 / G) - 1) / (256 / G);
    if (blocks > 65535 * 8) blocks = 65535 * 8;
    using V = point_t<D, T>;
    const V *yc = at<V>(ws, L.ycopy);
    const V *fr = at<V>(ws, L.frep);
    Header *hdr = at<Header>(ws, L.header);
    if (a.update)
        attract_kernel<G, true, D, T><<<unsigned(blocks), 256, 0, st>>>(
            row_ptr, col, val, yc, fr, hdr, n, nnz, a, reinterpret_cast<V *>(Y), reinterpret_cast<V *>(upd),
            reinterpret_cast<V *>(gains), reinterpret_cast<V *>(grad));
    else
        attract_kernel<G, false, D, T><<<unsigned(blocks), 256, 0, st>>>(row_ptr, col, val, yc, fr, hdr, n, nnz, a,
                                                                       nullptr, nullptr, nullptr,
                                                                       reinterpret_cast<V *>(grad));
}
template void launch_attract<2, float>(const int64_t *, const int32_t *, const float *, int64_t, int64_t,
                                       const StepArgsT<float> &, float *, float *, float *, float *, void *,
                                       const Layout &, hipStream_t);
template void launch_attract<2, double>(const int64_t *, const int32_t *, const double *, int64_t, int64_t,
                                        const StepArgsT<double> &, double *, double *, double *, double *, void *,
                                        const Layout &, hipStream_t);
template void launch_attract<3, float>(const int64_t *, const int32_t *, const float *, int64_t, int64_t,
                                       const StepArgsT<float> &, float *, float *, float *, float *, void *,
                                       const Layout &, hipStream_t);

} // namespace bht
