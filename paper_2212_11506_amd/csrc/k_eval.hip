// Evaluation of the t-SNE cost: the exact normaliser Z and the KL divergence
// (Background: the cost KL(P || Q) with q_ij = (1 + |y_i - y_j|^2)^-1 / Z, Z the
// sum over ordered pairs i != j).  Not part of an iteration: a run calls them to
// report its cost, so the exact Z (O(n^2) pairs) stays affordable at millions
// of points.
#include "common.hpp"
#include "kernels.hpp"

namespace bht {

constexpr int kZBlock = 256;
constexpr int kZPer = 8;                       // points of a lane
constexpr int kZPoints = kZBlock * kZPer;       // points of a block
static_assert(kZPoints == kZEvalPoints, "the workspace holds one partial per block");
constexpr int kZUnroll = 8;                     // j points per round of scalar loads
constexpr int kEvalBlock = 256;

// fixed-order sum of one double per block in the last block to finish;
// returns true in that block's thread 0 with the total in *out
__device__ inline bool last_block_sum(double mine, double *__restrict__ part, uint32_t nb,
                                      uint32_t *__restrict__ ticket, double *out)
{
    __shared__ double s_w[kEvalBlock / kWave];
    __shared__ bool s_last;
    const int w = threadIdx.x / kWave;
    double v = wave_sum(mine);
    if (lane_id() == 0) s_w[w] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        double b = 0.0;
        for (int k = 0; k < kEvalBlock / kWave; ++k) b += s_w[k];
        part[blockIdx.x] = b;
        __threadfence();
        s_last = atomicAdd(ticket, 1u) == nb - 1;
    }
    __syncthreads();
    if (!s_last) return false;
    __threadfence();
    // each thread a fixed contiguous chunk of the partials, then a fixed tree
    const uint32_t per = (nb + kEvalBlock - 1) / kEvalBlock;
    double t = 0.0;
    for (uint32_t k = threadIdx.x * per; k < (threadIdx.x + 1) * per && k < nb; ++k) t += part[k];
    t = wave_sum(t);
    __syncthreads();
    if (lane_id() == 0) s_w[w] = t;
    __syncthreads();
    if (threadIdx.x != 0) return false;
    double total = 0.0;
    for (int k = 0; k < kEvalBlock / kWave; ++k) total += s_w[k];
    *out = total;
    *ticket = 0; // ready for the next call
    return true;
}

// an evaluation call reports its own device conditions only, like a step
__global__ void eval_reset_kernel(Header *__restrict__ hdr)
{
    hdr->ticket_eval = 0;
    hdr->flags = 0;
}

// Z = sum over i != j of (1 + |y_i - y_j|^2)^-1.  A lane holds kZPer points i;
// the points j are the same for the whole wave, read with scalar loads, so a
// pair costs about seven vector instructions.  Each lane's pair with itself adds
// exactly 1 (d = 0), removed at the end.
__global__ __launch_bounds__(kZBlock) void z_exact_kernel(const float2 *__restrict__ Y, int64_t n,
                                                         double *__restrict__ part, Header *__restrict__ hdr)
{
    float2 yi[kZPer];
    double acc[kZPer];
#pragma unroll
    for (int q = 0; q < kZPer; ++q) {
        const int64_t i = int64_t(blockIdx.x) * kZPoints + q * kZBlock + threadIdx.x;
        yi[q] = i < n ? Y[i] : make_float2(0.0f, 0.0f);
        acc[q] = 0.0;
    }
    // eight pair terms at a time: a pairwise fp32 sum, then an fp64 add, so that
    // equal terms (coincident points) do not pile up fp32 rounding
    int64_t j = 0;
    for (; j + kZUnroll <= n; j += kZUnroll) {
        float2 yj[kZUnroll];
#pragma unroll
        for (int u = 0; u < kZUnroll; ++u) yj[u] = Y[j + u];
#pragma unroll
        for (int q = 0; q < kZPer; ++q) {
            float w[kZUnroll];
#pragma unroll
            for (int u = 0; u < kZUnroll; ++u) {
                const float dx = yi[q].x - yj[u].x, dy = yi[q].y - yj[u].y;
                w[u] = __builtin_amdgcn_rcpf(1.0f + fmaf(dx, dx, dy * dy));
            }
            static_assert(kZUnroll == 8, "pairwise sum of eight terms");
            acc[q] += double(((w[0] + w[1]) + (w[2] + w[3])) + ((w[4] + w[5]) + (w[6] + w[7])));
        }
    }
    for (; j < n; ++j) {
        const float2 yj = Y[j];
#pragma unroll
        for (int q = 0; q < kZPer; ++q) {
            const float dx = yi[q].x - yj.x, dy = yi[q].y - yj.y;
            acc[q] += double(__builtin_amdgcn_rcpf(1.0f + fmaf(dx, dx, dy * dy)));
        }
    }
    double mine = 0.0;
#pragma unroll
    for (int q = 0; q < kZPer; ++q) {
        const int64_t i = int64_t(blockIdx.x) * kZPoints + q * kZBlock + threadIdx.x;
        if (i < n) mine += acc[q] - 1.0;
    }
    double total;
    if (last_block_sum(mine, part, gridDim.x, &hdr->ticket_eval, &total)) hdr->eval = total;
}

// KL = sum over stored p_ij > 0 of p_ij (log p_ij + log(1 + |y_i - y_j|^2) + log Z),
// in fp64 from the fp32 inputs.  Eight lanes take a row (its entries in
// turn, then a fixed butterfly); blocks stride over the rows.
constexpr int kKlLanes = 8;

__global__ __launch_bounds__(kEvalBlock) void kl_kernel(const float2 *__restrict__ Y,
                                                       const int64_t *__restrict__ row_ptr,
                                                       const int32_t *__restrict__ col,
                                                       const float *__restrict__ val, int64_t n, int64_t nnz,
                                                       double log_z, double *__restrict__ part,
                                                       Header *__restrict__ hdr)
{
    const int j = threadIdx.x % kKlLanes;
    const int64_t groups = int64_t(gridDim.x) * (kEvalBlock / kKlLanes);
    double mine = 0.0;
    for (int64_t i = int64_t(blockIdx.x) * (kEvalBlock / kKlLanes) + threadIdx.x / kKlLanes; i < n; i += groups) {
        const float2 yi = Y[i];
        int64_t e0 = row_ptr[i], e1 = row_ptr[i + 1];
        if (e0 < 0 || e1 > nnz) { // malformed row: skip what lies outside the arrays
            if (j == 0) atomicOr(&hdr->flags, kErrRange);
            e0 = e0 < 0 ? 0 : e0;
            e1 = e1 > nnz ? nnz : e1;
        }
        double r = 0.0;
        for (int64_t e = e0 + j; e < e1; e += kKlLanes) {
            const double p = double(val[e]);
            if (!(p > 0.0)) continue;
            const int32_t c = col[e];
            if (c < 0 || int64_t(c) >= n) {
                atomicOr(&hdr->flags, kErrRange);
                continue;
            }
            const float2 yj = Y[c];
            const double dx = double(yi.x) - double(yj.x), dy = double(yi.y) - double(yj.y);
            r += p * (log(p) + log(1.0 + dx * dx + dy * dy) + log_z);
        }
#pragma unroll
        for (int s = kKlLanes / 2; s > 0; s >>= 1) r += __shfl_xor(r, s, kKlLanes);
        if (j == 0) mine += r;
    }
    double total;
    if (last_block_sum(mine, part, gridDim.x, &hdr->ticket_eval, &total)) hdr->eval = total;
}

// ------------------------------------------------------------------ launchers
int eval_blocks_z(int64_t n) { return int((n + kZPoints - 1) / kZPoints); }

void launch_z_exact(const float *Y, int64_t n, void *ws, const Layout &L, hipStream_t st)
{
    Header *hdr = at<Header>(ws, L.header);
    eval_reset_kernel<<<1, 1, 0, st>>>(hdr);
    z_exact_kernel<<<unsigned(eval_blocks_z(n)), kZBlock, 0, st>>>(reinterpret_cast<const float2 *>(Y), n,
                                                                    at<double>(ws, L.eval_part), hdr);
}

void launch_kl(const float *Y, const int64_t *row_ptr, const int32_t *col, const float *val, int64_t n,
               int64_t nnz, double log_z, void *ws, const Layout &L, hipStream_t st)
{
    Header *hdr = at<Header>(ws, L.header);
    eval_reset_kernel<<<1, 1, 0, st>>>(hdr);
    const int64_t want = (n + kEvalBlock / kKlLanes - 1) / (kEvalBlock / kKlLanes);
    const unsigned blocks = unsigned(want < kEvalMaxBlocks ? want : kEvalMaxBlocks);
    kl_kernel<<<blocks, kEvalBlock, 0, st>>>(reinterpret_cast<const float2 *>(Y), row_ptr, col, val, n, nnz, log_z,
                                             at<double>(ws, L.eval_part), hdr);
}

} // namespace bht
