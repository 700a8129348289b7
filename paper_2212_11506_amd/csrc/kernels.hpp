// Host-side launchers of the device kernels (internal to the library).
#pragma once

#include "common.hpp"

namespace bht {

struct StepArgs {
    float alpha;         // exaggeration of the attractive term
    float learning_rate; // eta
    float momentum;      // mu
    float min_gain;
    int update;          // 0: gradient only
};

// Optional per-node exports of the tree (device arrays of at least 2n entries).
struct TreeDebug {
    uint8_t *level = nullptr;
    uint8_t *kind = nullptr; // 0 internal, 1 bucket, 2 single point
    uint32_t *begin = nullptr;
    uint32_t *end = nullptr;
};

void launch_bbox(const float *Y, int64_t n, void *ws, const Layout &L, hipStream_t st);
void launch_morton(const float *Y, int64_t n, void *ws, const Layout &L, hipStream_t st);
void launch_sort(int64_t n, void *ws, const Layout &L, hipStream_t st);
void launch_tree(int64_t n, float theta, void *ws, const Layout &L, const TreeDebug &dbg, hipStream_t st);
void launch_repulsive(int64_t n, void *ws, const Layout &L, hipStream_t st);
void launch_attract(const int64_t *row_ptr, const int32_t *col, const float *val, int64_t n, int64_t nnz,
                    const StepArgs &a, float *Y, float *upd, float *gains, float *grad, void *ws, const Layout &L,
                    hipStream_t st);

} // namespace bht
