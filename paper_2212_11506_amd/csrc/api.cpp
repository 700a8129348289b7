// C ABI of the library: argument checks, workspace carving, launch order and
// per-phase timing.  See include/bhtsne.h for the contract of each call.
#include "bhtsne.h"

#include <array>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <vector>

#include "kernels.hpp"

using namespace bht;

namespace {

// ------------------------------------------------------------------ timing
struct Timing {
    std::mutex mu;
    bool enabled = false;
    uint32_t phases = (1u << BHTSNE_NUM_PHASES) - 1u; // phases that record events
    std::vector<hipEvent_t> pool;
    struct Pending {
        int phase;
        hipEvent_t a, b;
    };
    std::vector<Pending> pending;
    double ms[BHTSNE_NUM_PHASES] = {};
    int64_t count[BHTSNE_NUM_PHASES] = {};

    hipEvent_t get()
    {
        if (!pool.empty()) {
            hipEvent_t e = pool.back();
            pool.pop_back();
            return e;
        }
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        return e;
    }
};

Timing &timing()
{
    static Timing t;
    return t;
}

// Records an event pair around one phase when timing is on.
class PhaseTimer {
  public:
    PhaseTimer(int phase, hipStream_t st) : phase_(phase), st_(st)
    {
        Timing &t = timing();
        std::lock_guard<std::mutex> g(t.mu);
        if (!t.enabled || !((t.phases >> phase) & 1u)) return;
        a_ = t.get();
        b_ = t.get();
        if (a_ && b_) hipEventRecord(a_, st_);
    }
    ~PhaseTimer()
    {
        if (!a_ || !b_) return;
        hipEventRecord(b_, st_);
        Timing &t = timing();
        std::lock_guard<std::mutex> g(t.mu);
        t.pending.push_back({phase_, a_, b_});
    }

  private:
    int phase_;
    hipStream_t st_;
    hipEvent_t a_ = nullptr, b_ = nullptr;
};

bool finite_f(float x) { return std::isfinite(x); }

bool aligned(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 255u) == 0; }

int check_ws(int64_t n, int64_t nnz, void *ws, size_t bytes)
{
    if (!ws || !aligned(ws)) return BHTSNE_EWORKSPACE;
    size_t need = bhtsne_workspace_size(n, nnz);
    if (need == 0) return BHTSNE_EINVAL;
    if (bytes < need) return BHTSNE_EWORKSPACE;
    return BHTSNE_OK;
}

int check_csr(const bhtsne_csr *P)
{
    if (!P) return BHTSNE_EINVAL;
    if (P->n < 2 || P->n > kMaxPoints) return BHTSNE_EINVAL;
    if (P->nnz < 0 || !P->row_ptr) return BHTSNE_EINVAL;
    if (P->nnz > 0 && (!P->col || !P->val)) return BHTSNE_EINVAL;
    return BHTSNE_OK;
}

int flags_status(uint32_t flags)
{
    if (flags & kErrNonFinite) return BHTSNE_ENONFINITE;
    if (flags & (kErrLookback | kErrRange)) return BHTSNE_EDEVICE;
    return BHTSNE_OK;
}

int read_header(const void *ws, Header *h, hipStream_t st)
{
    if (hipMemcpyAsync(h, ws, sizeof(Header), hipMemcpyDeviceToHost, st) != hipSuccess) return BHTSNE_EDEVICE;
    if (hipStreamSynchronize(st) != hipSuccess) return BHTSNE_EDEVICE;
    return BHTSNE_OK;
}

// Box and codes.  `perm` (nullable; a layout's position -> caller's index)
// puts the private copy of Y in the layout's order.
void build_codes(const float *Y, int64_t n, const uint32_t *perm, void *ws, const Layout &L, hipStream_t st)
{
    PhaseTimer pt(BHTSNE_PHASE_BBOX_MORTON, st);
    launch_bbox(Y, n, ws, L, st);
    launch_morton(Y, n, perm, ws, L, st);
}

// Sort, tree and summaries.
void build_sorted_tree(const float *Y, int64_t n, float theta, void *ws, const Layout &L, const TreeDebug &dbg,
                       hipStream_t st)
{
    {
        PhaseTimer pt(BHTSNE_PHASE_SORT, st);
        launch_sort(n, Y, ws, L, st);
    }
    {
        PhaseTimer pt(BHTSNE_PHASE_TREE, st);
        launch_tree<2, float>(n, double(theta) * double(theta), ws, L, dbg, st);
    }
}

void build_tree(const float *Y, int64_t n, float theta, const uint32_t *perm, void *ws, const Layout &L,
                const TreeDebug &dbg, hipStream_t st)
{
    build_codes(Y, n, perm, ws, L, st);
    build_sorted_tree(Y, n, theta, ws, L, dbg, st);
}

// ------------------------------------------------------------------ side stream
// A second stream per device (default priority) for work that does not depend
// on the tree: the attractive forces of the layout calls.  Forked from the
// caller's stream with one event and joined back with another; the mutex keeps
// the enqueue of a fork .. join sequence whole when several threads call in.
struct Side {
    std::mutex mu;
    hipStream_t st = nullptr;
    hipEvent_t fork = nullptr, join = nullptr;
    bool failed = false;
};

constexpr int kMaxDevices = 64;

Side *side_stream()
{
    static Side sides[kMaxDevices];
    static std::mutex create_mu;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    Side &x = sides[dev];
    std::lock_guard<std::mutex> g(create_mu);
    if (x.failed) return nullptr;
    if (!x.st) {
        if (hipStreamCreateWithFlags(&x.st, hipStreamNonBlocking) != hipSuccess ||
            hipEventCreateWithFlags(&x.fork, hipEventDisableTiming) != hipSuccess ||
            hipEventCreateWithFlags(&x.join, hipEventDisableTiming) != hipSuccess) {
            x.failed = true;
            return nullptr;
        }
    }
    return &x;
}

// BHTSNE_OVERLAP=0 runs the attractive forces on the caller's stream instead
bool overlap_enabled()
{
    static bool v = [] {
        const char *e = std::getenv("BHTSNE_OVERLAP");
        return !(e && std::atoi(e) == 0);
    }();
    return v;
}

// Where a layout step forks the attractive forces off to the second stream:
// 0 after the codes, 1 after the sort, 2 after the tree (an environment
// variable, read once, else the default).
int env_fork(const char *name, int dflt)
{
    const char *e = std::getenv(name);
    const int x = e ? std::atoi(e) : dflt;
    return x < 0 ? 0 : (x > 2 ? 2 : x);
}

// fp32 2-D layouts (BHTSNE_FORK; default 0).  Measured at 1.3M points the
// sort, a chain of latency-bound passes, does best on the CUs the attractive
// kernel leaves free (its blocks cannot share a CU's LDS with one), and the
// tree and the repulsive walk lose more than they hide when forked later:
// 844 iterations/s, against 752 after the sort and 754 after the tree.
int fork_point()
{
    static const int v = env_fork("BHTSNE_FORK", 0);
    return v;
}

// 3-D layouts (BHTSNE_FORK3; default 2, after the tree).  The 3-D walk is four
// times longer than the 2-D one, so the attraction it absorbs costs it less
// than the attraction costs the sort and tree beside them: 337.9 iterations/s
// at 1.3M points, against 324.9 forked after the codes and 297.0 after the sort.
int fork_point3()
{
    static const int v = env_fork("BHTSNE_FORK3", 2);
    return v;
}

// fp64 layouts (BHTSNE_FORK64; default 2, after the tree): the fp64 tree phase
// slows from 0.14 to 0.51 ms beside the attraction, while the fp64 walk, 2.6
// times the fp32 one, absorbs it; 412.4 iterations/s at 1.3M points against
// 402.7 forked after the codes and 389.7 after the sort.
int fork_point64()
{
    static const int v = env_fork("BHTSNE_FORK64", 2);
    return v;
}

int device_cus()
{
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        return 256;
    return cus;
}

// Blocks of the persistent sliced attractive kernel (one per CU it holds):
// all CUs when it runs alone; beside the tree phases a share of them
// (BHTSNE_ATTRACT_CUS, percent of the CUs, default 75), so that the critical
// path keeps CUs of its own; 0 gives one block per item.  The windowed
// segments (no items) take all CUs: without tile locality the attraction is
// the longest phase (at 5M points 9.5 ms on 75% against 3.9 for the walk).
int attract_blocks(bool beside, int items)
{
    static int pct = [] {
        const char *e = std::getenv("BHTSNE_ATTRACT_CUS");
        int x = e ? std::atoi(e) : 75;
        return x < 0 ? 0 : (x > 100 ? 100 : x);
    }();
    if (items <= 0) return device_cus();
    if (beside && pct == 0) return items;
    const int cus = device_cus();
    const int b = beside ? cus * pct / 100 : cus;
    return b < 1 ? 1 : b;
}

int finish(double *Z, void *ws, hipStream_t st)
{
    if (hipGetLastError() != hipSuccess) return BHTSNE_EDEVICE;
    if (Z) {
        Header h;
        int rc = read_header(ws, &h, st);
        if (rc != BHTSNE_OK) return rc;
        *Z = h.Z;
        return flags_status(h.flags);
    }
    return BHTSNE_OK;
}

int run(float *Y, const bhtsne_csr *P, float theta, const StepArgs &a, float *update, float *gains, float *grad,
        double *Z, void *ws, hipStream_t st)
{
    const int64_t n = P->n;
    const Layout L = make_layout(n, P->nnz);
    build_tree(Y, n, theta, nullptr, ws, L, TreeDebug{}, st);
    {
        PhaseTimer pt(BHTSNE_PHASE_REPULSIVE, st);
        launch_repulsive<2, float>(n, repulsive_self_test(theta), ws, L, st);
    }
    {
        PhaseTimer pt(BHTSNE_PHASE_ATTRACTIVE, st);
        launch_attract<2>(P->row_ptr, P->col, P->val, n, P->nnz, a, Y, update, gains, grad, ws, L, st);
    }
    return finish(Z, ws, st);
}

// ------------------------------------------------------------------ fixed scratch
// Workspace of bhtsne_step_noalloc: one array per device, allocated when the
// code object is loaded and held until the process ends.  Host code never
// uses the symbol itself (on the host it names a stand-in, not device
// memory): the device address is looked up once per device, with that device
// current, and every launch takes that address.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

void *static_scratch()
{
    static std::mutex mu;
    static void *addr[kMaxDevices] = {};
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> g(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        addr[dev] = p;
    }
    return addr[dev];
}

constexpr uint64_t kLayoutMagic = 0x62687473654c3031ull; // "bhtseL01"

int stage_segments()
{
    static int v = [] {
        const char *e = std::getenv("BHTSNE_STAGE_SEGMENTS");
        int x = e ? std::atoi(e) : 16;
        return x < 0 ? 0 : x;
    }();
    return v;
}

// BHTSNE_TILES=0 keeps the row-block attractive kernel (for comparisons and tests)
bool tile_path_enabled()
{
    static bool v = [] {
        const char *e = std::getenv("BHTSNE_TILES");
        return !(e && std::atoi(e) == 0);
    }();
    return v;
}

// BHTSNE_WINDOWS=0 keeps the row-block attractive kernel where windowed
// segments would be built (for comparisons and tests)
bool window_path_enabled()
{
    static bool v = [] {
        const char *e = std::getenv("BHTSNE_WINDOWS");
        return !(e && std::atoi(e) == 0);
    }();
    return v;
}

constexpr uint64_t kLayoutMagic64 = 0x62687473654c3634ull; // "bhtseL64": an fp64 layout
constexpr uint64_t kLayoutMagic3 = 0x62687473654c3033ull;  // "bhtseL03": a 3-D layout

// vbytes: 4 for the fp32 calls' layouts, 8 for the fp64 variant's; dim 3 for
// the 3-D calls' layouts
int check_layout(const bhtsne_layout *lay, int vbytes = 4, int dim = 2)
{
    const uint64_t magic = dim == 3 ? kLayoutMagic3 : (vbytes == 8 ? kLayoutMagic64 : kLayoutMagic);
    if (!lay || lay->magic != magic || !lay->mem || !aligned(lay->mem)) return BHTSNE_EINVAL;
    if (lay->n < 2 || lay->n > kMaxPoints || lay->nnz < 0) return BHTSNE_EINVAL;
    const LayoutView v = layout_view(nullptr, lay->n, lay->nnz, vbytes, dim);
    if (lay->bytes < v.bytes) return BHTSNE_EINVAL;
    if (lay->tiles < 0 || lay->tiles > v.max_tiles) return BHTSNE_EINVAL;
    if (lay->items < 0 || lay->items > lay->tiles || (lay->tiles > 0) != (lay->items > 0)) return BHTSNE_EINVAL;
    if (lay->windows < 0 || lay->windows > kMaxWindows || (lay->windows > 0 && lay->tiles > 0)) return BHTSNE_EINVAL;
    // windowed segments need windows; windows without segments are a P with no
    // entries (F_attr = 0)
    if (lay->segments < 0 || lay->segments > v.max_segments || (lay->segments > 0 && lay->windows == 0))
        return BHTSNE_EINVAL;
    if (lay->order != BHTSNE_ORDER_MORTON && lay->order != BHTSNE_ORDER_BFS) return BHTSNE_EINVAL;
    return BHTSNE_OK;
}

// The fp64 variant (plain CSR): the same phases with fp64 coordinates,
// centres, thresholds, forces and optimiser state.
int run64(double *Y, const bhtsne_csr_f64 *P, double theta, const StepArgsT<double> &a, double *update,
          double *gains, double *grad, double *Z, void *ws, hipStream_t st)
{
    const int64_t n = P->n;
    const Layout L = make_layout(n, P->nnz, 8);
    {
        PhaseTimer pt(BHTSNE_PHASE_BBOX_MORTON, st);
        launch_bbox(Y, n, ws, L, st);
        launch_morton(Y, n, nullptr, ws, L, st);
    }
    {
        PhaseTimer pt(BHTSNE_PHASE_SORT, st);
        launch_sort(n, static_cast<const double *>(Y), ws, L, st);
    }
    {
        PhaseTimer pt(BHTSNE_PHASE_TREE, st);
        launch_tree<2, double>(n, theta * theta, ws, L, TreeDebug{}, st);
    }
    {
        PhaseTimer pt(BHTSNE_PHASE_REPULSIVE, st);
        launch_repulsive<2, double>(n, repulsive_self_test(theta), ws, L, st);
    }
    {
        PhaseTimer pt(BHTSNE_PHASE_ATTRACTIVE, st);
        launch_attract<2>(P->row_ptr, P->col, P->val, n, P->nnz, a, Y, update, gains, grad, ws, L, st);
    }
    return finish(Z, ws, st);
}

// The fp64 variant through a layout: the sliced or windowed-segment
// attraction on the second stream, by default forked after the tree, beside
// the walk.
int run_layout64(double *Y, const bhtsne_layout *lay, double theta, const StepArgsT<double> &a, double *update,
                 double *gains, double *grad, double *Z, void *ws, hipStream_t st)
{
    const int64_t n = lay->n;
    const Layout L = make_layout(n, lay->nnz, 8);
    const LayoutView lv = layout_view(lay->mem, n, lay->nnz, 8);
    {
        PhaseTimer pt(BHTSNE_PHASE_BBOX_MORTON, st);
        launch_bbox(Y, n, ws, L, st);
        launch_morton(static_cast<const double *>(Y), n, lv.perm, ws, L, st);
    }
    const int fork = fork_point64();
    if (fork >= 1) {
        PhaseTimer pt(BHTSNE_PHASE_SORT, st);
        launch_sort(n, static_cast<const double *>(Y), ws, L, st);
    }
    if (fork >= 2) {
        PhaseTimer pt(BHTSNE_PHASE_TREE, st);
        launch_tree<2, double>(n, theta * theta, ws, L, TreeDebug{}, st);
    }
    Side *side = overlap_enabled() ? side_stream() : nullptr;
    std::unique_lock<std::mutex> lk;
    if (side) {
        lk = std::unique_lock<std::mutex>(side->mu);
        if (hipEventRecord(side->fork, st) != hipSuccess || hipStreamWaitEvent(side->st, side->fork, 0) != hipSuccess)
            return BHTSNE_EDEVICE;
    }
    const hipStream_t sa = side ? side->st : st;
    {
        PhaseTimer pt(BHTSNE_PHASE_ATTRACTIVE, sa);
        launch_attract_layout<double>(lv, n, lay->nnz, int(lay->tiles), int(lay->items),
                                      attract_blocks(side != nullptr, int(lay->items)), stage_segments(),
                                      int(lay->windows), ws, L, sa);
    }
    if (side && hipEventRecord(side->join, sa) != hipSuccess) return BHTSNE_EDEVICE;
    if (fork < 1) {
        PhaseTimer pt(BHTSNE_PHASE_SORT, st);
        launch_sort(n, static_cast<const double *>(Y), ws, L, st);
    }
    if (fork < 2) {
        PhaseTimer pt(BHTSNE_PHASE_TREE, st);
        launch_tree<2, double>(n, theta * theta, ws, L, TreeDebug{}, st);
    }
    {
        PhaseTimer pt(BHTSNE_PHASE_REPULSIVE, st);
        launch_repulsive<2, double>(n, repulsive_self_test(theta), ws, L, st);
    }
    if (side && hipStreamWaitEvent(st, side->join, 0) != hipSuccess) return BHTSNE_EDEVICE;
    if (lk.owns_lock()) lk.unlock();
    {
        PhaseTimer pt(BHTSNE_PHASE_UPDATE, st);
        launch_update(lv, n, lay->tiles == 0 && lay->windows > 0, a, Y, update, gains, grad, ws, L, st);
    }
    return finish(Z, ws, st);
}

int run_layout(float *Y, const bhtsne_layout *lay, float theta, const StepArgs &a, float *update, float *gains,
               float *grad, double *Z, void *ws, hipStream_t st)
{
    const int64_t n = lay->n;
    const Layout L = make_layout(n, lay->nnz);
    const LayoutView lv = layout_view(lay->mem, n, lay->nnz);
    const int tiles = int(lay->tiles);
    // the attractive forces need only the layout-order copy of Y written with
    // the codes, so they can run beside the sort, tree and repulsive phases
    const int fork = fork_point();
    build_codes(Y, n, lv.perm, ws, L, st);
    if (fork >= 1) {
        PhaseTimer pt(BHTSNE_PHASE_SORT, st);
        launch_sort(n, Y, ws, L, st);
    }
    if (fork >= 2) {
        PhaseTimer pt(BHTSNE_PHASE_TREE, st);
        launch_tree<2, float>(n, double(theta) * double(theta), ws, L, TreeDebug{}, st);
    }
    Side *side = overlap_enabled() ? side_stream() : nullptr;
    std::unique_lock<std::mutex> lk;
    if (side) {
        lk = std::unique_lock<std::mutex>(side->mu);
        if (hipEventRecord(side->fork, st) != hipSuccess || hipStreamWaitEvent(side->st, side->fork, 0) != hipSuccess)
            return BHTSNE_EDEVICE;
    }
    const hipStream_t sa = side ? side->st : st;
    {
        PhaseTimer pt(BHTSNE_PHASE_ATTRACTIVE, sa);
        launch_attract_layout<float>(lv, n, lay->nnz, tiles, int(lay->items),
                                     attract_blocks(side != nullptr, int(lay->items)), stage_segments(),
                                     int(lay->windows), ws, L, sa);
    }
    if (side && hipEventRecord(side->join, sa) != hipSuccess) return BHTSNE_EDEVICE;
    if (fork < 1) {
        PhaseTimer pt(BHTSNE_PHASE_SORT, st);
        launch_sort(n, Y, ws, L, st);
    }
    if (fork < 2) {
        PhaseTimer pt(BHTSNE_PHASE_TREE, st);
        launch_tree<2, float>(n, double(theta) * double(theta), ws, L, TreeDebug{}, st);
    }
    {
        PhaseTimer pt(BHTSNE_PHASE_REPULSIVE, st);
        launch_repulsive<2, float>(n, repulsive_self_test(theta), ws, L, st);
    }
    if (side && hipStreamWaitEvent(st, side->join, 0) != hipSuccess) return BHTSNE_EDEVICE;
    if (lk.owns_lock()) lk.unlock();
    {
        PhaseTimer pt(BHTSNE_PHASE_UPDATE, st);
        launch_update(lv, n, tiles == 0 && lay->windows > 0, a, Y, update, gains, grad, ws, L, st);
    }
    return finish(Z, ws, st);
}

// A 3-D embedding (plain CSR P): the same phases on a cube, 63-bit codes, an
// octree with 32-byte records and three-component forces.
int run3(float *Y, const bhtsne_csr *P, float theta, const StepArgs &a, float *update, float *gains, float *grad,
         double *Z, void *ws, hipStream_t st)
{
    const int64_t n = P->n;
    const Layout L = make_layout(n, P->nnz, 4, 3);
    {
        PhaseTimer pt(BHTSNE_PHASE_BBOX_MORTON, st);
        launch_bbox_morton3(Y, n, nullptr, ws, L, st);
    }
    {
        PhaseTimer pt(BHTSNE_PHASE_SORT, st);
        launch_sort_points(n, reinterpret_cast<const float3 *>(Y), ws, L, st);
    }
    {
        PhaseTimer pt(BHTSNE_PHASE_TREE, st);
        launch_tree<3, float>(n, double(theta) * double(theta), ws, L, TreeDebug{}, st);
    }
    {
        PhaseTimer pt(BHTSNE_PHASE_REPULSIVE, st);
        launch_repulsive<3, float>(n, repulsive_self_test3(theta), ws, L, st);
    }
    {
        PhaseTimer pt(BHTSNE_PHASE_ATTRACTIVE, st);
        launch_attract<3>(P->row_ptr, P->col, P->val, n, P->nnz, a, Y, update, gains, grad, ws, L, st);
    }
    return finish(Z, ws, st);
}

// A 3-D embedding through a layout: the codes also write the layout-order copy
// of Y, the sliced attraction runs on the second stream (by default beside the
// walk), and the update joins F_attr (caller's order) with F_rep.
int run_layout3(float *Y, const bhtsne_layout *lay, float theta, const StepArgs &a, float *update, float *gains,
                float *grad, double *Z, void *ws, hipStream_t st)
{
    const int64_t n = lay->n;
    const Layout L = make_layout(n, lay->nnz, 4, 3);
    const LayoutView lv = layout_view(lay->mem, n, lay->nnz, 4, 3);
    {
        PhaseTimer pt(BHTSNE_PHASE_BBOX_MORTON, st);
        launch_bbox_morton3(Y, n, lv.perm, ws, L, st);
    }
    const int fork = fork_point3();
    if (fork >= 1) {
        PhaseTimer pt(BHTSNE_PHASE_SORT, st);
        launch_sort_points(n, reinterpret_cast<const float3 *>(Y), ws, L, st);
    }
    if (fork >= 2) {
        PhaseTimer pt(BHTSNE_PHASE_TREE, st);
        launch_tree<3, float>(n, double(theta) * double(theta), ws, L, TreeDebug{}, st);
    }
    Side *side = overlap_enabled() ? side_stream() : nullptr;
    std::unique_lock<std::mutex> lk;
    if (side) {
        lk = std::unique_lock<std::mutex>(side->mu);
        if (hipEventRecord(side->fork, st) != hipSuccess || hipStreamWaitEvent(side->st, side->fork, 0) != hipSuccess)
            return BHTSNE_EDEVICE;
    }
    const hipStream_t sa = side ? side->st : st;
    {
        PhaseTimer pt(BHTSNE_PHASE_ATTRACTIVE, sa);
        launch_attract_layout3(lv, n, int(lay->tiles), int(lay->items), attract_blocks(side != nullptr, int(lay->items)),
                               ws, L, sa);
    }
    if (side && hipEventRecord(side->join, sa) != hipSuccess) return BHTSNE_EDEVICE;
    if (fork < 1) {
        PhaseTimer pt(BHTSNE_PHASE_SORT, st);
        launch_sort_points(n, reinterpret_cast<const float3 *>(Y), ws, L, st);
    }
    if (fork < 2) {
        PhaseTimer pt(BHTSNE_PHASE_TREE, st);
        launch_tree<3, float>(n, double(theta) * double(theta), ws, L, TreeDebug{}, st);
    }
    {
        PhaseTimer pt(BHTSNE_PHASE_REPULSIVE, st);
        launch_repulsive<3, float>(n, repulsive_self_test3(theta), ws, L, st);
    }
    if (side && hipStreamWaitEvent(st, side->join, 0) != hipSuccess) return BHTSNE_EDEVICE;
    if (lk.owns_lock()) lk.unlock();
    {
        PhaseTimer pt(BHTSNE_PHASE_UPDATE, st);
        launch_update3(n, a, Y, update, gains, grad, ws, L, st);
    }
    return finish(Z, ws, st);
}

int check_step_args(float theta, float exaggeration, float learning_rate, float momentum, float min_gain)
{
    if (!finite_f(theta) || theta < 0.0f) return BHTSNE_EINVAL;
    if (!finite_f(exaggeration) || !(exaggeration > 0.0f)) return BHTSNE_EINVAL;
    if (!finite_f(learning_rate) || !(learning_rate > 0.0f)) return BHTSNE_EINVAL;
    if (!finite_f(momentum) || momentum < 0.0f || !(momentum < 1.0f)) return BHTSNE_EINVAL;
    if (!finite_f(min_gain) || min_gain < 0.0f) return BHTSNE_EINVAL;
    return BHTSNE_OK;
}

} // namespace

extern "C" {

size_t bhtsne_workspace_size(int64_t n, int64_t nnz)
{
    if (n < 2 || n > kMaxPoints || nnz < 0) return 0;
    return make_layout(n, nnz).total;
}

int bhtsne_gradient(const float *Y, const bhtsne_csr *P, float theta, float exaggeration, float *grad, double *Z,
                    void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    int rc = check_csr(P);
    if (rc != BHTSNE_OK) return rc;
    if (!Y || !grad) return BHTSNE_EINVAL;
    if (!finite_f(theta) || theta < 0.0f) return BHTSNE_EINVAL;
    if (!finite_f(exaggeration) || !(exaggeration > 0.0f)) return BHTSNE_EINVAL;
    rc = check_ws(P->n, P->nnz, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    StepArgs a{exaggeration, 0.0f, 0.0f, 0.0f, 0};
    return run(const_cast<float *>(Y), P, theta, a, nullptr, nullptr, grad, Z, workspace, stream);
}

int bhtsne_step(float *Y, const bhtsne_csr *P, float theta, float exaggeration, float learning_rate, float momentum,
                float min_gain, float *update, float *gains, float *grad, double *Z, void *workspace,
                size_t workspace_bytes, hipStream_t stream)
{
    int rc = check_csr(P);
    if (rc != BHTSNE_OK) return rc;
    if (!Y || !update || !gains) return BHTSNE_EINVAL;
    rc = check_step_args(theta, exaggeration, learning_rate, momentum, min_gain);
    if (rc != BHTSNE_OK) return rc;
    rc = check_ws(P->n, P->nnz, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    StepArgs a{exaggeration, learning_rate, momentum, min_gain, 1};
    return run(Y, P, theta, a, update, gains, grad, Z, workspace, stream);
}

size_t bhtsne_noalloc_max_bytes(void) { return kStaticScratchBytes; }

int bhtsne_step_noalloc(float *Y, const bhtsne_csr *P, float theta, float exaggeration, float learning_rate,
                        float momentum, float min_gain, float *update, float *gains, float *grad, double *Z,
                        hipStream_t stream)
{
    int rc = check_csr(P);
    if (rc != BHTSNE_OK) return rc;
    if (!Y || !update || !gains) return BHTSNE_EINVAL;
    rc = check_step_args(theta, exaggeration, learning_rate, momentum, min_gain);
    if (rc != BHTSNE_OK) return rc;
    const size_t need = bhtsne_workspace_size(P->n, P->nnz);
    if (need == 0 || need > kStaticScratchBytes) return BHTSNE_EINVAL;
    void *ws = static_scratch();
    if (!ws) return BHTSNE_EDEVICE;
    StepArgs a{exaggeration, learning_rate, momentum, min_gain, 1};
    return run(Y, P, theta, a, update, gains, grad, Z, ws, stream);
}

size_t bhtsne_workspace_size_f64(int64_t n, int64_t nnz)
{
    if (n < 2 || n > kMaxPoints || nnz < 0) return 0;
    return make_layout(n, nnz, 8).total;
}

static int check_csr_f64(const bhtsne_csr_f64 *P)
{
    if (!P) return BHTSNE_EINVAL;
    if (P->n < 2 || P->n > kMaxPoints) return BHTSNE_EINVAL;
    if (P->nnz < 0 || !P->row_ptr) return BHTSNE_EINVAL;
    if (P->nnz > 0 && (!P->col || !P->val)) return BHTSNE_EINVAL;
    return BHTSNE_OK;
}

static int check_ws_f64(int64_t n, int64_t nnz, void *ws, size_t bytes)
{
    if (!ws || !aligned(ws)) return BHTSNE_EWORKSPACE;
    size_t need = bhtsne_workspace_size_f64(n, nnz);
    if (need == 0) return BHTSNE_EINVAL;
    if (bytes < need) return BHTSNE_EWORKSPACE;
    return BHTSNE_OK;
}

int bhtsne_gradient_f64(const double *Y, const bhtsne_csr_f64 *P, double theta, double exaggeration, double *grad,
                        double *Z, void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    int rc = check_csr_f64(P);
    if (rc != BHTSNE_OK) return rc;
    if (!Y || !grad) return BHTSNE_EINVAL;
    if (!std::isfinite(theta) || theta < 0.0) return BHTSNE_EINVAL;
    if (!std::isfinite(exaggeration) || !(exaggeration > 0.0)) return BHTSNE_EINVAL;
    rc = check_ws_f64(P->n, P->nnz, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    StepArgsT<double> a{exaggeration, 0.0, 0.0, 0.0, 0};
    return run64(const_cast<double *>(Y), P, theta, a, nullptr, nullptr, grad, Z, workspace, stream);
}

int bhtsne_step_f64(double *Y, const bhtsne_csr_f64 *P, double theta, double exaggeration, double learning_rate,
                    double momentum, double min_gain, double *update, double *gains, double *grad, double *Z,
                    void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    int rc = check_csr_f64(P);
    if (rc != BHTSNE_OK) return rc;
    if (!Y || !update || !gains) return BHTSNE_EINVAL;
    if (!std::isfinite(theta) || theta < 0.0) return BHTSNE_EINVAL;
    if (!std::isfinite(exaggeration) || !(exaggeration > 0.0)) return BHTSNE_EINVAL;
    if (!std::isfinite(learning_rate) || !(learning_rate > 0.0)) return BHTSNE_EINVAL;
    if (!std::isfinite(momentum) || momentum < 0.0 || !(momentum < 1.0)) return BHTSNE_EINVAL;
    if (!std::isfinite(min_gain) || min_gain < 0.0) return BHTSNE_EINVAL;
    rc = check_ws_f64(P->n, P->nnz, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    StepArgsT<double> a{exaggeration, learning_rate, momentum, min_gain, 1};
    return run64(Y, P, theta, a, update, gains, grad, Z, workspace, stream);
}

size_t bhtsne_workspace_size_3d(int64_t n, int64_t nnz)
{
    if (n < 2 || n > kMaxPoints || nnz < 0) return 0;
    return make_layout(n, nnz, 4, 3).total;
}

static int check_ws_3d(int64_t n, int64_t nnz, void *ws, size_t bytes)
{
    if (!ws || !aligned(ws)) return BHTSNE_EWORKSPACE;
    const size_t need = bhtsne_workspace_size_3d(n, nnz);
    if (need == 0) return BHTSNE_EINVAL;
    if (bytes < need) return BHTSNE_EWORKSPACE;
    return BHTSNE_OK;
}

int bhtsne_gradient_3d(const float *Y, const bhtsne_csr *P, float theta, float exaggeration, float *grad, double *Z,
                       void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    int rc = check_csr(P);
    if (rc != BHTSNE_OK) return rc;
    if (!Y || !grad) return BHTSNE_EINVAL;
    if (!finite_f(theta) || theta < 0.0f) return BHTSNE_EINVAL;
    if (!finite_f(exaggeration) || !(exaggeration > 0.0f)) return BHTSNE_EINVAL;
    rc = check_ws_3d(P->n, P->nnz, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    StepArgs a{exaggeration, 0.0f, 0.0f, 0.0f, 0};
    return run3(const_cast<float *>(Y), P, theta, a, nullptr, nullptr, grad, Z, workspace, stream);
}

int bhtsne_step_3d(float *Y, const bhtsne_csr *P, float theta, float exaggeration, float learning_rate,
                   float momentum, float min_gain, float *update, float *gains, float *grad, double *Z,
                   void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    int rc = check_csr(P);
    if (rc != BHTSNE_OK) return rc;
    if (!Y || !update || !gains) return BHTSNE_EINVAL;
    rc = check_step_args(theta, exaggeration, learning_rate, momentum, min_gain);
    if (rc != BHTSNE_OK) return rc;
    rc = check_ws_3d(P->n, P->nnz, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    StepArgs a{exaggeration, learning_rate, momentum, min_gain, 1};
    return run3(Y, P, theta, a, update, gains, grad, Z, workspace, stream);
}

int bhtsne_debug_sort_3d(const float *Y, int64_t n, uint64_t *codes, uint64_t *sorted_codes, uint32_t *perm,
                         double *params, void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    if (!Y || n < 2 || n > kMaxPoints) return BHTSNE_EINVAL;
    int rc = check_ws_3d(n, 0, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    const Layout L = make_layout(n, 0, 4, 3);
    launch_bbox_morton3(Y, n, nullptr, workspace, L, stream);
    if (codes && hipMemcpyAsync(codes, at<void>(workspace, L.codes0), 8 * size_t(n), hipMemcpyDeviceToDevice,
                                stream) != hipSuccess)
        return BHTSNE_EDEVICE;
    launch_sort_points(n, reinterpret_cast<const float3 *>(Y), workspace, L, stream);
    if (sorted_codes && hipMemcpyAsync(sorted_codes, at<void>(workspace, L.codes0), 8 * size_t(n),
                                       hipMemcpyDeviceToDevice, stream) != hipSuccess)
        return BHTSNE_EDEVICE;
    if (perm && hipMemcpyAsync(perm, at<void>(workspace, L.idx0), 4 * size_t(n), hipMemcpyDeviceToDevice,
                               stream) != hipSuccess)
        return BHTSNE_EDEVICE;
    if (hipGetLastError() != hipSuccess) return BHTSNE_EDEVICE;
    if (params) {
        Header h;
        rc = read_header(workspace, &h, stream);
        if (rc != BHTSNE_OK) return rc;
        const double p[14] = {h.bmin[0], h.bmax[0], h.bmin[1],  h.bmax[1],  h.bmin[2],  h.bmax[2],  h.cent[0],
                              h.cent[1], h.cent[2], h.rspan,    h.yroot[0], h.yroot[1], h.yroot[2], h.scale};
        std::memcpy(params, p, sizeof(p));
        return flags_status(h.flags);
    }
    return BHTSNE_OK;
}

int bhtsne_debug_tree_3d(const float *Y, int64_t n, float theta, int64_t *n_nodes, uint8_t *level, uint8_t *kind,
                         uint32_t *begin, uint32_t *end, float *summary, float *threshold, uint32_t *meta,
                         void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    if (!Y || !n_nodes || n < 2 || n > kMaxPoints) return BHTSNE_EINVAL;
    if (!finite_f(theta) || theta < 0.0f) return BHTSNE_EINVAL;
    if ((level || kind || begin || end) && !(level && kind && begin && end)) return BHTSNE_EINVAL;
    int rc = check_ws_3d(n, 0, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    const Layout L = make_layout(n, 0, 4, 3);
    TreeDebug dbg;
    dbg.level = level;
    dbg.kind = kind;
    dbg.begin = begin;
    dbg.end = end;
    launch_bbox_morton3(Y, n, nullptr, workspace, L, stream);
    launch_sort_points(n, reinterpret_cast<const float3 *>(Y), workspace, L, stream);
    launch_tree<3, float>(n, double(theta) * double(theta), workspace, L, dbg, stream);
    if (summary || threshold || meta) launch_tree_unpack3(n, workspace, L, summary, threshold, meta, stream);
    if (hipGetLastError() != hipSuccess) return BHTSNE_EDEVICE;
    Header h;
    rc = read_header(workspace, &h, stream);
    if (rc != BHTSNE_OK) return rc;
    *n_nodes = int64_t(h.nodes);
    return flags_status(h.flags);
}

// The end of a layout build: its status, the device flags of the build's
// sort, and the handle (the forms the plan allows and the switches leave on;
// 3-D layouts have no windowed segments).
static int finish_layout(int built, const TilePlan &plan, int64_t n, int64_t nnz, void *layout_mem,
                         size_t layout_bytes, uint64_t magic, bhtsne_layout *out, void *workspace, hipStream_t stream)
{
    if (built == 1) return BHTSNE_EINPUT;
    if (built != 0) return BHTSNE_EDEVICE;
    Header h;
    const int rc = read_header(workspace, &h, stream);
    if (rc != BHTSNE_OK) return rc;
    if (h.flags & (kErrLookback | kErrRange)) return BHTSNE_EDEVICE;
    out->n = n;
    out->nnz = nnz;
    out->mem = layout_mem;
    out->bytes = layout_bytes;
    out->order = plan.order;
    const bool tiled = plan.tiled && tile_path_enabled();
    out->tiles = tiled ? plan.tiles : 0;
    out->items = tiled ? plan.items : 0;
    out->entries = tiled ? plan.entries : 0;
    const bool windowed = magic != kLayoutMagic3 && !tiled && plan.windows > 0 && window_path_enabled();
    out->windows = windowed ? plan.windows : 0;
    out->segments = windowed ? plan.segments : 0;
    out->magic = magic;
    return BHTSNE_OK;
}

size_t bhtsne_layout_size_3d(int64_t n, int64_t nnz)
{
    if (n < 2 || n > kMaxPoints || nnz < 0) return 0;
    return layout_view(nullptr, n, nnz, 4, 3).bytes;
}

int bhtsne_layout_build_3d(const bhtsne_csr *P, const float *Y, void *layout_mem, size_t layout_bytes,
                           bhtsne_layout *out, void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    int rc = check_csr(P);
    if (rc != BHTSNE_OK) return rc;
    if (!out || !layout_mem || !aligned(layout_mem)) return BHTSNE_EINVAL;
    if (layout_bytes < bhtsne_layout_size_3d(P->n, P->nnz)) return BHTSNE_EINVAL;
    if (P->nnz + 3 * P->n + 4 >= (int64_t(1) << 31)) return BHTSNE_EINVAL;
    rc = check_ws_3d(P->n, P->nnz, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    const Layout L = make_layout(P->n, P->nnz, 4, 3);
    const LayoutView lv = layout_view(layout_mem, P->n, P->nnz, 4, 3);
    TilePlan plan;
    const int built = launch_layout_build<float, 3>(P->row_ptr, P->col, P->val, P->n, P->nnz, Y, kOrderAuto, lv,
                                                    &plan, workspace, L, stream);
    return finish_layout(built, plan, P->n, P->nnz, layout_mem, layout_bytes, kLayoutMagic3, out, workspace, stream);
}

static int check_layout3_step(const bhtsne_layout *layout, const float *Y, float theta, float exaggeration,
                              void *workspace, size_t workspace_bytes)
{
    int rc = check_layout(layout, 4, 3);
    if (rc != BHTSNE_OK) return rc;
    // no sliced copy (no tile locality, or rows too long to sort): use the plain
    // 3-D calls; a P with no entries has no tiles and F_attr = 0
    if ((layout->tiles == 0 && layout->nnz > 0) || layout->windows != 0) return BHTSNE_EINVAL;
    if (!Y) return BHTSNE_EINVAL;
    if (!finite_f(theta) || theta < 0.0f) return BHTSNE_EINVAL;
    if (!finite_f(exaggeration) || !(exaggeration > 0.0f)) return BHTSNE_EINVAL;
    return check_ws_3d(layout->n, layout->nnz, workspace, workspace_bytes);
}

int bhtsne_gradient_layout_3d(const float *Y, const bhtsne_layout *layout, float theta, float exaggeration,
                              float *grad, double *Z, void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    int rc = check_layout3_step(layout, Y, theta, exaggeration, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    if (!grad) return BHTSNE_EINVAL;
    StepArgs a{exaggeration, 0.0f, 0.0f, 0.0f, 0};
    return run_layout3(const_cast<float *>(Y), layout, theta, a, nullptr, nullptr, grad, Z, workspace, stream);
}

int bhtsne_step_layout_3d(float *Y, const bhtsne_layout *layout, float theta, float exaggeration,
                          float learning_rate, float momentum, float min_gain, float *update, float *gains,
                          float *grad, double *Z, void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    int rc = check_layout3_step(layout, Y, theta, exaggeration, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    if (!update || !gains) return BHTSNE_EINVAL;
    rc = check_step_args(theta, exaggeration, learning_rate, momentum, min_gain);
    if (rc != BHTSNE_OK) return rc;
    StepArgs a{exaggeration, learning_rate, momentum, min_gain, 1};
    return run_layout3(Y, layout, theta, a, update, gains, grad, Z, workspace, stream);
}

size_t bhtsne_layout_size(int64_t n, int64_t nnz)
{
    if (n < 2 || n > kMaxPoints || nnz < 0) return 0;
    return layout_view(nullptr, n, nnz).bytes;
}

int bhtsne_layout_build(const bhtsne_csr *P, const float *Y, void *layout_mem, size_t layout_bytes,
                        bhtsne_layout *out, void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    return bhtsne_layout_build_ordered(P, Y, BHTSNE_ORDER_AUTO, layout_mem, layout_bytes, out, workspace,
                                       workspace_bytes, stream);
}

int bhtsne_layout_build_ordered(const bhtsne_csr *P, const float *Y, int order, void *layout_mem,
                                size_t layout_bytes, bhtsne_layout *out, void *workspace, size_t workspace_bytes,
                                hipStream_t stream)
{
    static_assert(BHTSNE_ORDER_MORTON == kOrderMorton && BHTSNE_ORDER_BFS == kOrderBfs &&
                      BHTSNE_ORDER_AUTO == kOrderAuto,
                  "the public order codes are the build's");
    if (order != BHTSNE_ORDER_MORTON && order != BHTSNE_ORDER_BFS && order != BHTSNE_ORDER_AUTO)
        return BHTSNE_EINVAL;
    int rc = check_csr(P);
    if (rc != BHTSNE_OK) return rc;
    if (!out || !layout_mem || !aligned(layout_mem)) return BHTSNE_EINVAL;
    if (layout_bytes < bhtsne_layout_size(P->n, P->nnz)) return BHTSNE_EINVAL;
    // padded entries are addressed with int32 offsets
    if (P->nnz + 3 * P->n + 4 >= (int64_t(1) << 31)) return BHTSNE_EINVAL;
    rc = check_ws(P->n, P->nnz, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    const Layout L = make_layout(P->n, P->nnz);
    const LayoutView lv = layout_view(layout_mem, P->n, P->nnz);
    TilePlan plan;
    const int built = launch_layout_build<float, 2>(P->row_ptr, P->col, P->val, P->n, P->nnz, Y, order, lv, &plan,
                                                    workspace, L, stream);
    return finish_layout(built, plan, P->n, P->nnz, layout_mem, layout_bytes, kLayoutMagic, out, workspace, stream);
}

size_t bhtsne_layout_size_f64(int64_t n, int64_t nnz)
{
    if (n < 2 || n > kMaxPoints || nnz < 0) return 0;
    return layout_view(nullptr, n, nnz, 8).bytes;
}

int bhtsne_layout_build_f64(const bhtsne_csr_f64 *P, const double *Y, void *layout_mem, size_t layout_bytes,
                            bhtsne_layout *out, void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    int rc = check_csr_f64(P);
    if (rc != BHTSNE_OK) return rc;
    if (!out || !layout_mem || !aligned(layout_mem)) return BHTSNE_EINVAL;
    if (layout_bytes < bhtsne_layout_size_f64(P->n, P->nnz)) return BHTSNE_EINVAL;
    if (P->nnz + 3 * P->n + 4 >= (int64_t(1) << 31)) return BHTSNE_EINVAL;
    rc = check_ws_f64(P->n, P->nnz, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    const Layout L = make_layout(P->n, P->nnz, 8);
    const LayoutView lv = layout_view(layout_mem, P->n, P->nnz, 8);
    TilePlan plan;
    const int built = launch_layout_build<double, 2>(P->row_ptr, P->col, P->val, P->n, P->nnz, Y, kOrderAuto, lv,
                                                     &plan, workspace, L, stream);
    return finish_layout(built, plan, P->n, P->nnz, layout_mem, layout_bytes, kLayoutMagic64, out, workspace,
                         stream);
}

static int check_layout64_step(const bhtsne_layout *layout, const double *Y, double theta, double exaggeration,
                               void *workspace, size_t workspace_bytes)
{
    int rc = check_layout(layout, 8);
    if (rc != BHTSNE_OK) return rc;
    // neither form (rows out of window order): use the plain fp64 calls
    if (layout->windows == 0 && layout->tiles == 0) return BHTSNE_EINVAL;
    if (!Y) return BHTSNE_EINVAL;
    if (!std::isfinite(theta) || theta < 0.0) return BHTSNE_EINVAL;
    if (!std::isfinite(exaggeration) || !(exaggeration > 0.0)) return BHTSNE_EINVAL;
    return check_ws_f64(layout->n, layout->nnz, workspace, workspace_bytes);
}

int bhtsne_gradient_layout_f64(const double *Y, const bhtsne_layout *layout, double theta, double exaggeration,
                               double *grad, double *Z, void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    int rc = check_layout64_step(layout, Y, theta, exaggeration, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    if (!grad) return BHTSNE_EINVAL;
    StepArgsT<double> a{exaggeration, 0.0, 0.0, 0.0, 0};
    return run_layout64(const_cast<double *>(Y), layout, theta, a, nullptr, nullptr, grad, Z, workspace, stream);
}

int bhtsne_step_layout_f64(double *Y, const bhtsne_layout *layout, double theta, double exaggeration,
                           double learning_rate, double momentum, double min_gain, double *update, double *gains,
                           double *grad, double *Z, void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    int rc = check_layout64_step(layout, Y, theta, exaggeration, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    if (!update || !gains) return BHTSNE_EINVAL;
    if (!std::isfinite(learning_rate) || !(learning_rate > 0.0)) return BHTSNE_EINVAL;
    if (!std::isfinite(momentum) || momentum < 0.0 || !(momentum < 1.0)) return BHTSNE_EINVAL;
    if (!std::isfinite(min_gain) || min_gain < 0.0) return BHTSNE_EINVAL;
    StepArgsT<double> a{exaggeration, learning_rate, momentum, min_gain, 1};
    return run_layout64(Y, layout, theta, a, update, gains, grad, Z, workspace, stream);
}

int bhtsne_gradient_layout(const float *Y, const bhtsne_layout *layout, float theta, float exaggeration, float *grad,
                           double *Z, void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    int rc = check_layout(layout);
    if (rc != BHTSNE_OK) return rc;
    if (!Y || !grad) return BHTSNE_EINVAL;
    if (!finite_f(theta) || theta < 0.0f) return BHTSNE_EINVAL;
    if (!finite_f(exaggeration) || !(exaggeration > 0.0f)) return BHTSNE_EINVAL;
    rc = check_ws(layout->n, layout->nnz, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    StepArgs a{exaggeration, 0.0f, 0.0f, 0.0f, 0};
    return run_layout(const_cast<float *>(Y), layout, theta, a, nullptr, nullptr, grad, Z, workspace, stream);
}

int bhtsne_step_layout(float *Y, const bhtsne_layout *layout, float theta, float exaggeration, float learning_rate,
                       float momentum, float min_gain, float *update, float *gains, float *grad, double *Z,
                       void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    int rc = check_layout(layout);
    if (rc != BHTSNE_OK) return rc;
    if (!Y || !update || !gains) return BHTSNE_EINVAL;
    rc = check_step_args(theta, exaggeration, learning_rate, momentum, min_gain);
    if (rc != BHTSNE_OK) return rc;
    rc = check_ws(layout->n, layout->nnz, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    StepArgs a{exaggeration, learning_rate, momentum, min_gain, 1};
    return run_layout(Y, layout, theta, a, update, gains, grad, Z, workspace, stream);
}

int bhtsne_get_stats(const void *workspace, bhtsne_stats *out, hipStream_t stream)
{
    if (!workspace || !out || !aligned(workspace)) return BHTSNE_EINVAL;
    Header h;
    int rc = read_header(workspace, &h, stream);
    if (rc != BHTSNE_OK) return rc;
    out->Z = h.Z;
    out->interactions = int64_t(h.interactions);
    out->nodes = int64_t(h.nodes);
    out->bbox[0] = h.bmin[0];
    out->bbox[1] = h.bmax[0];
    out->bbox[2] = h.bmin[1];
    out->bbox[3] = h.bmax[1];
    out->r_span = h.rspan;
    out->device_flags = h.flags;
    out->max_depth = int32_t(h.max_depth);
    return flags_status(h.flags);
}

size_t bhtsne_affinities_workspace_size(int64_t n, int32_t k)
{
    if (n < 2 || n > kMaxPoints || k < 1 || k > kAffMaxK || int64_t(k) >= n) return 0;
    return make_aff_layout(n, k).total;
}

int bhtsne_affinities(const int32_t *knn_idx, const float *knn_dist, int64_t n, int32_t k, double perplexity,
                      int64_t *row_ptr, int32_t *col, float *val, int64_t capacity, int64_t *nnz, double *sigma2,
                      void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    if (!knn_idx || !knn_dist || !row_ptr || !nnz || capacity < 0) return BHTSNE_EINVAL;
    if (capacity > 0 && (!col || !val)) return BHTSNE_EINVAL;
    if (!std::isfinite(perplexity) || !(perplexity > 0.0)) return BHTSNE_EINVAL;
    const size_t need = bhtsne_affinities_workspace_size(n, k);
    if (need == 0) return BHTSNE_EINVAL;
    if (!workspace || !aligned(workspace) || workspace_bytes < need) return BHTSNE_EWORKSPACE;
    const AffLayout A = make_aff_layout(n, k);
    launch_aff_clear(workspace, A, stream);
    // the index work and the search share the chip poorly (the search keeps
    // the VALU busy, the sort passes then wait for wave slots), so they run
    // one after the other
    launch_aff_index(knn_idx, n, k, row_ptr, workspace, A, stream);
    launch_aff_search(knn_dist, n, k, perplexity, sigma2, workspace, A, stream);
    if (hipGetLastError() != hipSuccess) return BHTSNE_EDEVICE;
    Header h;
    int64_t total = 0;
    if (hipMemcpyAsync(&total, row_ptr + n, sizeof(total), hipMemcpyDeviceToHost, stream) != hipSuccess)
        return BHTSNE_EDEVICE;
    int rc = read_header(static_cast<char *>(workspace) + A.header, &h, stream);
    if (rc != BHTSNE_OK) return rc;
    if (h.flags & kErrNonFinite) return BHTSNE_ENONFINITE;
    if (h.flags & kErrRange) return BHTSNE_EINPUT;
    if (h.flags) return BHTSNE_EDEVICE;
    *nnz = total;
    if (total > capacity) return BHTSNE_ECAPACITY;
    launch_aff_back(n, k, row_ptr, col, val, workspace, A, stream);
    if (hipGetLastError() != hipSuccess) return BHTSNE_EDEVICE;
    rc = read_header(static_cast<char *>(workspace) + A.header, &h, stream);
    if (rc != BHTSNE_OK) return rc;
    if (h.flags & kErrRange) return BHTSNE_EINPUT;
    return h.flags ? BHTSNE_EDEVICE : BHTSNE_OK;
}

const char *bhtsne_status_string(int status)
{
    switch (status) {
    case BHTSNE_OK: return "ok";
    case BHTSNE_EINVAL: return "invalid argument";
    case BHTSNE_EWORKSPACE: return "workspace missing, misaligned or too small";
    case BHTSNE_ENONFINITE: return "non-finite coordinate in Y";
    case BHTSNE_EDEVICE: return "HIP error or device-side consistency failure";
    case BHTSNE_EINPUT: return "invalid input data found on the GPU (malformed CSR row pointers, or neighbour lists with an index out of range, repeated or the point itself, or a point listed by more than 4096 others)";
    case BHTSNE_ECAPACITY: return "output arrays too small (the required entry count is returned)";
    default: return "unknown status";
    }
}

int bhtsne_timing_enable(int enable)
{
    Timing &t = timing();
    std::lock_guard<std::mutex> g(t.mu);
    t.enabled = enable != 0;
    return BHTSNE_OK;
}

int bhtsne_timing_phases(uint32_t phase_mask)
{
    if (phase_mask >> BHTSNE_NUM_PHASES) return BHTSNE_EINVAL;
    Timing &t = timing();
    std::lock_guard<std::mutex> g(t.mu);
    t.phases = phase_mask;
    return BHTSNE_OK;
}

int bhtsne_timing_read(bhtsne_timing *out, int reset)
{
    if (!out) return BHTSNE_EINVAL;
    Timing &t = timing();
    std::lock_guard<std::mutex> g(t.mu);
    int rc = BHTSNE_OK;
    for (auto &p : t.pending) {
        float ms = 0.0f;
        if (hipEventSynchronize(p.b) != hipSuccess || hipEventElapsedTime(&ms, p.a, p.b) != hipSuccess)
            rc = BHTSNE_EDEVICE;
        t.ms[p.phase] += ms;
        t.count[p.phase] += 1;
        t.pool.push_back(p.a);
        t.pool.push_back(p.b);
    }
    t.pending.clear();
    for (int k = 0; k < BHTSNE_NUM_PHASES; ++k) {
        out->ms[k] = t.ms[k];
        out->count[k] = t.count[k];
        if (reset) {
            t.ms[k] = 0.0;
            t.count[k] = 0;
        }
    }
    return rc;
}

int bhtsne_debug_sort(const float *Y, int64_t n, uint64_t *codes, uint64_t *sorted_codes, uint32_t *perm,
                      double *params, void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    if (!Y || n < 2 || n > kMaxPoints) return BHTSNE_EINVAL;
    int rc = check_ws(n, 0, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    const Layout L = make_layout(n, 0);
    launch_bbox(Y, n, workspace, L, stream);
    launch_morton(Y, n, nullptr, workspace, L, stream);
    if (codes && hipMemcpyAsync(codes, at<void>(workspace, L.codes0), 8 * size_t(n), hipMemcpyDeviceToDevice,
                                stream) != hipSuccess)
        return BHTSNE_EDEVICE;
    launch_sort(n, Y, workspace, L, stream);
    if (sorted_codes && hipMemcpyAsync(sorted_codes, at<void>(workspace, L.codes0), 8 * size_t(n),
                                       hipMemcpyDeviceToDevice, stream) != hipSuccess)
        return BHTSNE_EDEVICE;
    if (perm && hipMemcpyAsync(perm, at<void>(workspace, L.idx0), 4 * size_t(n), hipMemcpyDeviceToDevice,
                               stream) != hipSuccess)
        return BHTSNE_EDEVICE;
    if (hipGetLastError() != hipSuccess) return BHTSNE_EDEVICE;
    if (params) {
        Header h;
        rc = read_header(workspace, &h, stream);
        if (rc != BHTSNE_OK) return rc;
        double p[10] = {h.bmin[0], h.bmax[0], h.bmin[1], h.bmax[1], h.cent[0],
                        h.cent[1], h.rspan,   h.yroot[0], h.yroot[1], h.scale};
        std::memcpy(params, p, sizeof(p));
        return flags_status(h.flags);
    }
    return BHTSNE_OK;
}

int bhtsne_z_exact(const float *Y, int64_t n, double *Z, void *workspace, size_t workspace_bytes, hipStream_t stream)
{
    if (!Y || !Z || n < 2 || n > kMaxPoints) return BHTSNE_EINVAL;
    int rc = check_ws(n, 0, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    const Layout L = make_layout(n, 0);
    launch_z_exact(Y, n, workspace, L, stream);
    if (hipGetLastError() != hipSuccess) return BHTSNE_EDEVICE;
    Header h;
    rc = read_header(workspace, &h, stream);
    if (rc != BHTSNE_OK) return rc;
    *Z = h.eval;
    if (!std::isfinite(h.eval)) return BHTSNE_ENONFINITE;
    return flags_status(h.flags);
}

int bhtsne_kl(const float *Y, const bhtsne_csr *P, double Z, double *kl, void *workspace, size_t workspace_bytes,
              hipStream_t stream)
{
    if (!Y || !kl) return BHTSNE_EINVAL;
    int rc = check_csr(P);
    if (rc != BHTSNE_OK) return rc;
    if (!std::isfinite(Z) || !(Z > 0.0)) return BHTSNE_EINVAL;
    rc = check_ws(P->n, 0, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    const Layout L = make_layout(P->n, 0);
    launch_kl(Y, P->row_ptr, P->col, P->val, P->n, P->nnz, std::log(Z), workspace, L, stream);
    if (hipGetLastError() != hipSuccess) return BHTSNE_EDEVICE;
    Header h;
    rc = read_header(workspace, &h, stream);
    if (rc != BHTSNE_OK) return rc;
    *kl = h.eval;
    if (!std::isfinite(h.eval)) return BHTSNE_ENONFINITE;
    return flags_status(h.flags);
}

int bhtsne_debug_tree(const float *Y, int64_t n, float theta, int64_t *n_nodes, uint8_t *level, uint8_t *kind,
                      uint32_t *begin, uint32_t *end, float *summary, uint32_t *meta, void *workspace,
                      size_t workspace_bytes, hipStream_t stream)
{
    if (!Y || !n_nodes || n < 2 || n > kMaxPoints) return BHTSNE_EINVAL;
    if (!finite_f(theta) || theta < 0.0f) return BHTSNE_EINVAL;
    if ((level || kind || begin || end) && !(level && kind && begin && end)) return BHTSNE_EINVAL;
    int rc = check_ws(n, 0, workspace, workspace_bytes);
    if (rc != BHTSNE_OK) return rc;
    const Layout L = make_layout(n, 0);
    TreeDebug dbg;
    dbg.level = level;
    dbg.kind = kind;
    dbg.begin = begin;
    dbg.end = end;
    build_tree(Y, n, theta, nullptr, workspace, L, dbg, stream);
    if (summary || meta) launch_tree_unpack(n, workspace, L, summary, meta, stream);
    if (hipGetLastError() != hipSuccess) return BHTSNE_EDEVICE;
    Header h;
    rc = read_header(workspace, &h, stream);
    if (rc != BHTSNE_OK) return rc;
    *n_nodes = int64_t(h.nodes);
    return flags_status(h.flags);
}

} // extern "C"
