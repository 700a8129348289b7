/*
 * bhtsne.h - C ABI of the MI355X (gfx950) Barnes-Hut t-SNE gradient library.
 *
 * One call computes the gradient of the t-SNE cost for a 2-D embedding Y and a
 * sparse symmetric affinity matrix P, following the paper's per-iteration
 * steps (Background, "Brief overview of the Barnes Hut t-SNE Algorithm"):
 * quadtree building, summarization, attractive forces and repulsive forces,
 * then the gradient (Gradient Descent, split-gradient equation)
 *
 *     dC/dy_i = 4 (alpha F_attr,i - F_rep,i / Z)
 *     F_attr,i = sum_j p_ij (1 + |y_i - y_j|^2)^-1 (y_i - y_j)     (Algorithm 2)
 *     F_rep,i  ~ sum_j (1 + |y_i - y_j|^2)^-2 (y_i - y_j)         (Barnes-Hut)
 *     Z        ~ sum_{k != l} (1 + |y_k - y_l|^2)^-1                (q_ij definition)
 *
 * where the repulsive sums and Z are Barnes-Hut approximations: a quadtree
 * cell of side s whose centre of mass c lies at distance d from y_i stands in
 * for all of its points when s^2 < theta^2 d^2 (Repulsive Force Computation;
 * the cell "radius" read as the side of the square cell).  theta = 0 gives the
 * exact O(N^2) sums.  alpha is the early-exaggeration factor; it scales P.
 *
 * Conventions shared by every entry point:
 *  - Arrays named as device arrays are device pointers on the GPU that is
 *    current when the call is made; they stay owned by the caller.  The
 *    library never allocates or frees device memory: all scratch space is
 *    the caller's `workspace` (bhtsne_workspace_size bytes, 256-byte aligned).
 *  - Y, grad, update and gains are n x 2 float32, row-major ((x, y) per point).
 *  - All work is enqueued on `stream`; a call returns before it completes
 *    unless it must return a host value (Z or a node count), in which case it
 *    synchronises the stream first.  Calls that share a workspace must be
 *    ordered (same stream); distinct workspaces may run concurrently.
 *  - The gradient and step calls (plain and layout forms, fp32 and fp64)
 *    can be captured in a HIP graph when they return no host value: they
 *    allocate nothing, enqueue no memset (counters are cleared by kernels),
 *    and the layout forms' second stream joins the capture through the
 *    fork and join events.  Each replay recomputes the whole step.
 *  - Every call returns a bhtsne_status code and never throws.  Arguments are
 *    checked on the host before anything is enqueued; nothing is enqueued when
 *    a check fails.  Conditions found on the GPU (a non-finite coordinate, a
 *    corrupted intermediate) are latched in the workspace; they are reported
 *    by calls that synchronise and by bhtsne_get_stats.
 */
#ifndef BHTSNE_H
#define BHTSNE_H

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BHTSNE_OK = 0,
    BHTSNE_EINVAL = -1,     /* an argument failed a host-side check */
    BHTSNE_EWORKSPACE = -2, /* workspace missing, misaligned or too small */
    BHTSNE_ENONFINITE = -3, /* Y held a NaN or an infinity */
    BHTSNE_EDEVICE = -4,    /* a HIP call failed or the GPU flagged an internal error */
    BHTSNE_EINPUT = -5,     /* the GPU found invalid input data (bhtsne_affinities, bhtsne_layout_build) */
    BHTSNE_ECAPACITY = -6   /* output arrays too small; the required size is returned */
} bhtsne_status;

/* Sparse symmetric P in CSR form (0-based columns).  Expected, not checked:
 * p_ij = p_ji >= 0, p_ii = 0, sum p = 1 (Background, "Input similarity
 * computation").  row_ptr is non-decreasing with row_ptr[0] = 0 and
 * row_ptr[n] = nnz; columns outside [0, n) and entries outside [0, nnz) are
 * skipped on the GPU and flagged as a device error. */
typedef struct bhtsne_csr {
    int64_t n;              /* points; 2 <= n <= 16777215 */
    int64_t nnz;            /* stored entries, >= 0 */
    const int64_t *row_ptr; /* device, n + 1 entries */
    const int32_t *col;     /* device, nnz entries (may be NULL when nnz == 0) */
    const float *val;       /* device, nnz entries (may be NULL when nnz == 0) */
} bhtsne_csr;

/* A locality layout of P: a relabelled copy that speeds up the attractive
 * forces (Attractive Force Computation).  The struct is a host-side handle
 * filled by bhtsne_layout_build; `mem` is caller-owned device memory of at
 * least bhtsne_layout_size bytes that holds the copy. */
typedef struct bhtsne_layout {
    int64_t n, nnz;
    void *mem;
    size_t bytes;
    int64_t tiles;  /* tiles of the (row block x column segment) copy; 0 = row-block path */
    int64_t items;  /* work items of the tiled kernel (runs of tiles sharing a segment) */
    int64_t entries; /* entries of the sliced copy, padding included (0 without tiles) */
    int64_t windows; /* column windows of the windowed row segments (0 = none; only without tiles) */
    int64_t segments; /* (row, window) segments of that form */
    int64_t order;   /* point order of the copy: BHTSNE_ORDER_MORTON or BHTSNE_ORDER_BFS */
    uint64_t magic;
} bhtsne_layout;

/* Point orders of a layout, within each connected component of P's graph
 * (bhtsne_layout_build_ordered). */
enum {
    BHTSNE_ORDER_MORTON = 0, /* Morton code of Y (index order when Y is NULL) */
    BHTSNE_ORDER_BFS = 1,    /* breadth-first level from the component's root (its smallest point),
                                then index */
    BHTSNE_ORDER_AUTO = 2    /* Morton; the BFS levels when Morton gives no tiles and they do */
};

/* Scalars of the last call on a workspace (bhtsne_get_stats). */
typedef struct bhtsne_stats {
    double Z;             /* normaliser (ordered pairs) */
    int64_t interactions; /* accepted cell summaries + exact point pairs */
    int64_t nodes;        /* nodes of the compressed quadtree */
    double bbox[4];       /* min x, max x, min y, max y */
    double r_span;        /* half side of the square domain */
    uint32_t device_flags;/* 1 non-finite input, 2 look-back timeout, 4 index out of range */
    int32_t max_depth;    /* deepest leaf of the quadtree: the level of the deepest single-point
                             leaf, or 32 when identical points form a bucket (Quadtree Building:
                             a cell at level L has side 2 r_span 2^-L) */
} bhtsne_stats;

/* Kernel phases timed by bhtsne_timing_*. */
enum {
    BHTSNE_PHASE_BBOX_MORTON = 0, /* bounding box + Morton codes */
    BHTSNE_PHASE_SORT = 1,        /* radix sort of the codes + gather of Y */
    BHTSNE_PHASE_TREE = 2,        /* quadtree build + summaries */
    BHTSNE_PHASE_REPULSIVE = 3,   /* Barnes-Hut traversal + Z */
    BHTSNE_PHASE_ATTRACTIVE = 4,  /* attractive forces (plain CSR: with the gradient + update) */
    BHTSNE_PHASE_UPDATE = 5,      /* gradient + update of the layout calls */
    BHTSNE_NUM_PHASES = 6
};

typedef struct bhtsne_timing {
    double ms[BHTSNE_NUM_PHASES];   /* summed GPU time per phase (hipEvent pairs on the phase's stream) */
    int64_t count[BHTSNE_NUM_PHASES];
} bhtsne_timing;

/* Bytes of workspace needed for n points and nnz entries (0 if n is out of
 * range).  Pure host arithmetic; the same value for every call with these
 * sizes. */
size_t bhtsne_workspace_size(int64_t n, int64_t nnz);

/* Gradient of the t-SNE cost at Y (see the top of this file).
 *   Y      device, n x 2, read only.
 *   P      host struct describing the device CSR arrays; P->n is n.
 *   theta  Barnes-Hut angle, finite, >= 0 (0 = exact).
 *   exaggeration  alpha, finite, > 0.
 *   grad   device, n x 2, written.
 *   Z      host, nullable: when given, the stream is synchronised and the
 *          normaliser is stored; device flags are then checked as well.
 * Errors: BHTSNE_EINVAL (bad argument), BHTSNE_EWORKSPACE, BHTSNE_ENONFINITE,
 * BHTSNE_EDEVICE. */
int bhtsne_gradient(const float *Y, const bhtsne_csr *P, float theta, float exaggeration, float *grad,
                    double *Z, void *workspace, size_t workspace_bytes, hipStream_t stream);

/* One gradient-descent iteration in place: the gradient as above, then per
 * coordinate (the delta-bar-delta gains of the usual t-SNE optimiser; the
 * paper only states that the experiments keep scikit-learn's defaults,
 * Experimental setup)
 *     gain = (u * g < 0) ? gain + 0.2 : gain * 0.8;  gain = max(gain, min_gain)
 *     u    = momentum * u - learning_rate * gain * g
 *     y    = y + u
 *   Y       device, n x 2, read and overwritten with the new embedding.
 *   update  device, n x 2, momentum buffer u (zero before the first step).
 *   gains   device, n x 2 (one before the first step).
 *   grad    device, n x 2, nullable: the gradient at the old Y.
 *   learning_rate finite > 0; momentum in [0, 1); min_gain finite >= 0.
 * Other arguments and errors as bhtsne_gradient. */
int bhtsne_step(float *Y, const bhtsne_csr *P, float theta, float exaggeration, float learning_rate,
                float momentum, float min_gain, float *update, float *gains, float *grad, double *Z,
                void *workspace, size_t workspace_bytes, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation):
 * bhtsne_step with no workspace argument.  Its scratch space is a fixed
 * array of bhtsne_noalloc_max_bytes() bytes (64 MiB) in the library's device
 * image, one per GPU, reserved when the library is loaded and held until the
 * process ends; the call allocates nothing.  Sizes whose
 * bhtsne_workspace_size(n, nnz) exceeds it (n above about 168,000 points)
 * are BHTSNE_EINVAL.  Every call on a GPU shares that GPU's array: calls
 * that may overlap on one GPU (different streams or threads) race and must
 * be serialised by the caller; the kernels clear every counter they need,
 * so what a previous call left in the array does not matter.  Arguments,
 * results and other errors as bhtsne_step (plain CSR P). */
size_t bhtsne_noalloc_max_bytes(void);
int bhtsne_step_noalloc(float *Y, const bhtsne_csr *P, float theta, float exaggeration, float learning_rate,
                        float momentum, float min_gain, float *update, float *gains, float *grad, double *Z,
                        hipStream_t stream);

/* Bytes of device memory a layout of P needs (0 if n or nnz is out of range):
 * about 15.5 bytes per stored entry + 700 bytes per point (a row-sorted copy,
 * and room for a sliced copy with 16-bit column offsets and its tables). */
size_t bhtsne_layout_size(int64_t n, int64_t nnz);

/* Build a locality layout of P (once per matrix; may be rebuilt as Y evolves).
 * Points are renumbered by (connected component of P's graph, Morton code of
 * Y), or by the component's breadth-first levels when those give tiles and
 * the Morton order does not (bhtsne_layout_build_ordered, BHTSNE_ORDER_AUTO);
 * the copy stores P's rows in that order with renumbered columns, so the
 * columns of consecutive rows fall into compact index windows.  When every
 * block of 1024 rows spans at most 16 windows of 16384 columns, or at most
 * 128 with at most 32 tiles per row block on average holding at least 4096
 * entries each on average (the rows of large clusters), a second, sliced
 * copy is built: for each (row block, window) tile the rows are sorted by
 * their number of entries in the window and cut into slices of 64 rows,
 * stored entry-major, so that one window of Y in LDS serves many tiles and
 * every load is contiguous (out->tiles > 0, out->items > 0).  The copy is
 * skipped when its padding would exceed a quarter of nnz plus one chunk per
 * slice of 16 tiles per row block.  Without that copy (rows whose neighbours
 * spread sparsely over a large component), the build lists instead, for each column window of 2^18
 * points, the (row, entry range) segments of the rows with entries there
 * (out->windows > 0; out->segments = 0 for a P with no entries): the
 * attraction then takes one pass per window, with that window of Y held in
 * the L2 caches.  The gradient does not depend on the order; only the speed of the
 * attractive step does.
 *   P      the matrix (as for bhtsne_gradient; nnz < 2^31).
 *   Y      device, n x 2, nullable: without it points keep their index order
 *          inside a component.
 *   layout_mem, layout_bytes  caller device memory (256-byte aligned).
 *   out    host handle, filled on success.
 *   workspace  as for bhtsne_gradient (its contents are overwritten).
 * Synchronises the stream (the component search iterates until no label
 * changes).  P's row pointers are checked on the GPU before any entry is read
 * (row_ptr[0] = 0, non-decreasing, row_ptr[n] = nnz); a violation returns
 * BHTSNE_EINPUT and builds nothing.  Columns outside [0, n) are kept out of
 * the copy.  Errors: BHTSNE_EINVAL, BHTSNE_EWORKSPACE, BHTSNE_EINPUT,
 * BHTSNE_EDEVICE. */
int bhtsne_layout_build(const bhtsne_csr *P, const float *Y, void *layout_mem, size_t layout_bytes,
                        bhtsne_layout *out, void *workspace, size_t workspace_bytes, hipStream_t stream);

/* bhtsne_layout_build with the point order chosen by the caller; the plain
 * call is this one with BHTSNE_ORDER_AUTO.  The Morton order brings a row's
 * columns together when Y already reflects P (after the first iterations);
 * the breadth-first levels do when P itself has locality, whatever Y is (a
 * kNN graph of points on a low-dimensional set, from a random initial Y):
 * the neighbours of a point at level l lie at levels l - 1 to l + 1.  The
 * search runs from every component's root at once, one host synchronisation
 * per level; it gives up, and the Morton order is used, when a level holds
 * more than 65536 points or some point lies more than 16383 levels deep.
 * BHTSNE_ORDER_AUTO builds the Morton order first and, when that gives no
 * tiles, tries the levels, keeping whichever tiles (the Morton order if
 * neither does).  out->order reports the order taken.  Errors as
 * bhtsne_layout_build, and BHTSNE_EINVAL for another order code. */
int bhtsne_layout_build_ordered(const bhtsne_csr *P, const float *Y, int order, void *layout_mem,
                                size_t layout_bytes, bhtsne_layout *out, void *workspace, size_t workspace_bytes,
                                hipStream_t stream);

/* bhtsne_gradient / bhtsne_step taking P through a layout built by
 * bhtsne_layout_build (the original CSR arrays are not read).  Arguments,
 * outputs (in the caller's point order) and errors as the plain calls;
 * BHTSNE_EINVAL also for a handle that bhtsne_layout_build did not fill.
 * The attractive forces run on a stream the library keeps per device (default
 * priority), forked from `stream` after the Morton codes and joined back
 * before the gradient assembly, so they overlap the sort, tree and repulsive
 * phases; to the caller the call is ordered on `stream` as usual.  The
 * device is the current one, which must be the device of `stream`.  The
 * environment variable BHTSNE_FORK = 1 or 2 (read once) forks them after the
 * sort or the tree instead, and BHTSNE_OVERLAP = 0 keeps them on `stream`;
 * the results are the same bit for bit. */
int bhtsne_gradient_layout(const float *Y, const bhtsne_layout *layout, float theta, float exaggeration,
                           float *grad, double *Z, void *workspace, size_t workspace_bytes, hipStream_t stream);
int bhtsne_step_layout(float *Y, const bhtsne_layout *layout, float theta, float exaggeration, float learning_rate,
                       float momentum, float min_gain, float *update, float *gains, float *grad, double *Z,
                       void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Copy the scalars of the last call on `workspace` to *out; synchronises
 * `stream`.  Returns BHTSNE_ENONFINITE / BHTSNE_EDEVICE when the last call
 * latched a device flag (the stats are still filled in). */
int bhtsne_get_stats(const void *workspace, bhtsne_stats *out, hipStream_t stream);

/* Static English text for a status code. */
const char *bhtsne_status_string(int status);

/* Per-phase GPU timing.  While enabled, every later call records a hipEvent
 * pair around each selected phase on its stream (process-wide switch, thread
 * safe).  bhtsne_timing_read waits for the recorded events, returns the summed
 * milliseconds per phase, and with reset != 0 starts a new accumulation.
 * bhtsne_timing_phases selects the phases by bit (1 << BHTSNE_PHASE_*; all by
 * default): each event is a timestamp packet between two kernels, a few
 * microseconds of GPU time, so a throughput measurement times only the phases
 * it needs.  A mask with bits at or above BHTSNE_NUM_PHASES is BHTSNE_EINVAL. */
int bhtsne_timing_enable(int enable);
int bhtsne_timing_phases(uint32_t phase_mask);
int bhtsne_timing_read(bhtsne_timing *out, int reset);

/* Cost evaluation (Background: the KL divergence of P and Q), outside an
 * iteration; a run calls it to report its cost.  Both calls clear the device
 * flags of the workspace like a step, synchronise the stream and return their
 * result on the host.
 *
 * bhtsne_z_exact: the exact normaliser of q_ij, Z = sum over ordered pairs
 * i != j of (1 + |y_i - y_j|^2)^-1, over all n^2 pairs (fp32 pair terms, fp64
 * accumulation in a fixed order, so the result is reproducible).  Y: device,
 * n x 2 fp32; Z: host.  The workspace is sized as for
 * bhtsne_workspace_size(n, 0) or larger.  A non-finite result is
 * BHTSNE_ENONFINITE.
 *
 * bhtsne_kl: KL(P || Q) = sum over the stored entries with p_ij > 0 of
 * p_ij log(p_ij / q_ij), q_ij = (1 + |y_i - y_j|^2)^-1 / Z, for a given
 * Z > 0 (the exact one, or a step's Barnes-Hut estimate), in fp64 from the
 * fp32 inputs.  A column outside [0, n), or a row whose pointers reach outside
 * [0, nnz), is skipped (clamped) and reported as BHTSNE_EDEVICE. */
int bhtsne_z_exact(const float *Y, int64_t n, double *Z, void *workspace, size_t workspace_bytes,
                   hipStream_t stream);
int bhtsne_kl(const float *Y, const bhtsne_csr *P, double Z, double *kl, void *workspace, size_t workspace_bytes,
              hipStream_t stream);

/* Test export: bounding box, Morton codes and their sort (Quadtree Building,
 * Algorithm 1).  codes (original order), sorted_codes and perm (sorted
 * position -> original index) are device arrays of n entries, each nullable.
 * params is a host array of 10 doubles {min x, max x, min y, max y, cent x,
 * cent y, r_span, y_root x, y_root y, scale}, nullable; when given the
 * stream is synchronised. */
int bhtsne_debug_sort(const float *Y, int64_t n, uint64_t *codes, uint64_t *sorted_codes, uint32_t *perm,
                      double *params, void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Test export: the compressed quadtree and its summaries (Quadtree Building,
 * Parallel Summarization) in depth-first pre-order, i.e. sorted by (begin,
 * level).  Device arrays of 2n entries (summary: 2n x 4 floats {com x, com y,
 * count, threshold}), each nullable; *n_nodes (host, required) receives the
 * node count after a stream synchronisation.  kind: 0 internal, 1 bucket of
 * identical codes (level 32), 2 single point.  Every point has its own
 * single-point node; a bucket's points follow it as its children, at level
 * 33.  meta: skip index, the first node past the subtree (internal nodes and
 * buckets), or begin | 0xC0000000 (single points); threshold: -1 for single
 * points, else side^2 / theta^2. */
int bhtsne_debug_tree(const float *Y, int64_t n, float theta, int64_t *n_nodes, uint8_t *level, uint8_t *kind,
                      uint32_t *begin, uint32_t *end, float *summary, uint32_t *meta, void *workspace,
                      size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Input similarities (Background, "Input similarity computation": the sparse
 * approximation of p_{j|i} over the k nearest neighbours and the
 * symmetrisation p_ij = (p_{j|i} + p_{i|j}) / (2N); Binary Search
 * Perplexity).  For every point i, sigma_i^2 is found by bisection (the middle
 * point of the current interval each step, run to machine precision in fp64)
 * so that the perplexity exp(H) of
 *     p_{j|i} = exp(-d_ij^2 / 2 sigma_i^2) / sum_l exp(-d_il^2 / 2 sigma_i^2)
 * equals `perplexity`; then P is symmetrised over the union of the neighbour
 * relations in both directions.  With perplexity > k the row ends uniform
 * (sigma^2 = +inf); at or below the number of ties at the minimum distance it
 * ends uniform over those ties.
 *
 * knn_idx   [n * k] int32, device: row i lists k distinct neighbours of i (any
 *           order, none equal to i, all in [0, n)).
 * knn_dist  [n * k] float32, device: the matching distances (not squared),
 *           finite and >= 0.
 * row_ptr   [n + 1] int64, device, written: the CSR row pointers of P.
 * col, val  [capacity] device, written: columns (sorted within each row) and
 *           fp32 values of P; nullable when capacity == 0.
 * nnz       host out: the entry count of P (between n k and 2 n k), also
 *           when the call fails with BHTSNE_ECAPACITY, so the caller can size
 *           col and val and call again.
 * sigma2    [n] fp64, device, nullable: sigma_i^2.
 * Limits: 1 <= k <= 256, k < n <= 16777215; at most 4096 points may list
 * the same point.
 * The call synchronises `stream` twice (to learn nnz, then to report).
 * Errors: BHTSNE_EINVAL (arguments), BHTSNE_EWORKSPACE, BHTSNE_ENONFINITE (a
 * NaN, infinite or negative distance), BHTSNE_EINPUT (a neighbour index out of
 * range, equal to its row or repeated within a row, or a point listed by
 * more than 4096 others; col and val then hold no usable result), BHTSNE_ECAPACITY,
 * BHTSNE_EDEVICE.  The library allocates nothing. */
size_t bhtsne_affinities_workspace_size(int64_t n, int32_t k);
int bhtsne_affinities(const int32_t *knn_idx, const float *knn_dist, int64_t n, int32_t k, double perplexity,
                      int64_t *row_ptr, int32_t *col, float *val, int64_t capacity, int64_t *nnz, double *sigma2,
                      void *workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * The fp64 variant of the gradient step (the paper's default precision; its
 * supplementary fp32/fp64 comparison).  Same method, phases and readings as
 * bhtsne_gradient / bhtsne_step on a plain CSR P, with fp64 coordinates,
 * probabilities, tree centres and thresholds, forces, Z and optimiser state;
 * the Morton codes quantise the fp64 coordinates.  Y, grad, update, gains are
 * n x 2 row-major fp64 device arrays; P's values are fp64.  Its workspace
 * size is bhtsne_workspace_size_f64 (larger than the fp32 one: fp64 copies
 * of Y, 40-byte node records).  Same argument checks and errors as the fp32
 * calls (theta, exaggeration, learning_rate, momentum and min_gain are
 * doubles).  Its locality layout (bhtsne_layout_build_f64) follows below. */
typedef struct bhtsne_csr_f64 {
    int64_t n;              /* points; 2 <= n <= 16777215 */
    int64_t nnz;            /* stored entries, >= 0 */
    const int64_t *row_ptr; /* device, n + 1 entries */
    const int32_t *col;     /* device, nnz entries (may be NULL when nnz == 0) */
    const double *val;      /* device, nnz entries (may be NULL when nnz == 0) */
} bhtsne_csr_f64;

size_t bhtsne_workspace_size_f64(int64_t n, int64_t nnz);
int bhtsne_gradient_f64(const double *Y, const bhtsne_csr_f64 *P, double theta, double exaggeration, double *grad,
                        double *Z, void *workspace, size_t workspace_bytes, hipStream_t stream);
int bhtsne_step_f64(double *Y, const bhtsne_csr_f64 *P, double theta, double exaggeration, double learning_rate,
                    double momentum, double min_gain, double *update, double *gains, double *grad, double *Z,
                    void *workspace, size_t workspace_bytes, hipStream_t stream);

/* A locality layout for the fp64 variant (Attractive Force Computation: the
 * y_j reads of a row are what bound it).  bhtsne_layout_build_f64 renumbers
 * the points as bhtsne_layout_build does (BHTSNE_ORDER_AUTO: connected
 * component, then Morton order of the fp64 Y when given, or the breadth-first
 * levels when only those tile) and stores P's rows in that order with fp64
 * values and sorted columns.  It then builds the sliced copy as the fp32 build
 * does, with fp64 values over column windows of 8192 points (128 KB of fp64 Y
 * in LDS) and at most 32 tiles per block of 1024 rows (out->tiles > 0);
 * without it, the (row, entry range) segments of each column window of 2^18
 * points (out->windows > 0; out->segments > 0 unless P has no entries).  A row longer than 4096
 * entries keeps its order, which rules out the sliced copy and, with more
 * than one column window, the segments (out->tiles = out->windows = 0); such
 * a layout is refused by the two calls below (BHTSNE_EINVAL): use the plain
 * fp64 calls.  The workspace is bhtsne_workspace_size_f64; layout memory is
 * bhtsne_layout_size_f64 bytes.  The handle is tagged as an fp64 layout: the
 * fp32 layout calls refuse it, and these calls refuse an fp32 one.
 * bhtsne_gradient_layout_f64 / bhtsne_step_layout_f64 are bhtsne_gradient_f64
 * / bhtsne_step_f64 taking P through such a layout: the attraction runs on
 * the library's second stream beside the walk (BHTSNE_FORK64 = 0 or 1 forks
 * it after the codes or the sort instead); results come back in the caller's
 * order.  Errors as the plain fp64 calls, and
 * BHTSNE_EINPUT from the build for malformed row pointers. */
size_t bhtsne_layout_size_f64(int64_t n, int64_t nnz);
int bhtsne_layout_build_f64(const bhtsne_csr_f64 *P, const double *Y, void *layout_mem, size_t layout_bytes,
                            bhtsne_layout *out, void *workspace, size_t workspace_bytes, hipStream_t stream);
int bhtsne_gradient_layout_f64(const double *Y, const bhtsne_layout *layout, double theta, double exaggeration,
                               double *grad, double *Z, void *workspace, size_t workspace_bytes, hipStream_t stream);
int bhtsne_step_layout_f64(double *Y, const bhtsne_layout *layout, double theta, double exaggeration,
                           double learning_rate, double momentum, double min_gain, double *update, double *gains,
                           double *grad, double *Z, void *workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Three-dimensional embeddings (the problem statement allows a two- or
 * three-dimensional embedding; the paper works the method out in 2-D).  The
 * same method, readings and phases as bhtsne_gradient / bhtsne_step on a
 * plain CSR P, carried to three dimensions:
 *  - the domain is the cube centred on the bounding box whose half side
 *    r_span is the widest half extent;
 *  - each coordinate is quantised to 21 bits, trunc((y - y_root) 2^20 /
 *    r_span) clamped to [0, 2^21 - 1] (fp64), and bit k of dimension d goes
 *    to bit 3k + d of a 63-bit Morton code;
 *  - the compressed octree has cells at levels 0..21 of side 2 r_span 2^-L
 *    (identical codes form a bucket at level 21, whose points follow it one
 *    level below), and a cell stands in for its points when
 *    side^2 < theta^2 |y_i - c|^2;
 *  - Y, grad, update and gains are n x 3 float32, row-major (x, y, z).
 * The workspace is bhtsne_workspace_size_3d bytes.  Arguments, checks,
 * synchronisation and errors as the 2-D calls; bhtsne_get_stats reports Z,
 * the interaction and node counts and max_depth (bbox and r_span hold x, y
 * and the cube's r_span). */
size_t bhtsne_workspace_size_3d(int64_t n, int64_t nnz);
int bhtsne_gradient_3d(const float *Y, const bhtsne_csr *P, float theta, float exaggeration, float *grad,
                       double *Z, void *workspace, size_t workspace_bytes, hipStream_t stream);
int bhtsne_step_3d(float *Y, const bhtsne_csr *P, float theta, float exaggeration, float learning_rate,
                   float momentum, float min_gain, float *update, float *gains, float *grad, double *Z,
                   void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Locality layout for 3-D embeddings: the relabelled copy of P and its sliced
 * copy, as bhtsne_layout_build with the automatic order (Morton order of the
 * n x 3 Y when given, else the breadth-first order when Morton order gives no
 * tiles), over column windows of 8192 points (96 KB of LDS) and up to 32
 * tiles per row block.  There are no windowed segments: when no order gives
 * tiles (or a row is too long to sort) the build succeeds with tiles == 0 and
 * the 3-D layout calls refuse the handle with BHTSNE_EINVAL, unless P has no
 * entries (its attraction is zero); the plain 3-D calls serve such a P.  layout_mem holds bhtsne_layout_size_3d bytes (256-byte
 * aligned, owned by the caller and kept alive and unchanged while the handle
 * is used); the workspace is bhtsne_workspace_size_3d bytes.  The handle is
 * tagged as a 3-D layout: the 2-D layout calls refuse it and these calls
 * refuse a 2-D one.  bhtsne_gradient_layout_3d / bhtsne_step_layout_3d are
 * bhtsne_gradient_3d / bhtsne_step_3d taking P through such a layout: the
 * attractive forces run on the library's second stream beside the walk
 * (BHTSNE_FORK3 = 0 or 1 forks them after the codes or the sort instead);
 * results come back in the caller's order.  Errors as the
 * plain 3-D calls, and BHTSNE_EINPUT from the build for malformed row
 * pointers. */
size_t bhtsne_layout_size_3d(int64_t n, int64_t nnz);
int bhtsne_layout_build_3d(const bhtsne_csr *P, const float *Y, void *layout_mem, size_t layout_bytes,
                           bhtsne_layout *out, void *workspace, size_t workspace_bytes, hipStream_t stream);
int bhtsne_gradient_layout_3d(const float *Y, const bhtsne_layout *layout, float theta, float exaggeration,
                              float *grad, double *Z, void *workspace, size_t workspace_bytes, hipStream_t stream);
int bhtsne_step_layout_3d(float *Y, const bhtsne_layout *layout, float theta, float exaggeration,
                          float learning_rate, float momentum, float min_gain, float *update, float *gains,
                          float *grad, double *Z, void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Test exports for 3-D embeddings, as bhtsne_debug_sort / bhtsne_debug_tree:
 * params is a host array of 14 doubles {min x, max x, min y, max y, min z,
 * max z, cent x, cent y, cent z, r_span, y_root x, y_root y, y_root z,
 * scale}; summary is 2n x 4 floats {com x, com y, com z, count}, threshold
 * 2n floats (-1 for single points, else side^2 / theta^2), meta as for
 * bhtsne_debug_tree; bucket members sit at level 22. */
int bhtsne_debug_sort_3d(const float *Y, int64_t n, uint64_t *codes, uint64_t *sorted_codes, uint32_t *perm,
                         double *params, void *workspace, size_t workspace_bytes, hipStream_t stream);
int bhtsne_debug_tree_3d(const float *Y, int64_t n, float theta, int64_t *n_nodes, uint8_t *level, uint8_t *kind,
                         uint32_t *begin, uint32_t *end, float *summary, float *threshold, uint32_t *meta,
                         void *workspace, size_t workspace_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* BHTSNE_H */
