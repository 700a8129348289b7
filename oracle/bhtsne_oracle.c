/*
 * fp64 CPU oracle for one Barnes-Hut t-SNE gradient iteration.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the GPU library links, includes or
 * calls this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark load it.  It shares no code, header, table or constant
 * generator with the HIP path.
 *
 * Every quantity is computed in double precision (float32 inputs are promoted
 * exactly), in the plainest form the paper's definitions allow:
 *   - bounding box, centre and span radius  (Quadtree Building; Algorithm 1 inputs)
 *   - Morton codes                           (Quadtree Building; Algorithm 1, worked example)
 *   - stable sort of the codes               (Quadtree Building, "sorted Morton codes")
 *   - compressed quadtree, top-down          (Quadtree Building; cells = code prefixes)
 *   - centre of mass and count per cell      (Parallel Summarization) as direct sums
 *   - depth-first repulsive traversal with the acceptance test and the
 *     normaliser Z                           (Repulsive Force Computation; q_ij and Z)
 *   - attractive forces over P's stored      (Gradient Descent, first sum of the split
 *     entries                                 gradient; Attractive Force Computation)
 *   - gradient assembly                      (Gradient Descent, split-gradient equation)
 *   - gains / momentum update                (not specified by the paper; the standard
 *                                              t-SNE optimiser the experiments' defaults use)
 *   - KL divergence with an exact Z          (Gradient Descent, KL cost)
 *
 * Readings of points the paper leaves silent or garbles (each one is also
 * listed with its justification in the design notes of the repository):
 *   R1  square domain: r_span = max over both axes of the half extent.
 *   R2  quantised coordinate = trunc((y - y_root) * 2^31 / r_span), clamped to
 *       [0, 2^32 - 1]; r_span == 0 gives code 0 for every point.
 *   R3  ties in the sort are broken by original index.
 *   R4  the quadtree is compressed: cells with a single non-empty quadrant
 *       are not nodes (except the root, which always exists); identical codes
 *       form one bucket leaf at level 32.
 *   R5  acceptance test: side_L^2 < theta^2 * |y_i - c|^2 (strict), side_L =
 *       2 r_span 2^-L is the side of the square cell; buckets are tested like
 *       any cell, single-point leaves are always computed exactly.
 *   R6  self-interaction is excluded only at point level, by index.
 *   R7  Z sums ordered pairs (k != l); F_rep is accumulated with a positive
 *       sign and enters the gradient as g = 4 (alpha F_attr - F_rep / Z).
 *   R8  exaggeration alpha multiplies P (the attractive term) only.
 *   R9  update: gain += 0.2 if u*g < 0 else gain *= 0.8; gain >= min_gain;
 *       u = mu u - eta gain g; y += u.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_INTERNAL 0
#define ORC_BUCKET 1
#define ORC_SINGLE 2

/* ------------------------------------------------------------------ */
/* Bounding box, centre and span radius (Quadtree Building).          */
/* box = {min_x, max_x, min_y, max_y, cent_x, cent_y, r_span}          */
/* ------------------------------------------------------------------ */
void orc_bbox(const double *Y, int64_t n, double *box)
{
    double mn[2] = {Y[0], Y[1]}, mx[2] = {Y[0], Y[1]};
    for (int64_t i = 1; i < n; ++i)
        for (int d = 0; d < 2; ++d) {
            double v = Y[2 * i + d];
            if (v < mn[d]) mn[d] = v;
            if (v > mx[d]) mx[d] = v;
        }
    box[0] = mn[0];
    box[1] = mx[0];
    box[2] = mn[1];
    box[3] = mx[1];
    box[4] = (mn[0] + mx[0]) * 0.5;
    box[5] = (mn[1] + mx[1]) * 0.5;
    double ext0 = mx[0] - mn[0], ext1 = mx[1] - mn[1];
    box[6] = 0.5 * (ext0 > ext1 ? ext0 : ext1);
}

/* Morton code by definition: bit k of dimension d goes to bit 2k + d. */
uint64_t orc_interleave(uint32_t m0, uint32_t m1)
{
    uint64_t code = 0;
    for (int k = 0; k < 32; ++k) {
        code |= (uint64_t)((m0 >> k) & 1u) << (2 * k);
        code |= (uint64_t)((m1 >> k) & 1u) << (2 * k + 1);
    }
    return code;
}

/* Quantise one coordinate onto the 2^32 grid of the square domain (R2). */
static uint32_t orc_quantise(double y, double yroot, double scale)
{
    double q = (y - yroot) * scale;
    if (!(q > 0.0)) return 0u;
    if (q >= 4294967295.0) return 0xffffffffu;
    return (uint32_t)q; /* truncation toward zero */
}

/* Codes of all points; yrs = {y_root_x, y_root_y, scale} (scale 0 if r_span 0). */
void orc_morton(const double *Y, int64_t n, uint64_t *codes, uint32_t *grid, double *yrs)
{
    double box[7];
    orc_bbox(Y, n, box);
    double rspan = box[6];
    double yroot0 = box[4] - rspan, yroot1 = box[5] - rspan;
    double scale = rspan > 0.0 ? 2147483648.0 / rspan : 0.0;
    yrs[0] = yroot0;
    yrs[1] = yroot1;
    yrs[2] = scale;
    for (int64_t i = 0; i < n; ++i) {
        uint32_t m0 = 0, m1 = 0;
        if (rspan > 0.0) {
            m0 = orc_quantise(Y[2 * i], yroot0, scale);
            m1 = orc_quantise(Y[2 * i + 1], yroot1, scale);
        }
        if (grid) {
            grid[2 * i] = m0;
            grid[2 * i + 1] = m1;
        }
        codes[i] = orc_interleave(m0, m1);
    }
}

/* Stable ascending sort of the codes (R3): order by (code, index). */
typedef struct { uint64_t code; uint32_t idx; } orc_pair;

static int orc_pair_cmp(const void *a, const void *b)
{
    const orc_pair *x = (const orc_pair *)a, *y = (const orc_pair *)b;
    if (x->code != y->code) return x->code < y->code ? -1 : 1;
    return x->idx < y->idx ? -1 : (x->idx > y->idx);
}

void orc_sort(const uint64_t *codes, int64_t n, uint64_t *sorted, uint32_t *perm)
{
    orc_pair *p = (orc_pair *)malloc(sizeof(orc_pair) * (size_t)n);
    for (int64_t i = 0; i < n; ++i) {
        p[i].code = codes[i];
        p[i].idx = (uint32_t)i;
    }
    qsort(p, (size_t)n, sizeof(orc_pair), orc_pair_cmp);
    for (int64_t i = 0; i < n; ++i) {
        sorted[i] = p[i].code;
        perm[i] = p[i].idx;
    }
    free(p);
}

/* ------------------------------------------------------------------ */
/* Compressed quadtree over the sorted codes (R4).                     */
/* ------------------------------------------------------------------ */
typedef struct {
    int64_t n, cap, count;
    const uint64_t *codes;
    uint8_t *level, *kind;
    uint32_t *begin, *end;
    int32_t *parent;
} orc_builder;

static int64_t orc_emit(orc_builder *t, int level, uint32_t b, uint32_t e, int32_t parent, int kind)
{
    int64_t id = t->count++;
    t->level[id] = (uint8_t)level;
    t->begin[id] = b;
    t->end[id] = e;
    t->parent[id] = parent;
    t->kind[id] = (uint8_t)kind;
    return id;
}

/* Quadrant index of a code one level below level L: the 2-bit digit L+1. */
static int orc_digit(uint64_t code, int L) { return (int)((code >> (62 - 2 * L)) & 3u); }

static int orc_clz64(uint64_t x)
{
    int c = 0;
    if (x == 0) return 64;
    while (!(x & 0x8000000000000000ull)) {
        x <<= 1;
        ++c;
    }
    return c;
}

static void orc_build_internal(orc_builder *t, int L, uint32_t b, uint32_t e, int32_t parent);

/* A child range of a cell at level Lp: a point, a bucket or a deeper cell. */
static void orc_build_child(orc_builder *t, int Lp, uint32_t b, uint32_t e, int32_t parent)
{
    if (e - b == 1) {
        orc_emit(t, Lp + 1, b, e, parent, ORC_SINGLE);
    } else if (t->codes[b] == t->codes[e - 1]) {
        orc_emit(t, 32, b, e, parent, ORC_BUCKET);
    } else {
        /* the deepest cell still holding the whole (sorted) range */
        int L = orc_clz64(t->codes[b] ^ t->codes[e - 1]) / 2;
        orc_build_internal(t, L, b, e, parent);
    }
}

/* Emit the cell (L, [b,e)), then split its points into the non-empty quadrants. */
static void orc_build_internal(orc_builder *t, int L, uint32_t b, uint32_t e, int32_t parent)
{
    int32_t id = (int32_t)orc_emit(t, L, b, e, parent, ORC_INTERNAL);
    uint32_t s = b;
    while (s < e) {
        int d = orc_digit(t->codes[s], L);
        uint32_t u = s;
        while (u < e && orc_digit(t->codes[u], L) == d) ++u;
        orc_build_child(t, L, s, u, id);
        s = u;
    }
}

/* Node list in depth-first order with children in quadrant order, which is
 * the order sorted by (begin, level).  The root (level 0, [0,n)) always
 * exists.  Returns the node count (at most 2n). */
int64_t orc_tree(const uint64_t *sorted_codes, int64_t n, uint8_t *level, uint8_t *kind,
                 uint32_t *begin, uint32_t *end, int32_t *parent)
{
    orc_builder t = {n, 2 * n, 0, sorted_codes, level, kind, begin, end, parent};
    if (sorted_codes[0] == sorted_codes[n - 1]) {
        int32_t root = (int32_t)orc_emit(&t, 0, 0, (uint32_t)n, -1, ORC_INTERNAL);
        orc_emit(&t, 32, 0, (uint32_t)n, root, ORC_BUCKET);
    } else {
        orc_build_internal(&t, 0, 0, (uint32_t)n, -1);
    }
    return t.count;
}

/* Parallel Summarization: count and centre of mass of every node, here as
 * direct fp64 sums over the node's points (unit mass per point). */
void orc_summaries(const double *Y, const uint32_t *perm, int64_t nn, const uint32_t *begin,
                   const uint32_t *end, double *com, uint32_t *count)
{
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t v = 0; v < nn; ++v) {
        double sx = 0.0, sy = 0.0;
        for (uint32_t s = begin[v]; s < end[v]; ++s) {
            sx += Y[2 * (int64_t)perm[s]];
            sy += Y[2 * (int64_t)perm[s] + 1];
        }
        uint32_t c = end[v] - begin[v];
        count[v] = c;
        com[2 * v] = sx / (double)c;
        com[2 * v + 1] = sy / (double)c;
    }
}

/* ------------------------------------------------------------------ */
/* Whole tree state, kept between calls so tests can query points.    */
/* ------------------------------------------------------------------ */
typedef struct {
    int64_t n, nn;
    double box[7], yrs[3];
    uint64_t *codes, *sorted;
    uint32_t *perm, *inv;
    uint8_t *level, *kind;
    uint32_t *begin, *end, *count;
    int32_t *parent;
    int64_t *child_ptr;
    int32_t *child;
    double *com;
    double *ys; /* Y in sorted order, fp64 */
} orc_state;

void orc_state_free(orc_state *s)
{
    if (!s) return;
    free(s->codes); free(s->sorted); free(s->perm); free(s->inv);
    free(s->level); free(s->kind); free(s->begin); free(s->end); free(s->count);
    free(s->parent); free(s->child_ptr); free(s->child); free(s->com); free(s->ys);
    free(s);
}

orc_state *orc_state_build(const double *Y, int64_t n)
{
    orc_state *s = (orc_state *)calloc(1, sizeof(orc_state));
    s->n = n;
    s->codes = (uint64_t *)malloc(8 * (size_t)n);
    s->sorted = (uint64_t *)malloc(8 * (size_t)n);
    s->perm = (uint32_t *)malloc(4 * (size_t)n);
    s->inv = (uint32_t *)malloc(4 * (size_t)n);
    orc_bbox(Y, n, s->box);
    orc_morton(Y, n, s->codes, NULL, s->yrs);
    orc_sort(s->codes, n, s->sorted, s->perm);
    for (int64_t i = 0; i < n; ++i) s->inv[s->perm[i]] = (uint32_t)i;
    int64_t cap = 2 * n;
    s->level = (uint8_t *)malloc((size_t)cap);
    s->kind = (uint8_t *)malloc((size_t)cap);
    s->begin = (uint32_t *)malloc(4 * (size_t)cap);
    s->end = (uint32_t *)malloc(4 * (size_t)cap);
    s->parent = (int32_t *)malloc(4 * (size_t)cap);
    s->nn = orc_tree(s->sorted, n, s->level, s->kind, s->begin, s->end, s->parent);
    s->count = (uint32_t *)malloc(4 * (size_t)s->nn);
    s->com = (double *)malloc(16 * (size_t)s->nn);
    orc_summaries(Y, s->perm, s->nn, s->begin, s->end, s->com, s->count);
    /* explicit child lists from the parent pointers */
    s->child_ptr = (int64_t *)calloc((size_t)s->nn + 1, 8);
    s->child = (int32_t *)malloc(4 * (size_t)(s->nn > 1 ? s->nn - 1 : 1));
    for (int64_t v = 1; v < s->nn; ++v) s->child_ptr[s->parent[v] + 1]++;
    for (int64_t v = 0; v < s->nn; ++v) s->child_ptr[v + 1] += s->child_ptr[v];
    int64_t *fill = (int64_t *)malloc(8 * (size_t)s->nn);
    memcpy(fill, s->child_ptr, 8 * (size_t)s->nn);
    for (int64_t v = 1; v < s->nn; ++v) s->child[fill[s->parent[v]]++] = (int32_t)v;
    free(fill);
    s->ys = (double *)malloc(16 * (size_t)n);
    for (int64_t i = 0; i < n; ++i) {
        s->ys[2 * i] = Y[2 * (int64_t)s->perm[i]];
        s->ys[2 * i + 1] = Y[2 * (int64_t)s->perm[i] + 1];
    }
    return s;
}

int64_t orc_state_nodes(const orc_state *s) { return s->nn; }

void orc_state_export(const orc_state *s, double *box, double *yrs, uint64_t *codes,
                      uint64_t *sorted, uint32_t *perm, uint8_t *level, uint8_t *kind,
                      uint32_t *begin, uint32_t *end, int32_t *parent, double *com,
                      uint32_t *count)
{
    if (box) memcpy(box, s->box, sizeof(s->box));
    if (yrs) memcpy(yrs, s->yrs, sizeof(s->yrs));
    if (codes) memcpy(codes, s->codes, 8 * (size_t)s->n);
    if (sorted) memcpy(sorted, s->sorted, 8 * (size_t)s->n);
    if (perm) memcpy(perm, s->perm, 4 * (size_t)s->n);
    if (level) memcpy(level, s->level, (size_t)s->nn);
    if (kind) memcpy(kind, s->kind, (size_t)s->nn);
    if (begin) memcpy(begin, s->begin, 4 * (size_t)s->nn);
    if (end) memcpy(end, s->end, 4 * (size_t)s->nn);
    if (parent) memcpy(parent, s->parent, 4 * (size_t)s->nn);
    if (com) memcpy(com, s->com, 16 * (size_t)s->nn);
    if (count) memcpy(count, s->count, 4 * (size_t)s->nn);
}

/* ------------------------------------------------------------------ */
/* Repulsive Force Computation: depth-first traversal per point.      */
/* ------------------------------------------------------------------ */
typedef struct {
    double x, y;  /* the query point */
    uint32_t self; /* its sorted position */
    double fx, fy, z;
    int64_t inter;
} orc_query;

/* one exact pair: w = (1 + d^2)^-1; Z_i += w; F_rep,i += w^2 (y_i - y_j) */
static void orc_exact(const orc_state *s, orc_query *q, uint32_t j)
{
    double dx = q->x - s->ys[2 * (int64_t)j], dy = q->y - s->ys[2 * (int64_t)j + 1];
    double w = 1.0 / (1.0 + dx * dx + dy * dy);
    q->z += w;
    q->fx += w * w * dx;
    q->fy += w * w * dy;
    q->inter += 1;
}

static void orc_visit(const orc_state *s, orc_query *q, int32_t v, double theta2)
{
    if (s->kind[v] == ORC_SINGLE) {
        if (s->begin[v] != q->self) orc_exact(s, q, s->begin[v]);
        return;
    }
    double dx = q->x - s->com[2 * v], dy = q->y - s->com[2 * v + 1];
    double d2 = dx * dx + dy * dy;
    double side = ldexp(2.0 * s->box[6], -(int)s->level[v]);
    if (side * side < theta2 * d2) { /* the cell summary stands in for its points */
        double w = 1.0 / (1.0 + d2);
        double nv = (double)s->count[v];
        q->z += nv * w;
        q->fx += nv * w * w * dx;
        q->fy += nv * w * w * dy;
        q->inter += 1;
        return;
    }
    if (s->kind[v] == ORC_BUCKET) {
        for (uint32_t j = s->begin[v]; j < s->end[v]; ++j)
            if (j != q->self) orc_exact(s, q, j);
        return;
    }
    for (int64_t c = s->child_ptr[v]; c < s->child_ptr[v + 1]; ++c)
        orc_visit(s, q, s->child[c], theta2);
}

/* Repulsive sums for the points `pts` (original indices; NULL = all points in
 * index order).  frep[2k..] = sum n_v w^2 (y_i - c_v) (positive sign, R7),
 * zi[k] = sum n_v w, inter[k] = accepted cells + exact pairs. */
void orc_state_repulsive(const orc_state *s, double theta, const int64_t *pts, int64_t npts,
                         double *frep, double *zi, int64_t *inter)
{
    double theta2 = theta * theta;
#pragma omp parallel for schedule(dynamic, 256)
    for (int64_t k = 0; k < npts; ++k) {
        int64_t i = pts ? pts[k] : k;
        orc_query q;
        q.self = s->inv[i];
        q.x = s->ys[2 * (int64_t)q.self];
        q.y = s->ys[2 * (int64_t)q.self + 1];
        q.fx = q.fy = q.z = 0.0;
        q.inter = 0;
        orc_visit(s, &q, 0, theta2);
        frep[2 * k] = q.fx;
        frep[2 * k + 1] = q.fy;
        zi[k] = q.z;
        if (inter) inter[k] = q.inter;
    }
}

/* ------------------------------------------------------------------ */
/* Attractive forces: the first sum of the split gradient (Gradient    */
/* Descent), F_attr,i = sum_{j != i} p_ij q_ij Z (y_i - y_j), where    */
/* q_ij Z = (1 + |y_i - y_j|^2)^-1 is the Student-t kernel w_ij.  P is  */
/* zero outside its stored entries, so only the stored entries of row  */
/* i (0-based columns) contribute (Attractive Force Computation).      */
/* ------------------------------------------------------------------ */
static double orc_kernel_w(double dx, double dy) { return 1.0 / (1.0 + dx * dx + dy * dy); }

void orc_attractive(const double *Y, const int64_t *row_ptr, const int32_t *col, const float *val,
                    const int64_t *rows, int64_t nrows, double *fattr)
{
#pragma omp parallel for schedule(dynamic, 256)
    for (int64_t k = 0; k < nrows; ++k) {
        int64_t i = rows ? rows[k] : k;
        double f[2] = {0.0, 0.0};
        for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
            int64_t j = col[e];
            double diff[2] = {Y[2 * i] - Y[2 * j], Y[2 * i + 1] - Y[2 * j + 1]};
            double pw = (double)val[e] * orc_kernel_w(diff[0], diff[1]); /* p_ij q_ij Z */
            for (int d = 0; d < 2; ++d) f[d] += pw * diff[d];
        }
        fattr[2 * k] = f[0];
        fattr[2 * k + 1] = f[1];
    }
}

/* Sum in index order, so Z does not depend on the thread count. */
double orc_sum(const double *x, int64_t n)
{
    double s = 0.0;
    for (int64_t i = 0; i < n; ++i) s += x[i];
    return s;
}

/* ------------------------------------------------------------------ */
/* One full gradient (and optionally the update) over all points.     */
/* grad = 4 (alpha F_attr - F_rep / Z)                                 */
/* stats (nullable) = {Z, interactions, nodes}                         */
/* ------------------------------------------------------------------ */
void orc_gradient(const double *Y, int64_t n, const int64_t *row_ptr, const int32_t *col,
                  const float *val, double theta, double alpha, double *grad, double *stats)
{
    orc_state *s = orc_state_build(Y, n);
    double *frep = (double *)malloc(16 * (size_t)n);
    double *zi = (double *)malloc(8 * (size_t)n);
    int64_t *inter = (int64_t *)malloc(8 * (size_t)n);
    double *fattr = (double *)malloc(16 * (size_t)n);
    orc_state_repulsive(s, theta, NULL, n, frep, zi, inter);
    orc_attractive(Y, row_ptr, col, val, NULL, n, fattr);
    double Z = orc_sum(zi, n);
    int64_t tot = 0;
    for (int64_t i = 0; i < n; ++i) tot += inter[i];
    for (int64_t i = 0; i < 2 * n; ++i) grad[i] = 4.0 * (alpha * fattr[i] - frep[i] / Z);
    if (stats) {
        stats[0] = Z;
        stats[1] = (double)tot;
        stats[2] = (double)s->nn;
    }
    free(frep); free(zi); free(inter); free(fattr);
    orc_state_free(s);
}

/* Gains / momentum update of one step, elementwise over the n x 2 arrays. */
void orc_update(double *y, double *u, double *gains, const double *g, int64_t n2, double eta,
                double mu, double min_gain)
{
    for (int64_t k = 0; k < n2; ++k) {
        double gain = (u[k] * g[k] < 0.0) ? gains[k] + 0.2 : gains[k] * 0.8;
        if (gain < min_gain) gain = min_gain;
        gains[k] = gain;
        u[k] = mu * u[k] - eta * gain * g[k];
        y[k] += u[k];
    }
}

/* One iteration on an fp64 state: gradient of the current Y, then the update. */
void orc_step(double *y, int64_t n, const int64_t *row_ptr, const int32_t *col, const float *val,
              double theta, double alpha, double eta, double mu, double min_gain, double *u,
              double *gains, double *grad_out, double *stats)
{
    double *g = grad_out ? grad_out : (double *)malloc(16 * (size_t)n);
    orc_gradient(y, n, row_ptr, col, val, theta, alpha, g, stats);
    orc_update(y, u, gains, g, 2 * n, eta, mu, min_gain);
    if (!grad_out) free(g);
}

/* The same iteration as orc_step, with the wall time of each step of the
 * paper's per-step tables (Evaluating performance improvements of
 * individual steps): ms = {tree building (box, codes, sort, tree),
 * summarization, attractive, repulsive (with Z), gradient and update}.
 * stats (nullable) = {Z, interactions, nodes}. */
void orc_step_timed(double *y, int64_t n, const int64_t *row_ptr, const int32_t *col, const float *val,
                    double theta, double alpha, double eta, double mu, double min_gain, double *u, double *gains,
                    double *stats, double *ms)
{
#ifdef _OPENMP
#define ORC_NOW() omp_get_wtime()
#else
#define ORC_NOW() 0.0
#endif
    double t0 = ORC_NOW();
    orc_state *s = (orc_state *)calloc(1, sizeof(orc_state));
    s->n = n;
    s->codes = (uint64_t *)malloc(8 * (size_t)n);
    s->sorted = (uint64_t *)malloc(8 * (size_t)n);
    s->perm = (uint32_t *)malloc(4 * (size_t)n);
    s->inv = (uint32_t *)malloc(4 * (size_t)n);
    orc_bbox(y, n, s->box);
    orc_morton(y, n, s->codes, NULL, s->yrs);
    orc_sort(s->codes, n, s->sorted, s->perm);
    for (int64_t i = 0; i < n; ++i) s->inv[s->perm[i]] = (uint32_t)i;
    int64_t cap = 2 * n;
    s->level = (uint8_t *)malloc((size_t)cap);
    s->kind = (uint8_t *)malloc((size_t)cap);
    s->begin = (uint32_t *)malloc(4 * (size_t)cap);
    s->end = (uint32_t *)malloc(4 * (size_t)cap);
    s->parent = (int32_t *)malloc(4 * (size_t)cap);
    s->nn = orc_tree(s->sorted, n, s->level, s->kind, s->begin, s->end, s->parent);
    s->child_ptr = (int64_t *)calloc((size_t)s->nn + 1, 8);
    s->child = (int32_t *)malloc(4 * (size_t)(s->nn > 1 ? s->nn - 1 : 1));
    for (int64_t v = 1; v < s->nn; ++v) s->child_ptr[s->parent[v] + 1]++;
    for (int64_t v = 0; v < s->nn; ++v) s->child_ptr[v + 1] += s->child_ptr[v];
    int64_t *fill = (int64_t *)malloc(8 * (size_t)s->nn);
    memcpy(fill, s->child_ptr, 8 * (size_t)s->nn);
    for (int64_t v = 1; v < s->nn; ++v) s->child[fill[s->parent[v]]++] = (int32_t)v;
    free(fill);
    s->ys = (double *)malloc(16 * (size_t)n);
    for (int64_t i = 0; i < n; ++i) {
        s->ys[2 * i] = y[2 * (int64_t)s->perm[i]];
        s->ys[2 * i + 1] = y[2 * (int64_t)s->perm[i] + 1];
    }
    double t1 = ORC_NOW();
    s->count = (uint32_t *)malloc(4 * (size_t)s->nn);
    s->com = (double *)malloc(16 * (size_t)s->nn);
    orc_summaries(y, s->perm, s->nn, s->begin, s->end, s->com, s->count);
    double t2 = ORC_NOW();
    double *fattr = (double *)malloc(16 * (size_t)n);
    orc_attractive(y, row_ptr, col, val, NULL, n, fattr);
    double t3 = ORC_NOW();
    double *frep = (double *)malloc(16 * (size_t)n);
    double *zi = (double *)malloc(8 * (size_t)n);
    int64_t *inter = (int64_t *)malloc(8 * (size_t)n);
    orc_state_repulsive(s, theta, NULL, n, frep, zi, inter);
    double Z = orc_sum(zi, n);
    double t4 = ORC_NOW();
    double *g = (double *)malloc(16 * (size_t)n);
    for (int64_t i = 0; i < 2 * n; ++i) g[i] = 4.0 * (alpha * fattr[i] - frep[i] / Z);
    orc_update(y, u, gains, g, 2 * n, eta, mu, min_gain);
    double t5 = ORC_NOW();
    if (stats) {
        int64_t tot = 0;
        for (int64_t i = 0; i < n; ++i) tot += inter[i];
        stats[0] = Z;
        stats[1] = (double)tot;
        stats[2] = (double)s->nn;
    }
    if (ms) {
        ms[0] = 1e3 * (t1 - t0);
        ms[1] = 1e3 * (t2 - t1);
        ms[2] = 1e3 * (t3 - t2);
        ms[3] = 1e3 * (t4 - t3);
        ms[4] = 1e3 * (t5 - t4);
    }
    free(g); free(frep); free(zi); free(inter); free(fattr);
    orc_state_free(s);
#undef ORC_NOW
}

/* Threads of the OpenMP loops (the results do not depend on it). */
void orc_set_threads(int t)
{
#ifdef _OPENMP
    if (t > 0) omp_set_num_threads(t);
#else
    (void)t;
#endif
}

/* ------------------------------------------------------------------ */
/* KL divergence (Gradient Descent, KL cost) with an exact Z.         */
/* ------------------------------------------------------------------ */
/* Z = sum over ordered pairs i != j of (1 + |y_i - y_j|^2)^-1 (the q_ij
 * normaliser).  Each point's partial sum runs over j in index order; eight
 * points are swept together, each with its own accumulator, which changes no
 * rounding (the self pair adds an exact 0) and lets the compiler use vector
 * divisions.  The partials are then summed in index order. */
#define ORC_ZROWS 8
double orc_z_exact(const double *Y, int64_t n)
{
    double *part = (double *)calloc((size_t)n, 8);
    const int64_t blocks = (n + ORC_ZROWS - 1) / ORC_ZROWS;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t b = 0; b < blocks; ++b) {
        double xi[ORC_ZROWS], yi[ORC_ZROWS], z[ORC_ZROWS];
        int64_t id[ORC_ZROWS];
        for (int r = 0; r < ORC_ZROWS; ++r) {
            int64_t i = b * ORC_ZROWS + r;
            id[r] = i < n ? i : -1; /* rows past the end compute and discard */
            xi[r] = Y[2 * (i < n ? i : n - 1)];
            yi[r] = Y[2 * (i < n ? i : n - 1) + 1];
            z[r] = 0.0;
        }
        for (int64_t j = 0; j < n; ++j) {
            const double xj = Y[2 * j], yj = Y[2 * j + 1];
            for (int r = 0; r < ORC_ZROWS; ++r) {
                double dx = xi[r] - xj, dy = yi[r] - yj;
                double w = 1.0 / (1.0 + dx * dx + dy * dy);
                z[r] += (j == id[r]) ? 0.0 : w;
            }
        }
        for (int r = 0; r < ORC_ZROWS; ++r)
            if (id[r] >= 0) part[id[r]] = z[r];
    }
    double Z = orc_sum(part, n);
    free(part);
    return Z;
}

/* KL = sum over stored p_ij > 0 of p_ij log(p_ij / q_ij), q_ij = w_ij / Z. */
double orc_kl(const double *Y, int64_t n, const int64_t *row_ptr, const int32_t *col,
              const float *val, double Z)
{
    double *part = (double *)calloc((size_t)n, 8);
#pragma omp parallel for schedule(dynamic, 256)
    for (int64_t i = 0; i < n; ++i) {
        double acc = 0.0;
        for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
            double p = val[e];
            if (!(p > 0.0)) continue;
            int64_t j = col[e];
            double dx = Y[2 * i] - Y[2 * j];
            double dy = Y[2 * i + 1] - Y[2 * j + 1];
            double q = 1.0 / (1.0 + dx * dx + dy * dy) / Z;
            acc += p * log(p / q);
        }
        part[i] = acc;
    }
    double kl = orc_sum(part, n);
    free(part);
    return kl;
}

int orc_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
