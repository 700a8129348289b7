/*
 * fp64 CPU oracle for one Barnes-Hut t-SNE gradient iteration with a 3-D
 * embedding (the problem statement allows a two- or three-dimensional
 * embedding; the paper works the method out in 2-D).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the GPU library links, includes or
 * calls this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark load it.  It shares no code, header, table or constant
 * generator with the HIP path.
 *
 * The steps are the 2-D oracle's, carried to three dimensions:
 *   - bounding box, centre and span radius of a cube (Quadtree Building;
 *     Algorithm 1 inputs, with a third axis)
 *   - Morton codes: each coordinate quantised to 21 bits on the cube's grid
 *     and the three interleaved, bit k of dimension d at bit 3k + d, which
 *     fills 63 of the 64 bits (the Morton-code paragraph, three-way)
 *   - stable sort of the codes by (code, index)
 *   - compressed octree, top-down: a cell at level L is the set of codes that
 *     share their top 3L bits below the unused top bit; identical codes form
 *     one bucket leaf at level 21, the last level of 63-bit codes
 *   - centre of mass and count per cell as direct sums (Parallel Summarization)
 *   - depth-first repulsive traversal with the acceptance test and Z
 *     (Repulsive Force Computation; q_ij and Z)
 *   - attractive forces over P's stored entries (Gradient Descent, first sum
 *     of the split gradient)
 *   - gradient, gains / momentum update and KL with an exact Z
 *
 * Readings (the 2-D ones, R1-R12, carried over; the 3-D specifics):
 *   R13 cube domain: r_span = max over the three axes of the half extent;
 *       quantised coordinate = trunc((y - y_root) * 2^20 / r_span), clamped
 *       to [0, 2^21 - 1]; r_span == 0 gives code 0 for every point.
 *   R14 a cell at level L (0..21) has side 2 r_span 2^-L; the acceptance test
 *       is side_L^2 < theta^2 |y_i - c|^2 as in 2-D.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define O3_INTERNAL 0
#define O3_BUCKET 1
#define O3_SINGLE 2
#define O3_LEVELS 21

/* box = {min_x, max_x, min_y, max_y, min_z, max_z, cent_x, cent_y, cent_z, r_span} */
void orc3_bbox(const double *Y, int64_t n, double *box)
{
    double mn[3], mx[3];
    for (int d = 0; d < 3; ++d) mn[d] = mx[d] = Y[d];
    for (int64_t i = 1; i < n; ++i)
        for (int d = 0; d < 3; ++d) {
            double v = Y[3 * i + d];
            if (v < mn[d]) mn[d] = v;
            if (v > mx[d]) mx[d] = v;
        }
    double widest = 0.0;
    for (int d = 0; d < 3; ++d) {
        box[2 * d] = mn[d];
        box[2 * d + 1] = mx[d];
        box[6 + d] = (mn[d] + mx[d]) * 0.5;
        double ext = mx[d] - mn[d];
        if (ext > widest) widest = ext;
    }
    box[9] = 0.5 * widest;
}

/* Morton code by definition: bit k of dimension d goes to bit 3k + d. */
uint64_t orc3_interleave(uint32_t m0, uint32_t m1, uint32_t m2)
{
    const uint32_t m[3] = {m0, m1, m2};
    uint64_t code = 0;
    for (int k = 0; k < O3_LEVELS; ++k)
        for (int d = 0; d < 3; ++d) code |= (uint64_t)((m[d] >> k) & 1u) << (3 * k + d);
    return code;
}

/* One coordinate onto the 2^21 grid of the cube (R13). */
static uint32_t orc3_quantise(double y, double yroot, double scale)
{
    double q = (y - yroot) * scale;
    if (!(q > 0.0)) return 0u;
    if (q >= 2097151.0) return 2097151u;
    return (uint32_t)q; /* truncation toward zero */
}

/* yrs = {y_root_x, y_root_y, y_root_z, scale} (scale 0 if r_span is 0). */
void orc3_morton(const double *Y, int64_t n, uint64_t *codes, uint32_t *grid, double *yrs)
{
    double box[10];
    orc3_bbox(Y, n, box);
    const double rspan = box[9];
    const double scale = rspan > 0.0 ? 1048576.0 / rspan : 0.0;
    for (int d = 0; d < 3; ++d) yrs[d] = box[6 + d] - rspan;
    yrs[3] = scale;
    for (int64_t i = 0; i < n; ++i) {
        uint32_t m[3] = {0, 0, 0};
        if (rspan > 0.0)
            for (int d = 0; d < 3; ++d) m[d] = orc3_quantise(Y[3 * i + d], yrs[d], scale);
        if (grid)
            for (int d = 0; d < 3; ++d) grid[3 * i + d] = m[d];
        codes[i] = orc3_interleave(m[0], m[1], m[2]);
    }
}

/* The stable (code, index) sort of the 2-D oracle serves both. */
void orc_sort(const uint64_t *codes, int64_t n, uint64_t *sorted, uint32_t *perm);

/* ------------------------------------------------------------------ */
/* Compressed octree over the sorted codes.                           */
/* ------------------------------------------------------------------ */
typedef struct {
    int64_t count;
    const uint64_t *codes;
    uint8_t *level, *kind;
    uint32_t *begin, *end;
    int32_t *parent;
} orc3_builder;

static int64_t orc3_emit(orc3_builder *t, int level, uint32_t b, uint32_t e, int32_t parent, int kind)
{
    int64_t id = t->count++;
    t->level[id] = (uint8_t)level;
    t->begin[id] = b;
    t->end[id] = e;
    t->parent[id] = parent;
    t->kind[id] = (uint8_t)kind;
    return id;
}

/* Octant of a code one level below level L: the 3-bit digit L+1, counted
 * from the top below the unused bit 63. */
static int orc3_digit(uint64_t code, int L) { return (int)((code >> (60 - 3 * L)) & 7u); }

/* Deepest level whose cell holds both codes (a != b). */
static int orc3_common_level(uint64_t a, uint64_t b)
{
    uint64_t x = a ^ b;
    int top = 63;
    while (!((x >> top) & 1u)) --top; /* highest differing bit, 0..62 */
    return (62 - top) / 3;            /* bits 62..60 are level 1's digit, and so on */
}

static void orc3_build_internal(orc3_builder *t, int L, uint32_t b, uint32_t e, int32_t parent);

static void orc3_build_child(orc3_builder *t, int Lp, uint32_t b, uint32_t e, int32_t parent)
{
    if (e - b == 1)
        orc3_emit(t, Lp + 1, b, e, parent, O3_SINGLE);
    else if (t->codes[b] == t->codes[e - 1])
        orc3_emit(t, O3_LEVELS, b, e, parent, O3_BUCKET);
    else
        orc3_build_internal(t, orc3_common_level(t->codes[b], t->codes[e - 1]), b, e, parent);
}

static void orc3_build_internal(orc3_builder *t, int L, uint32_t b, uint32_t e, int32_t parent)
{
    int32_t id = (int32_t)orc3_emit(t, L, b, e, parent, O3_INTERNAL);
    uint32_t s = b;
    while (s < e) {
        int d = orc3_digit(t->codes[s], L);
        uint32_t u = s;
        while (u < e && orc3_digit(t->codes[u], L) == d) ++u;
        orc3_build_child(t, L, s, u, id);
        s = u;
    }
}

/* Nodes in depth-first order with children in octant order, i.e. sorted by
 * (begin, level); the root (level 0, [0, n)) always exists.  At most 2n. */
int64_t orc3_tree(const uint64_t *sorted_codes, int64_t n, uint8_t *level, uint8_t *kind, uint32_t *begin,
                  uint32_t *end, int32_t *parent)
{
    orc3_builder t = {0, sorted_codes, level, kind, begin, end, parent};
    if (sorted_codes[0] == sorted_codes[n - 1]) {
        int32_t root = (int32_t)orc3_emit(&t, 0, 0, (uint32_t)n, -1, O3_INTERNAL);
        orc3_emit(&t, O3_LEVELS, 0, (uint32_t)n, root, O3_BUCKET);
    } else {
        orc3_build_internal(&t, 0, 0, (uint32_t)n, -1);
    }
    return t.count;
}

/* ------------------------------------------------------------------ */
/* Tree state kept between calls.                                     */
/* ------------------------------------------------------------------ */
typedef struct {
    int64_t n, nn;
    double box[10], yrs[4];
    uint64_t *codes, *sorted;
    uint32_t *perm, *inv;
    uint8_t *level, *kind;
    uint32_t *begin, *end, *count;
    int32_t *parent;
    int64_t *child_ptr;
    int32_t *child;
    double *com; /* nn x 3 */
    double *ys;  /* Y in sorted order, n x 3 */
} orc3_state;

void orc3_state_free(orc3_state *s)
{
    if (!s) return;
    free(s->codes); free(s->sorted); free(s->perm); free(s->inv);
    free(s->level); free(s->kind); free(s->begin); free(s->end); free(s->count);
    free(s->parent); free(s->child_ptr); free(s->child); free(s->com); free(s->ys);
    free(s);
}

orc3_state *orc3_state_build(const double *Y, int64_t n)
{
    orc3_state *s = (orc3_state *)calloc(1, sizeof(orc3_state));
    s->n = n;
    s->codes = (uint64_t *)malloc(8 * (size_t)n);
    s->sorted = (uint64_t *)malloc(8 * (size_t)n);
    s->perm = (uint32_t *)malloc(4 * (size_t)n);
    s->inv = (uint32_t *)malloc(4 * (size_t)n);
    orc3_bbox(Y, n, s->box);
    orc3_morton(Y, n, s->codes, NULL, s->yrs);
    orc_sort(s->codes, n, s->sorted, s->perm);
    for (int64_t i = 0; i < n; ++i) s->inv[s->perm[i]] = (uint32_t)i;
    const int64_t cap = 2 * n;
    s->level = (uint8_t *)malloc((size_t)cap);
    s->kind = (uint8_t *)malloc((size_t)cap);
    s->begin = (uint32_t *)malloc(4 * (size_t)cap);
    s->end = (uint32_t *)malloc(4 * (size_t)cap);
    s->parent = (int32_t *)malloc(4 * (size_t)cap);
    s->nn = orc3_tree(s->sorted, n, s->level, s->kind, s->begin, s->end, s->parent);
    s->ys = (double *)malloc(24 * (size_t)n);
    for (int64_t i = 0; i < n; ++i)
        for (int d = 0; d < 3; ++d) s->ys[3 * i + d] = Y[3 * (int64_t)s->perm[i] + d];
    /* summaries: direct fp64 sums over each cell's points (unit masses) */
    s->count = (uint32_t *)malloc(4 * (size_t)s->nn);
    s->com = (double *)malloc(24 * (size_t)s->nn);
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t v = 0; v < s->nn; ++v) {
        double acc[3] = {0.0, 0.0, 0.0};
        for (uint32_t p = s->begin[v]; p < s->end[v]; ++p)
            for (int d = 0; d < 3; ++d) acc[d] += s->ys[3 * (int64_t)p + d];
        uint32_t c = s->end[v] - s->begin[v];
        s->count[v] = c;
        for (int d = 0; d < 3; ++d) s->com[3 * v + d] = acc[d] / (double)c;
    }
    s->child_ptr = (int64_t *)calloc((size_t)s->nn + 1, 8);
    s->child = (int32_t *)malloc(4 * (size_t)(s->nn > 1 ? s->nn - 1 : 1));
    for (int64_t v = 1; v < s->nn; ++v) s->child_ptr[s->parent[v] + 1]++;
    for (int64_t v = 0; v < s->nn; ++v) s->child_ptr[v + 1] += s->child_ptr[v];
    int64_t *fill = (int64_t *)malloc(8 * (size_t)s->nn);
    memcpy(fill, s->child_ptr, 8 * (size_t)s->nn);
    for (int64_t v = 1; v < s->nn; ++v) s->child[fill[s->parent[v]]++] = (int32_t)v;
    free(fill);
    return s;
}

int64_t orc3_state_nodes(const orc3_state *s) { return s->nn; }

void orc3_state_export(const orc3_state *s, double *box, double *yrs, uint64_t *codes, uint64_t *sorted,
                       uint32_t *perm, uint8_t *level, uint8_t *kind, uint32_t *begin, uint32_t *end,
                       int32_t *parent, double *com, uint32_t *count)
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
    if (com) memcpy(com, s->com, 24 * (size_t)s->nn);
    if (count) memcpy(count, s->count, 4 * (size_t)s->nn);
}

/* ------------------------------------------------------------------ */
/* Repulsive Force Computation: depth-first traversal per point.      */
/* ------------------------------------------------------------------ */
typedef struct {
    double y[3];
    uint32_t self;
    double f[3], z;
    int64_t inter;
} orc3_query;

/* w = (1 + d^2)^-1 of a displacement; a cell of c points adds c w to Z_i and
 * c w^2 (y_i - c_v) to F_rep,i (R7). */
static void orc3_add(orc3_query *q, const double *diff, double cnt)
{
    double d2 = 0.0;
    for (int d = 0; d < 3; ++d) d2 += diff[d] * diff[d];
    double w = 1.0 / (1.0 + d2);
    q->z += cnt * w;
    for (int d = 0; d < 3; ++d) q->f[d] += cnt * w * w * diff[d];
    q->inter += 1;
}

static void orc3_point(const orc3_state *s, orc3_query *q, uint32_t j)
{
    double diff[3];
    for (int d = 0; d < 3; ++d) diff[d] = q->y[d] - s->ys[3 * (int64_t)j + d];
    orc3_add(q, diff, 1.0);
}

static void orc3_visit(const orc3_state *s, orc3_query *q, int32_t v, double theta2)
{
    if (s->kind[v] == O3_SINGLE) {
        if (s->begin[v] != q->self) orc3_point(s, q, s->begin[v]);
        return;
    }
    double diff[3], d2 = 0.0;
    for (int d = 0; d < 3; ++d) {
        diff[d] = q->y[d] - s->com[3 * v + d];
        d2 += diff[d] * diff[d];
    }
    double side = ldexp(2.0 * s->box[9], -(int)s->level[v]);
    if (side * side < theta2 * d2) {
        orc3_add(q, diff, (double)s->count[v]);
        return;
    }
    if (s->kind[v] == O3_BUCKET) {
        for (uint32_t j = s->begin[v]; j < s->end[v]; ++j)
            if (j != q->self) orc3_point(s, q, j);
        return;
    }
    for (int64_t c = s->child_ptr[v]; c < s->child_ptr[v + 1]; ++c) orc3_visit(s, q, s->child[c], theta2);
}

/* frep[3k..] = sum n_v w^2 (y_i - c_v), zi[k] = sum n_v w, inter[k], for the
 * points `pts` (original indices; NULL = all points in index order). */
void orc3_state_repulsive(const orc3_state *s, double theta, const int64_t *pts, int64_t npts, double *frep,
                          double *zi, int64_t *inter)
{
    const double theta2 = theta * theta;
#pragma omp parallel for schedule(dynamic, 256)
    for (int64_t k = 0; k < npts; ++k) {
        int64_t i = pts ? pts[k] : k;
        orc3_query q;
        memset(&q, 0, sizeof(q));
        q.self = s->inv[i];
        for (int d = 0; d < 3; ++d) q.y[d] = s->ys[3 * (int64_t)q.self + d];
        orc3_visit(s, &q, 0, theta2);
        for (int d = 0; d < 3; ++d) frep[3 * k + d] = q.f[d];
        zi[k] = q.z;
        if (inter) inter[k] = q.inter;
    }
}

/* ------------------------------------------------------------------ */
/* Attractive forces over the stored entries of each row:             */
/* F_attr,i = sum_j p_ij (1 + |y_i - y_j|^2)^-1 (y_i - y_j).           */
/* ------------------------------------------------------------------ */
void orc3_attractive(const double *Y, const int64_t *row_ptr, const int32_t *col, const float *val,
                     const int64_t *rows, int64_t nrows, double *fattr)
{
#pragma omp parallel for schedule(dynamic, 256)
    for (int64_t k = 0; k < nrows; ++k) {
        int64_t i = rows ? rows[k] : k;
        double f[3] = {0.0, 0.0, 0.0};
        for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
            int64_t j = col[e];
            double diff[3], d2 = 0.0;
            for (int d = 0; d < 3; ++d) {
                diff[d] = Y[3 * i + d] - Y[3 * j + d];
                d2 += diff[d] * diff[d];
            }
            double pw = (double)val[e] * (1.0 / (1.0 + d2));
            for (int d = 0; d < 3; ++d) f[d] += pw * diff[d];
        }
        for (int d = 0; d < 3; ++d) fattr[3 * k + d] = f[d];
    }
}

double orc_sum(const double *x, int64_t n);

/* grad = 4 (alpha F_attr - F_rep / Z); stats (nullable) = {Z, interactions, nodes} */
void orc3_gradient(const double *Y, int64_t n, const int64_t *row_ptr, const int32_t *col, const float *val,
                   double theta, double alpha, double *grad, double *stats)
{
    orc3_state *s = orc3_state_build(Y, n);
    double *frep = (double *)malloc(24 * (size_t)n);
    double *zi = (double *)malloc(8 * (size_t)n);
    int64_t *inter = (int64_t *)malloc(8 * (size_t)n);
    double *fattr = (double *)malloc(24 * (size_t)n);
    orc3_state_repulsive(s, theta, NULL, n, frep, zi, inter);
    orc3_attractive(Y, row_ptr, col, val, NULL, n, fattr);
    const double Z = orc_sum(zi, n);
    int64_t tot = 0;
    for (int64_t i = 0; i < n; ++i) tot += inter[i];
    for (int64_t i = 0; i < 3 * n; ++i) grad[i] = 4.0 * (alpha * fattr[i] - frep[i] / Z);
    if (stats) {
        stats[0] = Z;
        stats[1] = (double)tot;
        stats[2] = (double)s->nn;
    }
    free(frep); free(zi); free(inter); free(fattr);
    orc3_state_free(s);
}

void orc_update(double *y, double *u, double *gains, const double *g, int64_t n2, double eta, double mu,
                double min_gain);

/* One iteration: gradient of the current Y, then the elementwise update. */
void orc3_step(double *y, int64_t n, const int64_t *row_ptr, const int32_t *col, const float *val, double theta,
               double alpha, double eta, double mu, double min_gain, double *u, double *gains, double *grad_out,
               double *stats)
{
    double *g = grad_out ? grad_out : (double *)malloc(24 * (size_t)n);
    orc3_gradient(y, n, row_ptr, col, val, theta, alpha, g, stats);
    orc_update(y, u, gains, g, 3 * n, eta, mu, min_gain);
    if (!grad_out) free(g);
}

/* Z = sum over ordered pairs i != j of (1 + |y_i - y_j|^2)^-1, each point's
 * partial in index order, the partials summed in index order. */
double orc3_z_exact(const double *Y, int64_t n)
{
    double *part = (double *)calloc((size_t)n, 8);
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t i = 0; i < n; ++i) {
        double z = 0.0;
        for (int64_t j = 0; j < n; ++j) {
            if (j == i) continue;
            double d2 = 0.0;
            for (int d = 0; d < 3; ++d) {
                double t = Y[3 * i + d] - Y[3 * j + d];
                d2 += t * t;
            }
            z += 1.0 / (1.0 + d2);
        }
        part[i] = z;
    }
    double Z = orc_sum(part, n);
    free(part);
    return Z;
}

/* KL = sum over stored p_ij > 0 of p_ij log(p_ij / q_ij), q_ij = w_ij / Z. */
double orc3_kl(const double *Y, int64_t n, const int64_t *row_ptr, const int32_t *col, const float *val, double Z)
{
    double *part = (double *)calloc((size_t)n, 8);
#pragma omp parallel for schedule(dynamic, 256)
    for (int64_t i = 0; i < n; ++i) {
        double acc = 0.0;
        for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
            double p = val[e];
            if (!(p > 0.0)) continue;
            int64_t j = col[e];
            double d2 = 0.0;
            for (int d = 0; d < 3; ++d) {
                double t = Y[3 * i + d] - Y[3 * j + d];
                d2 += t * t;
            }
            acc += p * log(p / (1.0 / (1.0 + d2) / Z));
        }
        part[i] = acc;
    }
    double kl = orc_sum(part, n);
    free(part);
    return kl;
}
