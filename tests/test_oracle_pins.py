"""Pins of the fp64 oracle against facts the paper and the mathematics fix.

None of these tests re-types an oracle formula and compares it with itself:
each checks the oracle against a worked example printed in the paper, a
different formulation of the same definition (dense exact gradient, finite
differences of the KL cost, a geometric top-down partition, an ancestor
enumeration instead of a depth-first walk), a closed form, or an invariant.
"""
import math
import os

import numpy as np
import pytest

import oracle
import synth


def _rows(path):
    out = []
    for line in open(path):
        line = line.strip()
        if line and not line.startswith("#"):
            out.append(line)
    return out


# ---------------------------------------------------------------- Morton codes
def test_morton_worked_example(golden_dir):
    for line in _rows(os.path.join(golden_dir, "morton_worked_example.txt")):
        m0, m1, code = (int(x) for x in line.split())
        assert oracle.interleave(m0, m1) == code


def _interleave_by_strings(m0, m1):
    a, b = format(m0, "032b"), format(m1, "032b")
    return int("".join(y + x for x, y in zip(a, b)), 2)  # dim 1 is the higher bit of each digit


def test_interleave_matches_string_interleave():
    rng = np.random.default_rng(1)
    for m0, m1 in [(0, 0), (0xFFFFFFFF, 0), (0, 0xFFFFFFFF), (0xFFFFFFFF, 0xFFFFFFFF)] + \
            [tuple(int(v) for v in rng.integers(0, 2**32, 2)) for _ in range(300)]:
        assert oracle.interleave(m0, m1) == _interleave_by_strings(m0, m1)


def test_quantisation_extremes():
    y = synth.random_y(257, seed=3, scale=5.0)
    codes, grid, yrs = oracle.morton(y)
    ext = y.max(0).astype(np.float64) - y.min(0)
    wide = int(np.argmax(ext))
    # the widest axis spans the whole grid: its extremes land on 0 and 2^32-1
    assert grid[np.argmin(y[:, wide]), wide] == 0
    assert grid[np.argmax(y[:, wide]), wide] == 0xFFFFFFFF
    # grid coordinates are monotone in the coordinate values
    for d in range(2):
        o = np.argsort(y[:, d], kind="stable")
        assert np.all(np.diff(grid[o, d].astype(np.int64)) >= 0)
    # narrow axis stays inside the grid and is centred
    nar = 1 - wide
    mid = (int(grid[:, nar].min()) + int(grid[:, nar].max())) / 2
    assert abs(mid - 2**31) < 2**31 * 1e-6 + 2


def test_quantisation_truncates_hand_worked_case(golden_dir):
    """Reading R2 fixed by a hand-worked case whose truncated and rounded grid
    values differ (tests/golden/quantisation_truncation.txt)."""
    rows = [line.split() for line in _rows(os.path.join(golden_dir, "quantisation_truncation.txt"))]
    y = np.array([[float(r[0]), float(r[1])] for r in rows], np.float32)
    codes, grid, yrs = oracle.morton(y)
    for k, r in enumerate(rows):
        assert int(grid[k, 0]) == int(r[2], 16) and int(grid[k, 1]) == int(r[3], 16), k
        assert int(codes[k]) == int(r[4], 16), k
    assert yrs[0] == 0.0 and yrs[1] == 0.0


def test_all_points_identical_gives_zero_codes():
    y = np.full((9, 2), 1.25, np.float32)
    codes, grid, yrs = oracle.morton(y)
    assert np.all(codes == 0) and yrs[2] == 0.0


def test_sort_is_stable_by_code_then_index():
    rng = np.random.default_rng(5)
    codes = rng.integers(0, 50, 2000).astype(np.uint64)  # many ties
    s, perm = oracle.sort_codes(codes)
    ref = np.argsort(codes, kind="stable")
    assert np.array_equal(perm, ref.astype(np.uint32))
    assert np.array_equal(s, codes[ref])


# ---------------------------------------------------------------- quadtree
def test_cell_ranges_from_paper(golden_dir):
    # all 64 cells of the paper's 3-level example occupied once: codes 0..63 in
    # the top 6 bits of a 64-bit code
    codes = (np.arange(64, dtype=np.uint64) << np.uint64(58))
    n = 64
    lv = np.empty(128, np.uint8)
    kd = np.empty(128, np.uint8)
    b = np.empty(128, np.uint32)
    e = np.empty(128, np.uint32)
    par = np.empty(128, np.int32)
    lib = oracle._load()
    nn = lib.orc_tree(codes.ctypes.data_as(oracle._u64), n, lv.ctypes.data_as(oracle._u8),
                      kd.ctypes.data_as(oracle._u8), b.ctypes.data_as(oracle._u32),
                      e.ctypes.data_as(oracle._u32), par.ctypes.data_as(oracle._i32))
    assert nn == 1 + 4 + 16 + 64
    nodes = {(int(b[v]), int(e[v]), int(lv[v])) for v in range(nn)}
    for line in _rows(os.path.join(golden_dir, "cell_ranges.txt")):
        lo, hi, level = line.split()
        assert (int(lo, 2), int(hi, 2) + 1, int(level)) in nodes


def _geometric_tree(grid):
    """Top-down partition of point sets by quadrant bits of the grid
    coordinates, level by level (the uncompressed tree of the paper's
    Quadtree Building description), then removal of single-child cells other
    than the root.  Returns {(level, frozenset(points), kind)}."""
    n = grid.shape[0]
    out = set()

    def rec(level, pts, is_root):
        if len(pts) == 1 and not is_root:
            out.add((level, frozenset(pts), oracle.SINGLE))
            return
        if level == 32:
            out.add((32, frozenset(pts), oracle.BUCKET))
            return
        bit = 31 - level
        quads = {}
        for p in pts:
            q = ((int(grid[p, 0]) >> bit) & 1) | (((int(grid[p, 1]) >> bit) & 1) << 1)
            quads.setdefault(q, []).append(p)
        if len(quads) > 1 or is_root:
            out.add((level, frozenset(pts), oracle.INTERNAL))
        # a cell with one non-empty quadrant is not emitted (chain collapse);
        # its only child is examined one level further down
        for q in sorted(quads):
            rec(level + 1, quads[q], False)

    rec(0, list(range(n)), True)
    return out


def _canonical_oracle_tree(t):
    return {(int(t.level[v]), frozenset(int(p) for p in t.perm[t.begin[v]:t.end[v]]),
             int(t.kind[v])) for v in range(t.nodes)}


@pytest.mark.parametrize("seed,n,scale,dups", [(1, 2, 1.0, 0), (2, 7, 1.0, 0), (3, 40, 1.0, 3),
                                               (4, 120, 1e-3, 10), (5, 200, 30.0, 0)])
def test_tree_matches_geometric_partition(seed, n, scale, dups):
    y = synth.random_y(n, seed=seed, scale=scale, dups=dups)
    # a few near-coincident points exercise deep levels
    y[-1] = y[0] + np.float32(1e-6) * scale
    t = oracle.tree(y)
    _, grid, _ = oracle.morton(y)
    geo = _geometric_tree(grid)
    assert _canonical_oracle_tree(t) == geo


def test_tree_invariants_and_order():
    y = synth.random_y(3000, seed=11, scale=2.0, dups=40)
    t = oracle.tree(y)
    nn = t.nodes
    assert t.level[0] == 0 and t.begin[0] == 0 and t.end[0] == 3000 and t.parent[0] == -1
    keys = t.begin.astype(np.int64) * 64 + t.level
    assert np.all(np.diff(keys) > 0)  # sorted by (begin, level), no duplicates
    internal = t.kind == oracle.INTERNAL
    assert internal.sum() <= 3000 - 1
    nchild = np.bincount(t.parent[1:], minlength=nn)
    assert np.all(nchild[internal][1:] >= 2)  # only the root may have one child
    for v in range(1, nn):
        p = t.parent[v]
        assert t.level[p] < t.level[v]
        assert t.begin[p] <= t.begin[v] and t.end[v] <= t.end[p]
    # children partition their parent's range
    cover = np.zeros(nn, np.int64)
    np.add.at(cover, t.parent[1:], (t.end[1:] - t.begin[1:]).astype(np.int64))
    assert np.array_equal(cover[internal], (t.end - t.begin)[internal].astype(np.int64))
    for v in np.nonzero(t.kind == oracle.BUCKET)[0]:
        assert np.all(t.sorted_codes[t.begin[v]:t.end[v]] == t.sorted_codes[t.begin[v]])


# ---------------------------------------------------------------- summaries
def test_summaries_root_mean_and_counts():
    y = synth.random_y(5000, seed=12, scale=3.0, dups=20)
    t = oracle.tree(y)
    assert t.count[0] == 5000
    assert np.allclose(t.com[0], y.astype(np.float64).mean(0), rtol=0, atol=1e-12)
    nn = t.nodes
    csum = np.zeros(nn, np.int64)
    np.add.at(csum, t.parent[1:], t.count[1:].astype(np.int64))
    internal = t.kind == oracle.INTERNAL
    assert np.array_equal(csum[internal], t.count[internal].astype(np.int64))
    ys = y.astype(np.float64)[t.perm]
    for v in range(0, nn, 37):
        pts = ys[t.begin[v]:t.end[v]]
        assert np.all(t.com[v] >= pts.min(0) - 1e-12) and np.all(t.com[v] <= pts.max(0) + 1e-12)


# ---------------------------------------------------------------- gradient pins
def _dense_p(n, row_ptr, col, val):
    P = np.zeros((n, n))
    for i in range(n):
        for k in range(row_ptr[i], row_ptr[i + 1]):
            P[i, col[k]] += val[k]
    return P


def _exact_gradient_single_sum(y, P, alpha=1.0):
    """dC/dy_i = 4 sum_j (alpha p_ij - q_ij) q_ij Z (y_i - y_j)  (Gradient Descent)."""
    y = y.astype(np.float64)
    diff = y[:, None, :] - y[None, :, :]
    w = 1.0 / (1.0 + (diff ** 2).sum(-1))
    np.fill_diagonal(w, 0.0)
    Z = w.sum()
    q = w / Z
    coef = (alpha * P - q) * q * Z
    return 4.0 * (coef[:, :, None] * diff).sum(1), Z


def _kl_dense(y, P):
    diff = y[:, None, :] - y[None, :, :]
    w = 1.0 / (1.0 + (diff ** 2).sum(-1))
    np.fill_diagonal(w, 0.0)
    q = w / w.sum()
    m = P > 0
    return float((P[m] * np.log(P[m] / q[m])).sum())


@pytest.mark.parametrize("n,seed,dups", [(2, 1, 0), (3, 2, 0), (60, 3, 0), (150, 4, 5)])
def test_theta0_equals_exact_gradient(n, seed, dups):
    y = synth.random_y(n, seed=seed, scale=2.0, dups=dups)
    rp, col, val = synth.random_p(n, seed=seed, k=6)
    P = _dense_p(n, rp, col, val)
    for alpha in (1.0, 12.0):
        g, Z, inter, _ = oracle.gradient(y, rp, col, val, theta=0.0, exaggeration=alpha)
        gref, Zref = _exact_gradient_single_sum(y, P, alpha)
        assert math.isclose(Z, Zref, rel_tol=1e-13)
        assert inter == n * (n - 1)
        assert np.allclose(g, gref, rtol=1e-11, atol=1e-14 * max(np.abs(gref).max(), 1.0))
        assert np.allclose(g.sum(0), 0.0, atol=1e-12 * max(np.abs(g).max(), 1.0))


def test_gradient_matches_finite_differences_of_kl():
    n = 25
    y = synth.random_y(n, seed=21, scale=1.5).astype(np.float64)
    rp, col, val = synth.random_p(n, seed=21, k=5)
    P = _dense_p(n, rp, col, val)
    g, _, _, _ = oracle.gradient(y, rp, col, val, theta=0.0)
    h = 1e-6
    fd = np.empty_like(y)
    for i in range(n):
        for d in range(2):
            yp, ym = y.copy(), y.copy()
            yp[i, d] += h
            ym[i, d] -= h
            fd[i, d] = (_kl_dense(yp, P) - _kl_dense(ym, P)) / (2 * h)
    assert np.allclose(g, fd, rtol=1e-5, atol=1e-7 * np.abs(fd).max())


def test_attractive_forces_sum_to_zero_for_symmetric_p():
    inp = synth.make_inputs(0)
    fa = oracle.attractive(inp.Y, inp.row_ptr, inp.col, inp.val)
    scale = np.abs(fa).sum()
    assert np.abs(fa.sum(0)).max() < 1e-12 * scale


def test_two_points_closed_form():
    a = 0.75
    y = np.array([[0.0, 0.0], [a, 0.0]], np.float32)
    rp = np.array([0, 1, 2], np.int64)
    col = np.array([1, 0], np.int32)
    val = np.array([0.5, 0.5], np.float32)
    g, Z, inter, nodes = oracle.gradient(y, rp, col, val, theta=0.5)
    w = 1.0 / (1.0 + a * a)
    assert math.isclose(Z, 2.0 * w, rel_tol=1e-15)
    # g_0 = 4 (p w (y0 - y1) - w^2 (y0 - y1) / Z)
    g0 = 4.0 * (0.5 * w * (-a) - w * w * (-a) / (2 * w))
    assert math.isclose(g[0, 0], g0, rel_tol=1e-14) and g[0, 1] == 0.0
    assert math.isclose(g[1, 0], -g0, rel_tol=1e-14)
    assert inter == 2


def test_z_bounds_and_exactness():
    y = synth.random_y(400, seed=31, scale=4.0)
    Zex = oracle.z_exact(y)
    n = 400
    D2 = float(((y.max(0).astype(np.float64) - y.min(0)) ** 2).sum())
    assert n * (n - 1) / (1 + D2) <= Zex <= n * (n - 1)
    with oracle.State(y) as s:
        _, zi, _ = s.repulsive(0.0)
        assert math.isclose(oracle.ordered_sum(zi), Zex, rel_tol=1e-13)
        _, zi5, _ = s.repulsive(0.5)
        assert oracle.ordered_sum(zi5) > 0


def test_identical_points():
    n = 6
    y = np.full((n, 2), -3.5, np.float32)
    rp, col, val = synth.random_p(n, seed=2, k=3)
    g, Z, inter, nodes = oracle.gradient(y, rp, col, val, theta=0.5)
    assert nodes == 2  # root and one bucket
    assert Z == n * (n - 1) and inter == n * (n - 1)
    assert np.all(g == 0.0)


def test_huge_theta_accepts_the_root():
    # with theta -> infinity every point (not at the centre of mass) accepts the
    # root summary: F_rep,i = N w^2 (y_i - mean), Z_i = N w, w = 1/(1+|y_i-mean|^2)
    y = synth.random_y(300, seed=41, scale=1.0)
    with oracle.State(y) as s:
        frep, zi, inter = s.repulsive(1e9)
    m = y.astype(np.float64).mean(0)
    d = y.astype(np.float64) - m
    w = 1.0 / (1.0 + (d ** 2).sum(1))
    assert np.all(inter == 1)
    assert np.allclose(zi, 300 * w, rtol=1e-12)
    assert np.allclose(frep, 300 * (w * w)[:, None] * d, rtol=1e-10, atol=1e-14)


def test_acceptance_uses_cell_side_over_distance():
    # four points on the corners of a square of side a far from a fifth point
    # at distance D: the square's points fill quadrant cells of the root, and
    # the cell enclosing them is found by the tree.  Accepting that cell needs
    # side < theta * D exactly (R5), so interactions of the far point drop from
    # 4 exact pairs to 1 summary when theta crosses side / D.
    a = 1.0
    D = 64.0
    y = np.array([[0, 0], [a, 0], [0, a], [a, a], [D, D]], np.float32)
    t = oracle.tree(y)
    far = 4
    # the deepest internal node holding exactly the four square points
    cand = [v for v in range(t.nodes) if t.kind[v] == oracle.INTERNAL and t.count[v] == 4]
    v = max(cand, key=lambda u: t.level[u])
    side = 2 * t.box[6] * 2.0 ** -int(t.level[v])
    dist = float(np.hypot(*(y[far].astype(np.float64) - t.com[v])))
    eps = 1e-9
    with oracle.State(y) as s:
        _, _, inter_lo = s.repulsive(side / dist * (1 - eps), points=[far])
        _, _, inter_hi = s.repulsive(side / dist * (1 + eps), points=[far])
    assert inter_lo[0] >= 4 and inter_hi[0] == 1


def _enumerate_interactions(t, y, theta):
    """BH interaction lists without a depth-first walk: node v serves point i
    iff v accepts i and no proper ancestor accepts i; exact pairs come from
    singletons and rejected buckets whose ancestors all reject."""
    ys = y.astype(np.float64)[t.perm]
    nn = t.nodes
    n = ys.shape[0]
    side = 2 * t.box[6] * np.exp2(-t.level.astype(np.float64))
    F = np.zeros((n, 2))
    Zi = np.zeros(n)
    inter = np.zeros(n, np.int64)
    anc = [[] for _ in range(nn)]
    for v in range(1, nn):
        anc[v] = anc[t.parent[v]] + [t.parent[v]]
    for s in range(n):
        d = ys[s] - t.com
        d2 = (d ** 2).sum(1)
        acc = (side ** 2 < theta ** 2 * d2) & (t.kind != oracle.SINGLE)
        for v in range(nn):
            if any(acc[u] for u in anc[v]):
                continue
            if acc[v]:
                w = 1.0 / (1.0 + d2[v])
                Zi[s] += t.count[v] * w
                F[s] += t.count[v] * w * w * d[v]
                inter[s] += 1
            elif t.kind[v] != oracle.INTERNAL:
                for j in range(t.begin[v], t.end[v]):
                    if j == s:
                        continue
                    dj = ys[s] - ys[j]
                    w = 1.0 / (1.0 + dj @ dj)
                    Zi[s] += w
                    F[s] += w * w * dj
                    inter[s] += 1
    inv = np.empty(n, np.int64)
    inv[t.perm] = np.arange(n)
    return F[inv], Zi[inv], inter[inv]


@pytest.mark.parametrize("theta", [0.2, 0.5, 0.8, 1.5])
def test_dfs_equals_ancestor_enumeration(theta):
    y = synth.random_y(90, seed=51, scale=3.0, dups=4)
    with oracle.State(y) as s:
        t = s.tree()
        frep, zi, inter = s.repulsive(theta)
    F, Z, I = _enumerate_interactions(t, y, theta)
    assert np.array_equal(inter, I)
    assert np.allclose(zi, Z, rtol=1e-13)
    assert np.allclose(frep, F, rtol=1e-12, atol=1e-15)


def test_bh_error_shrinks_with_theta():
    inp = synth.make_inputs(0)
    g0, Z0, i0, _ = oracle.gradient(inp.Y, inp.row_ptr, inp.col, inp.val, theta=0.0)
    errs, inters = [], []
    for th in (0.8, 0.5, 0.2):
        g, Z, inter, _ = oracle.gradient(inp.Y, inp.row_ptr, inp.col, inp.val, theta=th)
        errs.append(np.linalg.norm(g - g0) / np.linalg.norm(g0))
        inters.append(inter)
    assert errs[0] > errs[1] > errs[2] and errs[1] < 2e-2
    assert inters[0] < inters[1] < inters[2] < i0


# ---------------------------------------------------------------- update, KL
def test_update_hand_computed(golden_dir):
    for line in _rows(os.path.join(golden_dir, "update_steps.txt")):
        lhs, rhs = line.split("|")
        y0, u0, g0, g, eta, mu, mg = (float(x) for x in lhs.split())
        y1, u1, gain1 = (float(x) for x in rhs.split())
        y = np.array([y0]); u = np.array([u0]); gains = np.array([g0])
        oracle.update(y, u, gains, np.array([g]), eta, mu, mg)
        assert math.isclose(y[0], y1, abs_tol=1e-12)
        assert math.isclose(u[0], u1, abs_tol=1e-12)
        assert math.isclose(gains[0], gain1, abs_tol=1e-12)


def test_kl_matches_dense_and_is_nonnegative():
    n = 80
    y = synth.random_y(n, seed=61, scale=2.0)
    rp, col, val = synth.random_p(n, seed=61, k=7)
    P = _dense_p(n, rp, col, val).astype(np.float64)
    k = oracle.kl(y, rp, col, val)
    assert k >= 0
    assert math.isclose(k, _kl_dense(y.astype(np.float64), P), rel_tol=1e-12)


def test_oracle_step_descends_kl():
    inp = synth.make_inputs(0)
    y = inp.Y.astype(np.float64)
    u = np.zeros_like(y)
    gains = np.ones_like(y)
    kl0 = oracle.kl(y, inp.row_ptr, inp.col, inp.val)
    for it in range(20):
        oracle.step(y, u, gains, inp.row_ptr, inp.col, inp.val, 0.5, 1.0, 200.0, 0.5)
    assert oracle.kl(y, inp.row_ptr, inp.col, inp.val) < kl0
