"""Pins of the 3-D fp64 oracle against facts the paper and the mathematics fix.

As for the 2-D oracle, no test re-types an oracle formula and compares it
with itself: each checks the oracle against hand-worked fixtures, a
different formulation of the same definition (a string interleave, a
geometric top-down octant partition, the dense exact gradient, central
finite differences of the KL cost, an ancestor enumeration of the
interaction lists instead of a depth-first walk), a closed form or an
invariant.
"""
import math
import os

import numpy as np
import pytest

import oracle
import synth


def _rows(path):
    return [line.split() for line in open(path) if line.strip() and not line.startswith("#")]


# ---------------------------------------------------------------- Morton codes
def test_interleave3_worked_examples(golden_dir):
    for m0, m1, m2, code in _rows(os.path.join(golden_dir, "morton3_worked_example.txt")):
        assert oracle.interleave3(int(m0), int(m1), int(m2)) == int(code)


def _interleave3_by_strings(m0, m1, m2):
    a, b, c = (format(m, "021b") for m in (m0, m1, m2))
    # most significant first: each 3-bit digit reads (dim 2, dim 1, dim 0)
    return int("".join(z + y + x for x, y, z in zip(a, b, c)), 2)


def test_interleave3_matches_string_interleave():
    rng = np.random.default_rng(3)
    cases = [(0, 0, 0), (2**21 - 1, 0, 0), (0, 2**21 - 1, 0), (0, 0, 2**21 - 1)]
    cases += [tuple(int(v) for v in rng.integers(0, 2**21, 3)) for _ in range(300)]
    for m in cases:
        assert oracle.interleave3(*m) == _interleave3_by_strings(*m)


def test_quantisation3_truncates_hand_worked_case(golden_dir):
    rows = _rows(os.path.join(golden_dir, "quantisation3_truncation.txt"))
    y = np.array([[float(r[0]), float(r[1]), float(r[2])] for r in rows], np.float32)
    codes, grid, yrs = oracle.morton3(y)
    for k, r in enumerate(rows):
        assert [int(g) for g in grid[k]] == [int(r[3], 16), int(r[4], 16), int(r[5], 16)], k
        assert int(codes[k]) == int(r[6], 16), k
    assert list(yrs[:3]) == [0.0, 0.0, 0.0] and yrs[3] == 2.0**21 / 3.0


def test_quantisation3_extremes_and_centring():
    y = synth.random_y3(301, seed=4, scale=3.0)
    codes, grid, yrs = oracle.morton3(y)
    ext = y.max(0).astype(np.float64) - y.min(0)
    wide = int(np.argmax(ext))
    assert grid[np.argmin(y[:, wide]), wide] == 0
    assert grid[np.argmax(y[:, wide]), wide] == 2**21 - 1
    for d in range(3):
        o = np.argsort(y[:, d], kind="stable")
        assert np.all(np.diff(grid[o, d].astype(np.int64)) >= 0)
        mid = (int(grid[:, d].min()) + int(grid[:, d].max())) / 2
        assert abs(mid - 2**20) < 2**20 * 1e-6 + 2
    assert np.all(codes < np.uint64(1) << np.uint64(63))  # the top bit stays clear


# ---------------------------------------------------------------- octree
def _geometric_octree(grid):
    """Top-down partition by octant bits of the grid coordinates, level by
    level (the uncompressed tree), then removal of single-child cells other
    than the root.  Returns {(level, frozenset(points), kind)}."""
    out = set()

    def rec(level, pts, is_root):
        if len(pts) == 1 and not is_root:
            out.add((level, frozenset(pts), oracle.SINGLE))
            return
        if level == 21:
            out.add((21, frozenset(pts), oracle.BUCKET))
            return
        bit = 20 - level
        octs = {}
        for p in pts:
            o = sum(((int(grid[p, d]) >> bit) & 1) << d for d in range(3))
            octs.setdefault(o, []).append(p)
        if len(octs) > 1 or is_root:
            out.add((level, frozenset(pts), oracle.INTERNAL))
        for o in sorted(octs):
            rec(level + 1, octs[o], False)

    rec(0, list(range(grid.shape[0])), True)
    return out


@pytest.mark.parametrize("seed,n,scale,dups", [(1, 2, 1.0, 0), (2, 9, 1.0, 0), (3, 50, 1.0, 4),
                                               (4, 150, 1e-3, 12), (5, 220, 30.0, 0)])
def test_octree_matches_geometric_partition(seed, n, scale, dups):
    y = synth.random_y3(n, seed=seed, scale=scale, dups=dups)
    y[-1] = y[0] + np.float32(1e-6) * scale  # near-coincident points reach deep levels
    t = oracle.tree3(y)
    _, grid, _ = oracle.morton3(y)
    got = {(int(t.level[v]), frozenset(int(p) for p in t.perm[t.begin[v]:t.end[v]]), int(t.kind[v]))
           for v in range(t.nodes)}
    assert got == _geometric_octree(grid)


def test_octree_invariants_and_summaries():
    y = synth.random_y3(3000, seed=11, scale=2.0, dups=40)
    t = oracle.tree3(y)
    nn = t.nodes
    assert t.level[0] == 0 and t.begin[0] == 0 and t.end[0] == 3000 and t.parent[0] == -1
    assert np.all(np.diff(t.begin.astype(np.int64) * 64 + t.level) > 0)
    internal = t.kind == oracle.INTERNAL
    assert internal.sum() <= 3000 - 1
    nchild = np.bincount(t.parent[1:], minlength=nn)
    assert np.all(nchild[internal][1:] >= 2) and np.all(nchild <= 8)
    for v in range(1, nn):
        p = t.parent[v]
        assert t.level[p] < t.level[v] and t.begin[p] <= t.begin[v] and t.end[v] <= t.end[p]
    for v in np.nonzero(t.kind == oracle.BUCKET)[0]:
        assert t.level[v] == 21 and np.all(t.sorted_codes[t.begin[v]:t.end[v]] == t.sorted_codes[t.begin[v]])
    # summaries: the root holds every point at the mean; counts add up; centres lie in the hull
    assert t.count[0] == 3000
    assert np.allclose(t.com[0], y.astype(np.float64).mean(0), rtol=0, atol=1e-12)
    csum = np.zeros(nn, np.int64)
    np.add.at(csum, t.parent[1:], t.count[1:].astype(np.int64))
    assert np.array_equal(csum[internal], t.count[internal].astype(np.int64))
    ys = y.astype(np.float64)[t.perm]
    for v in range(0, nn, 29):
        pts = ys[t.begin[v]:t.end[v]]
        assert np.all(t.com[v] >= pts.min(0) - 1e-12) and np.all(t.com[v] <= pts.max(0) + 1e-12)


# ---------------------------------------------------------------- gradient pins
def _dense_p(n, row_ptr, col, val):
    P = np.zeros((n, n))
    for i in range(n):
        for k in range(row_ptr[i], row_ptr[i + 1]):
            P[i, col[k]] += val[k]
    return P


def _exact_gradient(y, P, alpha=1.0):
    """dC/dy_i = 4 sum_j (alpha p_ij - q_ij) q_ij Z (y_i - y_j)  (Gradient Descent)."""
    y = y.astype(np.float64)
    diff = y[:, None, :] - y[None, :, :]
    w = 1.0 / (1.0 + (diff ** 2).sum(-1))
    np.fill_diagonal(w, 0.0)
    Z = w.sum()
    q = w / Z
    return 4.0 * (((alpha * P - q) * q * Z)[:, :, None] * diff).sum(1), Z


def _kl_dense(y, P):
    diff = y[:, None, :] - y[None, :, :]
    w = 1.0 / (1.0 + (diff ** 2).sum(-1))
    np.fill_diagonal(w, 0.0)
    q = w / w.sum()
    m = P > 0
    return float((P[m] * np.log(P[m] / q[m])).sum())


@pytest.mark.parametrize("n,seed,dups", [(2, 1, 0), (3, 2, 0), (70, 3, 0), (160, 4, 6)])
def test_theta0_equals_exact_gradient(n, seed, dups):
    y = synth.random_y3(n, seed=seed, scale=2.0, dups=dups)
    rp, col, val = synth.random_p(n, seed=seed, k=6)
    P = _dense_p(n, rp, col, val)
    for alpha in (1.0, 12.0):
        g, Z, inter, _ = oracle.gradient3(y, rp, col, val, theta=0.0, exaggeration=alpha)
        gref, Zref = _exact_gradient(y, P, alpha)
        assert math.isclose(Z, Zref, rel_tol=1e-13)
        assert inter == n * (n - 1)
        assert np.allclose(g, gref, rtol=1e-11, atol=1e-14 * max(np.abs(gref).max(), 1.0))
        assert np.allclose(g.sum(0), 0.0, atol=1e-12 * max(np.abs(g).max(), 1.0))


def test_gradient_matches_finite_differences_of_kl():
    n = 22
    y = synth.random_y3(n, seed=21, scale=1.5).astype(np.float64)
    rp, col, val = synth.random_p(n, seed=21, k=5)
    P = _dense_p(n, rp, col, val)
    g, _, _, _ = oracle.gradient3(y, rp, col, val, theta=0.0)
    h = 1e-6
    fd = np.empty_like(y)
    for i in range(n):
        for d in range(3):
            yp, ym = y.copy(), y.copy()
            yp[i, d] += h
            ym[i, d] -= h
            fd[i, d] = (_kl_dense(yp, P) - _kl_dense(ym, P)) / (2 * h)
    assert np.allclose(g, fd, rtol=1e-5, atol=1e-7 * np.abs(fd).max())


def test_attractive_forces_sum_to_zero_for_symmetric_p():
    inp = synth.make_inputs(0, dim=3)
    fa = oracle.attractive3(inp.Y, inp.row_ptr, inp.col, inp.val)
    assert np.abs(fa.sum(0)).max() < 1e-12 * np.abs(fa).sum()


def test_two_points_closed_form():
    a = 0.6
    y = np.array([[0.0, 0.0, 0.0], [0.0, 0.0, a]], np.float32)
    rp = np.array([0, 1, 2], np.int64)
    col = np.array([1, 0], np.int32)
    val = np.array([0.5, 0.5], np.float32)
    g, Z, inter, nodes = oracle.gradient3(y, rp, col, val, theta=0.5)
    a = float(np.float32(a))
    w = 1.0 / (1.0 + a * a)
    assert math.isclose(Z, 2.0 * w, rel_tol=1e-15)
    g0 = 4.0 * (0.5 * w * (-a) - w * w * (-a) / (2 * w))
    assert math.isclose(g[0, 2], g0, rel_tol=1e-14) and g[0, 0] == 0.0 and g[0, 1] == 0.0
    assert math.isclose(g[1, 2], -g0, rel_tol=1e-14)
    assert inter == 2


def test_z_bounds_and_exactness():
    n = 350
    y = synth.random_y3(n, seed=31, scale=4.0)
    Zex = oracle.z_exact3(y)
    D2 = float(((y.max(0).astype(np.float64) - y.min(0)) ** 2).sum())
    assert n * (n - 1) / (1 + D2) <= Zex <= n * (n - 1)
    with oracle.State3(y) as s:
        _, zi, _ = s.repulsive(0.0)
        assert math.isclose(oracle.ordered_sum(zi), Zex, rel_tol=1e-13)


def test_identical_points():
    n = 6
    y = np.full((n, 3), 2.25, np.float32)
    rp, col, val = synth.random_p(n, seed=2, k=3)
    g, Z, inter, nodes = oracle.gradient3(y, rp, col, val, theta=0.5)
    assert nodes == 2 and Z == n * (n - 1) and inter == n * (n - 1) and np.all(g == 0.0)


def test_huge_theta_accepts_the_root():
    n = 300
    y = synth.random_y3(n, seed=41, scale=1.0)
    with oracle.State3(y) as s:
        frep, zi, inter = s.repulsive(1e9)
    d = y.astype(np.float64) - y.astype(np.float64).mean(0)
    w = 1.0 / (1.0 + (d ** 2).sum(1))
    assert np.all(inter == 1)
    assert np.allclose(zi, n * w, rtol=1e-12)
    assert np.allclose(frep, n * (w * w)[:, None] * d, rtol=1e-10, atol=1e-14)


def test_acceptance_uses_cell_side_over_distance():
    # eight corners of a cube of side a far from a ninth point at distance D:
    # accepting the cell around the cube needs side < theta * D exactly (R5)
    a, D = 1.0, 64.0
    corners = [[x, y, z] for x in (0, a) for y in (0, a) for z in (0, a)]
    y = np.array(corners + [[D, D, D]], np.float32)
    t = oracle.tree3(y)
    cand = [v for v in range(t.nodes) if t.kind[v] == oracle.INTERNAL and t.count[v] == 8]
    v = max(cand, key=lambda u: t.level[u])
    side = 2 * t.box[9] * 2.0 ** -int(t.level[v])
    dist = float(np.linalg.norm(y[8].astype(np.float64) - t.com[v]))
    with oracle.State3(y) as s:
        _, _, lo = s.repulsive(side / dist * (1 - 1e-9), points=[8])
        _, _, hi = s.repulsive(side / dist * (1 + 1e-9), points=[8])
    assert lo[0] >= 8 and hi[0] == 1


def _enumerate_interactions(t, y, theta):
    """Interaction lists without a walk: node v serves point i iff v accepts i
    and no proper ancestor does; exact pairs from singletons and rejected
    buckets whose ancestors all reject."""
    ys = y.astype(np.float64)[t.perm]
    nn, n = t.nodes, ys.shape[0]
    side = 2 * t.box[9] * np.exp2(-t.level.astype(np.float64))
    F = np.zeros((n, 3))
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
                    if j != s:
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
    y = synth.random_y3(90, seed=51, scale=3.0, dups=4)
    with oracle.State3(y) as s:
        t = s.tree()
        frep, zi, inter = s.repulsive(theta)
    F, Z, I = _enumerate_interactions(t, y, theta)
    assert np.array_equal(inter, I)
    assert np.allclose(zi, Z, rtol=1e-13)
    assert np.allclose(frep, F, rtol=1e-12, atol=1e-15)


def test_kl_matches_dense_and_steps_descend():
    n = 80
    y = synth.random_y3(n, seed=61, scale=2.0)
    rp, col, val = synth.random_p(n, seed=61, k=7)
    P = _dense_p(n, rp, col, val)
    k = oracle.kl3(y, rp, col, val)
    assert k >= 0 and math.isclose(k, _kl_dense(y.astype(np.float64), P), rel_tol=1e-12)
    inp = synth.make_inputs(0, dim=3)
    y = inp.Y.astype(np.float64)
    u, gains = np.zeros_like(y), np.ones_like(y)
    kl0 = oracle.kl3(y, inp.row_ptr, inp.col, inp.val)
    for _ in range(20):
        oracle.step3(y, u, gains, inp.row_ptr, inp.col, inp.val, 0.5, 1.0, 200.0, 0.5)
    assert oracle.kl3(y, inp.row_ptr, inp.col, inp.val) < kl0
