"""Pins of the fp64 similarity oracle (Background: input similarities and the
sparse approximation; Binary Search Perplexity).

Two facts fix each conditional row p_{.|i} completely: it has the Gaussian
form of the sparse-approximation equation (log p_{j|i} is affine in d_ij^2
with slope -1 / (2 sigma_i^2)), and its perplexity equals u (the entropy grows
strictly with sigma_i^2, so only one sigma_i^2 gives u).  The tests check both
facts on the oracle's output with library routines (scipy's entropy, a
least-squares line), plus closed and brute-force cases: a two-neighbour row
solved by root finding on the binary entropy, uniform rows, ties, and the
symmetrisation against dense matrix arithmetic.
"""
import numpy as np
import pytest
import scipy.optimize as so
import scipy.stats as ss

import synth
from oracle import affinities as A


def _rows(n=300, k=40, seed=7):
    rng = np.random.default_rng(seed)
    d = np.sort(rng.uniform(0.0, 3.0, size=(n, k)), axis=1).astype(np.float32)
    return d


@pytest.mark.parametrize("u", [5.0, 12.5, 30.0])
def test_perplexity_equals_u(u):
    d = _rows(k=90)
    s2, p = A.conditional(d, u)
    perp = np.exp(ss.entropy(p, axis=1))
    assert np.allclose(perp, u, rtol=1e-10, atol=0.0)
    assert np.allclose(p.sum(axis=1), 1.0, rtol=1e-14)


def test_gaussian_form_slope():
    d = _rows().astype(np.float64)
    s2, p = A.conditional(d, 10.0)
    for i in range(0, d.shape[0], 17):
        slope, icpt = np.polyfit(d[i] ** 2, np.log(p[i]), 1)
        assert abs(slope * (2.0 * s2[i]) + 1.0) < 1e-9
        resid = np.log(p[i]) - (slope * d[i] ** 2 + icpt)
        assert np.abs(resid).max() < 1e-9


def test_sigma_grows_with_perplexity():
    d = _rows()
    s_a = A.sigma2(d, 6.0)
    s_b = A.sigma2(d, 20.0)
    assert (s_b > s_a).all()


def test_two_neighbours_binary_entropy():
    # p = (q, 1 - q) with q the nearer neighbour's share; H(q) = log u fixes q
    for a, b, u in [(0.3, 1.1, 1.5), (0.0, 2.0, 1.9), (1.0, 1.2, 1.01)]:
        d = np.array([[a, b]], np.float32)
        _, p = A.conditional(d, u)
        h = lambda q: -(q * np.log(q) + (1 - q) * np.log(1 - q)) - np.log(u)
        q = so.brentq(h, 0.5 + 1e-15, 1.0 - 1e-15, xtol=1e-16, rtol=1e-15)
        assert abs(p[0, 0] - q) < 1e-12, (p, q)


def test_uniform_rows():
    d = np.full((3, 7), 0.8, np.float32)
    _, p = A.conditional(d, 4.0)
    assert np.array_equal(p, np.full((3, 7), 1.0 / 7))
    # no root when u > k: the search ends uniform
    d = _rows(n=5, k=6)
    s2, p = A.conditional(d, 7.0)
    assert np.isinf(s2).all() and np.allclose(p, 1.0 / 6, rtol=1e-15)


def test_ties_at_the_minimum():
    # three neighbours tie at the minimum; u below the tie count leaves them uniform
    d = np.array([[0.5, 0.5, 0.5, 1.0, 2.0, 2.5]], np.float32)
    _, p = A.conditional(d, 2.0)
    assert np.allclose(p[0, :3], 1.0 / 3, rtol=1e-12) and p[0, 3:].max() < 1e-300


def test_symmetrize_matches_dense():
    rng = np.random.default_rng(3)
    n, k = 12, 4
    idx = np.array([rng.choice(np.delete(np.arange(n), i), k, replace=False) for i in range(n)], np.int32)
    pc = rng.random((n, k))
    pc[5, 2] = 0.0  # an underflowed weight keeps its place in the pattern
    pc /= pc.sum(axis=1, keepdims=True)
    rp, col, val = A.symmetrize(idx, pc, n)
    pattern = {(i, int(j)) for i in range(n) for j in idx[i]}
    pattern |= {(j, i) for i, j in pattern}
    assert {(i, int(c)) for i in range(n) for c in col[rp[i]:rp[i + 1]]} == pattern
    dense = np.zeros((n, n))
    for i in range(n):
        dense[i, idx[i]] = pc[i]
    ref = (dense + dense.T) / (2 * n)
    got = np.zeros((n, n))
    for i in range(n):
        assert (np.diff(col[rp[i]:rp[i + 1]]) > 0).all()
        got[i, col[rp[i]:rp[i + 1]]] = val[rp[i]:rp[i + 1]]
    assert np.array_equal(got != 0, ref != 0)
    assert np.abs(got - ref).max() < 1e-16


def test_workload_affinities_are_a_joint_distribution():
    kn = synth.make_knn(0)
    rp, col, val, s2 = A.affinities(kn.idx, kn.dist, 30.0)
    n = kn.n
    assert abs(val.sum() - 1.0) < 1e-12
    rows = np.repeat(np.arange(n), np.diff(rp))
    assert not (rows == col).any()
    m = {(int(r), int(c)): v for r, c, v in zip(rows, col, val)}
    for (r, c), v in list(m.items())[::997]:
        assert m[(c, r)] == v
    # every neighbour relation appears, and nothing else
    assert rp[-1] == len({(min(i, int(j)), max(i, int(j))) for i in range(n) for j in kn.idx[i]}) * 2
