"""The ring generators used at the largest point count: their P is a valid
affinity matrix (symmetric, zero diagonal, sum 1, sorted distinct columns)
and their neighbour lists are valid kNN output (k distinct non-self
neighbours, ascending distances)."""
import numpy as np
import pytest
import scipy.sparse as sp

import synth


@pytest.mark.parametrize("n,m", [(5, 2), (7, 3), (50, 2), (1001, 4), (4096, 1)])
def test_ring_p_is_a_valid_affinity_matrix(n, m):
    rp, col, val = synth.ring_p(n, 3, m=m)
    assert rp.dtype == np.int64 and col.dtype == np.int32 and val.dtype == np.float32
    assert np.array_equal(rp, np.arange(0, 2 * m * n + 1, 2 * m))
    for i in range(n):
        c = col[rp[i]:rp[i + 1]]
        assert np.all(np.diff(c) > 0) and i not in c
    P = sp.csr_matrix((val.astype(np.float64), col, rp), shape=(n, n))
    assert abs(P - P.T).max() == 0
    assert abs(P.sum() - 1.0) < 1e-6


def test_ring_p_rejects_too_many_offsets():
    with pytest.raises(ValueError):
        synth.ring_p(6, 1, m=3)


@pytest.mark.parametrize("n,k", [(2, 1), (9, 8), (300, 5), (5000, 90)])
def test_ring_knn_lists(n, k):
    kn = synth.ring_knn(n, k, 4)
    assert kn.idx.shape == (n, k) and kn.dist.shape == (n, k)
    for i, r in enumerate(kn.idx.tolist()):
        assert len(set(r)) == k and i not in r and min(r) >= 0 and max(r) < n
    assert np.array_equal(np.bincount(kn.idx.ravel(), minlength=n), np.full(n, k))
    assert np.all(np.diff(kn.dist, axis=1) >= 0) and kn.dist.min() >= 0 and kn.dist.max() < 3
