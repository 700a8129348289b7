"""fp64 CPU oracle of the input similarities (test infrastructure only).

Only the tests, the smoke check and the CPU-baseline leg of the benchmark may
import this module; the GPU library never touches it.  It follows the
Background section ("Input similarity computation", the sparse approximation
equation and the symmetrisation under it) and the Binary Search Perplexity
subsection, in plain vectorised numpy:

* conditional similarities: for point i with neighbour set N_i (its k nearest
  neighbours, distances d_ij),
      p_{j|i} = exp(-d_ij^2 / 2 sigma_i^2) / sum_{l in N_i} exp(-d_il^2 / 2 sigma_i^2)
  and 0 outside N_i;
* sigma_i^2 is found by binary search: each step takes the middle point of
  the current interval of sigma_i^2 and keeps the half in which the
  perplexity of p_{.|i} crosses the target u.  The perplexity is exp(H) with
  H the Shannon entropy in nats (2^H in bits, the same number);
* symmetrisation: p_ij = (p_{j|i} + p_{i|j}) / (2N) over the union of the
  two sparsity patterns (one sparse-matrix addition, a library step).

Readings where the paper is silent:
* the search runs to machine precision: it stops when the midpoint of the
  interval equals one of its ends, and returns the upper end.  Its starting
  interval is [0, max_j D'_j] (D' below), doubled at the top until the
  perplexity there reaches u;
* the squared distances are shifted by their row minimum, D'_j = d_ij^2 -
  min_l d_il^2, before the exponentials; the ratios, hence p_{.|i}, do not
  change and no exponential underflows to an all-zero row;
* u > k has no root (the perplexity of k neighbours is at most k): the
  interval grows until sigma^2 is infinite and p_{.|i} is uniform; u at or
  below the number of ties at the minimum distance drives sigma^2 to the
  smallest double, which leaves p uniform over those ties;
* a row whose distances are all equal is uniform whatever sigma^2.
"""
from __future__ import annotations

import numpy as np
import scipy.sparse as sp

_MAX_STEPS = 2200  # enough to cross the whole fp64 range by halving


def _entropy(dp: np.ndarray, s2: np.ndarray) -> np.ndarray:
    """Entropy (nats) of the Gaussian weights over the shifted squared
    distances dp (rows x k) at sigma^2 = s2 (rows,); infinite s2 gives log k."""
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        a = dp / (2.0 * s2[:, None])
        a = np.where(np.isinf(s2)[:, None], 0.0, a)
        w = np.exp(-a)
        s = w.sum(axis=1)
        # a e^-a -> 0 where the weight underflows (a = inf)
        return np.log(s) + np.where(w > 0.0, a * w, 0.0).sum(axis=1) / s


def sigma2(dist: np.ndarray, u: float) -> np.ndarray:
    """sigma_i^2 of every row of the neighbour distances dist (n x k)."""
    d = np.asarray(dist, dtype=np.float64)
    dd = d * d
    dp = dd - dd.min(axis=1, keepdims=True)
    target = np.log(float(u))
    n = dp.shape[0]
    lo = np.zeros(n)
    top = dp.max(axis=1)
    flat = top == 0.0
    hi = np.where(flat, 1.0, top)
    # grow the top of the interval until the perplexity there reaches u
    grow = ~flat & (_entropy(dp, hi) < target)
    while grow.any():
        with np.errstate(over="ignore"):  # hi = inf ends the row (u above reach)
            hi[grow] *= 2.0
        grow &= np.isfinite(hi)
        idx = np.nonzero(grow)[0]
        if idx.size:
            grow[idx] = _entropy(dp[idx], hi[idx]) < target
    # halve: keep the half whose ends bracket the target
    live = ~flat & np.isfinite(hi)
    for _ in range(_MAX_STEPS):
        idx = np.nonzero(live)[0]
        if idx.size == 0:
            break
        mid = 0.5 * (lo[idx] + hi[idx])
        done = (mid <= lo[idx]) | (mid >= hi[idx])
        live[idx[done]] = False
        idx, mid = idx[~done], mid[~done]
        below = _entropy(dp[idx], mid) < target
        lo[idx[below]] = mid[below]
        hi[idx[~below]] = mid[~below]
    return hi


def conditional(dist: np.ndarray, u: float):
    """(sigma^2 [n], p_{j|i} [n x k]) for neighbour distances dist (n x k)."""
    d = np.asarray(dist, dtype=np.float64)
    s2 = sigma2(d, u)
    dd = d * d
    dp = dd - dd.min(axis=1, keepdims=True)
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):  # a = inf gives w = 0
        a = np.where(np.isinf(s2)[:, None], 0.0, dp / (2.0 * s2[:, None]))
    w = np.exp(-a)
    return s2, w / w.sum(axis=1, keepdims=True)


def symmetrize(idx: np.ndarray, pcond: np.ndarray, n: int):
    """p_ij = (p_{j|i} + p_{i|j}) / (2N) as CSR (row_ptr int64, col int32,
    val float64) with sorted columns.  The pattern is the union of the
    neighbour relations in both directions, zero values included: the
    entries (i, j, p_{j|i}) and (j, i, p_{j|i}) are summed by position."""
    k = idx.shape[1]
    r = np.repeat(np.arange(n, dtype=np.int64), k)
    c = np.asarray(idx, np.int64).ravel()
    v = np.asarray(pcond, np.float64).ravel()
    s = sp.coo_matrix((np.concatenate([v, v]), (np.concatenate([r, c]), np.concatenate([c, r]))),
                      shape=(n, n)).tocsr()  # duplicates summed, zeros kept
    s.sort_indices()
    return s.indptr.astype(np.int64), s.indices.astype(np.int32), s.data / (2.0 * n)


def affinities(idx: np.ndarray, dist: np.ndarray, u: float):
    """The symmetric P of the neighbour lists (idx, dist): (row_ptr, col, val
    fp64, sigma^2)."""
    s2, pc = conditional(dist, u)
    rp, col, val = symmetrize(idx, pc, idx.shape[0])
    return rp, col, val, s2
