"""Seeded synthetic inputs for the BH t-SNE gradient step.

This module only draws random inputs: an embedding Y (n x 2, float32) and a
sparse symmetric affinity matrix P in CSR form.  It holds none of the gradient
step's arithmetic, so both the fp64 oracle and the GPU library consume exactly
the same arrays.

Shapes follow the paper's workloads (Background, "Input similarity
computation"): every row of the conditional matrix keeps k = floor(3u) = 90
neighbours (perplexity u = 30), the conditional rows are normalised, and P is
the symmetrised (P + P^T) / (2N), so sum(P) = 1 and p_ii = 0.  The neighbour
sets are drawn inside synthetic clusters instead of coming from a kNN search
over a real dataset; cluster labels are assigned through a seeded random
permutation, so like a real dataset the index order carries no locality.

Recipe (per config c, ``seed = 22121150 + c``):
  1. cluster sizes: equal, Dirichlet(1) split or Zipf(1.1) ranks, rounded by
     largest remainder;
  2. labels: cluster c owns a contiguous slice of a random permutation;
  3. row i draws k distinct neighbours uniformly from its own cluster,
     excluding i (all m-1 members when the cluster size m <= k);
  4. weights exp(-d^2) with d ~ U(0, 3), row-normalised in fp64;
  5. P = (P + P^T) / (2N) in fp64, summed duplicates, sorted columns, then
     stored as fp32 values, int32 columns and int64 row pointers;
  6. Y ~ N(0, 1e-4 I) (early phase) or a late-phase clustered snapshot with
     centres ~ U(-50, 50)^2 and per-cluster spread sigma ~ U(0.1, 2);
     optionally a fraction of points copies another point of its cluster.
"""
from __future__ import annotations

import dataclasses
import hashlib
import time
from typing import Optional

import numpy as np
import scipy.sparse as sp
from numpy.random import PCG64, Generator, SeedSequence

SEED_BASE = 22121150
K_NEIGHBOURS = 90


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: sizes, P recipe, Y recipe and run schedule."""

    cid: int
    n: int
    clusters: int
    sizes: str              # "equal" | "dirichlet" | "zipf"
    y_kind: str             # "gauss" (N(0, 1e-4 I)) | "clustered"
    dup_frac: float = 0.0   # fraction of points that copy another point
    iters: int = 1000
    theta: float = 0.5
    description: str = ""

    def schedule(self, it: int) -> dict:
        """Optimiser parameters of iteration ``it`` (0-based).

        Early exaggeration 12 for the first 250 iterations and momentum
        0.5 -> 0.8 follow the usual t-SNE optimiser; the learning rate is
        max(N/12, 200).  The small workload uses a fixed 200/0.5/12 schedule
        and the late-phase workloads run without exaggeration.
        """
        if self.cid == 0:
            return dict(exaggeration=12.0, learning_rate=200.0, momentum=0.5)
        lr = max(self.n / 12.0, 200.0)
        if self.y_kind == "clustered":
            return dict(exaggeration=1.0, learning_rate=lr, momentum=0.8)
        early = it < 250
        return dict(exaggeration=12.0 if early else 1.0, learning_rate=lr,
                    momentum=0.5 if early else 0.8)


WORKLOADS = {
    0: Workload(0, 2_000, 10, "equal", "gauss", iters=50,
                description="2k points, 10 equal clusters, early-phase Y"),
    1: Workload(1, 70_000, 10, "equal", "gauss", iters=1000,
                description="70k points, 10 equal clusters, early-phase Y"),
    2: Workload(2, 1_300_000, 30, "dirichlet", "gauss", iters=1000,
                description="1.3M points, 30 Dirichlet(1) clusters, early-phase Y"),
    3: Workload(3, 5_000_000, 100, "zipf", "clustered", iters=200,
                description="5M points, 100 Zipf(1.1) clusters, late-phase Y"),
    4: Workload(4, 1_300_000, 30, "dirichlet", "clustered", dup_frac=0.05, iters=100,
                description="1.3M points, 30 Dirichlet(1) clusters, late-phase Y, 5% duplicates"),
}


def _streams(cid: int):
    ss = SeedSequence(SEED_BASE + cid)
    kids = ss.spawn(5)
    return [Generator(PCG64(k)) for k in kids]  # sizes, labels, neighbours, weights, Y


def _largest_remainder(fracs: np.ndarray, n: int) -> np.ndarray:
    raw = fracs / fracs.sum() * n
    base = np.floor(raw).astype(np.int64)
    rem = n - int(base.sum())
    order = np.argsort(-(raw - base), kind="stable")
    base[order[:rem]] += 1
    return base


def cluster_sizes(w: Workload, n: int, rng: Generator) -> np.ndarray:
    c = w.clusters
    if w.sizes == "equal":
        return _largest_remainder(np.ones(c), n)
    if w.sizes == "dirichlet":
        return _largest_remainder(rng.dirichlet(np.ones(c)), n)
    if w.sizes == "zipf":
        return _largest_remainder(np.arange(1, c + 1, dtype=np.float64) ** -1.1, n)
    raise ValueError(w.sizes)


def _neighbours_for_cluster(members: np.ndarray, k: int, rng: Generator):
    """Return (rows, cols) of k distinct within-cluster neighbours per member."""
    m = members.size
    if m <= 1:
        return np.empty(0, np.int64), np.empty(0, np.int64)
    if m - 1 <= k:  # take every other member
        pos = np.arange(m)
        nb = np.tile(np.arange(m - 1), (m, 1))
        nb = nb + (nb >= pos[:, None])
        rows = np.repeat(members, m - 1)
        return rows.astype(np.int64), members[nb.ravel()].astype(np.int64)
    pos = np.arange(m)
    if m <= 4096:  # random keys, keep the k smallest
        out = np.empty((m, k), np.int64)
        step = max(1, (1 << 24) // m)
        for s in range(0, m, step):
            keys = rng.random((min(step, m - s), m - 1))
            out[s:s + step] = np.argpartition(keys, k - 1, axis=1)[:, :k]
        nb = out
    else:  # rejection: redraw duplicated entries until every row is distinct
        nb = rng.integers(0, m - 1, size=(m, k), dtype=np.int64)
        nb.sort(axis=1)
        bad = np.nonzero((nb[:, 1:] == nb[:, :-1]).any(axis=1))[0]
        while bad.size:
            sub = nb[bad]
            dup = np.zeros_like(sub, dtype=bool)
            dup[:, 1:] = sub[:, 1:] == sub[:, :-1]
            sub[dup] = rng.integers(0, m - 1, size=int(dup.sum()), dtype=np.int64)
            sub.sort(axis=1)
            nb[bad] = sub
            still = (sub[:, 1:] == sub[:, :-1]).any(axis=1)
            bad = bad[still]
    nb = nb + (nb >= pos[:, None])  # skip self
    rows = np.repeat(members, k)
    return rows.astype(np.int64), members[nb.ravel()].astype(np.int64)


def make_p(w: Workload, n: int, labels_perm: np.ndarray, sizes: np.ndarray,
           rng_nb: Generator, rng_w: Generator, k: int = K_NEIGHBOURS):
    """Build the symmetric CSR matrix P = (P_cond + P_cond^T) / (2N)."""
    rows_l, cols_l = [], []
    off = 0
    for c in range(sizes.size):
        members = labels_perm[off:off + sizes[c]]
        off += sizes[c]
        r, cc = _neighbours_for_cluster(members, k, rng_nb)
        rows_l.append(r)
        cols_l.append(cc)
    rows = np.concatenate(rows_l)
    cols = np.concatenate(cols_l)
    del rows_l, cols_l
    d = rng_w.uniform(0.0, 3.0, size=rows.size)
    wts = np.exp(-d * d)
    del d
    cond = sp.csr_matrix((wts, (rows, cols)), shape=(n, n), dtype=np.float64)
    del rows, cols, wts
    rs = np.asarray(cond.sum(axis=1)).ravel()
    rs[rs == 0] = 1.0
    cond = sp.diags(1.0 / rs) @ cond
    sym = (cond + cond.T.tocsr()).tocsr()
    del cond
    sym.sum_duplicates()
    sym.sort_indices()
    val = (sym.data / (2.0 * n)).astype(np.float32)
    col = sym.indices.astype(np.int32)
    row_ptr = sym.indptr.astype(np.int64)
    return row_ptr, col, val


def make_y(w: Workload, n: int, labels_perm: np.ndarray, sizes: np.ndarray,
           rng: Generator) -> np.ndarray:
    if w.y_kind == "gauss":
        return (rng.standard_normal((n, 2)) * 1e-2).astype(np.float32)
    y = np.empty((n, 2), np.float64)
    centres = rng.uniform(-50.0, 50.0, size=(sizes.size, 2))
    sig = rng.uniform(0.1, 2.0, size=sizes.size)
    off = 0
    for c in range(sizes.size):
        members = labels_perm[off:off + sizes[c]]
        off += sizes[c]
        y[members] = centres[c] + sig[c] * rng.standard_normal((members.size, 2))
    y = y.astype(np.float32)
    if w.dup_frac > 0.0:
        ndup = int(round(w.dup_frac * n))
        off = 0
        # choose copiers per cluster proportionally, each copies a non-copier
        copier_mask = np.zeros(n, bool)
        copier_mask[rng.choice(n, size=ndup, replace=False)] = True
        for c in range(sizes.size):
            members = labels_perm[off:off + sizes[c]]
            off += sizes[c]
            cm = copier_mask[members]
            cop = members[cm]
            src_pool = members[~cm]
            if cop.size == 0:
                continue
            if src_pool.size == 0:  # whole cluster chosen: keep its first point
                src_pool = cop[:1]
                cop = cop[1:]
            y[cop] = y[src_pool[rng.integers(0, src_pool.size, size=cop.size)]]
    return y


def make_y3(w: Workload, n: int, labels_perm: np.ndarray, sizes: np.ndarray,
            rng: Generator) -> np.ndarray:
    """A 3-D embedding with the workload's recipe: N(0, 1e-4 I) (early phase)
    or clustered centres ~ U(-50, 50)^3 with spread sigma ~ U(0.1, 2) per
    cluster (late phase), and the same share of duplicated points."""
    if w.y_kind == "gauss":
        return (rng.standard_normal((n, 3)) * 1e-2).astype(np.float32)
    y = np.empty((n, 3), np.float64)
    centres = rng.uniform(-50.0, 50.0, size=(sizes.size, 3))
    sig = rng.uniform(0.1, 2.0, size=sizes.size)
    off = 0
    for c in range(sizes.size):
        members = labels_perm[off:off + sizes[c]]
        off += sizes[c]
        y[members] = centres[c] + sig[c] * rng.standard_normal((members.size, 3))
    y = y.astype(np.float32)
    if w.dup_frac > 0.0:
        ndup = int(round(w.dup_frac * n))
        copier = rng.choice(n, size=ndup, replace=False)
        mask = np.zeros(n, bool)
        mask[copier] = True
        off = 0
        for c in range(sizes.size):
            members = labels_perm[off:off + sizes[c]]
            off += sizes[c]
            cop, src = members[mask[members]], members[~mask[members]]
            if cop.size and src.size:
                y[cop] = y[src[rng.integers(0, src.size, size=cop.size)]]
    return y


@dataclasses.dataclass
class Inputs:
    workload: Workload
    n: int
    Y: np.ndarray          # (n, 2) float32
    row_ptr: np.ndarray    # (n+1,) int64
    col: np.ndarray        # (nnz,) int32
    val: np.ndarray        # (nnz,) float32
    labels: np.ndarray     # (n,) int32 cluster id
    gen_seconds: float = 0.0

    @property
    def nnz(self) -> int:
        return int(self.col.size)

    def hashes(self) -> dict:
        return {name: hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()[:16]
                for name, a in (("Y", self.Y), ("row_ptr", self.row_ptr),
                                ("col", self.col), ("val", self.val))}


def make_inputs(cid: int, n: Optional[int] = None, progress=None, k: int = K_NEIGHBOURS,
                dim: int = 2) -> Inputs:
    """Generate workload ``cid``; ``n`` overrides the size (cluster shares are kept),
    ``k`` the neighbours per row of the conditional matrix and ``dim`` (2 or 3)
    the embedding's dimension (P does not depend on it)."""
    t0 = time.time()
    w = WORKLOADS[cid]
    n = w.n if n is None else int(n)
    rng_sz, rng_lab, rng_nb, rng_w, rng_y = _streams(cid)
    sizes = cluster_sizes(w, n, rng_sz)
    perm = rng_lab.permutation(n)
    labels = np.empty(n, np.int32)
    off = 0
    for c in range(sizes.size):
        labels[perm[off:off + sizes[c]]] = c
        off += sizes[c]
    if progress:
        progress(f"[synth] workload {cid}: n={n}, drawing P")
    row_ptr, col, val = make_p(w, n, perm, sizes, rng_nb, rng_w, k=k)
    if progress:
        progress(f"[synth] workload {cid}: nnz={col.size}, drawing Y")
    Y = make_y(w, n, perm, sizes, rng_y) if dim == 2 else make_y3(w, n, perm, sizes, rng_y)
    return Inputs(w, n, Y, row_ptr, col, val, labels, time.time() - t0)


@dataclasses.dataclass
class Knn:
    """Neighbour lists as a k-nearest-neighbour search returns them."""
    n: int
    k: int
    idx: np.ndarray        # (n, k) int32, each row's neighbours by increasing distance
    dist: np.ndarray       # (n, k) float32, ascending within each row
    labels: np.ndarray     # (n,) int32 cluster id
    gen_seconds: float = 0.0


def make_knn(cid: int, n: Optional[int] = None, k: int = K_NEIGHBOURS, progress=None) -> Knn:
    """Neighbour lists of workload ``cid``: the same clusters and neighbour
    draw as its P (row i takes k distinct members of its own cluster), with
    distances d ~ U(0, 3) sorted ascending per row.  Every cluster must have
    more than k members."""
    t0 = time.time()
    w = WORKLOADS[cid]
    n = w.n if n is None else int(n)
    rng_sz, rng_lab, rng_nb, rng_w, _ = _streams(cid)
    sizes = cluster_sizes(w, n, rng_sz)
    if sizes.min() <= k:
        raise ValueError(f"a cluster of {sizes.min()} points cannot give {k} neighbours")
    perm = rng_lab.permutation(n)
    labels = np.empty(n, np.int32)
    idx = np.empty((n, k), np.int32)
    off = 0
    for c in range(sizes.size):
        members = perm[off:off + sizes[c]]
        off += sizes[c]
        labels[members] = c
        _, cols = _neighbours_for_cluster(members, k, rng_nb)
        idx[members] = cols.reshape(members.size, k)
        if progress and c % 10 == 9:
            progress(f"[synth] knn {cid}: cluster {c + 1}/{sizes.size}")
    dist = rng_w.uniform(0.0, 3.0, size=(n, k)).astype(np.float32)
    order = np.argsort(dist, axis=1, kind="stable")
    dist = np.take_along_axis(dist, order, axis=1)
    idx = np.take_along_axis(idx, order, axis=1)
    return Knn(n, k, idx, dist, labels, time.time() - t0)


def random_y(n: int, seed: int, scale: float = 1.0, dups: int = 0) -> np.ndarray:
    """Small free-form embeddings for edge-case tests (float32, n x 2)."""
    rng = Generator(PCG64(SeedSequence(seed)))
    y = (rng.standard_normal((n, 2)) * scale).astype(np.float32)
    for _ in range(dups):
        a, b = rng.integers(0, n, size=2)
        y[a] = y[b]
    return y


def random_y3(n: int, seed: int, scale: float = 1.0, dups: int = 0) -> np.ndarray:
    """Small free-form 3-D embeddings for edge-case tests (float32, n x 3)."""
    rng = Generator(PCG64(SeedSequence(seed + 3)))
    y = (rng.standard_normal((n, 3)) * scale).astype(np.float32)
    for _ in range(dups):
        a, b = rng.integers(0, n, size=2)
        y[a] = y[b]
    return y


def random_p(n: int, seed: int, k: int = 8) -> tuple:
    """Small symmetric CSR P over n points with up to k random neighbours per row."""
    rng = Generator(PCG64(SeedSequence(seed + 7)))
    k = min(k, n - 1)
    rows = np.repeat(np.arange(n), k)
    cols = np.concatenate([rng.choice(np.delete(np.arange(n), i), size=k, replace=False)
                           for i in range(n)]) if k > 0 else np.empty(0, np.int64)
    wts = rng.uniform(0.1, 1.0, size=rows.size)
    cond = sp.csr_matrix((wts, (rows, cols)), shape=(n, n), dtype=np.float64)
    rs = np.asarray(cond.sum(axis=1)).ravel()
    rs[rs == 0] = 1.0
    cond = sp.diags(1.0 / rs) @ cond
    sym = (cond + cond.T.tocsr()).tocsr()
    sym.sum_duplicates()
    sym.sort_indices()
    return (sym.indptr.astype(np.int64), sym.indices.astype(np.int32),
            (sym.data / (2.0 * n)).astype(np.float32))


def geometric_p(n: int, seed: int, k: int = K_NEIGHBOURS, blobs: int = 1) -> tuple:
    """Symmetric CSR P from the exact k nearest neighbours of n points drawn
    uniformly in the unit square (``blobs`` > 1: in that many disjoint squares
    side by side, one connected component each): the kNN graph of data on a
    low-dimensional set, whose locality lies in P itself and not in any
    embedding.  Weights exp(-(d / d_k)^2) with d_k the row's k-th neighbour
    distance, row-normalised in fp64, P = (P + P^T) / (2N).  The drawn order
    is the index order, so as in a real dataset it carries no locality."""
    from scipy.spatial import cKDTree
    rng = Generator(PCG64(SeedSequence(seed + 13)))
    x = rng.uniform(0.0, 1.0, size=(n, 2))
    if blobs > 1:
        x[:, 0] += 2.0 * rng.integers(0, blobs, size=n)   # gaps wider than any neighbour distance
    d, nb = cKDTree(x).query(x, k=k + 1, workers=-1)
    d, nb = d[:, 1:], nb[:, 1:]                         # column 0 is the point itself
    dk = np.maximum(d[:, -1:], 1e-300)
    wts = np.exp(-(d / dk) ** 2).ravel()
    rows = np.repeat(np.arange(n), k)
    cond = sp.csr_matrix((wts, (rows, nb.ravel())), shape=(n, n), dtype=np.float64)
    rs = np.asarray(cond.sum(axis=1)).ravel()
    rs[rs == 0] = 1.0
    cond = sp.diags(1.0 / rs) @ cond
    sym = (cond + cond.T.tocsr()).tocsr()
    sym.sum_duplicates()
    sym.sort_indices()
    return (sym.indptr.astype(np.int64), sym.indices.astype(np.int32),
            (sym.data / (2.0 * n)).astype(np.float32))


def _ring_offsets(n: int, m: int, rng: Generator) -> np.ndarray:
    """m distinct offsets in [1, n/2) (so i + o and i - o never meet mod n)."""
    half = (n - 1) // 2
    if m > half:
        raise ValueError(f"{n} points cannot give {m} distinct ring offsets")
    return np.sort(rng.choice(np.arange(1, half + 1, dtype=np.int64), size=m, replace=False)) \
        if half < 1 << 20 else _distinct_draw(rng, 1, half + 1, m)


def _distinct_draw(rng: Generator, lo: int, hi: int, m: int) -> np.ndarray:
    out = np.empty(0, np.int64)
    while out.size < m:
        out = np.unique(np.concatenate([out, rng.integers(lo, hi, size=m)]))
    return np.sort(rng.permutation(out)[:m])


def ring_p(n: int, seed: int, m: int = 2) -> tuple:
    """Symmetric CSR P for very large n, drawn in O(n m): row i lists the 2m
    points i +- o_j (mod n) for m random distinct offsets, with
    p_{i,i+o_j} = p_{i+o_j,i} = v_j and sum(P) = 1.  Index order and positions
    are unrelated, as in a real dataset."""
    rng = Generator(PCG64(SeedSequence(seed + 11)))
    off = _ring_offsets(n, m, rng)
    u = rng.uniform(0.1, 1.0, size=m)
    v = u / (2.0 * n * u.sum())
    d = np.concatenate([off, n - off])            # i + d (mod n) lists i +- o_j
    dv = np.concatenate([v, v])
    o = np.argsort(d)
    d, dv = d[o], dv[o]
    # row i in column order: the entries that wrap (d >= n - i) come first
    i = np.arange(n, dtype=np.int32)               # n < 2^30: int32 sums stay exact
    r = np.zeros(n, np.int32)
    for dd in d:
        r += i < n - dd
    j = np.arange(2 * m, dtype=np.int32)[None, :] + r[:, None]
    j[j >= 2 * m] -= 2 * m
    cols = i[:, None] + d.astype(np.int32)[j]
    cols[cols >= n] -= n
    vals = dv.astype(np.float32)[j]
    row_ptr = np.arange(0, 2 * m * n + 1, 2 * m, dtype=np.int64)
    return row_ptr, cols.ravel(), vals.ravel()


def ring_knn(n: int, k: int, seed: int) -> Knn:
    """Neighbour lists for very large n, drawn in O(n k): row i lists the
    points i + o_e (mod n) for k random distinct offsets in [1, n), so every
    point is listed by exactly k rows; distances d ~ U(0, 3), ascending."""
    t0 = time.time()
    rng = Generator(PCG64(SeedSequence(seed + 13)))
    off = rng.permutation(_distinct_draw(rng, 1, n, k))
    idx = np.arange(n, dtype=np.int32)[:, None] + off.astype(np.int32)
    idx[idx >= n] -= n
    dist = rng.random((n, k), dtype=np.float32) * np.float32(3.0)
    dist.sort(axis=1)
    return Knn(n, k, idx, dist, np.zeros(n, np.int32), time.time() - t0)
