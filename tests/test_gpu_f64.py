"""Parity of the fp64 variant (bhtsne_gradient_f64 / bhtsne_step_f64) with the
fp64 oracle.

Both sides quantise the same fp64 coordinates (Quadtree Building), so their
trees are identical (node counts equal); acceptance tests differ only where
a squared distance rounds differently in its last bit against a threshold,
so interaction counts agree to 1e-6 and gradients to a relative L2 of 1e-9
(the remaining differences are summation orders in fp64).  P's values are
fp32 numbers stored as fp64, which both sides read exactly.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2212_11506_amd as bh
import synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print(*a, flush=True)


def rel_l2(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def _y64(y32, seed):
    # genuinely fp64 coordinates: fp32 values plus an offset below fp32 resolution
    rng = np.random.default_rng(seed)
    y = y32.astype(np.float64)
    return y + rng.normal(0.0, 1.0, y.shape) * np.abs(y).max() * 2.0 ** -30


def _p64(rp, col, val):
    return bh.CsrF64.from_numpy(rp, col, val.astype(np.float64), device=DEV)


def _gpu_grad(y, rp, col, val, theta, alpha):
    P = _p64(rp, col, val)
    ws = torch.empty(bh.workspace_size_f64(y.shape[0], col.size), dtype=torch.uint8, device=DEV)
    g, Z = bh.gradient_f64(torch.from_numpy(y).to(DEV), P, theta, alpha, workspace=ws)
    return g.cpu().numpy(), Z, bh.get_stats(ws)


def _bucket_points(y):
    """Points in buckets: the library stores each as a node of its own."""
    with oracle.State(y) as s:
        t = s.tree()
    b = t.kind == oracle.BUCKET
    return int((t.end[b].astype(np.int64) - t.begin[b]).sum())


CASES = {
    "c0": lambda: _y64(synth.make_inputs(0).Y, 1),
    "late20k": lambda: _y64(synth.make_inputs(4, n=20000).Y, 2),
    "dups": lambda: np.repeat(_y64(synth.random_y(1500, seed=9), 3), 2, axis=0),
    "two": lambda: np.array([[0.25, -1.0], [1e-12, 3.0]], np.float64),
}


def _p_for(n, seed=3, k=8):
    rng = np.random.default_rng(seed)
    rows = np.repeat(np.arange(n), k)
    cols = rng.integers(0, n - 1, size=rows.size)
    cols = cols + (cols >= rows)
    import scipy.sparse as sp
    c = sp.csr_matrix((rng.random(rows.size), (rows, cols)), shape=(n, n))
    s = (c + c.T).tocsr()
    s.sum_duplicates()
    s.sort_indices()
    val = (s.data / s.data.sum()).astype(np.float32)
    return s.indptr.astype(np.int64), s.indices.astype(np.int32), val


@pytest.mark.parametrize("case,theta", [("c0", 0.5), ("c0", 0.0), ("late20k", 0.5), ("late20k", 0.8),
                                        ("dups", 0.5), ("dups", 1.0), ("two", 0.5)])
def test_gradient_f64_parity(case, theta):
    y = CASES[case]()
    if case == "c0":
        inp = synth.make_inputs(0)
        rp, col, val = inp.row_ptr, inp.col, inp.val
    else:
        rp, col, val = _p_for(y.shape[0])
    alpha = 12.0
    g, Z, st = _gpu_grad(y, rp, col, val, theta, alpha)
    go, Zo, inter_o, nodes_o = oracle.gradient(y, rp, col, val, theta, alpha)
    nodes_o += _bucket_points(y)
    err = rel_l2(g, go)
    say(f"[f64] {case} theta={theta}: rel-L2 {err:.2e}, Z rel {abs(Z - Zo) / Zo:.2e}, "
        f"interactions {st['interactions']} vs {inter_o}, nodes {st['nodes']} vs {nodes_o}")
    assert err <= 1e-9, err
    assert abs(Z - Zo) <= 1e-12 * Zo
    assert st["nodes"] == nodes_o
    assert abs(st["interactions"] - inter_o) <= 1e-6 * inter_o


def test_step_f64_tracks_oracle():
    inp = synth.make_inputs(0)
    w = inp.workload
    y = _y64(inp.Y, 5)
    P = _p64(inp.row_ptr, inp.col, inp.val)
    Y = torch.from_numpy(y).to(DEV)
    u = torch.zeros_like(Y)
    gains = torch.ones_like(Y)
    ws = torch.empty(bh.workspace_size_f64(inp.n, inp.nnz), dtype=torch.uint8, device=DEV)
    yo, uo, go = y.copy(), np.zeros_like(y), np.ones_like(y)
    for it in range(10):
        s = w.schedule(it)
        bh.step_f64(Y, P, 0.5, s["exaggeration"], s["learning_rate"], s["momentum"], 0.01, u, gains, workspace=ws)
        oracle.step(yo, uo, go, inp.row_ptr, inp.col, inp.val, 0.5, s["exaggeration"], s["learning_rate"],
                    s["momentum"], 0.01)
    err = rel_l2(Y.cpu().numpy() - y, yo - y)
    say(f"[f64] 10 steps: displacement rel-L2 {err:.2e}")
    assert err <= 1e-8


def test_f64_rejects_bad_arguments():
    inp = synth.make_inputs(0)
    P = _p64(inp.row_ptr, inp.col, inp.val)
    Y = torch.from_numpy(_y64(inp.Y, 6)).to(DEV)
    for theta, alpha in [(-0.1, 1.0), (float("nan"), 1.0), (0.5, 0.0), (0.5, float("inf"))]:
        with pytest.raises(bh.BhtsneError) as e:
            bh.gradient_f64(Y, P, theta, alpha)
        assert e.value.status == bh.BHTSNE_EINVAL
    small = torch.empty(16, dtype=torch.uint8, device=DEV)
    with pytest.raises(bh.BhtsneError) as e:
        bh.gradient_f64(Y, P, 0.5, 1.0, workspace=small)
    assert e.value.status == bh.BHTSNE_EWORKSPACE
    bad = Y.clone()
    bad[7, 1] = float("nan")
    with pytest.raises(bh.BhtsneError) as e:
        bh.gradient_f64(bad, P, 0.5, 1.0)
    assert e.value.status == bh.BHTSNE_ENONFINITE
