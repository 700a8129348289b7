"""GPU parity: the HIP path against the fp64 oracle on identical seeded inputs.

Bars (from the method's definition and the tolerances the library promises):
  * bounding box, quantisation parameters, Morton codes, sorted order and the
    tree topology: bit-exact;
  * cell summaries: fp32 rounding of the oracle's fp64 centre of mass;
  * gradient relative L2 <= 1e-4 at theta = 0 (exact) and <= 1e-3 at
    theta > 0 (against the oracle's Barnes-Hut on the same Y);
  * Z relative error <= 1e-5;
  * KL after a full run within 1% of the oracle's run.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2212_11506_amd as bh


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def dev_y(y):
    return torch.from_numpy(np.ascontiguousarray(y, np.float32)).cuda()


def dev_p(rp, col, val):
    return bh.Csr.from_numpy(rp, col, val)


# ------------------------------------------------------------------ edge-case embeddings
def _case(name):
    if name == "c0":
        return synth.make_inputs(0).Y
    if name.startswith("rand"):
        n = int(name[4:])
        return synth.random_y(n, seed=n, scale=1.0)
    if name == "dups":
        return synth.random_y(3000, seed=9, scale=1.0, dups=600)
    if name == "identical":
        return np.full((1000, 2), 0.375, np.float32)
    if name == "identical2":
        return np.array([[1.0, 2.0], [1.0, 2.0]], np.float32)
    if name == "huge":
        return synth.random_y(4000, seed=10, scale=1e35)
    if name == "tiny":
        return synth.random_y(4000, seed=11, scale=1e-20)
    if name == "outlier":
        y = synth.random_y(5000, seed=12, scale=1e-3)
        y[17] = (1e4, -3e3)
        return y
    if name == "line":
        t = np.linspace(-1, 1, 3001, dtype=np.float32)
        return np.stack([t, t], 1)
    if name == "late":
        return synth.make_inputs(4, n=20000).Y
    if name == "reps40":  # 3000 points, each 40 times, shuffled: 3000 runs of equal codes
        y = np.repeat(synth.random_y(3000, seed=13, scale=1.0), 40, axis=0)
        return y[np.random.default_rng(13).permutation(y.shape[0])]
    if name == "identical20k":  # one run of equal codes longer than a block sorts in LDS
        return np.full((20000, 2), -2.5, np.float32)
    if name.startswith("jitter"):  # places of m points 1e-6 apart, shuffled: runs of equal top halves
        places, m = {"jitter5": (1000, 5), "jitter100": (60, 100)}[name]
        y = np.repeat(synth.random_y(places, seed=15, scale=1.0), m, axis=0)
        y = y + synth.random_y(places * m, seed=16, scale=1e-6)
        return y[np.random.default_rng(15).permutation(places * m)].astype(np.float32)
    if name == "cloud6k":  # 6000 points within 1e-4 and one far away: a run of 6000 top halves
        y = synth.random_y(6000, seed=17, scale=1e-5)
        y[4321] = (1e3, 1e3)
        return y
    raise KeyError(name)


SORT_CASES = ["c0", "rand2", "rand3", "rand63", "rand64", "rand65", "rand2047", "rand2048",
              "rand2049", "rand4097", "rand70001", "dups", "identical", "identical2", "huge",
              "tiny", "outlier", "line", "late", "reps40", "identical20k", "jitter5", "jitter100", "cloud6k"]

# the longest run of codes with equal top 32 bits these cases are made to have
# (the sort's three ways of ordering such runs)
RUN_CASES = {"jitter5": (2, 32), "jitter100": (33, 4096), "cloud6k": (4097, 1 << 30)}


def longest_top_half_run(sorted_codes):
    hi = np.asarray(sorted_codes, np.uint64) >> np.uint64(32)
    starts = np.flatnonzero(np.r_[True, hi[1:] != hi[:-1]])
    return int(np.diff(np.r_[starts, hi.size]).max())


@pytest.mark.parametrize("case", SORT_CASES)
def test_morton_and_sort_bit_exact(case):
    y = _case(case)
    say(f"[sort] case={case} n={y.shape[0]}")
    codes, scodes, perm, params = bh.debug_sort(dev_y(y))
    with oracle.State(y) as s:
        t = s.tree()
    box = t.box
    assert params[0:4] == [box[0], box[1], box[2], box[3]]
    assert params[4] == box[4] and params[5] == box[5] and params[6] == box[6]
    assert params[7] == t.yrs[0] and params[8] == t.yrs[1]
    assert params[9] == t.yrs[2]
    assert np.array_equal(codes.cpu().numpy().view(np.uint64), t.codes)
    assert np.array_equal(scodes.cpu().numpy().view(np.uint64), t.sorted_codes)
    assert np.array_equal(perm.cpu().numpy().view(np.uint32), t.perm)
    if case in RUN_CASES:
        lo, hi = RUN_CASES[case]
        assert lo <= longest_top_half_run(t.sorted_codes) <= hi


def test_quantisation_truncates_like_the_hand_worked_case(golden_dir):
    """The hand-worked grid values and codes of tests/golden/quantisation_truncation.txt
    (reading R2: truncation, and the clamp at the top of the grid), on the GPU."""
    import os
    rows = []
    for line in open(os.path.join(golden_dir, "quantisation_truncation.txt")):
        if line.strip() and not line.startswith("#"):
            rows.append(line.split())
    y = np.array([[float(r[0]), float(r[1])] for r in rows], np.float32)
    codes, scodes, perm, params = bh.debug_sort(dev_y(y))
    got = codes.cpu().numpy().view(np.uint64)
    assert [int(c) for c in got] == [int(r[4], 16) for r in rows]
    assert params[7] == 0.0 and params[8] == 0.0 and params[6] == 1.5


def _bucket_points(y):
    """Points in buckets: the library stores each as a node of its own."""
    with oracle.State(y) as s:
        t = s.tree()
    b = t.kind == oracle.BUCKET
    return int((t.end[b].astype(np.int64) - t.begin[b]).sum())


def _with_members(t, y):
    """The oracle's tree laid out as the library stores it: every bucket leaf is
    followed by its points as single-point nodes (level 33), in sorted order."""
    from types import SimpleNamespace
    idx, lev, kind, beg, end, cnt, com = [], [], [], [], [], [], []
    ys = y.astype(np.float64)[t.perm.astype(np.int64)]
    for i in range(t.nodes):
        idx.append(i)
        lev.append(t.level[i]); kind.append(t.kind[i]); beg.append(t.begin[i]); end.append(t.end[i])
        cnt.append(t.count[i]); com.append(t.com[i])
        if t.kind[i] == oracle.BUCKET:
            for j in range(int(t.begin[i]), int(t.end[i])):
                lev.append(33); kind.append(oracle.SINGLE); beg.append(j); end.append(j + 1)
                cnt.append(1); com.append(ys[j])
    u = SimpleNamespace(**{k: getattr(t, k) for k in ("box", "perm", "codes", "sorted_codes", "yrs")})
    u.nodes = len(lev)
    u.level = np.array(lev, dtype=t.level.dtype)
    u.kind = np.array(kind, dtype=t.kind.dtype)
    u.begin = np.array(beg, dtype=t.begin.dtype)
    u.end = np.array(end, dtype=t.end.dtype)
    u.count = np.array(cnt, dtype=t.count.dtype)
    u.com = np.array(com, dtype=np.float64).reshape(-1, 2)
    return u


@pytest.mark.parametrize("case", SORT_CASES)
def test_tree_and_summaries(case):
    y = _case(case)
    theta = 0.5
    say(f"[tree] case={case} n={y.shape[0]}")
    ws = torch.empty(bh.workspace_size(y.shape[0], 0), dtype=torch.uint8, device="cuda")
    g = bh.debug_tree(dev_y(y), theta, workspace=ws)
    with oracle.State(y) as s:
        t = _with_members(s.tree(), y)
    assert g["nodes"] == t.nodes
    assert np.array_equal(g["level"].cpu().numpy(), t.level)
    assert np.array_equal(g["kind"].cpu().numpy(), t.kind)
    assert np.array_equal(g["begin"].cpu().numpy().view(np.uint32), t.begin)
    assert np.array_equal(g["end"].cpu().numpy().view(np.uint32), t.end)
    summ = g["summary"].cpu().numpy().astype(np.float64)
    assert np.array_equal(summ[:, 2], t.count.astype(np.float64))
    # centre of mass: the fp32 rounding of the fp64 definition, plus (cells of more
    # than 32 points) the rounding of a difference of two fp64 prefix sums of
    # (y - box centre), i.e. a few ulps of sum|y - centre| spread over the count
    err = np.abs(summ[:, :2] - t.com)
    smax = np.abs(y.astype(np.float64) - t.box[4:6]).sum(0)
    cnt = t.count.astype(np.float64)[:, None]
    tol = 7e-8 * np.abs(t.com) + np.where(cnt > 32, 8 * 2.0 ** -52 * smax / cnt, 0.0) + 1e-38
    assert np.all(err <= tol), float((err / tol).max())
    single = t.kind == oracle.SINGLE
    assert np.all(summ[single, 3] == -1.0)
    side2 = (2 * t.box[6] * np.exp2(-t.level[~single].astype(np.float64))) ** 2 / theta ** 2
    with np.errstate(over="ignore"):
        side2_f32 = side2.astype(np.float32).astype(np.float64)  # squared lengths live in fp32
    assert np.allclose(summ[~single, 3], side2_f32, rtol=1e-6, atol=1e-45)
    # skip pointers: cells (internal and buckets) -> first node past the subtree;
    # single points -> begin | leaf bit | single bit
    meta = g["meta"].cpu().numpy().view(np.uint32)
    cell = ~single
    order_end = np.searchsorted(t.begin.astype(np.int64) * 64 + t.level,
                                t.end.astype(np.int64) * 64, side="left")
    assert np.array_equal(meta[cell], order_end[cell].astype(np.uint32))
    assert np.array_equal(meta[single], t.begin[single] | np.uint32(0xC0000000))


# ------------------------------------------------------------------ gradients
def _p_for(y, seed=3, k=8):
    return synth.random_p(y.shape[0], seed=seed, k=k)


GRAD_CASES = ["c0", "rand2", "rand3", "rand65", "rand2049", "dups", "identical", "line", "late"]


@pytest.mark.parametrize("case", GRAD_CASES)
@pytest.mark.parametrize("theta", [0.0, 0.5])
def test_gradient_parity(case, theta):
    if case == "c0":
        inp = synth.make_inputs(0)
        y, (rp, col, val) = inp.Y, (inp.row_ptr, inp.col, inp.val)
    else:
        y = _case(case)
        rp, col, val = _p_for(y)
    alpha = 12.0
    say(f"[grad] case={case} theta={theta} n={y.shape[0]} nnz={col.size}")
    ws = torch.empty(bh.workspace_size(y.shape[0], col.size), dtype=torch.uint8, device="cuda")
    g, Z = bh.gradient(dev_y(y), dev_p(rp, col, val), theta, alpha, workspace=ws)
    g = g.cpu().numpy()
    stats = bh.get_stats(ws)
    go, Zo, inter_o, nodes_o = oracle.gradient(y, rp, col, val, theta, alpha)
    assert stats["nodes"] == nodes_o + _bucket_points(y)
    if theta == 0.0:
        assert stats["interactions"] == inter_o == y.shape[0] * (y.shape[0] - 1)
    else:  # an acceptance may flip where fp32 and fp64 distances straddle the threshold
        assert abs(stats["interactions"] - inter_o) <= 1e-3 * inter_o + 2
    tol = 1e-4 if theta == 0.0 else 1e-3
    if np.linalg.norm(go) == 0.0:
        assert np.abs(g).max() <= 1e-6
    else:
        assert rel_l2(g, go) <= tol, rel_l2(g, go)
    assert abs(Z - Zo) <= 1e-5 * Zo, (Z, Zo)


# 0.7 is the largest angle at which the walk drops the comparison with a
# point's own leaf (theta^2 <= 0.49: no point can accept a cell containing it,
# so each takes its own leaf once and its weight of 1 is removed afterwards);
# 0.71 and above compare positions instead.  "reps40" puts every point in a
# bucket of 40 identical points, so the own leaf sits among equal neighbours.
@pytest.mark.parametrize("case,theta", [("late", 0.2), ("late", 0.7), ("late", 0.71), ("late", 0.8), ("late", 1.2),
                                        ("reps40", 0.7), ("reps40", 0.71), ("dups", 1.0)])
def test_gradient_parity_other_angles(case, theta):
    y = _case(case)
    rp, col, val = _p_for(y, seed=5)
    say(f"[grad-angle] case={case} theta={theta}")
    ws = torch.empty(bh.workspace_size(y.shape[0], col.size), dtype=torch.uint8, device="cuda")
    g, Z = bh.gradient(dev_y(y), dev_p(rp, col, val), theta, 1.0, workspace=ws)
    stats = bh.get_stats(ws)
    go, Zo, inter_o, nodes_o = oracle.gradient(y, rp, col, val, theta, 1.0)
    nodes_o += _bucket_points(y)
    assert rel_l2(g.cpu().numpy(), go) <= 1e-3
    assert abs(Z - Zo) <= 1e-5 * Zo
    assert stats["nodes"] == nodes_o
    assert abs(stats["interactions"] - inter_o) <= 1e-3 * inter_o


def test_theta0_against_exact_definition():
    # theta = 0 must reproduce the exact O(n^2) gradient of the paper's equation
    inp = synth.make_inputs(0)
    say("[exact] c0 theta=0")
    g, Z = bh.gradient(dev_y(inp.Y), dev_p(inp.row_ptr, inp.col, inp.val), 0.0, 1.0)
    n = inp.n
    Zex = oracle.z_exact(inp.Y)
    assert abs(Z - Zex) <= 1e-5 * Zex
    go, _, inter, _ = oracle.gradient(inp.Y, inp.row_ptr, inp.col, inp.val, 0.0, 1.0)
    assert inter == n * (n - 1)
    assert rel_l2(g.cpu().numpy(), go) <= 1e-4


def test_empty_and_ragged_p():
    n = 3000
    y = synth.random_y(n, seed=21, scale=2.0)
    rp, col, val = synth.random_p(n, seed=21, k=6)
    # drop every entry touching points 0..499: those rows become empty, P stays symmetric
    r = np.repeat(np.arange(n), np.diff(rp))
    keep = (r >= 500) & (col >= 500)
    counts = np.bincount(r[keep], minlength=n)
    rp2 = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    col2, val2 = col[keep], val[keep]
    for (a, b, c) in [(rp2, col2, val2),
                      (np.zeros(n + 1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.float32))]:
        say(f"[ragged] nnz={b.size}")
        g, Z = bh.gradient(dev_y(y), dev_p(a, b, c), 0.5, 4.0)
        go, Zo, _, _ = oracle.gradient(y, a, b, c, 0.5, 4.0)
        assert rel_l2(g.cpu().numpy(), go) <= 1e-3
        assert abs(Z - Zo) <= 1e-5 * Zo


# ------------------------------------------------------------------ update / full runs
@pytest.mark.parametrize("form", ["plain", "layout"])
def test_step_matches_update_rule(form):
    """Each step's gains, momentum buffer and new Y equal the oracle's update
    rule applied to the GPU's own gradient, element by element: on the plain
    CSR path (update fused into the attraction) and through a locality layout
    (the separate update kernel the bench times)."""
    inp = synth.make_inputs(0)
    w = inp.workload
    Y = dev_y(inp.Y)
    P = dev_p(inp.row_ptr, inp.col, inp.val)
    if form == "layout":
        P = bh.Layout(P, Y)
    u = torch.zeros_like(Y)
    gains = torch.ones_like(Y)
    grad = torch.empty_like(Y)
    y64 = inp.Y.astype(np.float64)
    u64 = np.zeros_like(y64)
    g64 = np.ones_like(y64)
    for it in range(3):
        sch = w.schedule(it)
        say(f"[step] {form} it={it}")
        bh.step(Y, P, 0.5, sch["exaggeration"], sch["learning_rate"], sch["momentum"], 0.01, u,
                gains, grad=grad)
        gd = grad.cpu().numpy().astype(np.float64)
        oracle.update(y64, u64, g64, gd, sch["learning_rate"], sch["momentum"], 0.01)
        assert np.allclose(gains.cpu().numpy(), g64, rtol=1e-6, atol=0)
        assert np.allclose(u.cpu().numpy(), u64, rtol=2e-5, atol=1e-6 * np.abs(u64).max())
        assert np.allclose(Y.cpu().numpy(), y64, rtol=2e-5, atol=1e-6 * np.abs(y64).max())
        # keep the fp64 replay on the GPU's state so steps stay comparable
        y64 = Y.cpu().numpy().astype(np.float64)
        u64 = u.cpu().numpy().astype(np.float64)
        g64 = gains.cpu().numpy().astype(np.float64)


def _run_gpu(inp, iters, theta):
    w = inp.workload
    Y = dev_y(inp.Y)
    P = dev_p(inp.row_ptr, inp.col, inp.val)
    u = torch.zeros_like(Y)
    gains = torch.ones_like(Y)
    ws = torch.empty(bh.workspace_size(inp.n, inp.nnz), dtype=torch.uint8, device="cuda")
    for it in range(iters):
        s = w.schedule(it)
        bh.step(Y, P, theta, s["exaggeration"], s["learning_rate"], s["momentum"], 0.01, u, gains,
                workspace=ws)
    torch.cuda.synchronize()
    return Y.cpu().numpy()


def _run_oracle(inp, iters, theta):
    w = inp.workload
    y = inp.Y.astype(np.float64)
    u = np.zeros_like(y)
    gains = np.ones_like(y)
    for it in range(iters):
        s = w.schedule(it)
        oracle.step(y, u, gains, inp.row_ptr, inp.col, inp.val, theta, s["exaggeration"],
                    s["learning_rate"], s["momentum"], 0.01)
    return y


def test_full_run_kl_small_workload():
    inp = synth.make_inputs(0)
    say("[kl] workload 0, 50 iterations")
    yg = _run_gpu(inp, inp.workload.iters, 0.5)
    yo = _run_oracle(inp, inp.workload.iters, 0.5)
    klg = oracle.kl(yg, inp.row_ptr, inp.col, inp.val)
    klo = oracle.kl(yo, inp.row_ptr, inp.col, inp.val)
    kl0 = oracle.kl(inp.Y, inp.row_ptr, inp.col, inp.val)
    say(f"[kl] gpu={klg:.6f} oracle={klo:.6f} start={kl0:.6f}")
    assert klg < kl0 and klo < kl0
    assert abs(klg - klo) <= 0.01 * klo


# ------------------------------------------------------------------ robustness
def test_deterministic():
    inp = synth.make_inputs(0)
    Y, P = dev_y(inp.Y), dev_p(inp.row_ptr, inp.col, inp.val)
    g1, Z1 = bh.gradient(Y, P, 0.5, 12.0)
    g2, Z2 = bh.gradient(Y, P, 0.5, 12.0)
    assert Z1 == Z2
    assert torch.equal(g1, g2)


def test_nonfinite_input_is_reported():
    y = synth.random_y(500, seed=3)
    y[7, 1] = np.nan
    rp, col, val = _p_for(y)
    with pytest.raises(bh.BhtsneError) as e:
        bh.gradient(dev_y(y), dev_p(rp, col, val), 0.5, 1.0)
    assert e.value.status == bh.BHTSNE_ENONFINITE


def test_timing_records_every_phase():
    inp = synth.make_inputs(0)
    Y, P = dev_y(inp.Y), dev_p(inp.row_ptr, inp.col, inp.val)
    lay = bh.Layout(P, Y)
    bh.timing_read(reset=True)
    bh.timing_enable(True)
    try:
        for _ in range(3):
            bh.gradient(Y, P, 0.5, 12.0, return_z=False)
        plain = bh.timing_read(reset=True)
        for _ in range(3):
            bh.gradient(Y, lay, 0.5, 12.0, return_z=False)
        layout = bh.timing_read(reset=True)
    finally:
        bh.timing_enable(False)
    # the plain path assembles the gradient inside the attractive phase
    for name in bh.PHASES:
        ms, cnt = plain[name]
        assert (cnt == 0) if name == "update" else (cnt == 3 and ms > 0.0), (name, plain[name])
        ms, cnt = layout[name]
        assert cnt == 3 and ms > 0.0, (name, layout[name])
    # a phase mask limits the events to the selected phases
    bh.timing_phases(["repulsive", "attractive"])
    bh.timing_enable(True)
    try:
        for _ in range(2):
            bh.gradient(Y, lay, 0.5, 12.0, return_z=False)
        some = bh.timing_read(reset=True)
    finally:
        bh.timing_enable(False)
        bh.timing_phases(None)
    for name in bh.PHASES:
        ms, cnt = some[name]
        assert (cnt == 2 and ms > 0.0) if name in ("repulsive", "attractive") else cnt == 0, (name, some[name])
