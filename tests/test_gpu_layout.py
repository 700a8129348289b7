"""GPU tests of the locality layout of P and the LDS-staged attractive path.

The layout only renumbers points, so every result must match the oracle to
the same bars as the plain path; the layout itself must be an exact
relabelling of P."""
import os
import subprocess
import sys

import numpy as np
import pytest
import scipy.sparse as sp
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2212_11506_amd as bh

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def rel_l2(a, b):
    return float(np.linalg.norm(np.asarray(a, np.float64) - b) / np.linalg.norm(b))


from layout_tables import (CHUNK, ITEM_MAX_TILES, SLICE, SLICES, TILE_MAX_SEG, TILE_ROWS,  # noqa: E402,F401
                           TILE_NARROW_SEG, TILE_SEG, TILE_SLOTS, TILE_WIDE_ENTRIES,
                           check_sliced_copy)
from layout_tables import bfs_perm as _bfs_perm  # noqa: E402
from layout_tables import layout_arrays as _layout_arrays  # noqa: E402


NO_COLUMN = 0x7FFFFFFF


def _tcol_offset(n, nnz):
    """Byte offset of the sliced copy's column array in the layout memory (the
    windowed segments reuse that region), and the end of the layout."""
    off = 0

    def take(nbytes):
        nonlocal off
        o = off
        off = (off + nbytes + 255) // 256 * 256
        return o

    cap = nnz + 3 * n + 4
    for nbytes in (4 * n, 4 * n, 8 * (n + 1), 4 * cap, 4 * cap):
        take(nbytes)
    blocks = (n + TILE_ROWS - 1) // TILE_ROWS
    max_tiles = blocks * TILE_SLOTS
    max_units = max_tiles * SLICES
    max_entries = nnz + nnz // 4 + CHUNK * SLICES * blocks * TILE_NARROW_SEG + CHUNK
    for nbytes in (4 * blocks, 4 * blocks, 4 * blocks * TILE_MAX_SEG, 4 * max_tiles, 4 * max_tiles, 4 * max_tiles,
                   8 * max_tiles, 4 * max_tiles * TILE_ROWS, 2 * max_tiles * TILE_ROWS, 2 * max_tiles * TILE_ROWS,
                   4 * max_units, 4 * max_units, 4 * max_units, 4 * max_units, 16 * max_tiles, 16 * max_tiles * 16):
        take(nbytes)
    o_tc = take(2 * max_entries)
    take(4 * max_entries)
    return o_tc, off


def _window_region_offset(lay):
    return _tcol_offset(lay.n, lay.nnz)[0]


def _max_segments(lay):
    o_tc, end = _tcol_offset(lay.n, lay.nnz)
    return (end - o_tc - 8 * 65 - 4 * 256) // 12


def _hub_p(n, seed, sizes=(300, 450, 5000)):
    """Symmetric P whose first rows hold many more entries than the register slots
    (and one more than the in-LDS row sort takes)."""
    rp, col, val = synth.random_p(n, seed=seed, k=6)
    P = sp.csr_matrix((val.astype(np.float64), col, rp), shape=(n, n))
    rng = np.random.default_rng(seed)
    hubs = sp.lil_matrix((n, n))
    for h, size in enumerate(sizes):
        others = rng.choice(np.arange(len(sizes), n), size=size, replace=False)
        for o in others:
            hubs[h, o] = 1e-5
            hubs[o, h] = 1e-5
    P = (P + hubs.tocsr()).tocsr()
    P.sum_duplicates()
    P.sort_indices()
    P.data /= P.data.sum()
    return P.indptr.astype(np.int64), P.indices.astype(np.int32), P.data.astype(np.float32)


@pytest.mark.parametrize("with_y", [False, True])
def test_layout_is_a_relabelling(with_y):
    inp = synth.make_inputs(0)
    P = bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val)
    Y = torch.from_numpy(inp.Y).cuda()
    say(f"[layout] build with_y={with_y}")
    lay = bh.Layout(P, Y if with_y else None)
    perm, rank, rp, col, val = _layout_arrays(lay)
    n = inp.n
    assert np.array_equal(np.sort(perm), np.arange(n, dtype=np.uint32))
    assert np.array_equal(rank[perm], np.arange(n, dtype=np.uint32))
    # rows start on 16-byte boundaries and end with padding entries only
    assert np.all(rp % 4 == 0)
    used = rp[-1]
    assert np.all(col[used:used + 4] == NO_COLUMN) and np.all(val[used:used + 4] == 0)
    rows = np.repeat(np.arange(n), np.diff(rp))
    c, v = col[:used], val[:used]
    real = c != NO_COLUMN
    assert np.all(v[~real] == 0)
    Po = sp.csr_matrix((inp.val, inp.col, inp.row_ptr), shape=(n, n))
    Pn = sp.csr_matrix((v[real], (rows[real], c[real])), shape=(n, n))
    ref = Po[perm.astype(np.int64)][:, perm.astype(np.int64)]
    assert abs(Pn - ref).max() == 0.0
    assert Pn.nnz == inp.nnz
    # columns ascend within every row (padding last)
    ok = (np.diff(c.astype(np.int64)) > 0) | (np.diff(rows) != 0) | ((c[1:] == NO_COLUMN) & (c[:-1] == NO_COLUMN))
    assert np.all(ok)
    # each cluster (a connected component of this P) occupies one contiguous range
    lab = inp.labels[perm]
    changes = np.count_nonzero(lab[1:] != lab[:-1])
    assert changes == inp.workload.clusters - 1


@pytest.mark.parametrize("case", ["c0", "hubs", "late"])
@pytest.mark.parametrize("theta", [0.0, 0.5])
def test_gradient_through_layout(case, theta):
    if case == "c0":
        inp = synth.make_inputs(0)
        y, rp, col, val = inp.Y, inp.row_ptr, inp.col, inp.val
    elif case == "hubs":
        y = synth.random_y(6000, seed=4, scale=2.0)
        rp, col, val = _hub_p(6000, seed=4)
    else:  # late phase with 5% duplicates; at theta = 0 every pair is exact (4e8 pairs)
        inp = synth.make_inputs(4, n=20000)
        y, rp, col, val = inp.Y, inp.row_ptr, inp.col, inp.val
    say(f"[layout-grad] case={case} theta={theta} max row={np.diff(rp).max()}")
    Y = torch.from_numpy(np.ascontiguousarray(y)).cuda()
    P = bh.Csr.from_numpy(rp, col, val)
    lay = bh.Layout(P, Y)
    g, Z = bh.gradient(Y, lay, theta, 12.0)
    go, Zo, _, _ = oracle.gradient(y, rp, col, val, theta, 12.0)
    assert rel_l2(g.cpu().numpy(), go) <= (1e-4 if theta == 0.0 else 1e-3)
    assert abs(Z - Zo) <= 1e-5 * Zo
    gp, Zp = bh.gradient(Y, P, theta, 12.0)
    assert Zp == Z  # same tree, same repulsion
    assert rel_l2(g.cpu().numpy(), gp.cpu().numpy().astype(np.float64)) <= 1e-5


def test_layout_steps_track_plain_steps():
    inp = synth.make_inputs(0)
    w = inp.workload
    P = bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val)
    Ya = torch.from_numpy(inp.Y).cuda()
    Yb = Ya.clone()
    lay = bh.Layout(P, Ya)
    ua, ub = torch.zeros_like(Ya), torch.zeros_like(Ya)
    ga, gb = torch.ones_like(Ya), torch.ones_like(Ya)
    for it in range(5):
        s = w.schedule(it)
        bh.step(Ya, P, 0.5, s["exaggeration"], s["learning_rate"], s["momentum"], 0.01, ua, ga)
        bh.step(Yb, lay, 0.5, s["exaggeration"], s["learning_rate"], s["momentum"], 0.01, ub, gb)
    a, b = Ya.cpu().numpy(), Yb.cpu().numpy()
    assert np.abs(a - b).max() <= 1e-4 * np.abs(a).max()


def _ragged_and_empty_p(n, seed):
    """P with the rows (and columns) of its first 500 points emptied, and a P
    with no entries at all."""
    rp, col, val = synth.random_p(n, seed=seed, k=6)
    r = np.repeat(np.arange(n), np.diff(rp))
    keep = (r >= 500) & (col >= 500)
    rp2 = np.concatenate([[0], np.cumsum(np.bincount(r[keep], minlength=n))]).astype(np.int64)
    return [(rp2, col[keep], val[keep]),
            (np.zeros(n + 1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.float32))]


@pytest.mark.parametrize("form", ["fp32", "fp64", "3d"])
def test_layouts_of_ragged_and_empty_p(form):
    """Rows without entries, and a P without any, through the three layout
    forms: the oracle's gradient (zero attraction where rows are empty)."""
    n = 3000
    for rp, col, val in _ragged_and_empty_p(n, seed=21):
        say(f"[layout-ragged] form={form} nnz={col.size}")
        if form == "3d":
            y = synth.random_y3(n, seed=21, scale=2.0)
            Y = torch.from_numpy(y).cuda()
            lay = bh.Layout3(bh.Csr.from_numpy(rp, col, val), Y)
            g, Z = bh.gradient_3d(Y, lay, 0.5, 4.0)
            go, Zo, _, _ = oracle.gradient3(y, rp, col, val, 0.5, 4.0)
            tol = 1e-3
        elif form == "fp64":
            y = synth.random_y(n, seed=21, scale=2.0).astype(np.float64)
            Y = torch.from_numpy(y).cuda()
            lay = bh.LayoutF64(bh.CsrF64.from_numpy(rp, col, val.astype(np.float64)), Y)
            g, Z = bh.gradient_f64(Y, lay, 0.5, 4.0)
            go, Zo, _, _ = oracle.gradient(y, rp, col, val.astype(np.float64), 0.5, 4.0)
            tol = 1e-9
        else:
            y = synth.random_y(n, seed=21, scale=2.0)
            Y = torch.from_numpy(y).cuda()
            lay = bh.Layout(bh.Csr.from_numpy(rp, col, val), Y)
            g, Z = bh.gradient(Y, lay, 0.5, 4.0)
            go, Zo, _, _ = oracle.gradient(y, rp, col, val, 0.5, 4.0)
            tol = 1e-3
        say(f"[layout-ragged] tiles {lay.tiles} windows {lay.windows} segments {lay.segments}")
        assert lay.tiles > 0 or col.size == 0
        assert rel_l2(g.cpu().numpy(), go) <= tol
        assert abs(Z - Zo) <= (1e-12 if form == "fp64" else 1e-5) * Zo


def test_direct_gather_fallback_in_subprocess():
    # with LDS staging disabled every block takes y_j straight from memory
    code = (
        "import sys; sys.path.insert(0, %r)\n"
        "import numpy as np, torch, synth, oracle, paper_2212_11506_amd as bh\n"
        "inp = synth.make_inputs(0)\n"
        "Y = torch.from_numpy(inp.Y).cuda(); P = bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val)\n"
        "g, Z = bh.gradient(Y, bh.Layout(P, Y), 0.5, 12.0)\n"
        "go, Zo, _, _ = oracle.gradient(inp.Y, inp.row_ptr, inp.col, inp.val, 0.5, 12.0)\n"
        "e = np.linalg.norm(g.cpu().numpy() - go) / np.linalg.norm(go)\n"
        "print('relL2', e); assert e <= 1e-3 and abs(Z - Zo) <= 1e-5 * Zo\n" % ROOT)
    env = dict(os.environ, BHTSNE_STAGE_SEGMENTS="0")
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=300)
    say(r.stdout, r.stderr[-2000:])
    assert r.returncode == 0


def test_layout_rejects_bad_handles():
    inp = synth.make_inputs(0)
    Y = torch.from_numpy(inp.Y).cuda()
    P = bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val)
    lay = bh.Layout(P, Y)
    lay._s.magic = 0
    with pytest.raises(bh.BhtsneError) as e:
        bh.gradient(Y, lay, 0.5, 1.0)
    assert e.value.status == bh.BHTSNE_EINVAL


@pytest.mark.parametrize("fault", ["first", "decreasing", "past_end", "short_end"])
def test_layout_rejects_malformed_row_pointers(fault):
    """The build checks P's row pointers on the GPU before it reads any entry
    (row_ptr[0] = 0, non-decreasing, row_ptr[n] = nnz) and returns
    BHTSNE_EINPUT; the KL evaluation clamps such rows to the arrays and reports
    BHTSNE_EDEVICE."""
    inp = synth.make_inputs(0)
    rp = inp.row_ptr.copy()
    n, nnz = inp.n, inp.nnz
    if fault == "first":
        rp[0] = 1
    elif fault == "decreasing":
        rp[n // 2] = rp[n // 2 + 1] + 7
    elif fault == "past_end":
        rp[n - 1] = nnz + 1000
        rp[n] = nnz + 1000
    else:
        rp[n] = nnz - 5
    say(f"[malformed] {fault}")
    Y = torch.from_numpy(inp.Y).cuda()
    P = bh.Csr.from_numpy(rp, inp.col, inp.val)
    with pytest.raises(bh.BhtsneError) as e:
        bh.Layout(P, Y)
    assert e.value.status == bh.BHTSNE_EINPUT
    if fault == "past_end":
        with pytest.raises(bh.BhtsneError) as e:
            bh.kl(Y, P, 1.0)
        assert e.value.status == bh.BHTSNE_EDEVICE
    # a well-formed P still builds and runs on the same workspace afterwards
    ws = torch.empty(bh.workspace_size(n, nnz), dtype=torch.uint8, device="cuda")
    good = bh.Layout(bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val), Y, workspace=ws)
    g, Z = bh.gradient(Y, good, 0.5, 12.0, workspace=ws)
    assert torch.isfinite(g).all() and Z > 0


def test_tiled_copy_reproduces_p():
    inp = synth.make_inputs(1, n=40000)
    P = bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val)
    Y = torch.from_numpy(inp.Y).cuda()
    lay = bh.Layout(P, Y)
    assert lay.tiles > 0
    check_sliced_copy(lay, inp.row_ptr, inp.col, inp.val)


def _subprocess_gradient(env_extra, n=None, wide=False):
    code = (
        "import sys; sys.path.insert(0, %r)\n"
        "import numpy as np, torch, synth, oracle, paper_2212_11506_amd as bh\n"
        "wide = %r\n"
        "if wide:\n"
        "    y = synth.random_y(300000, seed=8, scale=3.0); rp, col, val = synth.random_p(300000, seed=8, k=6)\n"
        "else:\n"
        "    inp = synth.make_inputs(1, n=%r); y, rp, col, val = inp.Y, inp.row_ptr, inp.col, inp.val\n"
        "Y = torch.from_numpy(y).cuda(); P = bh.Csr.from_numpy(rp, col, val)\n"
        "lay = bh.Layout(P, Y); print('tiles', lay.tiles, 'windows', lay.windows, 'segments', lay.segments)\n"
        "g, Z = bh.gradient(Y, lay, 0.5, 12.0)\n"
        "go, Zo, _, _ = oracle.gradient(y, rp, col, val, 0.5, 12.0)\n"
        "e = np.linalg.norm(g.cpu().numpy() - go) / np.linalg.norm(go)\n"
        "print('relL2', e); assert e <= 1e-3 and abs(Z - Zo) <= 1e-5 * Zo\n"
        "sys.exit(3 if lay.tiles > 0 else (5 if lay.windows > 0 else 4))\n" % (ROOT, wide, n))
    env = dict(os.environ, **env_extra)
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=300)
    say(r.stdout, r.stderr[-2000:])
    return r.returncode


def test_row_block_path_when_tiles_disabled():
    assert _subprocess_gradient({"BHTSNE_TILES": "0"}, n=40000) == 4


def test_wide_row_blocks_take_windowed_segments():
    # random columns: every block of 1024 rows spans all ~19 windows of 16384
    # points, so no sliced copy; the rows are cut into segments of the two
    # column windows of 2^18 points instead
    assert _subprocess_gradient({}, wide=True) == 5


def test_wide_row_blocks_fall_back_to_row_blocks_without_windows():
    assert _subprocess_gradient({"BHTSNE_WINDOWS": "0"}, wide=True) == 4


def test_wide_dense_row_blocks_take_the_sliced_copy():
    """Uniform random neighbours (48 drawn per row, about 96 per row after
    symmetrisation) over 300,000 points with a random Y: a block of 1024 rows
    in Morton order reaches all 19 column windows of 16384 points, more than
    the 16 every layout may tile, but its tiles hold about 5,200 entries each
    (a wide layout needs 4,096 on average) and 19 tiles per row block fit the
    32 partial slots per row.  So the sliced copy is built over 19 windows per
    row block, holds exactly P, and the gradient matches the oracle.  With six
    neighbours per row (the tests above) the tiles are too sparse and the
    windowed segments serve the layout."""
    n, k = 300_000, 48
    rng = np.random.default_rng(51)
    rows = np.repeat(np.arange(n), k)
    cols = rng.integers(0, n - 1, size=rows.size)
    cols += cols >= rows  # no self-pairs
    A = sp.csr_matrix((rng.uniform(0.1, 1.0, rows.size), (rows, cols)), shape=(n, n))
    A = (A + A.T).tocsr()
    A.sum_duplicates()
    A.sort_indices()
    A.data /= A.data.sum()
    rp, col, val = A.indptr.astype(np.int64), A.indices.astype(np.int32), A.data.astype(np.float32)
    y = synth.random_y(n, seed=51, scale=3.0)
    Y = torch.from_numpy(np.ascontiguousarray(y)).cuda()
    lay = bh.Layout(bh.Csr.from_numpy(rp, col, val), Y)
    blocks, windows = (n + TILE_ROWS - 1) // TILE_ROWS, (n + TILE_SEG - 1) // TILE_SEG
    say(f"[wide] n={n} nnz={col.size}: order {lay.order}, tiles {lay.tiles}, items {lay.items}, "
        f"entries {lay.entries}, windows {lay.windows}")
    assert lay.order == bh.ORDER_MORTON and lay.tiles == blocks * windows and lay.windows == 0
    assert windows > 16 and col.size >= TILE_WIDE_ENTRIES * lay.tiles
    check_sliced_copy(lay, rp, col, val)
    g, Z = bh.gradient(Y, lay, 0.5, 12.0)
    go, Zo, _, _ = oracle.gradient(y, rp, col, val, 0.5, 12.0)
    err = rel_l2(g.cpu().numpy(), go)
    say(f"[wide] rel-L2 {err:.2e}, Z rel {abs(Z - Zo) / Zo:.2e}")
    assert err <= 1e-3 and abs(Z - Zo) <= 1e-5 * Zo


def test_rows_longer_than_the_row_sort_keep_the_row_block_kernel():
    """A row of 9000 entries is longer than the layout's in-LDS row sort takes,
    so its columns stay out of window order: no segments are built, the
    row-block kernel runs, and the gradient still matches the oracle."""
    n = 400_000
    y = synth.random_y(n, seed=34, scale=2.0)
    rp, col, val = _ring_hubs(n, seed=34, sizes=(9000,))
    say(f"[windows] long row: n={n} nnz={col.size} longest={np.diff(rp).max()}")
    Y = torch.from_numpy(np.ascontiguousarray(y)).cuda()
    lay = bh.Layout(bh.Csr.from_numpy(rp, col, val), Y)
    assert lay.tiles == 0 and lay.windows == 0
    g, Z = bh.gradient(Y, lay, 0.5, 12.0)
    go, Zo, _, _ = oracle.gradient(y, rp, col, val, 0.5, 12.0)
    assert rel_l2(g.cpu().numpy(), go) <= 1e-3 and abs(Z - Zo) <= 1e-5 * Zo


def _ring_hubs(n, seed, sizes=(300, 450, 5000)):
    """A ring P (6 entries per row) plus hub rows longer than any register budget."""
    rp, col, val = synth.ring_p(n, seed, m=3)
    P = sp.csr_matrix((val.astype(np.float64), col, rp), shape=(n, n))
    rng = np.random.default_rng(seed)
    r, c = [], []
    for h, size in enumerate(sizes):
        others = rng.choice(np.arange(len(sizes), n), size=size, replace=False)
        r += [h] * size + list(others)
        c += list(others) + [h] * size
    H = sp.csr_matrix((np.full(len(r), 1e-7), (r, c)), shape=(n, n))
    P = (P + H).tocsr()
    P.sum_duplicates()
    P.sort_indices()
    P.data /= P.data.sum()
    return P.indptr.astype(np.int64), P.indices.astype(np.int32), P.data.astype(np.float32)


@pytest.mark.parametrize("case", ["ring6", "ring40", "hubs"])
def test_windowed_segments_are_p_and_match_the_oracle(case):
    """Layouts without tile locality at several column windows: the segments
    cover every real entry of the relabelled copy exactly once, in window order
    within each row and in row order within each window, and the gradient
    matches the oracle.  Ring P over a random Y, relabelled by the Morton code
    of Y (asked for: a ring with few offsets is a lattice whose breadth-first
    levels would tile it): a row's columns spread over the whole range (one
    component).  ring6: 700k points, 6 entries per row (3 windows); ring40:
    600k points, 40 per row; hubs: 540k points plus rows of 300, 450 and 5000
    entries."""
    if case == "ring6":
        n = 700_000
        y = synth.random_y(n, seed=31, scale=3.0)
        rp, col, val = synth.ring_p(n, 31, m=3)
    elif case == "ring40":
        n = 600_000
        y = synth.random_y(n, seed=32, scale=4.0)
        rp, col, val = synth.ring_p(n, 32, m=20)
    else:
        n = 540_000
        y = synth.random_y(n, seed=33, scale=2.0)
        rp, col, val = _ring_hubs(n, seed=33)
    say(f"[windows] {case}: n={n} nnz={col.size}")
    Y = torch.from_numpy(np.ascontiguousarray(y)).cuda()
    P = bh.Csr.from_numpy(rp, col, val)
    lay = bh.Layout(P, Y, order=bh.ORDER_MORTON)
    assert lay.tiles == 0 and lay.windows == (n + (1 << 18) - 1) >> 18 and lay.segments > 0
    (perm, rank, lrp, lcol, lval) = _layout_arrays(lay)
    mem = lay.mem.cpu().numpy()
    base = _window_region_offset(lay)
    wstart = mem[base:base + 8 * 65].view(np.int64)
    S = lay.segments
    o = base + ((8 * 65 + 255) // 256) * 256
    cap = _max_segments(lay)
    seg_row = mem[o:o + 4 * cap].view(np.uint32)[:S]
    o += ((4 * cap + 255) // 256) * 256
    seg_start = mem[o:o + 4 * cap].view(np.uint32)[:S]
    o += ((4 * cap + 255) // 256) * 256
    seg_len = mem[o:o + 4 * cap].view(np.uint32)[:S]
    assert wstart[0] == 0 and wstart[lay.windows] == S and np.all(np.diff(wstart[:lay.windows + 1]) >= 0)
    win = np.repeat(np.arange(lay.windows), np.diff(wstart[:lay.windows + 1]))
    rows = seg_row.astype(np.int64)
    st = seg_start.astype(np.int64)
    ln = seg_len.astype(np.int64)
    for w in range(lay.windows):  # row order, one segment per row and window
        assert np.all(np.diff(rows[wstart[w]:wstart[w + 1]]) > 0)
    assert np.all(ln > 0) and np.all(lrp[rows] <= st) and np.all(st + ln <= lrp[rows + 1])
    idx = np.repeat(st, ln) + (np.arange(ln.sum()) - np.repeat(np.cumsum(ln) - ln, ln))
    assert np.all((lcol[idx] >> 18) == np.repeat(win, ln))
    covered = np.bincount(idx, minlength=lcol.size)
    real = lcol != NO_COLUMN
    real[lrp[-1]:] = False
    assert np.all(covered[real] == 1) and np.all(covered[~real] == 0)
    g, Z = bh.gradient(Y, lay, 0.5, 12.0)
    go, Zo, _, _ = oracle.gradient(y, rp, col, val, 0.5, 12.0)
    err = rel_l2(g.cpu().numpy(), go)
    say(f"[windows] {case}: {lay.windows} windows, {S} segments, rel-L2 {err:.2e}")
    assert err <= 1e-3 and abs(Z - Zo) <= 1e-5 * Zo


# ------------------------------------------------------------------ point orders
@pytest.mark.parametrize("blobs", [1, 2])
def test_bfs_order_tiles_a_geometric_p_from_a_random_y(blobs):
    """P from the 30 nearest neighbours of 400,000 points uniform in the unit
    square (one component; two squares apart: two), Y a random initial
    embedding.  Morton order of Y brings nothing together: a block of 1024
    rows then reaches all 25 column windows of its component (one component:
    about 1,330 entries per tile; two: 13 windows, 25 for the block across
    both, about 2,550 entries per tile), more than 16 and too sparse for a
    wide layout (4,096 entries per tile).  So the automatic build takes the
    breadth-first levels of P's
    graph (250 or 180 levels of at most 3,700 points: a row block reaches two
    windows): the sliced tiles engage.  The copy's order is exactly
    (component, level, index), and both layouts give the oracle's
    gradient."""
    n = 400_000
    rp, col, val = synth.geometric_p(n, 41 + blobs, k=30, blobs=blobs)
    y = synth.random_y(n, seed=41 + blobs, scale=1e-2)
    Y = torch.from_numpy(np.ascontiguousarray(y)).cuda()
    P = bh.Csr.from_numpy(rp, col, val)
    lay = bh.Layout(P, Y)
    say(f"[order] geometric blobs={blobs}: order {lay.order}, tiles {lay.tiles}, windows {lay.windows}")
    assert lay.order == bh.ORDER_BFS and lay.tiles > 0
    perm = _layout_arrays(lay)[0]
    assert np.array_equal(perm, _bfs_perm(rp, col, n))
    morton = bh.Layout(P, Y, order=bh.ORDER_MORTON)
    assert morton.order == bh.ORDER_MORTON and morton.tiles == 0
    go, Zo, _, _ = oracle.gradient(y, rp, col, val, 0.5, 12.0)
    for lt in (lay, morton):
        g, Z = bh.gradient(Y, lt, 0.5, 12.0)
        err = rel_l2(g.cpu().numpy(), go)
        say(f"[order] order {lt.order}: rel-L2 {err:.2e}")
        assert err <= 1e-3 and abs(Z - Zo) <= 1e-5 * Zo


def test_bfs_order_gives_up_without_locality():
    """A ring P with 40 random offsets per row over 700,000 points: the
    breadth-first levels grow fortyfold and pass 65,536 points at the fourth,
    so an explicit request for them, like the automatic build, falls back to
    the Morton order (and the windowed segments), and the gradient is
    unchanged."""
    n = 700_000
    rp, col, val = synth.ring_p(n, 43, m=20)
    y = synth.random_y(n, seed=43, scale=3.0)
    Y = torch.from_numpy(np.ascontiguousarray(y)).cuda()
    P = bh.Csr.from_numpy(rp, col, val)
    gp, _ = bh.gradient(Y, P, 0.5, 12.0)
    for order in (bh.ORDER_BFS, bh.ORDER_AUTO):
        lay = bh.Layout(P, Y, order=order)
        assert lay.order == bh.ORDER_MORTON and lay.tiles == 0 and lay.windows > 0
        g, _ = bh.gradient(Y, lay, 0.5, 12.0)
        assert rel_l2(g.cpu().numpy(), gp.cpu().numpy().astype(np.float64)) <= 1e-5


def test_explicit_orders_on_a_clustered_p():
    """Workload 0 (2k points, 10 clusters): the automatic build keeps the Morton
    order, which tiles; the breadth-first order is exact and tiles too; an
    unknown order code is rejected."""
    inp = synth.make_inputs(0)
    P = bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val)
    Y = torch.from_numpy(inp.Y).cuda()
    auto = bh.Layout(P, Y)
    assert auto.order == bh.ORDER_MORTON and auto.tiles > 0
    bfs = bh.Layout(P, Y, order=bh.ORDER_BFS)
    assert bfs.order == bh.ORDER_BFS and bfs.tiles > 0
    assert np.array_equal(_layout_arrays(bfs)[0], _bfs_perm(inp.row_ptr, inp.col, inp.n))
    ga, _ = bh.gradient(Y, auto, 0.5, 12.0)
    gb, _ = bh.gradient(Y, bfs, 0.5, 12.0)
    assert rel_l2(gb.cpu().numpy(), ga.cpu().numpy().astype(np.float64)) <= 1e-5
    with pytest.raises(bh.BhtsneError) as e:
        bh.Layout(P, Y, order=7)
    assert e.value.status == bh.BHTSNE_EINVAL


def test_a_row_too_long_to_sort_rules_out_the_sliced_copy():
    """40,000 points of workload 1's clusters (which tile) plus one point
    linked to 9,000 others: that row is longer than the in-LDS row sort
    (8192) and stays unsorted, so the sliced copy, which finds a row's runs
    by binary search, is not built.  With one column window of 2^18 points a
    row is a single segment, whose order does not matter, so the windowed
    segments serve the layout; the gradient matches the oracle."""
    inp = synth.make_inputs(1, n=40000)
    n = inp.n
    P = sp.csr_matrix((inp.val.astype(np.float64), inp.col, inp.row_ptr), shape=(n, n))
    others = np.random.default_rng(17).choice(np.arange(1, n), size=9000, replace=False)
    H = sp.csr_matrix((np.full(18000, 1e-7), (np.r_[np.zeros(9000, int), others], np.r_[others, np.zeros(9000, int)])),
                      shape=(n, n))
    P = (P + H).tocsr()
    P.sum_duplicates()
    P.sort_indices()
    P.data /= P.data.sum()
    rp, col, val = P.indptr.astype(np.int64), P.indices.astype(np.int32), P.data.astype(np.float32)
    assert np.diff(rp).max() > 8192
    Y = torch.from_numpy(inp.Y).cuda()
    lay = bh.Layout(bh.Csr.from_numpy(rp, col, val), Y)
    assert lay.tiles == 0 and lay.windows == 1
    g, Z = bh.gradient(Y, lay, 0.5, 12.0)
    go, Zo, _, _ = oracle.gradient(inp.Y, rp, col, val, 0.5, 12.0)
    assert rel_l2(g.cpu().numpy(), go) <= 1e-3 and abs(Z - Zo) <= 1e-5 * Zo
    # without the long row the same P tiles
    assert bh.Layout(bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val), Y).tiles > 0
