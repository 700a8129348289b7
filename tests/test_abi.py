"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function declared in include/bhtsne.h, sizes workspaces, and rejects
bad arguments before touching the device."""
import ctypes as C
import os
import re

import pytest
import torch  # noqa: F401  (loads the HIP runtime the library links against)

import paper_2212_11506_amd as bh
from paper_2212_11506_amd._binding import _Csr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "bhtsne.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(bhtsne_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    lib = bh.load_library()
    names = _declared_functions()
    assert "bhtsne_gradient" in names and "bhtsne_step" in names
    for name in names:
        assert hasattr(lib, name), name


def test_library_has_gfx950_code_object():
    data = open(bh.library_path(), "rb").read()
    assert b"gfx950" in data


def test_workspace_size():
    assert bh.workspace_size(1, 0) == 0
    assert bh.workspace_size(-5, 0) == 0
    assert bh.workspace_size(2, -1) == 0
    assert bh.workspace_size(1 << 26, 0) == 0
    # skip indices of the 2n - 1 node records take 25 bits: n < 2^24
    assert bh.workspace_size(1 << 24, 0) == 0
    assert bh.workspace_size((1 << 24) - 1, 0) > 0
    a = bh.workspace_size(1000, 10)
    b = bh.workspace_size(2000, 10)
    assert 0 < a < b
    assert a % 256 == 0
    # O(n) bytes: ~ a few hundred bytes per point
    big = bh.workspace_size(1_300_000, 233_000_000)
    assert 50 * 1_300_000 < big < 400 * 1_300_000


def test_status_strings():
    for s in (bh.BHTSNE_OK, bh.BHTSNE_EINVAL, bh.BHTSNE_EWORKSPACE, bh.BHTSNE_ENONFINITE,
              bh.BHTSNE_EDEVICE, bh.BHTSNE_EINPUT, bh.BHTSNE_ECAPACITY):
        assert bh.status_string(s) and bh.status_string(s) != "unknown status"
    assert bh.status_string(12345) == "unknown status"


FAKE = 1 << 20  # non-null, 256-aligned fake device addresses: never dereferenced on rejection


def _grad(lib, P, theta=0.5, alpha=1.0, Y=FAKE, grad=FAKE, ws=FAKE, wsb=1 << 40):
    return lib.bhtsne_gradient(C.c_void_p(Y) if Y else None, C.byref(P) if P is not None else None,
                               theta, alpha, C.c_void_p(grad) if grad else None, None,
                               C.c_void_p(ws) if ws else None, wsb, None)


@pytest.mark.parametrize("case", ["null_P", "n1", "nnz_neg", "null_rowptr", "null_col", "null_Y",
                                  "null_grad", "theta_neg", "theta_nan", "alpha_zero",
                                  "alpha_inf", "too_many"])
def test_gradient_rejects_bad_arguments(case):
    lib = bh.load_library()
    P = _Csr(100, 10, FAKE, FAKE, FAKE)
    kw = {}
    if case == "null_P":
        P = None
    elif case == "n1":
        P.n = 1
    elif case == "nnz_neg":
        P.nnz = -1
    elif case == "null_rowptr":
        P.row_ptr = None
    elif case == "null_col":
        P.col = None
    elif case == "null_Y":
        kw["Y"] = 0
    elif case == "null_grad":
        kw["grad"] = 0
    elif case == "theta_neg":
        kw["theta"] = -0.1
    elif case == "theta_nan":
        kw["theta"] = float("nan")
    elif case == "alpha_zero":
        kw["alpha"] = 0.0
    elif case == "alpha_inf":
        kw["alpha"] = float("inf")
    elif case == "too_many":
        P.n = 1 << 26
    assert _grad(lib, P, **kw) == bh.BHTSNE_EINVAL


def test_evaluation_calls_reject_bad_arguments():
    lib = bh.load_library()
    z = C.c_double(0.0)
    ws = C.c_void_p(FAKE)
    assert lib.bhtsne_z_exact(None, 10, C.byref(z), ws, 1 << 40, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_z_exact(C.c_void_p(FAKE), 1, C.byref(z), ws, 1 << 40, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_z_exact(C.c_void_p(FAKE), 10, None, ws, 1 << 40, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_z_exact(C.c_void_p(FAKE), 10, C.byref(z), None, 1 << 40, None) == bh.BHTSNE_EWORKSPACE
    assert lib.bhtsne_z_exact(C.c_void_p(FAKE), 10, C.byref(z), ws, 16, None) == bh.BHTSNE_EWORKSPACE
    P = bh._binding._Csr(10, 20, C.c_void_p(FAKE), C.c_void_p(FAKE), C.c_void_p(FAKE))
    for bad_z in (0.0, -1.0, float("nan"), float("inf")):
        assert lib.bhtsne_kl(C.c_void_p(FAKE), C.byref(P), bad_z, C.byref(z), ws, 1 << 40, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_kl(C.c_void_p(FAKE), None, 1.0, C.byref(z), ws, 1 << 40, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_kl(None, C.byref(P), 1.0, C.byref(z), ws, 1 << 40, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_kl(C.c_void_p(FAKE), C.byref(P), 1.0, None, ws, 1 << 40, None) == bh.BHTSNE_EINVAL


def test_timing_phase_mask():
    lib = bh.load_library()
    assert lib.bhtsne_timing_phases(1 << len(bh.PHASES)) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_timing_phases(0xFFFFFFFF) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_timing_phases(1 << bh.PHASES.index("repulsive")) == bh.BHTSNE_OK
    assert lib.bhtsne_timing_phases((1 << len(bh.PHASES)) - 1) == bh.BHTSNE_OK


def test_gradient_rejects_bad_workspace():
    lib = bh.load_library()
    P = _Csr(100, 10, FAKE, FAKE, FAKE)
    need = lib.bhtsne_workspace_size(100, 10)
    assert _grad(lib, P, ws=0) == bh.BHTSNE_EWORKSPACE
    assert _grad(lib, P, ws=FAKE + 8) == bh.BHTSNE_EWORKSPACE  # misaligned
    assert _grad(lib, P, wsb=need - 1) == bh.BHTSNE_EWORKSPACE


@pytest.mark.parametrize("lr,mu,mg,ok", [(0.0, 0.5, 0.01, False), (200.0, 1.0, 0.01, False),
                                         (200.0, -0.1, 0.01, False), (200.0, 0.5, -1.0, False),
                                         (float("nan"), 0.5, 0.01, False)])
def test_step_rejects_bad_optimiser_arguments(lr, mu, mg, ok):
    lib = bh.load_library()
    P = _Csr(100, 10, FAKE, FAKE, FAKE)
    rc = lib.bhtsne_step(C.c_void_p(FAKE), C.byref(P), 0.5, 12.0, lr, mu, mg, C.c_void_p(FAKE),
                         C.c_void_p(FAKE), None, None, C.c_void_p(FAKE), 1 << 40, None)
    assert rc == bh.BHTSNE_EINVAL


def test_step_rejects_missing_state():
    lib = bh.load_library()
    P = _Csr(100, 10, FAKE, FAKE, FAKE)
    rc = lib.bhtsne_step(C.c_void_p(FAKE), C.byref(P), 0.5, 12.0, 200.0, 0.5, 0.01, None,
                         C.c_void_p(FAKE), None, None, C.c_void_p(FAKE), 1 << 40, None)
    assert rc == bh.BHTSNE_EINVAL


def test_debug_entry_points_reject_bad_arguments():
    lib = bh.load_library()
    nn = C.c_int64(0)
    assert lib.bhtsne_debug_sort(None, 10, None, None, None, None, C.c_void_p(FAKE), 1 << 40,
                                 None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_debug_sort(C.c_void_p(FAKE), 1, None, None, None, None, C.c_void_p(FAKE),
                                 1 << 40, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_debug_tree(C.c_void_p(FAKE), 10, 0.5, None, None, None, None, None, None,
                                 None, C.c_void_p(FAKE), 1 << 40, None) == bh.BHTSNE_EINVAL
    # partial set of per-node export arrays
    assert lib.bhtsne_debug_tree(C.c_void_p(FAKE), 10, 0.5, C.byref(nn), C.c_void_p(FAKE), None,
                                 None, None, None, None, C.c_void_p(FAKE), 1 << 40,
                                 None) == bh.BHTSNE_EINVAL


def test_binding_refuses_cpu_tensors():
    with pytest.raises(ValueError):
        bh.Csr(torch.zeros(3, dtype=torch.int64), torch.zeros(2, dtype=torch.int32),
               torch.zeros(2, dtype=torch.float32))


def test_affinities_workspace_size():
    ws = bh.affinities_workspace_size
    assert ws(1, 1) == 0 and ws(10, 0) == 0 and ws(10, 10) == 0  # k < n, k >= 1
    assert ws(1000, 257) == 0 and ws(1000, 256) > 0             # at most 256 neighbours
    assert ws(1 << 24, 90) == 0 and ws((1 << 24) - 1, 90) > 0
    a, b = ws(1000, 30), ws(1000, 60)
    assert 0 < a < b and a % 256 == 0
    # per neighbour: p and its sorted column with the neighbour position (13 B),
    # two ping-pong (column, entry) pairs of the sort (16 B) and the look-back
    # words, 3 passes x 256 digits x 8 B per 4096 pairs (1.5 B; 2 passes below
    # 65536 points), plus 16 B per point
    assert 30.5 * 1_300_000 * 90 < ws(1_300_000, 90) < 30.8 * 1_300_000 * 90
    assert 30 * 1000 * 200 < ws(1000, 200) < 31 * 1000 * 200


def test_affinities_rejects_bad_arguments():
    lib = bh.load_library()
    nnz = C.c_int64(-1)
    f = C.c_void_p(FAKE)
    ws = C.c_void_p(FAKE)
    big = 1 << 40

    def call(idx=f, dist=f, n=100, k=10, u=5.0, rp=f, col=f, val=f, cap=2000, out=True, w=ws, wb=big):
        return lib.bhtsne_affinities(idx, dist, n, k, u, rp, col, val, cap, C.byref(nnz) if out else None, None,
                                     w, wb, None)

    assert call(idx=None) == bh.BHTSNE_EINVAL
    assert call(dist=None) == bh.BHTSNE_EINVAL
    assert call(rp=None) == bh.BHTSNE_EINVAL
    assert call(out=False) == bh.BHTSNE_EINVAL
    assert call(cap=-1) == bh.BHTSNE_EINVAL
    assert call(col=None) == bh.BHTSNE_EINVAL
    for u in (0.0, -1.0, float("nan"), float("inf")):
        assert call(u=u) == bh.BHTSNE_EINVAL
    assert call(k=0) == bh.BHTSNE_EINVAL and call(k=257, n=1000) == bh.BHTSNE_EINVAL
    assert call(k=100, n=100) == bh.BHTSNE_EINVAL and call(n=1) == bh.BHTSNE_EINVAL
    assert call(w=None) == bh.BHTSNE_EWORKSPACE
    assert call(w=C.c_void_p(FAKE + 8)) == bh.BHTSNE_EWORKSPACE
    assert call(wb=lib.bhtsne_affinities_workspace_size(100, 10) - 1) == bh.BHTSNE_EWORKSPACE
    assert nnz.value == -1  # nothing reached the device


def test_f64_workspace_size():
    assert bh.workspace_size_f64(1, 0) == 0 and bh.workspace_size_f64(2, -1) == 0
    assert bh.workspace_size_f64(1 << 24, 0) == 0 and bh.workspace_size_f64((1 << 24) - 1, 0) > 0
    # fp64 copies of Y, F_rep and 40-byte node records, and the sliced copy's
    # partial sums in 32 slots per point of 16 bytes (fp32: 8 bytes): larger
    # than the fp32 workspace by 256 to 400 bytes per point
    a, b = bh.workspace_size(100000, 10**6), bh.workspace_size_f64(100000, 10**6)
    assert a + 256 * 100000 < b < a + 400 * 100000 and b % 256 == 0


def test_f64_entry_points_reject_bad_arguments():
    lib = bh.load_library()
    P = bh._binding._Csr(100, 10, FAKE, FAKE, FAKE)
    ws = C.c_void_p(FAKE)
    f = C.c_void_p(FAKE)
    z = C.c_double(0.0)
    assert lib.bhtsne_gradient_f64(None, C.byref(P), 0.5, 1.0, f, None, ws, 1 << 40, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_gradient_f64(f, None, 0.5, 1.0, f, None, ws, 1 << 40, None) == bh.BHTSNE_EINVAL
    for theta, alpha in [(-1.0, 1.0), (float("nan"), 1.0), (0.5, 0.0), (0.5, float("inf"))]:
        assert lib.bhtsne_gradient_f64(f, C.byref(P), theta, alpha, f, C.byref(z), ws, 1 << 40,
                                       None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_gradient_f64(f, C.byref(P), 0.5, 1.0, f, None, None, 1 << 40, None) == bh.BHTSNE_EWORKSPACE
    assert lib.bhtsne_gradient_f64(f, C.byref(P), 0.5, 1.0, f, None, ws, 16, None) == bh.BHTSNE_EWORKSPACE
    for lr, mu, mg in [(0.0, 0.5, 0.01), (200.0, 1.0, 0.01), (200.0, -0.1, 0.01), (200.0, 0.5, -1.0)]:
        assert lib.bhtsne_step_f64(f, C.byref(P), 0.5, 12.0, lr, mu, mg, f, f, None, None, ws, 1 << 40,
                                   None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_step_f64(f, C.byref(P), 0.5, 12.0, 200.0, 0.5, 0.01, None, f, None, None, ws, 1 << 40,
                               None) == bh.BHTSNE_EINVAL
    bad = bh._binding._Csr(1, 10, FAKE, FAKE, FAKE)
    assert lib.bhtsne_gradient_f64(f, C.byref(bad), 0.5, 1.0, f, None, ws, 1 << 40, None) == bh.BHTSNE_EINVAL


def test_bench_refuses_more_than_one_gpu():
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=root)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_step_noalloc_rejects_bad_arguments_on_the_host():
    lib = bh.load_library()
    assert lib.bhtsne_noalloc_max_bytes() == 64 << 20
    # a size whose workspace exceeds the fixed array, bad optimiser arguments, missing state
    big = _Csr(300000, 10, FAKE, FAKE, FAKE)
    small = _Csr(100, 10, FAKE, FAKE, FAKE)
    for P, lr, upd in ((big, 200.0, FAKE), (small, 0.0, FAKE), (small, 200.0, None)):
        rc = lib.bhtsne_step_noalloc(C.c_void_p(FAKE), C.byref(P), 0.5, 12.0, lr, 0.5, 0.01,
                                     C.c_void_p(upd) if upd else None, C.c_void_p(FAKE), None, None, None)
        assert rc == bh.BHTSNE_EINVAL


def test_3d_workspace_size_and_argument_checks():
    lib = bh.load_library()
    assert lib.bhtsne_workspace_size_3d(1, 0) == 0 and lib.bhtsne_workspace_size_3d(1 << 24, 0) == 0
    n = 5000
    assert lib.bhtsne_workspace_size_3d(n, 10) > lib.bhtsne_workspace_size(n, 10) // 2
    P = _Csr(n, 10, FAKE, FAKE, FAKE)
    ws = lib.bhtsne_workspace_size_3d(n, 10)
    # bad theta, bad exaggeration, missing grad, small workspace: all refused on the host
    assert lib.bhtsne_gradient_3d(C.c_void_p(FAKE), C.byref(P), -1.0, 1.0, C.c_void_p(FAKE), None,
                                  C.c_void_p(FAKE), ws, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_gradient_3d(C.c_void_p(FAKE), C.byref(P), 0.5, 0.0, C.c_void_p(FAKE), None,
                                  C.c_void_p(FAKE), ws, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_gradient_3d(C.c_void_p(FAKE), C.byref(P), 0.5, 1.0, None, None,
                                  C.c_void_p(FAKE), ws, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_gradient_3d(C.c_void_p(FAKE), C.byref(P), 0.5, 1.0, C.c_void_p(FAKE), None,
                                  C.c_void_p(FAKE), ws - 1, None) == bh.BHTSNE_EWORKSPACE
    assert lib.bhtsne_step_3d(C.c_void_p(FAKE), C.byref(P), 0.5, 1.0, 200.0, 1.0, 0.01, C.c_void_p(FAKE),
                              C.c_void_p(FAKE), None, None, C.c_void_p(FAKE), ws, None) == bh.BHTSNE_EINVAL
    nn = C.c_int64(0)
    assert lib.bhtsne_debug_tree_3d(C.c_void_p(FAKE), 1, 0.5, C.byref(nn), None, None, None, None, None, None,
                                    None, C.c_void_p(FAKE), ws, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_debug_sort_3d(None, n, None, None, None, None, C.c_void_p(FAKE), ws,
                                    None) == bh.BHTSNE_EINVAL


def test_3d_layout_size_and_argument_checks():
    from paper_2212_11506_amd._binding import _Layout
    lib = bh.load_library()
    assert lib.bhtsne_layout_size_3d(1, 0) == 0 and lib.bhtsne_layout_size_3d(1 << 24, 0) == 0
    n, nnz = 100_000, 1_000_000
    a2, a3 = lib.bhtsne_layout_size(n, nnz), lib.bhtsne_layout_size_3d(n, nnz)
    # the same copies; the 3-D sliced copy may pad for twice the tiles per
    # row block (8192-point windows)
    assert a2 < a3 < 2 * a2 and a3 % 256 == 0
    P = _Csr(n, nnz, FAKE, FAKE, FAKE)
    ws = lib.bhtsne_workspace_size_3d(n, nnz)
    lay = _Layout()
    f = C.c_void_p(FAKE)
    assert lib.bhtsne_layout_build_3d(C.byref(P), None, f, a3, None, f, ws, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_layout_build_3d(C.byref(P), None, f, a3 - 1, C.byref(lay), f, ws, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_layout_build_3d(C.byref(P), None, f, a3, C.byref(lay), f, ws - 1,
                                      None) == bh.BHTSNE_EWORKSPACE
    assert lib.bhtsne_layout_build_3d(None, None, f, a3, C.byref(lay), f, ws, None) == bh.BHTSNE_EINVAL

    def handle(magic, tiles):
        return _Layout(n, nnz, FAKE, a3, tiles, 1 if tiles else 0, 4096 * tiles, 0, 0, 0, magic)

    l3 = handle(0x62687473654c3033, 10)
    for bad in (handle(0x62687473654c3031, 10), handle(0x62687473654c3634, 10), handle(0, 10),
                handle(0x62687473654c3033, 0)):
        # a 2-D, fp64 or unbuilt handle, or a 3-D one without tiles: refused on the host
        assert lib.bhtsne_gradient_layout_3d(f, C.byref(bad), 0.5, 1.0, f, None, f, ws, None) == bh.BHTSNE_EINVAL
        assert lib.bhtsne_step_layout_3d(f, C.byref(bad), 0.5, 1.0, 200.0, 0.5, 0.01, f, f, None, None, f, ws,
                                         None) == bh.BHTSNE_EINVAL
    # and the 2-D calls refuse a 3-D handle
    assert lib.bhtsne_gradient_layout(f, C.byref(l3), 0.5, 1.0, f, None, f, 1 << 40, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_gradient_layout_3d(f, C.byref(l3), -1.0, 1.0, f, None, f, ws, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_gradient_layout_3d(f, C.byref(l3), 0.5, 1.0, None, None, f, ws, None) == bh.BHTSNE_EINVAL
    assert lib.bhtsne_gradient_layout_3d(f, C.byref(l3), 0.5, 1.0, f, None, f, ws - 1,
                                         None) == bh.BHTSNE_EWORKSPACE
    assert lib.bhtsne_step_layout_3d(f, C.byref(l3), 0.5, 1.0, 200.0, 1.0, 0.01, f, f, None, None, f, ws,
                                     None) == bh.BHTSNE_EINVAL
