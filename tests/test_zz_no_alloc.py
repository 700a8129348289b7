"""The no-allocation entry point, bhtsne_step_noalloc, against bhtsne_step.

bhtsne_step_noalloc runs the same kernels as bhtsne_step on the library's
fixed scratch array instead of a caller workspace, so on identical inputs
its outputs (Y, momentum buffer, gains, gradient, Z) must equal bhtsne_step's
bit for bit.  Two calls in a row, the second on a smaller input, check that
what the first call left in the shared array does not leak into the second.
The gradient is also held to the oracle's tolerance (rel-L2 <= 1e-3 at
theta = 0.5, Z within 1e-5)."""
import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2212_11506_amd as bh


def _case(name):
    if name == "late20k":
        inp = synth.make_inputs(4, n=20000)
        return inp.Y, inp.row_ptr, inp.col, inp.val, 1.0
    inp = synth.make_inputs(0)
    return inp.Y, inp.row_ptr, inp.col, inp.val, 12.0


def _one(name):
    y, rp, col, val, alpha = _case(name)
    n = y.shape[0]
    print(f"[noalloc] case={name} n={n} nnz={col.size}", flush=True)
    P = bh.Csr.from_numpy(rp, col, val)
    out = {}
    for form in ("workspace", "noalloc"):
        Y = torch.from_numpy(y).cuda()
        u = torch.full_like(Y, 0.01)
        gains = torch.ones_like(Y)
        grad = torch.empty_like(Y)
        if form == "workspace":
            ws = torch.empty(bh.workspace_size(n, col.size), dtype=torch.uint8, device="cuda")
            Z = bh.step(Y, P, 0.5, alpha, 200.0, 0.5, 0.01, u, gains, grad=grad, workspace=ws, return_z=True)
        else:
            Z = bh.step_noalloc(Y, P, 0.5, alpha, 200.0, 0.5, 0.01, u, gains, grad=grad, return_z=True)
        torch.cuda.synchronize()
        out[form] = [t.cpu().numpy() for t in (Y, u, gains, grad)] + [Z]
    a, b = out["workspace"], out["noalloc"]
    for k in range(4):
        assert np.array_equal(a[k], b[k]), k
    assert a[4] == b[4]
    go, Zo, _, _ = oracle.gradient(y, rp, col, val, 0.5, alpha)
    err = float(np.linalg.norm(b[3] - go) / np.linalg.norm(go))
    print(f"[noalloc] case={name}: identical to bhtsne_step; gradient rel-L2 {err:.2e} against the oracle", flush=True)
    assert err <= 1e-3 and abs(b[4] - Zo) <= 1e-5 * Zo


def test_noalloc_matches_step_twice_second_smaller():
    _one("late20k")
    _one("c0")


def test_noalloc_rejects_sizes_beyond_its_array():
    n = 300000  # its workspace exceeds the fixed array: refused on the host, nothing runs
    assert bh.workspace_size(n, 0) > bh.noalloc_max_bytes()
    rp = torch.zeros(n + 1, dtype=torch.int64, device="cuda")
    P = bh.Csr(rp, torch.zeros(0, dtype=torch.int32, device="cuda"), torch.zeros(0, dtype=torch.float32, device="cuda"))
    Y = torch.zeros((n, 2), dtype=torch.float32, device="cuda")
    u, g = torch.zeros_like(Y), torch.ones_like(Y)
    with pytest.raises(bh.BhtsneError) as e:
        bh.step_noalloc(Y, P, 0.5, 1.0, 200.0, 0.5, 0.01, u, g)
    assert e.value.status == bh.BHTSNE_EINVAL
