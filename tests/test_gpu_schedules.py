"""The layout steps' stream schedules change only how the kernels overlap:
where the attractive forces fork off to the second stream (after the codes,
the sort or the tree: BHTSNE_FORK, BHTSNE_FORK3, BHTSNE_FORK64) and one
stream only (BHTSNE_OVERLAP=0).  The settings are read once per process, so
each runs in a child process; every one must give the default schedule's
gradient and Z bit for bit (the kernels and their inputs are the same)."""
import os
import subprocess
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import sys
sys.path.insert(0, sys.argv[1])
import numpy as np, torch
import synth, paper_2212_11506_amd as bh
form, out = sys.argv[2], sys.argv[3]
inp = synth.make_inputs(1, n=40000, dim=3 if form == "3d" else 2)
if form == "fp64":
    Y = torch.from_numpy(inp.Y.astype(np.float64)).cuda()
    P = bh.CsrF64.from_numpy(inp.row_ptr, inp.col, inp.val.astype(np.float64))
    lay = bh.LayoutF64(P, Y)
    g, Z = bh.gradient_f64(Y, lay, 0.5, 12.0)
elif form == "3d":
    Y = torch.from_numpy(inp.Y).cuda()
    lay = bh.Layout3(bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val), Y)
    g, Z = bh.gradient_3d(Y, lay, 0.5, 12.0)
else:
    Y = torch.from_numpy(inp.Y).cuda()
    lay = bh.Layout(bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val), Y)
    g, Z = bh.gradient(Y, lay, 0.5, 12.0)
assert lay.tiles > 0
np.save(out, g.cpu().numpy())
print(repr(float(Z)), flush=True)
"""


def _run(form, env_extra, out):
    env = dict(os.environ)
    for k in ("BHTSNE_FORK", "BHTSNE_FORK3", "BHTSNE_FORK64", "BHTSNE_OVERLAP"):
        env.pop(k, None)
    env.update(env_extra)
    r = subprocess.run([sys.executable, "-c", CHILD, ROOT, form, out], env=env, capture_output=True, text=True,
                       timeout=300)
    print(form, env_extra, r.stdout.strip(), r.stderr[-500:], flush=True)
    assert r.returncode == 0
    return np.load(out), float(r.stdout.strip().splitlines()[-1])


@pytest.mark.parametrize("form,var", [("fp32", "BHTSNE_FORK"), ("3d", "BHTSNE_FORK3"), ("fp64", "BHTSNE_FORK64")])
def test_schedules_give_the_same_gradient(form, var, tmp_path):
    g0, z0 = _run(form, {}, str(tmp_path / "default.npy"))
    for extra in ({var: "0"}, {var: "1"}, {var: "2"}, {"BHTSNE_OVERLAP": "0"}):
        g, z = _run(form, extra, str(tmp_path / "other.npy"))
        assert z == z0, (extra, z, z0)
        assert np.array_equal(g.view(np.uint8), g0.view(np.uint8)), extra
