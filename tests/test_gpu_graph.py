"""A gradient step captured in a HIP graph (through torch.cuda.graph) and
replayed: the layout step (with the attractive forces forked to the second
stream and joined back by events), the plain CSR step, the fp64 step and
the 3-D layout step.
A step allocates nothing, never synchronises unless Z is requested and
clears its counters with kernels, so each replay must give bit for bit the
eager trajectory's Y, update and gains, with eager work on the same
workspace and synchronisations between the replays."""
import numpy as np
import pytest
import torch

import paper_2212_11506_amd as bh
import synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
ARGS = (0.5, 12.0, 200.0, 0.5, 0.01)
STEPS = 4


def say(*a):
    print(*a, flush=True)


@pytest.mark.parametrize("form", ["layout", "plain", "fp64", "layout3d"])
def test_step_replays_in_a_graph(form):
    inp = synth.make_inputs(1, dim=3 if form == "layout3d" else 2)
    dev = torch.device(DEV)
    if form == "layout3d":
        Y0 = torch.from_numpy(inp.Y).to(dev)
        P = bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val, device=dev)
        ws = torch.empty(bh.workspace_size_3d(inp.n, inp.nnz), dtype=torch.uint8, device=dev)
        step, grad, other = bh.step_3d, bh.gradient_3d, P
        P = bh.Layout3(P, Y0, workspace=ws)
        assert P.tiles > 0
    elif form == "fp64":
        Y0 = torch.from_numpy(inp.Y.astype(np.float64)).to(dev)
        P = bh.CsrF64.from_numpy(inp.row_ptr, inp.col, inp.val.astype(np.float64), device=dev)
        ws = torch.empty(bh.workspace_size_f64(inp.n, inp.nnz), dtype=torch.uint8, device=dev)
        step, grad, other = bh.step_f64, bh.gradient_f64, P
    else:
        Y0 = torch.from_numpy(inp.Y).to(dev)
        P = bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val, device=dev)
        ws = torch.empty(bh.workspace_size(inp.n, inp.nnz), dtype=torch.uint8, device=dev)
        step, grad, other = bh.step, bh.gradient, P
        if form == "layout":
            P = bh.Layout(P, Y0, workspace=ws)

    def fresh():
        return Y0.clone(), torch.zeros_like(Y0), torch.ones_like(Y0)

    Ye, ue, ge = fresh()
    eager = []
    for _ in range(STEPS):
        step(Ye, P, *ARGS, ue, ge, workspace=ws)
        torch.cuda.synchronize()
        eager.append((Ye.clone(), ue.clone(), ge.clone()))

    Yg, ug, gg = fresh()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(Yg, P, *ARGS, ug, gg, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(Yg, Y0), "capture must not run the step"
    Yo = Y0.flip(0).contiguous()
    for k in range(STEPS):
        graph.replay()
        torch.cuda.synchronize()
        for got, want, name in zip((Yg, ug, gg), eager[k], ("Y", "update", "gains")):
            assert torch.equal(got, want), f"{form} replay {k}: {name} differs"
        g, _ = grad(Yo, other, 0.5, 1.0, workspace=ws)  # eager work on the same workspace
        torch.cuda.synchronize()
        assert torch.isfinite(g).all()
    say(f"[graph] {form}: {STEPS} replays match the eager steps")
