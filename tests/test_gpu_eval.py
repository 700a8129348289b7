"""Cost evaluation on the GPU (Background: KL(P || Q) and the normaliser Z of
q_ij) against the oracle's definitions, and closed forms at full size."""
import numpy as np
import pytest
import torch

import oracle
import paper_2212_11506_amd as bh
import synth

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


@pytest.mark.parametrize("n", [2, 3, 63, 1000, 2047, 2048, 2049, 20001])
def test_z_exact_matches_oracle(n):
    y = synth.random_y(n, seed=n, scale=2.0)
    z = bh.z_exact(dev(y))
    zo = oracle.z_exact(y)
    say(f"[z] n={n}: {z:.12e} vs {zo:.12e}")
    assert abs(z - zo) <= 1e-6 * zo


def test_z_exact_two_points_closed_form():
    a = 1.75
    y = np.array([[0.0, 0.0], [a, 0.0]], np.float32)
    assert abs(bh.z_exact(dev(y)) - 2.0 / (1.0 + a * a)) <= 1e-7


def test_z_exact_full_size_closed_forms():
    n = synth.WORKLOADS[2].n
    # all points coincide: every ordered pair contributes exactly 1
    y = np.full((n, 2), 3.25, np.float32)
    assert bh.z_exact(dev(y)) == float(n) * (n - 1)
    # two coincident groups of m points at distance a
    m, a = n // 2, 0.5
    y = np.zeros((2 * m, 2), np.float32)
    y[m:, 0] = a
    want = 2.0 * m * (m - 1) + 2.0 * m * m / (1.0 + a * a)
    z = bh.z_exact(dev(y))
    say(f"[z] two groups of {m}: {z:.12e} vs {want:.12e}")
    assert abs(z - want) <= 1e-6 * want


def test_z_exact_deterministic():
    y = dev(synth.random_y(70001, seed=4))
    assert bh.z_exact(y) == bh.z_exact(y)


@pytest.mark.parametrize("cid", [0, 1])
def test_kl_matches_oracle(cid):
    inp = synth.make_inputs(cid)
    Y = dev(inp.Y)
    P = bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val)
    zo = oracle.z_exact(inp.Y)
    # the same Z on both sides: the KL sum itself
    k = bh.kl(Y, P, zo)
    ko = oracle.kl(inp.Y, inp.row_ptr, inp.col, inp.val, Z=zo)
    say(f"[kl] workload {cid}: {k:.12f} vs {ko:.12f}")
    assert abs(k - ko) <= 1e-9 * abs(ko)
    # with the GPU's exact Z
    z = bh.z_exact(Y)
    assert abs(bh.kl(Y, P, z) - ko) <= 1e-6 * abs(ko)


def test_kl_skips_zero_entries_and_reports_bad_columns():
    y = synth.random_y(100, seed=2)
    rp, col, val = synth.random_p(100, seed=2, k=5)
    val = val.copy()
    val[::7] = 0.0
    zo = oracle.z_exact(y)
    k = bh.kl(dev(y), bh.Csr.from_numpy(rp, col, val), zo)
    assert abs(k - oracle.kl(y, rp, col, val, Z=zo)) <= 1e-9 * abs(k)
    bad = col.copy()
    bad[3] = 100
    with pytest.raises(bh.BhtsneError) as e:
        bh.kl(dev(y), bh.Csr.from_numpy(rp, bad, val), zo)
    assert e.value.status == bh.BHTSNE_EDEVICE


def test_z_exact_nonfinite_input():
    y = synth.random_y(500, seed=3)
    y[10, 0] = np.inf
    with pytest.raises(bh.BhtsneError) as e:
        bh.z_exact(dev(y))
    assert e.value.status == bh.BHTSNE_ENONFINITE
