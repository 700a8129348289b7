#!/usr/bin/env python3
"""Write tests/golden/full_runs.json: the fp64 oracle's own full runs of the
large workloads, for the GPU's full-run KL checks.

Calls only the seeded input generator (synth) and the oracle.  For each run
it records the input hashes, the schedule, the KL divergence (Gradient
Descent, the KL cost; the exact O(n^2) normaliser Z, reading R11) of the
initial and the final embedding, the Barnes-Hut Z and interaction count of
the last step, and the wall time.

Runs (each from the workload's initial embedding):
  workload 2  1000 iterations of the schedule (exaggeration 12 and momentum
              0.5 for iterations 0-249, then 1 and 0.8; learning rate N/12)
  workload 4  100 steps at each theta in {0.2, 0.5, 0.8} (exaggeration 1,
              momentum 0.8), and, on the initial embedding, the gradient
              error of the oracle's Barnes-Hut gradient at each theta against
              the exact (theta = 0) gradient on a seeded 20,000-point sample,
              with the exact Z of that embedding
  workload 3  200 steps (exaggeration 1, momentum 0.8)

Usage: python tests/golden/make_full_runs.py [2] [4] [3]   (default: 2 4 3)
Takes hours on 8 cores; progress goes to stdout.  Each finished run is
merged into the JSON file at once.
"""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import synth  # noqa: E402

OUT = os.path.join(HERE, "full_runs.json")
SAMPLE = 20000
SAMPLE_SEED = 2212
THETAS = (0.2, 0.5, 0.8)


def say(*a):
    print(f"[{time.strftime('%H:%M:%S')}]", *a, flush=True)


def merge(key, value):
    data = json.load(open(OUT)) if os.path.exists(OUT) else {}
    data[key] = value
    tmp = OUT + ".tmp"
    with open(tmp, "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
        f.write("\n")
    os.replace(tmp, OUT)


def run(inp, iters, theta, schedule, tag):
    y = inp.Y.astype(np.float64)
    u = np.zeros_like(y)
    g = np.ones_like(y)
    t0 = time.time()
    Z = inter = None
    for it in range(iters):
        s = schedule(it)
        _, Z, inter, _ = oracle.step(y, u, g, inp.row_ptr, inp.col, inp.val, theta, s["exaggeration"],
                                     s["learning_rate"], s["momentum"], 0.01)
        if it % 25 == 24 or it == iters - 1:
            say(f"{tag}: iteration {it + 1}/{iters}, BH Z {Z:.6e}, interactions {inter}, "
                f"{(time.time() - t0) / (it + 1):.2f} s/iteration")
    return y, Z, inter, time.time() - t0


def kl_exact(inp, y, tag):
    t0 = time.time()
    z = oracle.z_exact(y)
    kl = oracle.kl(y, inp.row_ptr, inp.col, inp.val, Z=z)
    say(f"{tag}: exact Z {z:.9e}, KL {kl:.6f} ({time.time() - t0:.0f} s)")
    return kl, z


def schedule_doc(w, it):
    s = w.schedule(it)
    return {k: float(v) for k, v in s.items()}


def workload_2():
    inp = synth.make_inputs(2, progress=say)
    w = inp.workload
    kl0, z0 = kl_exact(inp, inp.Y.astype(np.float64), "workload 2 initial")
    y, Z, inter, secs = run(inp, w.iters, 0.5, w.schedule, "workload 2")
    kl1, z1 = kl_exact(inp, y, "workload 2 final")
    merge("workload_2", {
        "n": inp.n, "nnz": inp.nnz, "hashes": inp.hashes(), "theta": 0.5, "iterations": w.iters,
        "schedule": {"0": schedule_doc(w, 0), "250": schedule_doc(w, 250)},
        "kl_initial": kl0, "z_exact_initial": z0, "kl_final": kl1, "z_exact_final": z1,
        "z_bh_last_step": Z, "interactions_last_step": inter, "seconds": secs, "threads": oracle.threads()})


def workload_3():
    inp = synth.make_inputs(3, progress=say)
    w = inp.workload
    y, Z, inter, secs = run(inp, w.iters, 0.5, w.schedule, "workload 3")
    kl1, z1 = kl_exact(inp, y, "workload 3 final")
    merge("workload_3", {
        "n": inp.n, "nnz": inp.nnz, "hashes": inp.hashes(), "theta": 0.5, "iterations": w.iters,
        "schedule": {"0": schedule_doc(w, 0)}, "kl_final": kl1, "z_exact_final": z1,
        "z_bh_last_step": Z, "interactions_last_step": inter, "seconds": secs, "threads": oracle.threads()})


def workload_4():
    inp = synth.make_inputs(4, progress=say)
    w = inp.workload
    n = inp.n
    y0 = inp.Y.astype(np.float64)
    # gradient error of Barnes-Hut against the exact gradient, initial embedding
    sample = np.sort(np.random.default_rng(SAMPLE_SEED).choice(n, size=SAMPLE, replace=False))
    alpha = w.schedule(0)["exaggeration"]
    t0 = time.time()
    z_exact = oracle.z_exact(y0)
    say(f"workload 4: exact Z of the initial embedding {z_exact:.9e} ({time.time() - t0:.0f} s)")
    fattr = oracle.attractive(y0, inp.row_ptr, inp.col, inp.val, rows=sample)
    errors = {}
    with oracle.State(y0) as s:
        frep0, _, _ = s.repulsive(0.0, points=sample)
        g_exact = 4.0 * (alpha * fattr - frep0 / z_exact)
        for theta in THETAS:
            frep, zi, inter = s.repulsive(theta)
            z_bh = oracle.ordered_sum(zi)
            g_bh = 4.0 * (alpha * fattr - frep[sample] / z_bh)
            err = float(np.linalg.norm(g_bh - g_exact) / np.linalg.norm(g_exact))
            errors[str(theta)] = {"rel_l2": err, "z_bh": z_bh, "z_rel_err": abs(z_bh - z_exact) / z_exact,
                                  "interactions": int(inter.sum())}
            say(f"workload 4 theta={theta}: BH gradient rel-L2 {err:.3e} against exact, Z rel "
                f"{abs(z_bh - z_exact) / z_exact:.2e}, interactions {int(inter.sum())}")
    runs = {}
    kl0 = oracle.kl(y0, inp.row_ptr, inp.col, inp.val, Z=z_exact)
    for theta in THETAS:
        y, Z, inter, secs = run(inp, w.iters, theta, w.schedule, f"workload 4 theta={theta}")
        kl1, z1 = kl_exact(inp, y, f"workload 4 theta={theta} final")
        runs[str(theta)] = {"kl_final": kl1, "z_exact_final": z1, "z_bh_last_step": Z,
                            "interactions_last_step": inter, "seconds": secs}
        merge("workload_4", {
            "n": n, "nnz": inp.nnz, "hashes": inp.hashes(), "iterations": w.iters,
            "schedule": {"0": schedule_doc(w, 0)}, "kl_initial": kl0, "z_exact_initial": z_exact,
            "gradient_error": {"sample": SAMPLE, "sample_seed": SAMPLE_SEED, "exaggeration": alpha,
                               "by_theta": errors},
            "runs": runs, "threads": oracle.threads()})


if __name__ == "__main__":
    which = [int(a) for a in sys.argv[1:]] or [2, 4, 3]
    for cid in which:
        say(f"workload {cid}: start ({oracle.threads()} threads)")
        {2: workload_2, 3: workload_3, 4: workload_4}[cid]()
