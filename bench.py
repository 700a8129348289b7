#!/usr/bin/env python3
"""Throughput of the BH t-SNE gradient iteration on one MI355X.

A step is one full iteration of the library (bounding box, Morton codes,
radix sort, quadtree build and summaries, Barnes-Hut repulsion with Z, CSR
attraction, gradient and gains/momentum update) on the 1.3M-point workload
with 30 Dirichlet(1) clusters and 90 within-cluster neighbours per point
(about 2.34e8 stored entries of P), theta = 0.5, following the 1000-iteration
schedule (exaggeration 12 and momentum 0.5 for the first 250 iterations, then
1 and 0.8; learning rate N/12).  Inputs are seeded synthetic data resident in
HBM before timing starts.

Prints one JSON line on stdout.  Progress goes to stderr.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "BH t-SNE gradient iterations/s at N=1.3M, theta=0.5; repulsive interactions/s"
HBM_PEAK_GBS = 8000.0
# MI355X's published fp32 vector peak (it counts packed fp32: two lanes' worth
# per instruction) and the rate without packed math, which this build
# disables: 256 CUs x 64 lanes x 2 flops (FMA) x 2.4 GHz
ALU_PEAK_TFLOPS = 157.3
ALU_PEAK_NONPACKED_TFLOPS = 256 * 64 * 2 * 2.4e9 / 1e12
# algorithmic flops of one interaction (summary or exact pair): dx, dy (2),
# d^2 (3), 1 + d^2 (1), reciprocal (1), count x w and w^2 (2), Z (1), forces (4)
FLOPS_PER_INTERACTION = 14
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_1p3M.md")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", type=int, default=2)
    ap.add_argument("--n", type=int, default=None, help="override the workload size")
    ap.add_argument("--theta", type=float, default=0.5)
    ap.add_argument("--cpu-iters", type=int, default=16, help="oracle iterations for the CPU baseline")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-count", action="store_true", help="skip the interaction-counting replay")
    ap.add_argument("--no-affinities", action="store_true", help="skip the input-similarity measurement")
    ap.add_argument("--affinities-only", action="store_true", help="measure only the input similarities")
    ap.add_argument("--no-fp64", action="store_true", help="skip the fp64-variant measurement")
    ap.add_argument("--fp64-only", action="store_true", help="measure only the fp64 variant")
    ap.add_argument("--plain", action="store_true",
                    help="attractive step straight from the CSR arrays (no locality layout)")
    ap.add_argument("--no-overlap", action="store_true",
                    help="attractive forces on the main stream, not beside the sort, tree and walk "
                         "(for counter collection, which takes one dispatch at a time)")
    ap.add_argument("--copy-calibrate", action="store_true",
                    help="only run device-to-device copies of 1 GiB (for scaling HBM counters)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other workloads (0, 1, 3 and 4 at each theta) of the headline run")
    ap.add_argument("--no-3d", action="store_true", help="skip the 3-D embedding measurement")
    ap.add_argument("--3d-only", dest="only_3d", action="store_true", help="measure only the 3-D embedding path")
    ap.add_argument("--no-locality", action="store_true",
                    help="skip the layout-order measurement on a geometric P with a random Y")
    ap.add_argument("--locality-only", action="store_true", help="measure only the layout orders")
    ap.add_argument("--configs-only", action="store_true", help="measure only the other workloads")
    ap.add_argument("--save-y", default=None,
                    help="run --save-after iterations of the schedule, save Y there (.npy) and stop")
    ap.add_argument("--save-after", type=int, default=900)
    ap.add_argument("--load-y", default=None,
                    help="start from a Y saved by --save-y (layout built from it), at schedule iteration "
                         "--iter0, with zero momentum and unit gains (for counters on late iterations)")
    ap.add_argument("--iter0", type=int, default=900)
    return ap.parse_args()


def copy_calibrate():
    """Ten copies of 1 GiB on the device: the known bytes that FETCH_SIZE and
    WRITE_SIZE are scaled by."""
    import torch
    nbytes = 1 << 30
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(10):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration": True, "bytes_read_per_copy": nbytes, "bytes_written_per_copy": nbytes,
                      "copies": 10}), flush=True)


def source_hash(*names):
    import hashlib
    h = hashlib.sha256()
    for name in names:
        with open(os.path.join(ROOT, "paper_2212_11506_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel, sources):
    """HBM bytes per launch of `kernel` from the committed counter summary,
    or None when the summary is missing or the kernel's sources changed since."""
    try:
        lines = open(TRAFFIC_FILE).read().splitlines()
    except OSError:
        return None
    for line in lines:
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if len(cells) >= 4 and cells[0] == kernel:
            try:
                traffic = float(cells[1])
            except ValueError:
                return None
            return traffic if cells[3] == source_hash(*sources) else None
    return None


def attractive_path(lay):
    """Which attractive kernel a layout takes."""
    if lay.tiles > 0:
        return "sliced tiles"
    return "windowed segments" if lay.windows > 0 else "row blocks"


def gpu_run(inp, theta, steps, warmup, schedule, layout=True, order=None, graph=False):
    """Iterations of `schedule` on the GPU through the locality layout (the
    launch configuration of the headline run), inputs resident in HBM: the
    rate over `steps` timed iterations after `warmup` untimed ones (from the
    initial state again), the walk's and the attraction's event times, and
    the interactions per iteration from a replay of the same (deterministic)
    trajectory with a sync per step."""
    import numpy as np
    import torch

    import paper_2212_11506_amd as bh

    dev = torch.device("cuda:0")
    n, nnz = inp.n, inp.nnz
    Y0 = torch.from_numpy(inp.Y).to(dev)
    P = bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val, device=dev)
    ws = torch.empty(bh.workspace_size(n, nnz), dtype=torch.uint8, device=dev)
    build_s = None
    if layout:
        torch.cuda.synchronize()
        tb = time.perf_counter()
        P = bh.Layout(P, Y0, workspace=ws, order=order)
        torch.cuda.synchronize()
        build_s = time.perf_counter() - tb
    Y, u, g = Y0.clone(), torch.zeros_like(Y0), torch.ones_like(Y0)

    def reset():
        Y.copy_(Y0)
        u.zero_()
        g.fill_(1.0)

    def run(k, per_step=None):
        for it in range(k):
            s = schedule(it)
            bh.step(Y, P, theta, s["exaggeration"], s["learning_rate"], s["momentum"], 0.01, u, g, workspace=ws)
            if per_step:
                per_step(it)

    run(warmup)
    torch.cuda.synchronize()
    reset()
    bh.timing_read(reset=True)
    bh.timing_phases(["repulsive", "attractive"])
    bh.timing_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(steps)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    bh.timing_enable(False)
    bh.timing_phases(None)
    ph = bh.timing_read(reset=True)
    y_final = Y.cpu().numpy()
    reset()
    counts = []
    run(steps, per_step=lambda it: counts.append(bh.get_stats(ws)["interactions"]))
    torch.cuda.synchronize()
    same = bool(np.array_equal(Y.cpu().numpy(), y_final))
    inter = float(np.mean(counts)) if same else None
    graph_rate = graph_same = None
    if graph:
        # the same iterations replayed from HIP graphs, one per set of the
        # schedule's parameters (a step never synchronises without Z)
        graphs = {}
        keys = [tuple(schedule(it)[k] for k in ("exaggeration", "learning_rate", "momentum")) for it in range(steps)]
        reset()
        torch.cuda.synchronize()
        for key in dict.fromkeys(keys):
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr):
                bh.step(Y, P, theta, key[0], key[1], key[2], 0.01, u, g, workspace=ws)
            graphs[key] = gr
        torch.cuda.synchronize()
        for gr in graphs.values():  # warm replays, then the initial state again
            gr.replay()
        torch.cuda.synchronize()
        reset()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for key in keys:
            graphs[key].replay()
        torch.cuda.synchronize()
        graph_rate = steps / (time.perf_counter() - t0)
        graph_same = bool(np.array_equal(Y.cpu().numpy(), y_final))
        del graphs
    rep_ms = ph["repulsive"][0] / max(ph["repulsive"][1], 1)
    att_ms = ph["attractive"][0] / max(ph["attractive"][1], 1)
    out = {"n": n, "nnz": nnz, "theta": theta, "steps": steps, "iterations_per_s": steps / dt,
           "ms_per_step": 1e3 * dt / steps, "interactions_per_iteration": inter,
           "interactions_per_s": inter * steps / dt if inter else None,
           "repulsive_ms": rep_ms, "attractive_ms": att_ms,
           "attractive_path": attractive_path(P) if layout else "plain CSR"}
    if layout:
        out["layout_order"] = "bfs levels" if P.order == bh.ORDER_BFS else "morton"
        out["layout_build_s"] = build_s
    if graph:
        out["graph_iterations_per_s"] = graph_rate
        out["graph_matches_eager"] = graph_same
    if inter:
        tf = FLOPS_PER_INTERACTION * inter / (rep_ms * 1e-3) / 1e12
        out["repulsive_tflops"] = tf
        out["repulsive_frac_alu"] = tf / ALU_PEAK_TFLOPS
        out["repulsive_frac_alu_nonpacked"] = tf / ALU_PEAK_NONPACKED_TFLOPS
    out["attractive_model_gbs"] = (8.0 * nnz + 32.0 * n) / (att_ms * 1e-3) / 1e9
    out["attractive_model_frac_hbm"] = out["attractive_model_gbs"] / HBM_PEAK_GBS
    del P, ws, Y0, Y, u, g
    torch.cuda.empty_cache()
    return out


def oracle_sample(inp, theta, iters, schedule, threads=None):
    """The fp64 oracle (as it stands) on the first `iters` iterations of the
    same schedule, with the wall time of each of the paper's steps."""
    import numpy as np

    import oracle

    all_threads = oracle.threads()
    if threads:
        oracle.set_threads(threads)
    try:
        y = inp.Y.astype(np.float64)
        u, g = np.zeros_like(y), np.ones_like(y)
        tot = dict.fromkeys(oracle.STEP_PHASES, 0.0)
        t0 = time.perf_counter()
        inter = 0
        for it in range(iters):
            s = schedule(it)
            _, k, _, ms = oracle.step_timed(y, u, g, inp.row_ptr, inp.col, inp.val, theta, s["exaggeration"],
                                            s["learning_rate"], s["momentum"], 0.01)
            inter += k
            for key in tot:
                tot[key] += ms[key]
        dt = time.perf_counter() - t0
        cores = oracle.threads()
    finally:
        oracle.set_threads(all_threads)
    return {"iterations_per_s": iters / dt, "cores": cores, "iterations": iters, "seconds": dt,
            "interactions_per_s": inter / dt, "step_ms": {k: v / iters for k, v in tot.items()}}


def bench_locality(args, n=1_300_000, k=90, steps=100, seed=2212):
    """A P whose locality lies in P alone: the 90 nearest neighbours of 1.3M
    points uniform in the unit square (one connected component), from a
    random initial Y (N(0, 1e-4 I)), iterations 0..99 of the headline
    schedule.  The layout's automatic order (the breadth-first levels of P's
    graph, which tile) against the Morton order of Y (no tiles: windowed
    segments)."""
    import types

    import synth

    t0 = time.time()
    rp, col, val = synth.geometric_p(n, seed, k=k)
    y = synth.random_y(n, seed=seed, scale=1e-2)
    log(f"[bench] locality: geometric P, n={n} nnz={col.size} drawn in {time.time() - t0:.0f}s")
    inp = types.SimpleNamespace(n=n, nnz=int(col.size), Y=y, row_ptr=rp, col=col, val=val)
    w = synth.WORKLOADS[2]
    out = {"workload": f"kNN graph (k = {k}) of {n} points uniform in the unit square, one component, "
                       f"random initial Y, iterations 0..{steps - 1} of the workload-2 schedule",
           "n": n, "nnz": int(col.size)}
    import paper_2212_11506_amd as bh
    for tag, order in (("auto", bh.ORDER_AUTO), ("morton", bh.ORDER_MORTON)):
        r = gpu_run(inp, args.theta, steps, 5, w.schedule, order=order)
        log(f"[bench] locality {tag}: {r['iterations_per_s']:.1f} it/s, {r['attractive_path']} "
            f"({r['layout_order']}), attraction {r['attractive_ms']:.3f} ms")
        out[tag] = r
    return out


def bench_configs(args, log_every=None):
    """Every workload besides the headline one, each with its own schedule:
    iterations/s and interactions/s on the GPU, walk and attraction
    fractions, and the oracle on the host (all cores, single thread for the
    two small workloads) on a bounded sample of the same run."""
    import gc

    import synth

    out = {}
    plan = [(0, [0.5], 50, 10, 2), (1, [0.5], 1000, 3, 1), (4, [0.2, 0.5, 0.8], 100, 1, 0), (3, [0.5], 200, 1, 0)]
    for cid, thetas, steps, cpu_iters, cpu_single in plan:
        t0 = time.time()
        inp = synth.make_inputs(cid, progress=log)
        w = inp.workload
        log(f"[bench] workload {cid}: n={inp.n} nnz={inp.nnz} generated in {time.time() - t0:.1f}s")
        entry = {"workload": f"{w.description} (workload {cid})", "n": inp.n, "nnz": inp.nnz,
                 "schedule": f"iterations 0..{steps - 1}", "by_theta": {}}
        for theta in thetas:
            # the small workloads are launch-bound: also replayed from HIP graphs
            r = gpu_run(inp, theta, steps, 5 if steps >= 50 else 1, w.schedule, graph=cid in (0, 1))
            log(f"[bench] workload {cid} theta={theta}: {r['iterations_per_s']:.1f} it/s, "
                f"{r['interactions_per_s'] or 0:.3e} interactions/s")
            if not args.no_cpu and cpu_iters:
                r["oracle"] = oracle_sample(inp, theta, cpu_iters, w.schedule)
                if cpu_single:
                    r["oracle_single_thread"] = oracle_sample(inp, theta, cpu_single, w.schedule, threads=1)
                log(f"[bench] workload {cid} theta={theta}: oracle {r['oracle']['iterations_per_s']:.3f} it/s "
                    f"on {r['oracle']['cores']} threads")
            entry["by_theta"][str(theta)] = r
        out[f"workload_{cid}"] = entry
        del inp
        gc.collect()
    return out


def bench_3d(args, steps=200, warmup=5):
    """The 3-D embedding path on workload 2's P with a 3-D early-phase Y
    (N(0, 1e-4 I3)): iterations/s over the first `steps` iterations of the
    schedule with P through the 3-D locality layout (the sliced attraction
    beside the sort, tree and walk), then on the plain CSR P; each with the
    phases' event times."""
    import numpy as np
    import torch

    import paper_2212_11506_amd as bh
    import synth

    inp = synth.make_inputs(2, dim=3)
    w = inp.workload
    n, nnz = inp.n, inp.nnz
    dev = torch.device("cuda:0")
    P = bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val, device=dev)
    ws = torch.empty(bh.workspace_size_3d(n, nnz), dtype=torch.uint8, device=dev)
    Y0 = torch.from_numpy(inp.Y).to(dev)
    Y, u, g = Y0.clone(), torch.zeros_like(Y0), torch.ones_like(Y0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    lay = bh.Layout3(P, Y0, workspace=ws)
    torch.cuda.synchronize()
    build_s = time.perf_counter() - t0

    def reset():
        Y.copy_(Y0)
        u.zero_()
        g.fill_(1.0)

    def run(PP, k, per_step=None):
        for it in range(k):
            s = w.schedule(it)
            bh.step_3d(Y, PP, args.theta, s["exaggeration"], s["learning_rate"], s["momentum"], 0.01, u, g,
                       workspace=ws)
            if per_step:
                per_step(it)

    def measure(PP):
        run(PP, warmup)
        torch.cuda.synchronize()
        reset()
        bh.timing_read(reset=True)
        bh.timing_phases(None)
        bh.timing_enable(True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        run(PP, steps)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        bh.timing_enable(False)
        ph = bh.timing_read(reset=True)
        reset()
        return {"iterations_per_s": steps / dt, "ms_per_step": 1e3 * dt / steps,
                "phases_ms": {k: v[0] / v[1] for k, v in ph.items() if v[1]}}

    tiled = lay.tiles > 0
    out = {"workload": "workload 2's P (1.3M points) with a 3-D early-phase Y ~ N(0, 1e-4 I3)",
           "n": n, "nnz": nnz, "theta": args.theta, "steps": steps,
           "attractive_path": "sliced tiles" if tiled else "plain CSR (the layout has no tiles)",
           "layout_tiles": lay.tiles, "layout_entries": lay.entries,
           "layout_order": "bfs levels" if lay.order == bh.ORDER_BFS else "morton", "layout_build_s": build_s}
    out.update(measure(lay if tiled else P))
    out["plain_csr"] = measure(P)
    counts = []
    run(P, steps, per_step=lambda it: counts.append(bh.get_stats(ws)["interactions"]))
    torch.cuda.synchronize()
    reset()
    inter = float(np.mean(counts))
    out["interactions_per_iteration"] = inter
    out["interactions_per_s_walk"] = inter / (out["phases_ms"]["repulsive"] * 1e-3)
    del P, ws, Y0, Y, u, g, lay
    torch.cuda.empty_cache()
    return out


def bench_affinities(args, cpu_rows=20000):
    """bhtsne_affinities on the workload's neighbour lists (k = 90, u = 30):
    the input similarities, computed once before the iterations.  Inputs are
    resident on the GPU when timing starts; each call synchronises twice (it
    returns nnz), so the time is host wall-clock per call."""
    import numpy as np
    import torch

    import paper_2212_11506_amd as bh
    import synth

    kn = synth.make_knn(args.workload, n=args.n)
    n, k, u = kn.n, kn.k, 30.0
    log(f"[bench] affinities: n={n} k={k}, lists drawn in {kn.gen_seconds:.1f}s")
    idx = torch.from_numpy(kn.idx).cuda()
    dist = torch.from_numpy(kn.dist).cuda()
    ws = torch.empty(bh.affinities_workspace_size(n, k), dtype=torch.uint8, device="cuda")
    P, _ = bh.affinities(idx, dist, u, workspace=ws)  # warm-up
    torch.cuda.synchronize()
    calls = 5
    t0 = time.perf_counter()
    for _ in range(calls):
        P, _ = bh.affinities(idx, dist, u, workspace=ws)
    torch.cuda.synchronize()
    ms = 1e3 * (time.perf_counter() - t0) / calls
    nnz = P.nnz
    out = {"workload": f"neighbour lists of workload {args.workload}: k = {k} per point within its cluster, "
                       f"d ~ U(0, 3) sorted per row; perplexity {u}",
           "n": n, "k": k, "perplexity": u, "nnz": nnz, "calls": calls, "ms_per_call": ms,
           "points_per_s": n / (ms * 1e-3),
           # bytes the step must move: the lists in (8 B per neighbour), P out
           # (8 B per entry + 8 B per row pointer)
           "algorithmic_gbs": (8.0 * n * k + 8.0 * nnz + 8.0 * (n + 1)) / (ms * 1e-3) / 1e9}
    del P, ws, idx, dist
    torch.cuda.empty_cache()
    if not args.no_cpu and cpu_rows > 0:
        from oracle import affinities as A

        rows = np.random.default_rng(5).choice(n, min(cpu_rows, n), replace=False)
        tc = time.perf_counter()
        A.conditional(kn.dist[rows], u)
        dt = time.perf_counter() - tc
        out["cpu_oracle"] = {"value": rows.size / dt, "unit": "points/s", "kind": "oracle",
                             "sample": f"sigma search and p_(j|i) of {rows.size} random rows (numpy fp64, "
                                       f"{dt:.1f}s); the symmetrisation is not in this figure"}
    return out


def bench_fp64(args, inp, steps=200, warmup=5):
    """The fp64 variant against the fp32 path on the same workload:
    iterations/s over the first `steps` iterations of the schedule, inputs
    resident, with the per-phase event times.  fp64: through its locality
    layout (the sliced copy over 8192-point windows, or windowed segments);
    fp64_plain and fp32: both on the plain CSR P, for the like-for-like
    precision ratio."""
    import numpy as np
    import torch

    import paper_2212_11506_amd as bh

    w = inp.workload
    n, nnz = inp.n, inp.nnz
    dev = torch.device("cuda:0")
    out = {"workload": f"{w.description} (workload {w.cid}), iterations 0..{steps - 1}",
           "steps": steps}
    for name, dt in (("fp64", torch.float64), ("fp64_plain", torch.float64), ("fp32", torch.float32)):
        if dt == torch.float64:
            P = bh.CsrF64.from_numpy(inp.row_ptr, inp.col, inp.val.astype(np.float64), device=dev)
            ws = torch.empty(bh.workspace_size_f64(n, nnz), dtype=torch.uint8, device=dev)
            if name == "fp64":
                P = bh.LayoutF64(P, torch.from_numpy(inp.Y).to(dev).double(), workspace=ws)
            fn = bh.step_f64
        else:
            P = bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val, device=dev)
            ws = torch.empty(bh.workspace_size(n, nnz), dtype=torch.uint8, device=dev)
            fn = bh.step
        Y0 = torch.from_numpy(inp.Y).to(dev).to(dt)
        Y = Y0.clone()
        u = torch.zeros_like(Y)
        g = torch.ones_like(Y)

        def run(k):
            for it in range(k):
                s = w.schedule(it)
                fn(Y, P, args.theta, s["exaggeration"], s["learning_rate"], s["momentum"], 0.01, u, g, workspace=ws)

        run(warmup)
        torch.cuda.synchronize()
        Y.copy_(Y0)
        u.zero_()
        g.fill_(1.0)
        bh.timing_phases(None)
        bh.timing_read(reset=True)
        bh.timing_enable(True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        run(steps)
        torch.cuda.synchronize()
        dt_s = time.perf_counter() - t0
        bh.timing_enable(False)
        ph = bh.timing_read(reset=True)
        out[name] = {"iterations_per_s": steps / dt_s, "ms_per_step": 1e3 * dt_s / steps,
                     "phases_ms": {k: v[0] / v[1] for k, v in ph.items() if v[1]},
                     "attractive_path": attractive_path(P) if name == "fp64" else "plain CSR"}
        if name == "fp64":
            out[name].update(layout_tiles=P.tiles, layout_entries=P.entries, layout_windows=P.windows)
        del P, ws, Y0, Y, u, g
        torch.cuda.empty_cache()
    out["fp64_over_fp32_time"] = out["fp64_plain"]["ms_per_step"] / out["fp32"]["ms_per_step"]
    return out


def main():
    args = parse()
    if args.no_overlap:
        os.environ["BHTSNE_OVERLAP"] = "0"  # read once by the library, at its first step
    if args.copy_calibrate:
        copy_calibrate()
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the multi-GPU path is a design note, "
              "not a built component (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2212_11506_amd as bh
    import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    bh.load_library()
    if args.affinities_only:
        print(json.dumps({"affinities": bench_affinities(args)}), flush=True)
        return
    if args.configs_only:
        print(json.dumps({"configs": bench_configs(args)}), flush=True)
        return
    if args.locality_only:
        print(json.dumps({"locality": bench_locality(args)}), flush=True)
        return
    if args.only_3d:
        print(json.dumps({"embedding_3d": bench_3d(args)}), flush=True)
        return
    w = synth.WORKLOADS[args.workload]
    t0 = time.time()
    inp = synth.make_inputs(args.workload, n=args.n, progress=log)
    log(f"[bench] inputs: n={inp.n} nnz={inp.nnz} generated in {time.time() - t0:.1f}s")
    if args.fp64_only:
        print(json.dumps({"fp64_variant": bench_fp64(args, inp)}), flush=True)
        return
    iter0 = 0
    if args.load_y:
        y = np.load(args.load_y)
        if y.shape != inp.Y.shape or y.dtype != np.float32:
            raise SystemExit(f"{args.load_y}: expected float32 {inp.Y.shape}, found {y.dtype} {y.shape}")
        inp.Y = y
        iter0 = args.iter0
        log(f"[bench] starting from {args.load_y} at schedule iteration {iter0}")

    def sched(it):
        return w.schedule(it + iter0)

    n, nnz = inp.n, inp.nnz
    dev = torch.device("cuda:0")
    Y0 = torch.from_numpy(inp.Y).to(dev)
    P = bh.Csr.from_numpy(inp.row_ptr, inp.col, inp.val, device=dev)
    Pcsr = P  # kept for the KL evaluation
    ws = torch.empty(bh.workspace_size(n, nnz), dtype=torch.uint8, device=dev)
    layout_s = None
    if not args.plain:
        # one-time renumbering of the points for locality of P's columns (outside the timed loop)
        torch.cuda.synchronize()
        tl = time.perf_counter()
        Pl = bh.Layout(P, Y0, workspace=ws)
        torch.cuda.synchronize()
        layout_s = time.perf_counter() - tl
        log(f"[bench] layout built in {layout_s:.3f}s, {Pl.tiles} column tiles")
        P = Pl
    Y = Y0.clone()
    u = torch.zeros_like(Y)
    gains = torch.ones_like(Y)

    def reset():
        Y.copy_(Y0)
        u.zero_()
        gains.fill_(1.0)

    def run(k, per_step=None):
        for it in range(k):
            s = sched(it)
            bh.step(Y, P, args.theta, s["exaggeration"], s["learning_rate"], s["momentum"], 0.01, u,
                    gains, workspace=ws)
            if per_step:
                per_step(it)

    if args.save_y:
        run(args.save_after)
        np.save(args.save_y, Y.cpu().numpy())
        print(json.dumps({"saved_y": args.save_y, "iterations": args.save_after}), flush=True)
        return

    # warm-up (code-object loading, caches), then back to the initial state
    run(args.warmup)
    torch.cuda.synchronize()
    reset()
    torch.cuda.synchronize()

    # the timed run records hipEvents around the two force phases only (the
    # roofline's kernels): each event is a timestamp packet of a few
    # microseconds between kernels, and all six phases cost 3.5% of a step
    bh.timing_read(reset=True)
    bh.timing_phases(["repulsive", "attractive"])
    bh.timing_enable(True)
    # stream events at the schedule's switch (exaggeration off, momentum 0.8 from
    # iteration 250): the two stretches' means, without a sync in the loop
    split = 250 if args.steps > 250 else None
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    torch.cuda.synchronize()
    ev[0].record()
    t1 = time.perf_counter()
    run(args.steps, per_step=(lambda it: ev[1].record() if it == split - 1 else None) if split else None)
    ev[2].record()
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    segments = None
    if split:
        a, b = ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2])
        segments = {f"0..{split - 1}": split / (a * 1e-3), f"{split}..{args.steps - 1}": (args.steps - split) / (b * 1e-3)}
    bh.timing_enable(False)
    bh.timing_phases(None)
    phases = bh.timing_read(reset=True)
    elapsed = t2 - t1
    its = args.steps / elapsed
    log(f"[bench] {args.steps} steps in {elapsed:.3f}s -> {its:.1f} it/s")
    stats_last = bh.get_stats(ws)
    y_final = Y.cpu().numpy()

    # the run's cost: KL of the first and last embedding with the exact Z (all
    # n^2 pairs), the exact-Z kernel timed on the stream
    Pc = Pcsr
    kl_initial = bh.kl(Y0, Pc, bh.z_exact(Y0, workspace=ws), workspace=ws)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    z_final = bh.z_exact(Y, workspace=ws)
    e1.record()
    torch.cuda.synchronize()
    z_ms = e0.elapsed_time(e1)
    cost = {"kl_initial": kl_initial, "kl_final": bh.kl(Y, Pc, z_final, workspace=ws), "z_exact_final": z_final,
            "z_exact_ms": z_ms, "z_pair_terms_per_s": float(n) * n / (z_ms * 1e-3)}
    log(f"[bench] KL {cost['kl_initial']:.5f} -> {cost['kl_final']:.5f}, exact Z in {z_ms:.1f} ms")

    # the other phases: a replay of the first iterations with every phase timed
    reset()
    bh.timing_enable(True)
    breakdown_steps = min(args.steps, 200)
    run(breakdown_steps)
    torch.cuda.synchronize()
    bh.timing_enable(False)
    breakdown = bh.timing_read(reset=True)

    inter_total = None
    if not args.no_count:
        # deterministic kernels: replaying the same trajectory gives the same trees,
        # so the per-step interaction counts belong to the timed run
        reset()
        counts = []
        run(args.steps, per_step=lambda it: counts.append(bh.get_stats(ws)["interactions"]))
        torch.cuda.synchronize()
        same = np.array_equal(Y.cpu().numpy(), y_final)
        log(f"[bench] replay identical to timed run: {same}")
        inter_total = int(sum(counts)) if same else None

    # per phase: time per launch from the library's hipEvent pairs; with a
    # layout the attractive phase runs on a second stream beside the sort, tree
    # and repulsive phases, so phase times add up to more than a step
    kernels = {}
    for name, (ms, cnt) in phases.items():
        if cnt == 0:
            ms, cnt = breakdown[name]
            if cnt == 0:
                continue
            kernels[name] = {"ms_per_launch": ms / cnt, "launches": cnt,
                             "timed": f"replay of iterations 0..{breakdown_steps - 1}, every phase timed"}
            continue
        kernels[name] = {"ms_per_launch": ms / cnt, "launches": cnt, "timed": "timed run"}
    rep_ms = kernels["repulsive"]["ms_per_launch"]
    att_ms = kernels["attractive"]["ms_per_launch"]
    # sources whose change invalidates the committed traffic counters
    rep_src = ("k_forces.hip", "k_tree.hip", "common.hpp")
    att_src = ("k_layout.hip", "common.hpp") if not args.plain else ("k_forces.hip", "common.hpp")
    rep = kernels["repulsive"]
    rep_traffic = measured_traffic("repulsive_kernel", rep_src)
    if inter_total is not None:
        per_launch = inter_total / args.steps
        rep["interactions_per_s"] = per_launch / (rep_ms * 1e-3)
        rep["tflops"] = FLOPS_PER_INTERACTION * rep["interactions_per_s"] / 1e12
        rep["frac_alu"] = rep["tflops"] / ALU_PEAK_TFLOPS
        rep["frac_alu_nonpacked"] = rep["tflops"] / ALU_PEAK_NONPACKED_TFLOPS
        # the per-interaction byte model (16 B per summary or point + 20 B per
        # point) counts cache hits: the node records stay in the caches, so it
        # exceeds what HBM can move and is no measure of HBM use
        rep["model16_gbs"] = (16.0 * per_launch + 20.0 * n) / (rep_ms * 1e-3) / 1e9
    if rep_traffic:
        # what the walk really moves through HBM (committed FETCH + WRITE counters)
        rep["measured_gbs"] = rep_traffic / (rep_ms * 1e-3) / 1e9
        rep["measured_frac_hbm"] = rep["measured_gbs"] / HBM_PEAK_GBS
    # attraction: 8 B per stored entry (column, value) and 32 B per point (row
    # pointers, y_i, output); with the plain CSR path the phase also holds the
    # gradient assembly and update, 72 B per point, which the layout path times
    # as its own phase
    att_bytes = 8.0 * nnz + (104.0 if args.plain else 32.0) * n
    att = kernels["attractive"]
    att["model_gbs"] = att_bytes / (att_ms * 1e-3) / 1e9
    att["model_frac_hbm"] = att["model_gbs"] / HBM_PEAK_GBS
    att_kernels = ("attract_sell_kernel", "attract_rows_kernel") if not args.plain else ("attract_kernel",)
    att_traffic = [measured_traffic(k, att_src) for k in att_kernels]
    att["traffic"] = sum(att_traffic) if all(t is not None for t in att_traffic) else None
    if att["traffic"]:
        # measured HBM bytes of the phase's kernels over the phase's time
        att["measured_gbs"] = att["traffic"] / (att_ms * 1e-3) / 1e9
        att["measured_frac_hbm"] = att["measured_gbs"] / HBM_PEAK_GBS
    if kernels.get("update", {}).get("launches"):
        upd = kernels["update"]
        # reads F_attr, F_rep, Y, update and gains (8 B each), writes the last
        # three; the windowed segments leave F_attr in layout order and add the
        # 4-byte rank read
        upd_bytes = (68.0 if not args.plain and attractive_path(P) == "windowed segments" else 64.0) * n
        upd["gbs"] = upd_bytes / (upd["ms_per_launch"] * 1e-3) / 1e9
        upd["frac_hbm"] = upd["gbs"] / HBM_PEAK_GBS
        upd["traffic"] = measured_traffic("update_kernel", att_src)
    dominant = max(("repulsive", "attractive"), key=lambda k: kernels[k]["ms_per_launch"])
    if dominant == "repulsive" and inter_total is not None:
        roof = {"kernel": "repulsive", "bound": "alu", "achieved": rep["tflops"], "peak": ALU_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": rep["frac_alu"], "traffic": rep_traffic,
                "peak_nonpacked": ALU_PEAK_NONPACKED_TFLOPS, "frac_nonpacked": rep["frac_alu_nonpacked"],
                "measured_frac_hbm": rep.get("measured_frac_hbm"),
                "model": f"{FLOPS_PER_INTERACTION} fp32 flops per interaction (summary or exact pair); peak: the "
                         "published fp32 vector rate (packed); peak_nonpacked: 256 CUs x 64 lanes x 2 x 2.4 GHz, "
                         "the rate without packed fp32, which this build disables"}
    else:
        achieved = att.get("measured_gbs") or att["model_gbs"]
        roof = {"kernel": "attractive", "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS, "traffic": att["traffic"],
                "model": ("measured FETCH_SIZE + WRITE_SIZE bytes" if att.get("measured_gbs") else
                          "8 B per stored entry + %d B per point" % (104 if args.plain else 32))}

    cpu = None
    if not args.no_cpu and args.cpu_iters > 0:
        o = oracle_sample(inp, args.theta, args.cpu_iters, w.schedule)
        log(f"[bench] oracle: {o['iterations_per_s']:.3f} it/s on {o['cores']} threads ({o['seconds']:.1f}s)")
        cpu = {"value": o["iterations_per_s"], "unit": "iterations/s", "cores": o["cores"], "kind": "oracle",
               "sample": f"first {args.cpu_iters} iterations of the same workload and schedule, "
                         f"fp64 oracle, {o['seconds']:.1f}s",
               "interactions_per_s": o["interactions_per_s"], "step_ms": o["step_ms"]}
    layout_tiles = None if args.plain else P.tiles
    layout_entries = None if args.plain else P.entries
    path = "plain CSR" if args.plain else attractive_path(P)
    del P, Pcsr, ws, Y0, Y, u, gains
    torch.cuda.empty_cache()

    out = {
        "metric": METRIC,
        "value": its,
        "unit": "iterations/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * elapsed / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{w.description} (workload {w.cid})", "n": n, "nnz": nnz,
                   "theta": args.theta, "iterations": f"0..{args.steps - 1} of the schedule"},
        "iterations_per_s_by_stretch": segments,
        "cost": cost,
        "interactions_per_s": (inter_total / elapsed) if inter_total is not None else None,
        "interactions_per_iteration": (inter_total / args.steps) if inter_total is not None else None,
        "nodes_last": stats_last["nodes"],
        "attractive_path": path,
        "layout_build_s": layout_s,
        "layout_tiles": layout_tiles,
        "layout_entries": layout_entries,
        "kernels": kernels,
        "roofline": roof,
        "cpu_baseline": cpu,
        "affinities": None if args.no_affinities else bench_affinities(args),
        "fp64_variant": None if args.no_fp64 else bench_fp64(args, inp),
        "embedding_3d": None if (args.no_3d or args.workload != 2 or args.n) else bench_3d(args),
        "configs": None if (args.no_configs or args.workload != 2 or args.n) else bench_configs(args),
        "locality": None if (args.no_locality or args.workload != 2 or args.n) else bench_locality(args),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
