#!/usr/bin/env python3
"""Throughput of the fused slice -> token mix -> deslice path, forward + backward, on one MI355X.

One step = fs_slice_fwd, fs_mix, fs_deslice_fwd and fs_slice_deslice_bwd (which includes the
mix backward) over one batch of seeded synthetic inputs already resident in device memory.
The default workload is the large-mesh volume layer (bf16 storage with fp32 accumulation,
B=1, N=2^20 points, H=8 heads, dh=32, G=64 slices, fixed G x G token matrix). Prints ONE JSON line. A forward-only
workload (``--workload infer``: bf16, N = 2^24) times fs_slice_fwd, fs_mix and fs_deslice_fwd
with no saved normaliser instead.

Besides the step time it reports, for the dominant kernel (backward pass B), the roofline
point from algorithmic bytes or MFMA flops per launch over its average duration measured with
HIP events recorded around its launch on the stream it runs on, and the fp64 oracle timed on
the host cores as a CPU baseline. ``valu`` sets the vector ALU, which binds before the matrix
cores at large G, beside them: the VALU issue time and the MFMA busy time one step needs, from
the committed rocprofv3 SQ-counter record of the workload (``profiles/issue_<workload>.json``,
used only while the kernel sources match it), over the measured step time.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("points/sec fused slice+deslice fwd+bwd; % HBM BW (small G) / % MFMA (large G)")
METRIC_FWD = "points/sec fused slice+deslice forward (inference, no saved normaliser)"
HBM_PEAK = 8.0e12
MFMA_PEAK = {"f32": 157.3e12, "bf16": 2.5e15}
PASS_NAMES = ("slice", "deslice", "bwd_a", "bwd_b")
KERNEL_NAMES = {"slice": "k_slice", "deslice": "k_deslice", "bwd_a": "k_bwd_a", "bwd_b": "k_bwd_b"}
MIX_NAMES = {0: "identity", 1: "fixed GxG matrix", 2: "per-token channel map",
             3: "single-head GxG self-attention"}


def pass_work(w, pass_name):
    """Algorithmic HBM bytes and MFMA flops of one streaming pass per (point, head).

    bytes: the pass's point-tensor reads and writes in the storage dtype plus the 4-byte lse
    (none in the forward-only path, which neither writes nor reads it);
    flops: its dense contractions (logits 2DG, each token contraction 2GV or 2DG).
    """
    elt = 2 if w.dtype == "bf16" else 4
    D, V, G = w.D, w.V, w.G
    lse = 0 if w.forward_only else 4
    if pass_name == "slice":      # read x, fx; write lse; logits + U
        return (D + V) * elt + lse, 2 * D * G + 2 * G * V
    if pass_name == "deslice":    # read x, lse; write out; logits + w zmix
        return (D + V) * elt + lse, 2 * D * G + 2 * G * V
    if pass_name == "bwd_a":      # read x, dout, lse; logits + w^T dout
        return (D + V) * elt + 4, 2 * D * G + 2 * G * V
    # bwd_b: read x, fx, dout, lse; write dx, dfx; logits, dw (2 GV), dfx, dx, dW_s
    return (2 * D + 3 * V) * elt + 4, 6 * D * G + 6 * G * V


def measured_traffic(workload, kernel):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it was taken on
    the current kernel sources; otherwise None."""
    path = os.path.join(ROOT, "profiles", f"pmc_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        d = json.load(fh)
    from paper_2609_32525_amd.profiling import kernel_source_hash
    if d.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return d.get("traffic_bytes_per_launch")


def measured_issue(workload):
    """The vector-ALU and matrix-core time per step from the committed rocprofv3 issue record
    (SQ instruction counters), if it was taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", f"issue_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        d = json.load(fh)
    from paper_2609_32525_amd.profiling import kernel_source_hash
    if d.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return d


# State the forked oracle workers read (set before the pool starts, shared copy-on-write).
_ORACLE_JOB = {}


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def _mem_available():
    """Bytes of host memory available to this run (MemAvailable, at most 256 GiB)."""
    try:
        with open("/proc/meminfo") as fh:
            for line in fh:
                if line.startswith("MemAvailable:"):
                    return min(int(line.split()[1]) * 1024, 256 << 30)
    except OSError:
        pass
    return 16 << 30


def _oracle_pair(pair):
    """One (sample, head) pair of the unchanged oracle, forward (+ backward); returns its
    wall time. Runs in a forked worker with its BLAS pool capped to its share of the cores."""
    from threadpoolctl import threadpool_limits
    import oracle
    job = _ORACLE_JOB
    w, inp, args = job["w"], job["inp"], job["args"]
    pairs = [pair]
    with threadpool_limits(job["blas"]):
        t0 = time.perf_counter()
        if w.variant == "untied":
            f = oracle.untied_forward(*args, eps=w.eps, pairs=pairs)
            oracle.untied_backward(*args, inp["dout"], eps=w.eps, fwd=f, pairs=pairs)
        elif w.variant == "linearno":
            f = oracle.linearno_forward(*args, pairs=pairs)
            oracle.linearno_backward(*args, inp["dout"], fwd=f, pairs=pairs)
        else:
            oracle.run_inputs(inp, w.mix, w.eps, backward_too=not w.forward_only, pairs=pairs)
        return time.perf_counter() - t0


def cpu_baseline(w, inp, budget_s=12.0, max_cores=16):
    """The fp64 oracle (unchanged) on the same workload, timed on the host cores: its (sample,
    head) pairs are independent, so a pool of forked workers runs them side by side, one pair
    per worker at a time, each worker's BLAS pool taking its share of the cores. The pool
    covers the cores this process may run on (os.sched_getaffinity), at most ``max_cores``
    (the host share of one GPU). Whole passes over all pairs repeat until ``budget_s`` of wall
    time has passed. Runs before the GPU is initialised (the workers are forked). A workload
    built from a repeated block is sampled on one block (its points per second)."""
    import multiprocessing as mp
    try:
        libc = ctypes.CDLL("libc.so.6")
        libc.mallopt(-4, 0)
        libc.mallopt(-1, 2 ** 31 - 1)
    except OSError:
        pass
    import workloads
    visible = len(os.sched_getaffinity(0))
    cores = max(1, min(visible, max_cores))
    pairs = [(b, h) for b in range(w.B) for h in range(w.H)]
    # each worker touches every page of its own full-size fp64 point outputs (a pair's
    # (N, V) slice is strided across them) and holds a few N x G fp64 temporaries: run no
    # more workers than half the available host memory holds
    n = w.block_N or w.N
    per_worker = 8 * w.B * n * w.H * (w.D + 2 * w.V) + 8 * 12 * n * (w.G + max(w.D, w.V))
    nproc = max(1, min(cores, len(pairs), int(0.5 * _mem_available() // per_worker)))
    blas = max(1, cores // nproc)
    args = None
    if w.variant != "tied":
        ut = workloads.untied_params(w)
        prm = {k: inp.get(k) for k in ("A", "Wc", "Wq", "Wk", "Wv", "scale")}
        args = (inp["x"], inp["fx"], inp["Ws"], inp["b"], inp["tau"], ut["Wd"], ut["bd"],
                ut["taud"], w.mix, prm)
    _ORACLE_JOB.update(w=w, inp=inp, args=args, blas=blas)
    runs, t_total, t_said = 0, 0.0, 0.0
    ctx = mp.get_context("fork")
    with ctx.Pool(nproc) as pool:
        while runs == 0 or (t_total < budget_s and runs < 500):
            t0 = time.perf_counter()
            pool.map(_oracle_pair, pairs, chunksize=1)
            t_total += time.perf_counter() - t0
            runs += 1
            if t_total - t_said > 5.0 or runs == 1:
                print(f"[bench] oracle: {runs} pass(es), {t_total:.1f} s", file=sys.stderr,
                      flush=True)
                t_said = t_total
    _ORACLE_JOB.clear()
    n = w.block_N or w.N
    pts = w.B * n * runs
    what = "whole workload" if not w.block_N else "one seeded block"
    return {"value": pts / t_total, "unit": "points/s", "cores": nproc * blas, "kind": "oracle",
            "sample": f"{what} (B={w.B}, N={n}, all {w.H} heads), "
                      f"{'forward' if w.forward_only else 'forward + backward'} in fp64, "
                      f"{runs} pass(es) over the {len(pairs)} (sample, head) pairs in "
                      f"{t_total:.1f} s; {nproc} worker processes x {blas} BLAS thread(s)",
            "cores_visible": visible, "cpu": _cpu_model()}


def stack_flops_per_point(spec):
    """fp32 flops of one training step per point: per layer three C x C projections and the
    C -> 4C -> C MLP (2 * 11 C^2 forward, twice that backward), plus the path's contractions
    12 G (D + V) per head."""
    C, H, G, L = spec["C"], spec["H"], spec["G"], spec["L"]
    D = C // H
    return L * (66 * C * C + H * 12 * G * 2 * D)


def stack_cpu_baseline(name, spec, budget_s=12.0, max_cores=16):
    """The CPU reference of the stack (float64 torch layers around the oracle's path, unchanged)
    timed on a sample of the workload's points: one sample of 4096 points, training steps
    repeated until ``budget_s``; points per second. Runs before the GPU is initialised."""
    import torch
    import workloads
    from oracle.stack import reference_step
    cores = max(1, min(len(os.sched_getaffinity(0)), max_cores))
    torch.set_num_threads(cores)
    n = 4096
    h, R = workloads.make_stack_inputs(name, B=1, N=n)
    torch.manual_seed(workloads.SEED)
    from paper_2609_32525_amd.layer import SliceStack
    state = SliceStack(spec["L"], spec["C"], spec["H"], spec["G"]).state_dict()
    runs, t_total = 0, 0.0
    while runs == 0 or t_total < budget_s:
        t0 = time.perf_counter()
        reference_step(state, spec["L"], spec["C"], spec["H"], spec["G"], h, R)
        t_total += time.perf_counter() - t0
        runs += 1
    return {"value": n * runs / t_total, "unit": "points/s", "cores": cores, "kind": "oracle",
            "sample": f"one sample of {n} points (B=1), {runs} training step(s) of the float64 "
                      f"reference stack (oracle path) in {t_total:.1f} s; {cores} threads",
            "cores_visible": len(os.sched_getaffinity(0)), "cpu": _cpu_model()}


def bench_stack(args):
    """The full slicing stack: one training step (forward, loss sum(out * R), backward, plain
    SGD update) over a batch resident in device memory."""
    import numpy as np
    import workloads
    spec = workloads.STACKS[args.workload]
    cpu = None if args.no_cpu_baseline else stack_cpu_baseline(args.workload, spec)
    h_np, R_np = workloads.make_stack_inputs(args.workload)
    import torch
    from paper_2609_32525_amd.layer import SliceStack, training_step
    dev = torch.device("cuda:0")
    torch.manual_seed(workloads.SEED)
    model = SliceStack(spec["L"], spec["C"], spec["H"], spec["G"]).to(dev)
    h = torch.from_numpy(h_np).to(dev)
    R = torch.from_numpy(R_np).to(dev)
    del h_np, R_np
    lr = 1e-6
    for _ in range(args.warmup):
        training_step(model, h, R, lr)
    torch.cuda.synchronize(dev)
    stream = torch.cuda.current_stream(dev)
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize(dev)
    wall0 = time.perf_counter()
    t0.record(stream)
    for _ in range(args.steps):
        training_step(model, h, R, lr)
    t1.record(stream)
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - wall0
    ms_step = t0.elapsed_time(t1) / args.steps
    # the path's share: events around every path call (forward and backward) of a few more
    # steps, against those steps' own time
    nshare = max(1, min(args.steps, 5))
    model.space.events = []
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(nshare):
        training_step(model, h, R, lr)
    b.record(stream)
    torch.cuda.synchronize(dev)
    path_ms = sum(x.elapsed_time(y) for x, y in model.space.events) / nshare
    share_ms = a.elapsed_time(b) / nshare
    model.space.events = None
    points = spec["B"] * spec["N"]
    flops = stack_flops_per_point(spec) * points
    t_step = ms_step * 1e-3
    out = {
        "metric": "points/sec of one training step of the 8-layer slicing stack "
                  "(forward + backward + SGD update)",
        "value": points / t_step, "unit": "points/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": args.workload, "L": spec["L"], "B": spec["B"], "N": spec["N"],
                   "C": spec["C"], "H": spec["H"], "dh": spec["C"] // spec["H"], "G": spec["G"],
                   "mix": MIX_NAMES[1], "storage": "f32"},
        "roofline": {"bound": "mfma", "achieved": flops / t_step / 1e12,
                     "peak": MFMA_PEAK["f32"] / 1e12, "unit": "TFLOP/s",
                     "frac": flops / t_step / MFMA_PEAK["f32"], "traffic": None,
                     "kernel": "whole step (fp32 GEMMs of the projections and MLPs dominate)",
                     "per_launch": {"units": points, "algorithmic_flops": flops,
                                    "avg_duration_us": ms_step * 1e3}},
        "path": {"ms_per_step": path_ms, "share": path_ms / share_ms,
                 "calls_per_step": 2 * spec["L"]},
        "wall_s_timed": wall,
    }
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)


def copy_bandwidth(torch, mib=1024, reps=5):
    """HBM bytes per second of a plain device-to-device copy (read + write) of ``mib`` MiB,
    measured before the timed region: the streaming rate this GPU reaches in practice, as
    context for the roofline fraction (which is taken against the 8 TB/s peak)."""
    src = torch.empty(mib << 18, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    sec = a.elapsed_time(b) * 1e-3 / reps
    del src, dst
    return 2 * (mib << 20) / sec / 1e9


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="volume")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="replay each step as one captured HIP graph")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="first copy this many MiB device to device three times (a known "
                         "amount of traffic for calibrating rocprofv3 byte counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (sharding the points "
              "would add one all-reduce of the token partials per pass); run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import workloads

    if args.workload in workloads.STACKS:
        bench_stack(args)
        return
    w = workloads.WORKLOADS[args.workload]
    fwd_only = w.forward_only
    inp = workloads.make_inputs(w, with_grad=not fwd_only)
    # the oracle's CPU baseline runs first, in forked workers, before anything touches the GPU
    cpu = None if args.no_cpu_baseline else cpu_baseline(w, inp)

    import torch
    import paper_2609_32525_amd as fs
    from paper_2609_32525_amd.runner import PathBuffers

    if args.copy_calibration_mib > 0:
        src = torch.ones(args.copy_calibration_mib << 18, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # (skipped in counter runs, whose only large copy must be the calibration one)
    copy_gbps = copy_bandwidth(torch) if args.copy_calibration_mib == 0 else None

    pb = PathBuffers(inp, w.mix, w.dtype, w.eps, with_backward=not fwd_only, repeat=w.repeat,
                     keep_lse=not fwd_only,
                     untied=workloads.untied_params(w) if w.variant != "tied" else None,
                     linearno=w.variant == "linearno")
    del inp
    dev = pb.dev
    stream = torch.cuda.current_stream(dev)

    graph = None
    if args.graph:
        s = torch.cuda.Stream(dev)
        s.wait_stream(stream)
        with torch.cuda.stream(s):
            for _ in range(3):
                pb.step()
        stream.wait_stream(s)
        torch.cuda.synchronize(dev)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            pb.step()
        torch.cuda.synchronize(dev)

    def step():
        if graph is not None:
            graph.replay()
        else:
            pb.step()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize(dev)

    # timed region: exactly K steps, synchronised on both sides
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize(dev)
    wall0 = time.perf_counter()
    t0.record(stream)
    for _ in range(args.steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - wall0
    ms_step = t0.elapsed_time(t1) / args.steps

    # per-kernel durations: events recorded around each streaming kernel's launch, on its
    # stream, over the same number of eager steps
    npass = 2 if fwd_only else 4
    ev = {p: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)] for p in range(npass)}
    for p in range(npass):  # torch creates the underlying hipEvent_t on first record
        for a, b in ev[p]:
            a.record(stream)
            b.record(stream)
    torch.cuda.synchronize(dev)
    for k in range(args.steps):
        for p in range(npass):
            fs.set_pass_events(p, ev[p][k][0], ev[p][k][1])
        pb.step()
    fs.set_pass_events(-1)
    torch.cuda.synchronize(dev)
    pass_us = {PASS_NAMES[p]: 1e3 * float(np.mean([a.elapsed_time(b) for a, b in ev[p]]))
               for p in range(npass)}

    units = w.B * w.N * w.H   # (point, head) pairs per launch
    dom = max(pass_us, key=pass_us.get)
    byt, flp = pass_work(w, dom)
    t_dom = pass_us[dom] * 1e-6
    t_hbm = byt * units / HBM_PEAK
    t_mfma = flp * units / MFMA_PEAK[w.dtype]
    if t_hbm >= t_mfma:
        roof = {"bound": "hbm", "achieved": byt * units / t_dom / 1e9, "peak": HBM_PEAK / 1e9,
                "unit": "GB/s"}
    else:
        roof = {"bound": "mfma", "achieved": flp * units / t_dom / 1e12,
                "peak": MFMA_PEAK[w.dtype] / 1e12, "unit": "TFLOP/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["hbm_copy_gbps"] = copy_gbps  # measured device copy, context for the HBM peak
    roof["traffic"] = measured_traffic(args.workload, KERNEL_NAMES[dom])
    roof["kernel"] = KERNEL_NAMES[dom]
    roof["per_launch"] = {"units": units, "algorithmic_bytes": byt * units,
                          "algorithmic_flops": flp * units, "avg_duration_us": pass_us[dom]}

    # whole step against the path's own ceilings (4 passes; 2 in the forward-only path)
    elt = 2 if w.dtype == "bf16" else 4
    if fwd_only:
        step_bytes = (2 * w.D + 2 * w.V) * elt * units
        step_flops = 4 * w.G * (w.D + w.V) * units
    else:
        step_bytes = ((5 * w.D + 6 * w.V) * elt + 12) * units
        step_flops = 12 * w.G * (w.D + w.V) * units
    t_step = ms_step * 1e-3
    step_roof = {"hbm_frac": step_bytes / t_step / HBM_PEAK,
                 "mfma_frac": step_flops / t_step / MFMA_PEAK[w.dtype],
                 "t_hbm_us": step_bytes / HBM_PEAK * 1e6,
                 "t_mfma_us": step_flops / MFMA_PEAK[w.dtype] * 1e6}

    # the vector ALU beside the matrix cores (it binds first at large G): the VALU issue time
    # and the MFMA busy time one step needs, from the counters, over the measured step time
    iss = measured_issue(args.workload)
    valu = None
    if iss is not None:
        valu = {"frac": iss["t_valu_us_per_step"] * 1e-6 / t_step,
                "mfma_busy_frac": iss["t_mfma_us_per_step"] * 1e-6 / t_step,
                "t_valu_us": iss["t_valu_us_per_step"],
                "t_mfma_busy_us": iss["t_mfma_us_per_step"],
                "source": f"profiles/issue_{args.workload}.json"}

    value = w.B * w.N / t_step
    out = {
        "metric": METRIC_FWD if fwd_only else METRIC, "value": value, "unit": "points/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "N": w.N, "H": w.H, "dh": w.D, "G": w.G,
                   "mix": MIX_NAMES[w.mix], "storage": w.dtype, "graph": bool(args.graph)},
        "roofline": roof,
        "step_roofline": step_roof,
        "valu": valu,
        "passes_us": pass_us,
        "wall_s_timed": wall,
    }
    if fwd_only:
        out["config"]["forward_only"] = True
    if w.variant != "tied":
        out["config"]["variant"] = w.variant
    if w.block_N:
        out["config"]["points"] = f"{w.repeat} copies of one seeded {w.block_N}-point block"
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
