"""Benchmark of the TopoEP planner on one MI355X.

A step plans every MoE layer of one microbatch: for each layer the plan's
kernels (one launch when the single-workgroup solver fits, else histogram,
solver and reroute) run on one stream, all layers captured in one HIP graph
(the layers are planned one after another, as they would be in a forward
pass).  Inputs (the synthetic routing matrix and this rank's top-k ids of
every layer) are resident in HBM before the timed region.  A workload of
fewer than 32 layers is captured several times over in the graph
(passes_per_replay), so that the host's cost of submitting a replay does
not stand in for the plan's latency; times are per pass.

Printed JSON line: value = rerouted assignments per second over the whole
step; plan_latency_us_per_layer = step time / layers.  ``roofline`` covers
the kernel with the longest average duration, timed with HIP events on the
stream it runs on; ``launch_floor_us_per_layer`` is the same graph of empty
kernels with the plan's grid, threads and LDS; ``cpu_baseline`` times the
CPU oracle on a bounded sample of the same workload on this host (one
thread, then every core, then the host-planning path of Eq. 1: copy the
inputs to the host, plan there, copy the outputs back).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--config dsv3]
       python bench.py --sweep    (histogram/reroute/layout bandwidth sweep; with
                                   --pmc-pass it ends with the counter calibration copy)
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workload  # noqa: E402

HBM_PEAK_GBS = 8000.0
METRIC = "plan latency (us) per MoE layer at EP32/256e/top-8; rerouted assignments/s"
DESCR = {
    "tiny": "Tiny: 2 nodes x 4 GPUs (R=8), E=16, top-2, T=512, 1 slot, 1 layer",
    "mixtral": "Mixtral-like: 1 node x 8 GPUs (R=8), E=8, top-2, T=4096, 1 slot, 32 layers",
    "qwen3": "Qwen3-MoE-like: 4 nodes x 8 GPUs (R=32), E=128, top-8, T=4096, 2 slots, 48 layers",
    "dsv3": "DeepSeek-V3-like: 4 nodes x 8 GPUs (R=32), E=256, top-8, T=8192, 2 slots, 58 layers",
    "stress": "Stress: 32 nodes x 8 GPUs (R=256), E=512, top-8, T=16384, 4 slots, 16 layers",
}


def _gen(args):
    name, layer, mb = args
    cfg = workload.get(name)
    return workload.make_layer(cfg, layer, mb, 0)


def make_inputs(cfg, layers, mb=0, workers=None):
    jobs = [(cfg.name, l, mb) for l in range(layers)]
    workers = workers or min(16, os.cpu_count() or 1, layers)
    if workers > 1 and layers > 1:
        import multiprocessing as mp
        with mp.get_context("fork").Pool(workers) as pool:
            return pool.map(_gen, jobs)
    return [_gen(j) for j in jobs]


STAGE_NAMES = {1: ("plan",), 3: ("hist", "solve", "reroute")}


def algorithmic_bytes(cfg, N, kernels):
    """Bytes the method must move per layer (the plan's algorithmic traffic),
    by kernel: 4 per assignment to count the ids, 8 per assignment to read
    them again and write the destinations, Omega (4 R E) and the outputs
    (4 R (N + 1): replica slots and send counts); in all 12 B per assignment
    + 4 R E + 4 R (N + 1).  One launch does all of it.  The kernels' own
    count (``kernel_bytes``) differs: the one-launch kernel keeps the ids in
    registers and reads them once, and every plan writes two status words."""
    a = cfg.T * cfg.k
    omega = 4 * cfg.R * cfg.E
    outs = 4 * cfg.R * (N + 1)
    if kernels == 1:
        return {"plan": 12 * a + omega + outs}
    return {"hist": 4 * a, "solve": omega + outs, "reroute": 8 * a}


def kernel_bytes(cfg, N, kernels):
    """Bytes each kernel itself must read and write (its own count)."""
    a = cfg.T * cfg.k
    omega = 4 * cfg.R * cfg.E
    outs = 4 * cfg.R * (N + 1) + 8
    if kernels == 1:
        return {"plan": 8 * a + omega + outs}
    return {"hist": 4 * a, "solve": omega + outs, "reroute": 8 * a}


KERNEL_SRCS = [os.path.join(ROOT, "paper_2609_35481_amd", "csrc", n) for n in ("topoep.hip", "wave.h")]


def source_digest() -> str:
    """Digest of the plan kernels' code: their source and the wave helpers
    they include, with // comments and blank lines left out (a comment edit
    keeps the committed counters valid, a code edit does not)."""
    import hashlib
    h = hashlib.sha1()
    for path in KERNEL_SRCS:
        with open(path, encoding="utf-8") as f:
            for line in f:
                code = line.split("//", 1)[0].rstrip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()[:12]


def measured_traffic(workload_name, kernel):
    """HBM bytes per launch of a kernel from the committed counter summary
    (profiles/traffic_<workload>.txt), or None when there is none or the
    kernels changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "traffic_%s.txt" % workload_name)
    if not os.path.exists(path):
        return None
    digest, val = None, None
    with open(path) as f:
        for line in f:
            parts = line.split()
            if len(parts) >= 2 and parts[0] == "kernel_source_sha1:":
                digest = parts[1]
            if len(parts) >= 2 and parts[0] == "%s_kernel_bytes_per_launch:" % kernel:
                val = float(parts[1])
    if digest != source_digest() or val is None:
        return None
    return val


def launch_from_args(args):
    """The launch shape the options ask for (None = the library's choice)."""
    if args.solver or args.ipt or args.block_threads or args.tiles_per_block or args.solve_threads:
        return (args.ipt, args.block_threads, args.tiles_per_block, args.solve_threads, args.solver)
    return None


def run_pmc_pass(args):
    """Workload for counter runs: one plan of every layer, then each kernel
    of the plan alone over every layer (--stage-reps times), then a plain
    device-to-device copy of 256 MiB (the counter calibration)."""
    import torch
    from paper_2609_35481_amd import topoep

    cfg = workload.get(args.config)
    layers = cfg.layers if args.layers <= 0 else args.layers
    dev = torch.device("cuda:0")
    inputs = make_inputs(cfg, layers)
    topo = topoep.topology(cfg.R, cfg.G, cfg.E, 0, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W)
    dev_inputs = [(torch.from_numpy(gl.copy()).to(dev), torch.from_numpy(tk.copy()).to(dev))
                  for gl, tk in inputs]
    launch = launch_from_args(args)
    planners = [topoep.Planner(topo, cfg.T, cfg.k, cfg.N, device=dev, launch=launch) for _ in range(layers)]
    for p, (g, t) in zip(planners, dev_inputs):
        p.plan(g, t)
    for sid in range(planners[0].shape.kernels):
        for _ in range(args.stage_reps):
            for p, (g, t) in zip(planners, dev_inputs):
                p.stage(sid, g, t)
    src = torch.ones(64 << 20, dtype=torch.int32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(4):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"pmc_pass": cfg.name, "layers": layers, "stage_reps": args.stage_reps,
                      "copy_bytes": src.numel() * 4, "kernel_source_sha1": source_digest()}), flush=True)


def _host_cpu():
    """nproc and the lscpu model name of this host (None where unavailable)."""
    import subprocess
    out = {"nproc": None, "lscpu_model_name": None}
    try:
        out["nproc"] = int(subprocess.run(["nproc"], capture_output=True, text=True, timeout=10).stdout.strip())
    except Exception:
        out["nproc"] = os.cpu_count()
    try:
        for line in subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout.splitlines():
            if line.startswith("Model name:"):
                out["lscpu_model_name"] = line.split(":", 1)[1].strip()
                break
    except Exception:
        pass
    return out


def cpu_baseline(cfg, inputs, budget_s=15.0, dev_inputs=None):
    """The oracle timed on this host: (i) one thread, layers back to back
    (the reported value); (ii) layers spread over every core this process
    may use (threads: the oracle call releases the GIL); (iii) the
    host-planning path of Eq. 1 for the same layers: synchronise and copy
    Omega and the ids to pinned host memory, plan on the CPU, copy the
    outputs back to the GPU."""
    import concurrent.futures as cf

    import oracle
    # (i) one thread: the layers back to back, cycling through them until
    # the budget (about half of budget_s) is spent
    n = 0
    t0 = time.perf_counter()
    while True:
        gl, tk = inputs[n % len(inputs)]
        oracle.plan_cfg(cfg, gl, tk, 0)
        n += 1
        if time.perf_counter() - t0 > 0.5 * budget_s:
            break
    dt = time.perf_counter() - t0
    per_layer = dt / n
    out = {"value": n * cfg.T * cfg.k / dt, "unit": "assignments/s", "cores": 1, "kind": "oracle",
           "sample": "%d layer plans (the %d layers of the %s workload, cycled, back to back, one "
                     "thread): %.0f us per layer, %.1f s" % (n, len(inputs), cfg.name, per_layer * 1e6, dt),
           **_host_cpu()}
    # (ii) every core: about budget/2 seconds of work
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    cores = max(1, min(cores, 64))
    tasks = max(cores, min(200000, int(0.25 * budget_s / per_layer * cores)))
    jobs = [inputs[i % len(inputs)] for i in range(tasks)]
    t0 = time.perf_counter()
    with cf.ThreadPoolExecutor(cores) as ex:
        list(ex.map(lambda a: oracle.plan_cfg(cfg, a[0], a[1], 0), jobs))
    dt2 = time.perf_counter() - t0
    out["all_cores"] = {"value": tasks * cfg.T * cfg.k / dt2, "unit": "assignments/s", "threads": cores,
                        "us_per_layer": dt2 / tasks * 1e6, "layers_planned": tasks}
    # (iii) Eq. 1 host-planning path
    if dev_inputs is not None:
        import torch
        dev = dev_inputs[0][0].device
        m = min(200, max(1, int(0.2 * budget_s / per_layer)))   # the layers, cycled
        gl_h = torch.empty(dev_inputs[0][0].shape, dtype=torch.int32, pin_memory=True)
        tk_h = torch.empty(dev_inputs[0][1].shape, dtype=torch.int32, pin_memory=True)
        slots_d = torch.empty((cfg.R, cfg.N), dtype=torch.int32, device=dev)
        dest_d = torch.empty(dev_inputs[0][1].shape, dtype=torch.int32, device=dev)
        sc_d = torch.empty((cfg.R,), dtype=torch.int32, device=dev)
        t_sync = t_cpu = t_ret = 0.0
        cpu_each, cpu_again = [], []
        for i in range(m):
            gd, td = dev_inputs[i % len(dev_inputs)]
            torch.cuda.synchronize()
            a = time.perf_counter()
            gl_h.copy_(gd, non_blocking=True)
            tk_h.copy_(td, non_blocking=True)
            torch.cuda.synchronize()
            # out of the pinned staging buffers into ordinary (cached) host
            # memory, which the CPU planner reads many times
            gl_c = np.array(gl_h.numpy())
            tk_c = np.array(tk_h.numpy())
            b = time.perf_counter()
            ref = oracle.plan_cfg(cfg, gl_c, tk_c, 0)
            c = time.perf_counter()
            # the same plan once more on the same arrays, outside the path's
            # total: separates a slow first touch from the planner's own time
            oracle.plan_cfg(cfg, gl_c, tk_c, 0)
            cpu_again.append(time.perf_counter() - c)
            cpu_each.append(c - b)
            c = time.perf_counter()
            slots_d.copy_(torch.from_numpy(ref["replica_slots"]))
            dest_d.copy_(torch.from_numpy(ref["token_dest"]))
            sc_d.copy_(torch.from_numpy(ref["send_counts"]))
            torch.cuda.synchronize()
            d = time.perf_counter()
            t_sync += b - a
            t_cpu += cpu_each[-1]
            t_ret += d - c
        out["host_plan_path"] = {"us_per_layer": (t_sync + t_cpu + t_ret) / m * 1e6,
                                 "t_sync_us": t_sync / m * 1e6, "t_cpu_us": t_cpu / m * 1e6,
                                 "t_return_us": t_ret / m * 1e6, "layers": m,
                                 "t_cpu_us_min_median_max": [float(np.min(cpu_each)) * 1e6,
                                                             float(np.median(cpu_each)) * 1e6,
                                                             float(np.max(cpu_each)) * 1e6],
                                 "t_cpu_repeat_us_median": float(np.median(cpu_again)) * 1e6}
    return out


def time_stage(torch, planners, dev_inputs, stage, reps):
    """Average duration of one kernel of the plan: a HIP graph of reps x layers
    back-to-back launches of that kernel alone (every workspace holds a full
    plan of its layer), timed with HIP events on the stream the graph runs
    on.  Includes the dispatch gap between consecutive launches."""
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(stream):
        with torch.cuda.graph(g, stream=stream):
            for _ in range(reps):
                for p, (gl, tk) in zip(planners, dev_inputs):
                    p.stage(stage, gl, tk, stream=stream)
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        g.replay()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(3):
            g.replay()
        b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) * 1e3 / (3 * reps * len(planners))   # microseconds


# Phase stamps of the instrumented library (slot: what was just done), in
# the one-launch plan; the solver's slots come from workgroup 0, the chunk
# slots from chunk 0 except "last arrival done" (the last chunk).
PHASE_SLOTS = [(0, "solver start"), (1, "Omega in LDS"), (23, "plan start"), (22, "stage 1 candidates"),
               (2, "stage 1"), (3, "setup"), (4, "routing"), (5, "refinement"), (6, "outputs"),
               (7, "instance list"), (10, "flags released"), (8, "speculative plan returned"),
               (9, "verdict handled"),
               (12, "chunk 0 arrived"), (19, "last arrival start"), (13, "last arrival done"),
               (16, "chunk 0 offsets"), (14, "chunk 0 sees flag"), (15, "chunk 0 done"),
               (24, "s1: candidates"), (26, "s1: ranks"), (27, "ff: lists and hosting"), (28, "ff: counts"), (30, "ff: entries")]


# the per-domain solver (three-kernel plan): workgroup 0's phases, then the
# last workgroup's instance list
SOLVE_SLOTS = [(0, "solver start"), (1, "stage 1"), (2, "grid barrier passed"), (3, "row self and hosting masks"),
               (4, "domain instances"), (5, "q columns"), (6, "routing"), (7, "refinement"), (8, "outputs"),
               (9, "drained"), (10, "list start (last workgroup)"), (11, "list counted"), (12, "list placed"),
               (13, "list done"), (14, "s1: rows copied"), (15, "s1: row self"), (16, "s1: candidates")]

REFINE_SECTIONS = ["busiest and levels", "scoring", "selection", "target instance", "transfer", "updates"]


def run_phases(args):
    """Phase timeline of the one-launch plan from the stamped library (run
    with TOPOEP_STAMPS=1): every layer planned in one HIP graph, replayed;
    each slot's median over layers and replays, in microseconds after the
    solver's start (the stamps read the 100 MHz constant clock)."""
    import torch
    from paper_2609_35481_amd import topoep
    if not topoep.LIB_PATH.endswith("libtopoep_stamps.so"):
        raise SystemExit("--phases needs TOPOEP_STAMPS=1 (the instrumented library)")
    cfg = workload.get(args.config)
    layers = cfg.layers if args.layers <= 0 else args.layers
    dev = torch.device("cuda:0")
    inputs = make_inputs(cfg, layers)
    topo = topoep.topology(cfg.R, cfg.G, cfg.E, 0, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W)
    dev_inputs = [(torch.from_numpy(gl.copy()).to(dev), torch.from_numpy(tk.copy()).to(dev)) for gl, tk in inputs]
    launch = launch_from_args(args)
    N = cfg.N if args.slots < 0 else args.slots
    planners = [topoep.Planner(topo, cfg.T, cfg.k, N, device=dev, launch=launch) for _ in range(layers)]
    slots = PHASE_SLOTS if planners[0].shape.kernels == 1 else SOLVE_SLOTS
    samples, refine = [], []
    for rep in range(args.steps):
        for p, (g, t) in zip(planners, dev_inputs):
            p.plan(g, t)
        torch.cuda.synchronize()
        if rep < args.warmup:
            continue
        for p in planners:
            w = p.workspace_view()[64:256].cpu().numpy().view(np.uint32).astype(np.int64)
            samples.append([((int(w[i]) - int(w[0])) & 0xFFFFFFFF) if i < 20 or i > 21 else 0
                            for i, _ in slots])
            if w[38] > 0:
                refine.append([w[32 + k] / w[38] for k in range(6)] + [w[38]])
    clk = []
    for p in planners:
        w = p.workspace_view()[64:256].cpu().numpy().view(np.uint32).astype(np.int64)
        dt = (int(w[10]) - int(w[0])) & 0xFFFFFFFF
        if dt and slots is PHASE_SLOTS:
            clk.append(((int(w[21]) - int(w[20])) & 0xFFFFFFFF) / (dt * 0.01))
    arr = np.array(samples, dtype=np.float64) * 0.01   # 100 MHz ticks -> microseconds
    med = np.median(arr, axis=0)
    out = {"phases": cfg.name, "replica_slots": N, "layers": layers, "samples": len(samples),
           "us_after_solver_start_median": {name: round(float(v), 3) for (_, name), v in zip(slots, med)},
           "us_p10": {name: round(float(v), 3) for (_, name), v in zip(slots, np.percentile(arr, 10, axis=0))},
           "us_p90": {name: round(float(v), 3) for (_, name), v in zip(slots, np.percentile(arr, 90, axis=0))},
           "core_clock_MHz_median": round(float(np.median(clk)), 1) if clk else None,
           # domain 0's refinement loop: core-clock cycles per iteration by
           # section (median over the plans that refined it)
           "refine_cycles_per_iteration": (
               {name: round(float(v), 1) for name, v in zip(REFINE_SECTIONS + ["iterations"],
                                                             np.median(np.array(refine, dtype=np.float64), axis=0))}
               if refine else None),
           "plan_shape": planners[0].shape.as_dict()}
    return out


def measure(torch, topoep, cfg, N, inputs, steps, warmup, stage_reps, launch=None):
    """Time every layer's plan of one microbatch as one HIP graph (inputs
    resident in HBM), then each kernel of the plan alone and the launch
    floor.  Returns the measurement and the planners (each holding a full
    plan of its layer)."""
    layers = len(inputs)
    dev = torch.device("cuda:0")
    topo = topoep.topology(cfg.R, cfg.G, cfg.E, 0, cfg.c_intra, cfg.c_inter, cfg.S, cfg.W)
    dev_inputs = [(torch.from_numpy(gl.copy()).to(dev), torch.from_numpy(tk.copy()).to(dev)) for gl, tk in inputs]
    planners = [topoep.Planner(topo, cfg.T, cfg.k, N, device=dev, launch=launch) for _ in range(layers)]
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        for p, (g, t) in zip(planners, dev_inputs):
            p.plan(g, t)
    torch.cuda.synchronize()
    # a workload of few layers is captured several times over, so that each
    # replay holds at least 32 plans and the host's cost of submitting a
    # replay stays hidden behind the GPU work; a step is still one pass over
    # every layer
    copies = max(1, -(-32 // layers))
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(copies):
            for p, (g, t) in zip(planners, dev_inputs):
                p.plan(g, t)
    torch.cuda.synchronize()
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for a, b in ev:
        a.record()
        graph.replay()
        b.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = np.array([a.elapsed_time(b) for a, b in ev]) / copies
    ms_per_step = wall / (steps * copies) * 1e3
    value = layers * cfg.T * cfg.k / (ms_per_step / 1e3)
    # every plan of the last replay must be a valid plan (status 0)
    st = torch.stack([p.status for p in planners]).cpu().numpy()
    if (st[:, 0] & ~topoep.ST_SELF_DIFF).any():
        raise SystemExit("%s: plan status bits set: %s" % (cfg.name, np.unique(st[:, 0])))
    moves = st[:, 1].astype(np.int64)
    # per-kernel durations (a graph of back-to-back launches of one kernel,
    # HIP events on its stream), and the launch floor (empty kernels, same
    # shapes, same graph structure)
    shape = planners[0].shape
    kernels = shape.kernels
    stages = {}
    for sid, name in enumerate(STAGE_NAMES[kernels]):
        stages[name] = time_stage(torch, planners, dev_inputs, sid, max(stage_reps, copies))
    floor_us = time_stage(torch, planners, dev_inputs, topoep.STAGE_FLOOR, max(stage_reps, copies))
    for p, (g, t) in zip(planners, dev_inputs):
        p.plan(g, t)
    torch.cuda.synchronize()
    nbytes = algorithmic_bytes(cfg, N, kernels)
    own = kernel_bytes(cfg, N, kernels)
    dom = max(stages, key=lambda k: stages[k])
    avg_us = stages[dom]
    achieved = nbytes[dom] / (avg_us * 1e-6) / 1e9
    roof = {"bound": "hbm", "kernel": dom + "_kernel", "achieved": achieved, "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
            # (the counters were taken at the workload's own slot count and
            # the library's launch shape only)
            "traffic": measured_traffic(cfg.name, dom) if N == cfg.N and launch is None else None,
            "algorithmic_bytes_per_launch": nbytes[dom], "kernel_own_bytes_per_launch": own[dom],
            "frac_kernel_own_bytes": own[dom] / (avg_us * 1e-6) / 1e9 / HBM_PEAK_GBS, "avg_kernel_us": avg_us,
            "floor_ratio": avg_us / (floor_us / kernels) if floor_us > 0 else None}
    per_layer = ms_per_step * 1e3 / layers
    layer_bytes = sum(nbytes.values())
    res = {
        "workload": DESCR.get(cfg.name, cfg.name), "layers": layers, "replica_slots": N,
        "passes_per_replay": copies, "plan_shape": shape.as_dict(), "ms_per_step": ms_per_step,
        "assignments_per_s": value, "plan_latency_us_per_layer": per_layer,
        "plan_latency_us_per_layer_p10_p50_p90": [float(np.percentile(step_ms, q)) * 1e3 / layers
                                                  for q in (10, 50, 90)],
        "kernel_avg_us": {k: round(v, 3) for k, v in stages.items()},
        "launch_floor_us_per_layer": round(floor_us, 3),
        "floor_ratio": per_layer / floor_us if floor_us > 0 else None,
        "refinement_moves_per_layer": {"mean": float(moves.mean()), "max": int(moves.max()),
                                       "layers_with_moves": int((moves > 0).sum())},
        "algorithmic_bytes_per_layer": layer_bytes,
        "hbm_frac_per_layer": layer_bytes / (per_layer * 1e-6) / 1e9 / HBM_PEAK_GBS,
        "roofline": roof,
    }
    return res, planners, dev_inputs, topo


# extra workloads of the all-configs object: name, configuration, replica
# slots (the refinement-heavy cases: DeepSeek-V3-like with 4 slots, where
# stage 1 leaves slots free, and Mixtral-like, which refines every layer)
ALL_CONFIGS = [("tiny", "tiny", None), ("mixtral", "mixtral", None), ("qwen3", "qwen3", None),
               ("dsv3", "dsv3", None), ("stress", "stress", None), ("dsv3_N4", "dsv3", 4)]


def all_configs(torch, topoep, args, headline=None):
    """Every configuration (first microbatch, all its layers) and the
    refinement-heavy DeepSeek-V3-like case with 4 slots, fewer steps each."""
    out = {}
    for key, name, N in ALL_CONFIGS:
        cfg = workload.get(name)
        n_slots = cfg.N if N is None else N
        if headline is not None and key == args.config:
            res = headline
        else:
            t = time.perf_counter()
            inputs = workload.make_layers(cfg, [(l, 0) for l in range(cfg.layers)],
                                          workers=min(16, os.cpu_count() or 1))
            gen_s = time.perf_counter() - t
            res, _, _, _ = measure(torch, topoep, cfg, n_slots, inputs, args.all_steps, max(3, args.warmup // 4),
                                   args.stage_reps)
            res["input_generation_s"] = round(gen_s, 2)
        out[key] = {k: res[k] for k in ("workload", "layers", "replica_slots", "plan_shape",
                                        "plan_latency_us_per_layer", "plan_latency_us_per_layer_p10_p50_p90",
                                        "assignments_per_s", "kernel_avg_us", "launch_floor_us_per_layer",
                                        "floor_ratio", "refinement_moves_per_layer", "algorithmic_bytes_per_layer",
                                        "hbm_frac_per_layer", "roofline")}
        print("all_configs %s: %.2f us per layer" % (key, res["plan_latency_us_per_layer"]), file=sys.stderr,
              flush=True)
        torch.cuda.empty_cache()
    return out


def run_bench(args):
    import torch
    from paper_2609_35481_amd import topoep

    cfg = workload.get(args.config)
    N = cfg.N
    layers = cfg.layers if args.layers <= 0 else args.layers
    t_gen = time.perf_counter()
    inputs = make_inputs(cfg, layers)
    t_gen = time.perf_counter() - t_gen
    launch = launch_from_args(args)
    res, planners, dev_inputs, topo = measure(torch, topoep, cfg, N, inputs, args.steps, args.warmup,
                                              args.stage_reps, launch)
    res["input_generation_s"] = round(t_gen, 2)
    out = {
        "metric": METRIC,
        "value": res["assignments_per_s"],
        "unit": "assignments/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "launch": launch,
        "passes_per_replay": res["passes_per_replay"],
        "plan_shape": res["plan_shape"],
        "config": {"workload": DESCR[cfg.name], "layers_per_step": layers, "tokens_per_rank": cfg.T,
                   "top_k": cfg.k, "ranks": cfg.R, "experts": cfg.E, "replica_slots": N,
                   "assignments_per_layer": cfg.T * cfg.k},
        "plan_latency_us_per_layer": res["plan_latency_us_per_layer"],
        "plan_latency_us_per_layer_p10_p50_p90": res["plan_latency_us_per_layer_p10_p50_p90"],
        "kernel_avg_us": res["kernel_avg_us"],
        "launch_floor_us_per_layer": res["launch_floor_us_per_layer"],
        "floor_ratio": res["floor_ratio"],
        "refinement_moves_per_layer": res["refinement_moves_per_layer"],
        "roofline": res["roofline"],
        "input_generation_s": res["input_generation_s"],
    }
    if not args.no_dispatch:
        out["dispatch"] = bench_dispatch(torch, topoep, cfg, topo, planners, dev_inputs, args)
    if not args.no_gather:
        out["replica_gather"] = bench_gather(torch, topoep, cfg, topo, planners)
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(cfg, inputs, args.cpu_seconds, dev_inputs)
    if not args.no_all_configs and args.layers <= 0 and launch is None:
        out["all_configs"] = all_configs(torch, topoep, args, headline=res)
    return out


def _graph_us(torch, enqueue, reps, per):
    """Microseconds per unit of a HIP graph holding `enqueue()` (per units),
    replayed reps times between events on the graph's stream."""
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        enqueue(stream)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(stream):
        with torch.cuda.graph(g, stream=stream):
            enqueue(stream)
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        g.replay()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            g.replay()
        b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) * 1e3 / (reps * per)


def bench_gather(torch, topoep, cfg, topo, planners, reps=20):
    """Replica-slot parameter gather: rank 0's slots (as many as the first
    layer's plan fills) receive bf16 experts of ||W_e|| bytes from a buffer
    holding every expert's parameters.  Each repetition gathers a different
    set of experts, so the sources are never resident in the 256 MB
    Infinity Cache; a plain device copy of the same bytes from the same
    rotating sources is timed beside it."""
    dev = planners[0].replica_slots.device
    n_copied = int((planners[0].replica_slots[0] >= 0).sum().item())
    if n_copied == 0:
        return {"slots_copied": 0}
    elems = cfg.W // 2
    params = torch.empty((cfg.E, elems), dtype=torch.bfloat16, device=dev)
    out = torch.empty((cfg.N, elems), dtype=torch.bfloat16, device=dev)
    sets = []
    for r in range(reps):
        sl = torch.full((cfg.R, cfg.N), -1, dtype=torch.int32)
        sl[0, :n_copied] = torch.tensor([(r * n_copied + j) % cfg.E for j in range(n_copied)], dtype=torch.int32)
        sets.append(sl.to(dev))
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    topoep.gather_replicas(topo, sets[-1], params, out)
    a.record()
    for sl in sets:
        topoep.gather_replicas(topo, sl, params, out)
    b.record()
    torch.cuda.synchronize()
    us = a.elapsed_time(b) * 1e3 / reps
    a.record()
    for r in range(reps):
        e0 = (r * n_copied) % cfg.E
        if e0 + n_copied <= cfg.E:
            out[:n_copied].copy_(params[e0:e0 + n_copied])
        else:
            for j in range(n_copied):
                out[j].copy_(params[(e0 + j) % cfg.E])
    b.record()
    torch.cuda.synchronize()
    copy_us = a.elapsed_time(b) * 1e3 / reps
    del params, out
    torch.cuda.empty_cache()
    moved = 2 * n_copied * cfg.W
    achieved = moved / (us * 1e-6) / 1e9
    return {"slots_copied": n_copied, "bytes_per_expert": cfg.W, "gather_us": round(us, 2),
            "device_copy_us": round(copy_us, 2),
            "roofline": {"bound": "hbm", "kernel": "gather_kernel", "achieved": achieved, "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "algorithmic_bytes_per_launch": moved},
            "device_copy_GBps": moved / (copy_us * 1e-6) / 1e9}


def bench_dispatch(torch, topoep, cfg, topo, planners, dev_inputs, args):
    """The dispatch side of the plan: the plan with receive counts and the
    send-buffer layout (topoep_plan_dispatch) per layer, and the layout
    kernel alone on each layer's destinations (its HBM roofline)."""
    layers = len(planners)
    dps = [topoep.DispatchPlanner(topo, cfg.T, cfg.k, cfg.N, device=dev_inputs[0][0].device)
           for _ in range(layers)]

    def plan_all(stream):
        for d, (g, t) in zip(dps, dev_inputs):
            d.plan(g, t, stream=stream)
    per_layer = _graph_us(torch, plan_all, max(5, args.steps // 4), layers)
    st = torch.stack([d.status for d in dps]).cpu().numpy()
    if (st[:, 0] & ~topoep.ST_SELF_DIFF).any():
        raise SystemExit("dispatch plan status bits set: %s" % np.unique(st[:, 0]))
    lps = [topoep.LayoutPlanner(topo, cfg.T, cfg.k, device=dev_inputs[0][0].device) for _ in range(layers)]

    def layout_all(stream):
        for lp, p in zip(lps, planners):
            lp.layout(p.token_dest, p.send_counts, stream=stream)
    reps = max(1, args.stage_reps)
    layout_us = _graph_us(torch, lambda s: [layout_all(s) for _ in range(reps)], 3, reps * layers)
    n = cfg.T * cfg.k
    nbytes = 8 * n + 4 * cfg.R + 4 * (cfg.R + 1)
    achieved = nbytes / (layout_us * 1e-6) / 1e9
    return {"plan_dispatch_latency_us_per_layer": per_layer,
            "layout_kernel_avg_us": round(layout_us, 3),
            "layout_roofline": {"bound": "hbm", "kernel": "layout_kernel", "achieved": achieved,
                                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                                "algorithmic_bytes_per_launch": nbytes}}


def run_sweep(args):
    """Histogram, reroute and send-buffer layout alone over synthetic id arrays of growing size,
    past the 256 MB Infinity Cache, with a fixed plan."""
    import torch
    from paper_2609_35481_amd import topoep

    dev = torch.device("cuda:0")
    rows = []
    for E in [int(x) for x in args.sweep_experts.split(",")]:
        R, G = 32, 8
        for lg in range(args.sweep_min_log2, args.sweep_max_log2 + 1, 2):
            n = 1 << lg
            k = 8
            T = n // k
            rng = np.random.default_rng(lg)
            p = workload.generate.zipf_weights(E, 1.0)
            tk = torch.from_numpy(rng.choice(E, size=(T, k), p=p).astype(np.int32)) if n <= (1 << 22) else None
            if tk is None:
                small = torch.from_numpy(rng.choice(E, size=(1 << 22,), p=p).astype(np.int32)).to(dev)
                tk_d = small.repeat(n // (1 << 22)).view(T, k)
            else:
                tk_d = tk.to(dev)
            hist = torch.bincount(tk_d.view(-1).long(), minlength=E).to(torch.int32)
            # other ranks' rows stay small so that the total load fits int32
            gl = torch.randint(0, 1000, (R, E), dtype=torch.int32, device=dev)
            gl[0] = hist
            topo = topoep.topology(R, G, E, 0, 1, 8, 4096, 9 << 20)
            # the three-kernel path, so the histogram and reroute kernels run
            # alone (the per-domain solver where one workgroup's LDS is too small)
            shape = (args.ipt, args.block_threads, args.tiles_per_block, 0)
            try:
                pl = topoep.Planner(topo, T, k, 2, device=dev, launch=shape + (topoep.SOLVER_SINGLE,))
            except topoep.TopoepError:
                pl = topoep.Planner(topo, T, k, 2, device=dev, launch=shape + (topoep.SOLVER_PER_DOMAIN,))
            pl.plan(gl, tk_d)
            torch.cuda.synchronize()
            st = int(pl.status[0].item())
            res = {}
            lp = topoep.LayoutPlanner(topo, T, k, device=dev)
            runs = (("hist", lambda: pl.stage(0, gl, tk_d), 4), ("reroute", lambda: pl.stage(2, gl, tk_d), 8),
                    ("layout", lambda: lp.layout(pl.token_dest, pl.send_counts), 8))
            for name, fn, bpa in runs:
                reps = 5 if n >= (1 << 26) else 20
                a = torch.cuda.Event(enable_timing=True)
                b = torch.cuda.Event(enable_timing=True)
                fn()
                a.record()
                for _ in range(reps):
                    fn()
                b.record()
                torch.cuda.synchronize()
                us = a.elapsed_time(b) * 1e3 / reps
                res[name] = {"us": round(us, 2), "GB/s": round(bpa * n / us / 1e3, 1)}
            if int(lp.status[0].item()) != 0:
                raise SystemExit("layout status %d" % int(lp.status[0].item()))
            rows.append({"E": E, "ids": n, "status": st, **res})
            print(json.dumps(rows[-1]), flush=True)
            del pl, lp, tk_d, gl
            torch.cuda.empty_cache()
    if args.pmc_pass:
        # counter calibration in the same run: a plain device copy of 256 MiB
        src = torch.ones(64 << 20, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(4):
            dst.copy_(src)
        torch.cuda.synchronize()
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="dsv3", choices=sorted(DESCR))
    ap.add_argument("--layers", type=int, default=0, help="0 = the configuration's layer count")
    ap.add_argument("--slots", type=int, default=-1, help="replica slots per rank for --phases (-1: the configuration's)")
    ap.add_argument("--stage-reps", type=int, default=5)
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="CPU baseline budget: half for one thread, a quarter for every core")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-dispatch", action="store_true", help="skip the dispatch-side measurement")
    ap.add_argument("--no-gather", action="store_true", help="skip the replica-slot gather measurement")
    ap.add_argument("--no-all-configs", action="store_true", help="skip the all-configurations object")
    ap.add_argument("--all-steps", type=int, default=50, help="timed steps per configuration of all_configs")
    ap.add_argument("--sweep", action="store_true")
    ap.add_argument("--sweep-min-log2", type=int, default=16)
    ap.add_argument("--sweep-max-log2", type=int, default=28)
    ap.add_argument("--sweep-experts", default="128,512")
    ap.add_argument("--pmc-pass", action="store_true", help="workload for rocprofv3 counter runs")
    ap.add_argument("--phases", action="store_true",
                    help="phase timeline of the one-launch plan (needs TOPOEP_STAMPS=1)")
    ap.add_argument("--solver", type=int, default=0,
                    help="0 auto, 1 one solver workgroup, 2 one per domain, 3 one launch")
    ap.add_argument("--ipt", type=int, default=0, help="ids per thread per tile (0 = default)")
    ap.add_argument("--block-threads", type=int, default=0)
    ap.add_argument("--tiles-per-block", type=int, default=0)
    ap.add_argument("--solve-threads", type=int, default=0)
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the planner is replicated per rank and has no "
              "cross-GPU step in this build (--gpus %d requested)" % args.gpus, file=sys.stderr)
        raise SystemExit(2)
    if args.sweep:
        run_sweep(args)
        return
    if args.pmc_pass:
        run_pmc_pass(args)
        return
    if args.phases:
        print(json.dumps(run_phases(args)), flush=True)
        return
    print(json.dumps(run_bench(args)), flush=True)


if __name__ == "__main__":
    main()
