#!/usr/bin/env python3
"""Throughput of the fused local update + P-Reduce step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config C]

A step is one pass of the whole hot path over one batch of synthetic input:
the host group schedule for step t, then one launch of the fused kernel that
applies every active worker's local update and the P-Reduce of every group.
The default workload (--config 5) is the largest of the five: 8 replicas of
1.3 B parameters stored as bf16 (fp32 arithmetic), a seeded static schedule
of two groups of four, plain SGD.  --config 1..4 select the others.

Prints one JSON line (stdout).  ``value`` is algorithmic HBM bytes of the K
timed steps divided by their wall time, inputs resident in HBM before timing
starts.  ``roofline.achieved`` is the same bytes over the GPU time of the
timed launches: one pair of HIP events on the launch stream brackets the
whole timed window, and the span is spread evenly over the launches in it
(the next launch is queued before the previous kernel ends, so the span is
kernel time plus the dispatch gaps between launches; it can never exceed the
wall time; the library reports how many kernels each step enqueued, one or
two).  ``cpu_baseline`` times the CPU oracle on a bounded sample of the
same workload, pinned to one core.  Progress goes to stderr.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "P-Reduce+update effective HBM GB/s and % of MI355X HBM peak"
KERNEL_SOURCES = ["paper_1909_08029_amd/csrc/rip_kernels.hip",
                  "paper_1909_08029_amd/csrc/rip_api.hip",
                  "paper_1909_08029_amd/csrc/rip_kernel_args.h",
                  "paper_1909_08029_amd/csrc/rip_launch_policy.h"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
SCHEDULE_NAMES = ["table", "static", "random_gb", "global_division", "scripted", "rule",
                  "inter_intra", "adpsgd"]


def err(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_hash() -> str:
    """First 16 hex digits of sha256 over the kernel and launch sources with
    comments and whitespace removed, so an edit to a comment does not
    orphan counters taken on the same code."""
    import re
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def load_traffic(workload: str, alg_bytes_per_launch: float):
    """HBM bytes per launch from the rocprofv3 FETCH_SIZE/WRITE_SIZE passes
    (scaled by a copy of known size), if they were taken on the current
    kernel source for this workload: the measured traffic/algorithmic ratio
    times this run's algorithmic bytes per launch (the two agree for
    workloads whose launches all move the same bytes)."""
    try:
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    ent = data.get(workload)
    if not ent or ent.get("kernel_hash") != kernel_hash():
        return None
    return int(round(ent["traffic_over_alg"] * alg_bytes_per_launch))


def host_cpu() -> str:
    """CPU model, logical CPUs and the CPUs this process may run on."""
    model = "unknown CPU"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        allowed = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        allowed = os.cpu_count()
    return f"{model}, {os.cpu_count()} logical CPUs, {allowed} in this process's affinity"


def cpu_baseline(w, seconds: float = 12.0):
    """The oracle as it stands (numpy) on one window of every replica, for as
    many steps of the workload's schedule as fit the budget (at least 2; the
    schedule runs on past the workload's step count if time is left),
    timed on the update + group averaging only.  It runs on one core: the
    calling thread is pinned to one CPU and numpy's thread pools are limited
    to one thread for the duration (numpy's element-wise operations are
    single-threaded anyway)."""
    import numpy as np  # noqa: F401
    from threadpoolctl import threadpool_limits
    from oracle import preduce as op
    from oracle import sched as osd
    from seedgen import DTYPE_BF16
    from seedgen import workloads as wl

    width = min(w.numel, 1 << 22)
    a, b = 0, width
    kw = dict(w.sched)
    mode = kw.pop("mode")
    sch = osd.Scheduler(w.n, mode, **kw)
    p, grad, v = wl.host_inputs(w, a, b)
    dt = op.BF16 if w.dtype == DTYPE_BF16 else op.F32
    sub = wl.scaled(w, [width])
    spent, nbytes, steps = 0.0, 0, 0
    before = os.sched_getaffinity(0)
    cpu = min(before)
    os.sched_setaffinity(0, {cpu})           # this thread only
    try:
        with threadpool_limits(limits=1):
            while steps < 2 or spent < seconds:
                active, groups = sch.step(steps, w.eligible(steps))
                g = grad(w.grad_slot(steps))
                t0 = time.perf_counter()
                p, v = op.step(p, g, v, groups, active, w.lr, w.momentum or None, dt, True,
                               w.weight_decay, w.nesterov)
                spent += time.perf_counter() - t0
                nbytes += sub.alg_bytes(active, groups)
                steps += 1
    finally:
        os.sched_setaffinity(0, before)
    return dict(value=round(nbytes / spent / 1e9, 4), unit="GB/s", cores=1, kind="oracle",
                sample=f"{steps} steps of the workload schedule on elements [0, {width}) of all "
                       f"{w.n} replicas ({100.0 * width / w.numel:.2f}% of each replica), "
                       f"numpy pinned to CPU {cpu} with thread pools limited to 1, on "
                       f"{host_cpu()}; {spent:.1f} s timed, update+average only")


def graph_steps(args, w, rip, handles, sched, t, stream, stats):
    """Times args.steps fused steps as replays of one captured period.

    Only a schedule that repeats is replayable: the steps of one period
    (a multiple of the gradient ring) are scheduled by the library, their
    launches captured into a HIP graph, and a second scheduler checks that the
    next period schedules exactly the same groups.  Every replay then runs
    those steps, as a static schedule prescribes.  Returns (period,
    bytes per step, GPU span in ms of all replays, wall seconds, kernel
    launches replayed)."""
    import math
    import torch
    from seedgen import workloads as wl
    if args.unfused or w.sched["mode"] not in (wl.TABLE, wl.STATIC, wl.RULE) \
            or w.straggler_every is not None:
        err("--graph needs a fused step with a fixed (table, static or rule) schedule and "
            "no straggler")
        sys.exit(2)
    rows = {wl.TABLE: len(w.sched.get("table", [[]])), wl.STATIC: w.sched.get("period", 4),
            wl.RULE: 4}[w.sched["mode"]]
    L = rows * w.grad_ring // math.gcd(rows, w.grad_ring)
    while L < 8 and args.steps % (2 * L) == 0:   # a few steps per replay, whole periods
        L *= 2
    if args.steps % L:
        err(f"--graph replays {L} steps at a time; --steps must be a multiple of {L}")
        sys.exit(2)
    period = [rip.rip_schedule_groups(sched, t + i) for i in range(L)]
    kw = dict(w.sched)
    check = rip.Scheduler(w.n, kw.pop("mode"), **kw)
    seen = [rip.rip_schedule_groups(check, i) for i in range(t + 2 * L)]
    if seen[t:t + L] != period or seen[t + L:] != period:
        err("--graph: the schedule does not repeat with the captured period")
        sys.exit(2)
    opt = dict(momentum=w.momentum, weight_decay=w.weight_decay, nesterov=w.nesterov)
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    kernels = 0
    with torch.cuda.graph(g):
        cap = torch.cuda.current_stream()
        for i, (active, groups) in enumerate(period):
            rip.rip_preduce(handles[w.grad_slot(t + i)], groups, active, lr=w.lr, stream=cap,
                            **opt)
            kernels += rip.rip_last_launch_count()
    torch.cuda.synchronize()
    g.replay()                                     # first execution, untimed
    torch.cuda.synchronize()
    step_bytes = [w.alg_bytes(a, gr) for a, gr in period]
    reps = args.steps // L
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(reps):
        g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    span_ms = e0.elapsed_time(e1)
    per_step_bytes = []
    for _ in range(reps):
        for (active, groups), b in zip(period, step_bytes):
            per_step_bytes.append(b)
            stats["steps"] += 1
            stats["updates"] += len(active)
            stats["groups"] += sum(1 for x in groups if len(x) > 1)
            stats["members"] += sum(len(x) for x in groups if len(x) > 1)
            stats["empty"] += 0 if (active or any(len(x) > 1 for x in groups)) else 1
    del g
    return L, per_step_bytes, span_ms, wall, kernels * reps


def sweep_caps(args, w, rip, handles, stream):
    """Kernel GB/s of the workload's steps at each residency cap (resident
    waves per CU), measured in one process: three rounds, each timing
    args.steps steps (after two untimed ones) at every cap in turn, each cap
    with a scheduler of its own.  Prints one JSON line per cap with the
    median over the rounds."""
    import torch
    caps = [int(x) for x in args.sweep_caps.split(",") if x.strip()]
    if not caps or min(caps) < 1:
        err("--sweep-caps needs positive waves per CU")
        sys.exit(2)
    kw = dict(w.sched)
    mode = kw.pop("mode")
    scheds = {c: rip.Scheduler(w.n, mode, **kw) for c in caps}
    t_next = {c: 0 for c in caps}
    res = {c: [] for c in caps}
    for rnd in range(3):
        for c in caps:
            rip.rip_set_blocks_per_cu(c)
            evs, nbytes = [], 0
            for i in range(args.steps + 2):
                t = t_next[c]
                active, groups = rip.rip_schedule_groups(scheds[c], t, w.eligible(t))
                h = handles[w.grad_slot(t)]
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                if args.average_only:
                    active = []
                    rip.rip_preduce(h, groups, [], stream=stream)
                else:
                    rip.rip_preduce(h, groups, active, lr=w.lr, momentum=w.momentum,
                                    stream=stream, weight_decay=w.weight_decay,
                                    nesterov=w.nesterov)
                e1.record(stream)
                t_next[c] += 1
                b = w.alg_bytes(active, groups)
                if i >= 2 and b:
                    evs.append((e0, e1))
                    nbytes += b
            torch.cuda.synchronize()
            ms = sum(a.elapsed_time(b) for a, b in evs)
            res[c].append(nbytes / (ms * 1e-3) / 1e9 if ms > 0 else 0.0)
        err(f"[bench] sweep round {rnd}: " +
            "  ".join(f"{c}: {res[c][-1]:.0f}" for c in caps))
    rip.rip_set_blocks_per_cu(0)
    for c in caps:
        print(json.dumps({"sweep": "resident waves per CU", "workload": w.name,
                          "pass": "average only" if args.average_only else "fused",
                          "waves_per_cu": c, "gbps_median": round(sorted(res[c])[1], 1),
                          "gbps_rounds": [round(x, 1) for x in res[c]],
                          "steps_per_round": args.steps}), flush=True)


def run_program(name, argv):
    """Builds one of the measurement programs beside bench.py (before any GPU
    work in this process) and runs it as a child process."""
    import importlib.util
    spec = importlib.util.spec_from_file_location(
        "rip_build", os.path.join(ROOT, "paper_1909_08029_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    exe = mod.build_bench_program(name)
    sys.exit(subprocess.run([exe, *argv]).returncode)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=5, choices=[1, 2, 3, 4, 5],
                    help="workload (default 5, the largest: 8 x 1.3B bf16, two groups of four)")
    ap.add_argument("--layout", default="flat", choices=["flat", "separate"])
    ap.add_argument("--grad-ring", type=int, default=None)
    ap.add_argument("--schedule", default=None,
                    help="replace the workload's schedule by one of the paper's policies: "
                         "random_gb, gd, gd_filter, inter_intra, static, adpsgd, allreduce")
    ap.add_argument("--max-blocks", type=int, default=0)
    ap.add_argument("--blocks-per-cu", type=int, default=0,
                    help="resident workgroups per CU (0 = the library's per-shape default)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--unfused", action="store_true",
                    help="ablation: rip_local_step then a pure rip_preduce per step "
                         "(two passes over memory; reported with its own bytes)")
    ap.add_argument("--graph", action="store_true",
                    help="fixed schedules only (static, rule, table; no straggler): capture "
                         "one period of fused steps into a HIP graph and replay it, so the "
                         "host launches once per period instead of once per step")
    ap.add_argument("--groups", type=int, default=0,
                    help="replace the schedule by one table row of consecutive groups of this "
                         "size, everyone eligible: every unit of one shape")
    ap.add_argument("--momentum", type=float, default=None,
                    help="override the workload's momentum")
    ap.add_argument("--average-only", action="store_true",
                    help="with --sweep-caps: pure P-Reduce launches, no local update")
    ap.add_argument("--sweep-caps", default=None,
                    help="comma-separated resident waves per CU: time --steps steps at each "
                         "cap in one process, interleaved over three rounds; one JSON line "
                         "per cap instead of the benchmark line")
    ap.add_argument("--native", action="store_true",
                    help="only run bench_native.hip (the C ABI from a C++ loop, no Python or "
                         "torch) on the workload's shape: configs 1, 2, 3 and 5")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain device copy of known size (to scale HBM counters)")
    ap.add_argument("--ceiling", action="store_true",
                    help="only run bench_ceiling.hip, bare HBM streams of the kernel's access "
                         "shapes (random vs zero data)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: every replica of the P-Reduce path lives in one "
              "MI355X's HBM and this library has no multi-GPU path; run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    if args.ceiling:
        run_program("bench_ceiling", [])

    if args.native:
        shapes = {1: ["--replicas", "4", "--params", "1048576", "--fixed", "0,1,2"],
                  2: ["--replicas", "16", "--params", "25600000", "--group", "4"],
                  3: ["--replicas", "16", "--params", "138357544", "--group", "8",
                      "--momentum", "0.9"],
                  5: ["--replicas", "8", "--params", "1300000000", "--group", "4", "--bf16"]}
        if args.config not in shapes:
            err("--native runs the fixed-schedule workloads only (configs 1, 2, 3, 5)")
            sys.exit(2)
        run_program("bench_native", [*shapes[args.config], "--steps", str(args.steps),
                                     "--warmup", str(args.warmup)])

    import torch
    import paper_1909_08029_amd as rip
    from seedgen import DTYPE_BF16
    from seedgen import workloads as wl

    if not torch.cuda.is_available():
        err("no GPU visible")
        sys.exit(1)
    torch.cuda.set_device(0)
    if args.calibrate_copy:
        n = 1 << 30                                    # 4 GiB of fp32 each way
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "copy", "bytes_read_per_launch": 4 * n,
                          "bytes_written_per_launch": 4 * n, "launches": 5}), flush=True)
        return
    w = wl.WORKLOADS[args.config]
    if args.grad_ring:
        w = wl.scaled(w, w.seg_numel, grad_ring=args.grad_ring)
    if args.schedule:
        w = wl.with_schedule(w, args.schedule)
    if args.groups:
        k = args.groups
        w = wl.scaled(w, w.seg_numel, name=f"{w.name}_groups{k}", straggler_every=None,
                      sched=dict(mode=wl.TABLE, table=[[tuple(range(i, i + k))
                                                        for i in range(0, w.n - w.n % k, k)]]))
    if args.momentum is not None:
        w = wl.scaled(w, w.seg_numel, name=f"{w.name}_mom{args.momentum:g}",
                      momentum=args.momentum)
    err(f"[bench] workload {w.name}: N={w.n} P={w.numel} layout={args.layout}")
    if args.max_blocks:
        rip.rip_set_max_blocks(args.max_blocks)
    if args.blocks_per_cu:
        rip.rip_set_blocks_per_cu(args.blocks_per_cu)

    st = wl.DeviceState(w, args.layout)
    st.fill()
    handles = [rip.Replicas(st.param, gs, st.mom) for gs in st.grad_sets]
    sched_kw = dict(w.sched)
    sched = rip.Scheduler(w.n, sched_kw.pop("mode"), **sched_kw)
    torch.cuda.synchronize()
    err("[bench] inputs resident")

    stream = torch.cuda.current_stream()
    t = 0
    if args.sweep_caps:
        sweep_caps(args, w, rip, handles, stream)
        return

    stats = dict(steps=0, updates=0, groups=0, members=0, empty=0)

    opt = dict(momentum=w.momentum, stream=stream, weight_decay=w.weight_decay,
               nesterov=w.nesterov)
    eligible = [w.eligible(i) for i in range(args.warmup + args.steps)]

    def one_step():
        """One step; returns its (active, groups).  Bytes and statistics are
        worked out after the timed window, so the loop holds only the calls."""
        nonlocal t
        h = handles[w.grad_slot(t)]
        kernels = 0
        if args.unfused:
            active, groups = rip.rip_schedule_groups(sched, t, eligible[t])
            if active:
                rip.rip_local_step(h, active, w.lr, **opt)
                kernels += rip.rip_last_launch_count()
            rip.rip_preduce(h, groups, stream=stream)
        else:
            # group generation and the fused launch in one library call
            active, groups = rip.rip_step(sched, h, t, w.lr, eligible=eligible[t], **opt)
        kernels += rip.rip_last_launch_count()
        t += 1
        return active, groups, kernels

    def account(done):
        """Algorithmic bytes and kernel launches of the timed steps."""
        total, launched = 0, 0
        for active, groups, kernels in done:
            stats["steps"] += 1
            stats["updates"] += len(active)
            stats["groups"] += sum(1 for g in groups if len(g) > 1)
            stats["members"] += sum(len(g) for g in groups if len(g) > 1)
            work = bool(active) or any(len(g) > 1 for g in groups)
            stats["empty"] += 0 if work else 1
            total += (w.alg_bytes_unfused if args.unfused else w.alg_bytes)(active, groups)
            launched += kernels
        return total, launched

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    err(f"[bench] {args.warmup} warmup steps done")

    graph_period = 0
    if args.graph:
        graph_period, per_step_bytes, span_ms, wall, launches = graph_steps(
            args, w, rip, handles, sched, t, stream, stats)
        total_bytes = sum(per_step_bytes)
    else:
        # One event pair brackets the whole timed window on the launch
        # stream: markers between steps would add packets to the stream.
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        done = [None] * args.steps
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        e0.record(stream)
        for i in range(args.steps):
            done[i] = one_step()
        e1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        span_ms = e0.elapsed_time(e1)
        total_bytes, launches = account(done)
    err(f"[bench] {args.steps} timed steps: {wall * 1e3:.2f} ms wall, "
        f"{span_ms:.2f} ms GPU span, {launches} launches")

    # host scheduling cost alone (fresh scheduler, same steps)
    sched_kw = dict(w.sched)
    sch2 = rip.Scheduler(w.n, sched_kw.pop("mode"), **sched_kw)
    h0 = time.perf_counter()
    for i in range(args.steps):
        rip.rip_schedule_groups(sch2, i, w.eligible(i))
    sched_us = (time.perf_counter() - h0) / args.steps * 1e6

    value = total_bytes / wall / 1e9
    mean_launch_bytes = total_bytes / max(1, launches)
    mean_kernel_ms = span_ms / max(1, launches)
    achieved = total_bytes / (span_ms * 1e-3) / 1e9 if span_ms > 0 else 0.0
    traffic = None
    if args.layout == "flat" and not args.grad_ring and not args.unfused:
        traffic = load_traffic(w.name, mean_launch_bytes)

    cpu = None
    if not args.no_cpu_baseline:
        err("[bench] timing the CPU oracle on a bounded sample")
        cpu = cpu_baseline(w)

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # the arithmetic type: every value is computed in fp32, whatever the
        # storage type (config.storage)
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "n_replicas": w.n,
            "params_per_replica": w.numel,
            "segments": len(w.seg_numel),
            "layout": args.layout,
            "storage": "bf16" if w.dtype == DTYPE_BF16 else "fp32",
            "optimizer": f"sgd lr={w.lr}" + (f" momentum={w.momentum}" if w.momentum else ""),
            "schedule": args.schedule or SCHEDULE_NAMES[w.sched["mode"]],
            "schedule_stats": {
                "local_updates_per_step": round(stats["updates"] / max(1, stats["steps"]), 3),
                "groups_per_step": round(stats["groups"] / max(1, stats["steps"]), 3),
                "mean_group_size": round(stats["members"] / max(1, stats["groups"]), 3),
                "steps_without_work": stats["empty"],
                "local_updates_per_s": round(stats["updates"] / wall, 1),
            },
            "grad_ring": w.grad_ring,
            "pct_of_hbm_peak": round(100.0 * value / HBM_PEAK_GBPS, 2),
            "host_schedule_us_per_step": round(sched_us, 2),
            "parallelism": "single-gpu",
            "pass": "unfused (local step, then P-Reduce)" if args.unfused else "fused",
            "launch": (f"hip graph of {graph_period} steps, replayed" if graph_period
                       else "one library call per step"),
            **({"note": w.note} if w.note else {}),
        },
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": traffic,
            "alg_bytes_per_launch": int(round(mean_launch_bytes)),
            "mean_kernel_us": round(mean_kernel_ms * 1e3, 2),
            "launches_timed": launches,
            "kernel_time": "GPU span of the timed window (one HIP event pair on the launch "
                           "stream) / kernel launches in it",
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
