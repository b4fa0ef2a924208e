#!/usr/bin/env python3
"""Throughput of the fused local update + P-Reduce step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config C]

A step is one pass of the whole hot path over one batch of synthetic input:
the host group schedule for step t, then one launch of the fused kernel that
applies every active worker's local update and the P-Reduce of every group.
The default workload is 16 fp32 replicas of a 25.6M-parameter (ResNet-50
sized) model with a seeded static schedule of four groups of four (the
configuration the headline metric is quoted on).

Prints one JSON line (stdout).  ``value`` is algorithmic HBM bytes of the K
timed steps divided by their wall time, inputs resident in HBM before timing
starts.  ``roofline.achieved`` is the algorithmic bytes of one launch over the
kernel's mean duration measured with HIP events on its stream, around every
fifth timed step (``--event-every``).
``cpu_baseline`` times the CPU oracle on a bounded sample of the same
workload.  Progress goes to stderr.
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
    """The oracle as it stands, single-threaded numpy, on one window of every
    replica, for as many steps of the workload's schedule as fit the budget
    (at least 2).  Times the update + group averaging only."""
    import numpy as np
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
    while steps < 2 or (spent < seconds and steps < w.steps):
        active, groups = sch.step(steps, w.eligible(steps))
        g = grad(w.grad_slot(steps))
        t0 = time.perf_counter()
        p, v = op.step(p, g, v, groups, active, w.lr, w.momentum or None, dt, True,
                       w.weight_decay, w.nesterov)
        spent += time.perf_counter() - t0
        nbytes += sub.alg_bytes(active, groups)
        steps += 1
    return dict(value=round(nbytes / spent / 1e9, 4), unit="GB/s", cores=1, kind="oracle",
                sample=f"{steps} steps of the workload schedule on elements [0, {width}) of all "
                       f"{w.n} replicas ({100.0 * width / w.numel:.1f}% of each replica), "
                       f"numpy single-threaded on {host_cpu()}; "
                       f"{spent:.1f} s timed, update+average only")


def graph_steps(args, w, rip, handles, sched, t, stream, stats):
    """Times args.steps fused steps as replays of one captured period.

    Only a schedule that repeats is replayable: the steps of one period
    (a multiple of the gradient ring) are scheduled by the library, their
    launches captured into a HIP graph, and a second scheduler checks that the
    next period schedules exactly the same groups.  Every replay then runs
    those steps, as a static schedule prescribes.  Returns (period, total
    bytes, bytes per step, kernel ms per step, wall seconds)."""
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
    with torch.cuda.graph(g):
        cap = torch.cuda.current_stream()
        for i, (active, groups) in enumerate(period):
            rip.rip_preduce(handles[w.grad_slot(t + i)], groups, active, lr=w.lr, stream=cap,
                            **opt)
    torch.cuda.synchronize()
    g.replay()                                     # first execution, untimed
    torch.cuda.synchronize()
    step_bytes = [w.alg_bytes(a, gr) for a, gr in period]
    reps = args.steps // L
    events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(reps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1 in events:
        e0.record(stream)
        g.replay()
        e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_step_bytes, kern_ms = [], []
    for e0, e1 in events:
        ms = e0.elapsed_time(e1) / L               # graph time spread over its launches
        for (active, groups), b in zip(period, step_bytes):
            per_step_bytes.append(b)
            kern_ms.append(ms)
            stats["steps"] += 1
            stats["updates"] += len(active)
            stats["groups"] += sum(1 for x in groups if len(x) > 1)
            stats["members"] += sum(len(x) for x in groups if len(x) > 1)
            stats["empty"] += 0 if (active or any(len(x) > 1 for x in groups)) else 1
    del g
    return L, sum(per_step_bytes), per_step_bytes, kern_ms, wall


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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=2, choices=[1, 2, 3, 4, 5])
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
    ap.add_argument("--event-every", type=int, default=5,
                    help="bracket every n-th timed step with HIP events for the kernel's "
                         "launch duration (1 = every step; each event pair costs wall time)")
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
                    help="only run the C-ABI-only program (no Python or torch in the loop) on "
                         "the workload's shape: configs 1, 2, 3 and 5")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain device copy of known size (to scale HBM counters)")
    ap.add_argument("--ceiling", action="store_true",
                    help="only run the bare-stream HBM ceiling program (random vs zero data)")
    ap.add_argument("--ceiling-xcd", action="store_true",
                    help="only run the ceiling program's XCD tile-placement sweep")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: every replica of the P-Reduce path lives in one "
              "MI355X's HBM and this library has no multi-GPU path; run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    if args.ceiling or args.ceiling_xcd:
        exe = os.path.join(ROOT, "paper_1909_08029_amd", "stream_ceiling")
        if not os.path.exists(exe):
            err("stream_ceiling is not built; run __graft_entry__.build()")
            sys.exit(1)
        sys.exit(subprocess.run([exe] + (["xcd"] if args.ceiling_xcd else [])).returncode)

    if args.native:
        exe = os.path.join(ROOT, "paper_1909_08029_amd", "rip_bench_native")
        if not os.path.exists(exe):
            err("rip_bench_native is not built; run __graft_entry__.build()")
            sys.exit(1)
        shapes = {1: ["--replicas", "4", "--params", "1048576", "--fixed", "0,1,2"],
                  2: ["--replicas", "16", "--params", "25600000", "--group", "4"],
                  3: ["--replicas", "16", "--params", "138357544", "--group", "8",
                      "--momentum", "0.9"],
                  5: ["--replicas", "8", "--params", "1300000000", "--group", "4", "--bf16"]}
        if args.config not in shapes:
            err("--native runs the fixed-schedule workloads only (configs 1, 2, 3, 5)")
            sys.exit(2)
        sys.exit(subprocess.run([exe, *shapes[args.config], "--steps", str(args.steps),
                                 "--warmup", str(args.warmup)]).returncode)

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

    def one_step(ev=None, timed=False):
        nonlocal t
        h = handles[w.grad_slot(t)]
        opt = dict(momentum=w.momentum, stream=stream, weight_decay=w.weight_decay,
                   nesterov=w.nesterov)
        if ev is not None:
            ev[0].record(stream)
        if args.unfused:
            active, groups = rip.rip_schedule_groups(sched, t, w.eligible(t))
            if active:
                rip.rip_local_step(h, active, w.lr, **opt)
            rip.rip_preduce(h, groups, stream=stream)
        else:
            # group generation and the fused launch in one library call
            active, groups = rip.rip_step(sched, h, t, w.lr, eligible=w.eligible(t), **opt)
        if ev is not None:
            ev[1].record(stream)
        if timed:
            stats["steps"] += 1
            stats["updates"] += len(active)
            stats["groups"] += sum(1 for g in groups if len(g) > 1)
            stats["members"] += sum(len(g) for g in groups if len(g) > 1)
            stats["empty"] += 0 if (active or any(len(g) > 1 for g in groups)) else 1
        t += 1
        if args.unfused:
            return w.alg_bytes_unfused(active, groups)
        return w.alg_bytes(active, groups)

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    err(f"[bench] {args.warmup} warmup steps done")

    graph_period = 0
    if args.graph:
        graph_period, total_bytes, per_step_bytes, kern_ms, wall = graph_steps(
            args, w, rip, handles, sched, t, stream, stats)
        launched = [(b, ms) for b, ms in zip(per_step_bytes, kern_ms) if b > 0]
    else:
        # Every event is a marker packet in the stream; bracketing every step
        # cost about 1% of the wall-clock rate, so only every n-th step is
        # bracketed (its launch duration is the kernel's, as before).
        every = max(1, args.event_every)
        events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  if i % every == 0 else None for i in range(args.steps)]
        total_bytes = 0
        per_step_bytes = []
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            b = one_step(events[i], timed=True)
            per_step_bytes.append(b)
            total_bytes += b
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        launched = [(b, ev[0].elapsed_time(ev[1])) for b, ev in zip(per_step_bytes, events)
                    if ev is not None and b > 0]
    err(f"[bench] {args.steps} timed steps: {wall * 1e3:.2f} ms wall")

    # host scheduling cost alone (fresh scheduler, same steps)
    sched_kw = dict(w.sched)
    sch2 = rip.Scheduler(w.n, sched_kw.pop("mode"), **sched_kw)
    h0 = time.perf_counter()
    for i in range(args.steps):
        rip.rip_schedule_groups(sch2, i, w.eligible(i))
    sched_us = (time.perf_counter() - h0) / args.steps * 1e6

    value = total_bytes / wall / 1e9
    mean_launch_bytes = sum(b for b, _ in launched) / max(1, len(launched))
    mean_kernel_ms = sum(ms for _, ms in launched) / max(1, len(launched))
    median_kernel_ms = sorted(ms for _, ms in launched)[len(launched) // 2] if launched else 0.0
    achieved = mean_launch_bytes / (mean_kernel_ms * 1e-3) / 1e9 if launched else 0.0
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
        },
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": traffic,
            "alg_bytes_per_launch": int(mean_launch_bytes),
            "mean_kernel_us": round(mean_kernel_ms * 1e3, 2),
            "median_kernel_us": round(median_kernel_ms * 1e3, 2),
            "launches_timed": len(launched),
            "timed_every_nth_step": 1 if graph_period else max(1, args.event_every),
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
