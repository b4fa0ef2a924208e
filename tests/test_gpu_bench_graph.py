"""The benchmark's HIP-graph mode computes the same steps as the oracle.

``bench.py --graph`` schedules one period of a fixed schedule, captures its
fused launches into a HIP graph and replays it; its numbers only mean
something if every replay runs the steps the schedule prescribes.  This runs
that code on small fixed-schedule workloads (a table with a lone updater,
a static schedule over a gradient ring of two, momentum in bf16) and compares
every element of every replica with the oracle after all replays.
"""
import argparse

import numpy as np
import pytest

from seedgen import DTYPE_BF16, DTYPE_F32
from seedgen import workloads as wl

from gpu_util import compare, log, oracle_windows

pytestmark = pytest.mark.gpu

CASES = [
    ("table", wl.Workload("graph_table", 4, [3 * 4096 + 7], DTYPE_F32, 0.1, 0.0, 0.01,
                          dict(mode=wl.TABLE, table=[[(0, 1, 2)]]), 1, 71)),
    ("static", wl.Workload("graph_static", 8, [5000, 4099], DTYPE_F32, 0.1, 0.0, 0.01,
                           dict(mode=wl.STATIC, seed=9, group_size=4, period=4), 1, 72)),
    ("static_bf16_mom", wl.Workload("graph_static_bf16", 8, [8 * 1024 + 3], DTYPE_BF16, 2.0, 0.9,
                                    0.01, dict(mode=wl.STATIC, seed=10, group_size=2, period=2),
                                    1, 73, param_sigma=0.05)),
]


@pytest.mark.parametrize("name,w", CASES, ids=[c[0] for c in CASES])
def test_graph_replays_match_oracle(name, w):
    import torch
    import bench
    import paper_1909_08029_amd as rip
    torch.cuda.set_device(0)
    st = wl.DeviceState(w)
    st.fill()
    handles = [rip.Replicas(st.param, gs, st.mom) for gs in st.grad_sets]
    kw = dict(w.sched)
    sched = rip.Scheduler(w.n, kw.pop("mode"), **kw)
    stats = dict(steps=0, updates=0, groups=0, members=0, empty=0)
    args = argparse.Namespace(steps=8, unfused=False)
    torch.cuda.synchronize()
    L, per_step, span_ms, _, kernels = bench.graph_steps(args, w, rip, handles, sched, 0,
                                                         torch.cuda.current_stream(), stats)
    torch.cuda.synchronize()
    log(f"case graph {name}: period {L}, {args.steps} timed steps")
    assert len(per_step) == args.steps and stats["steps"] == args.steps
    assert span_ms > 0
    assert kernels >= sum(1 for b in per_step if b > 0)
    total = sum(per_step)
    # one untimed replay, then steps / L timed ones: the schedule of steps 0 .. L + steps - 1
    ref = rip.Scheduler(w.n, dict(w.sched)["mode"],
                        **{k: v for k, v in w.sched.items() if k != "mode"})
    schedule = [rip.rip_schedule_groups(ref, t) for t in range(L + args.steps)]
    assert total == sum(w.alg_bytes(a, g) for a, g in schedule[L:])
    (po, vo), = oracle_windows(w, schedule, [(0, w.numel)])
    for r in range(w.n):
        compare(st.window("param", r, 0, w.numel), po[r], w.dtype, f"{name} param r={r}")
        if w.momentum:
            compare(st.window("mom", r, 0, w.numel), vo[r], w.dtype, f"{name} mom r={r}")
    for h in handles:
        h.close()


@pytest.mark.parametrize("average_only", [False, True])
def test_sweep_caps_mode_reports_every_cap(average_only, capsys):
    """bench.py --sweep-caps runs the steps at each residency cap and prints
    one JSON line per cap, with the rate of each of its three rounds."""
    import json
    import torch
    import bench
    import paper_1909_08029_amd as rip
    torch.cuda.set_device(0)
    w = CASES[1][1]
    st = wl.DeviceState(w)
    st.fill()
    handles = [rip.Replicas(st.param, gs, st.mom) for gs in st.grad_sets]
    args = argparse.Namespace(steps=3, sweep_caps="6,10", average_only=average_only)
    log(f"case sweep caps average_only={average_only}")
    bench.sweep_caps(args, w, rip, handles, torch.cuda.current_stream())
    torch.cuda.synchronize()
    lines = [json.loads(l) for l in capsys.readouterr().out.splitlines() if l.startswith("{")]
    assert [d["waves_per_cu"] for d in lines] == [6, 10]
    assert all(d["gbps_median"] > 0 and len(d["gbps_rounds"]) == 3 for d in lines)
    for h in handles:
        h.close()
