"""Shared helpers of the GPU parity tests: drive the HIP path through the
C-ABI binding, drive the oracle on the same seeded inputs, compare."""
from __future__ import annotations

import sys
from typing import List, Optional, Sequence, Tuple

import numpy as np

from seedgen import DTYPE_BF16
from seedgen import workloads as wl

TOL = {0: 1e-6, 1: 1e-2}     # max relative error: fp32 storage, bf16 storage


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def to_f32(x: np.ndarray, dtype: int) -> np.ndarray:
    if dtype == DTYPE_BF16:
        return (x.astype(np.uint32) << np.uint32(16)).view(np.float32)
    return x


def max_ulp(gpu: np.ndarray, ora: np.ndarray, dtype: int) -> int:
    """Largest distance in units in the last place between matching elements
    (bit patterns mapped to a monotone integer order; +0 and -0 are 0 apart)."""
    if gpu.size == 0:
        return 0
    if dtype == DTYPE_BF16:
        bg, bo, sign = gpu.view(np.uint16).astype(np.int64), ora.view(np.uint16).astype(np.int64), 1 << 15
    else:
        bg, bo, sign = gpu.view(np.uint32).astype(np.int64), ora.view(np.uint32).astype(np.int64), 1 << 31

    def order(b):
        return np.where(b >= sign, sign - b, b)
    return int(np.abs(order(bg) - order(bo)).max())


def compare(gpu: np.ndarray, ora: np.ndarray, dtype: int, what: str = ""):
    """Returns (max relative error, bit mismatches); asserts the tolerance and
    bit-exactness (the kernels follow the oracle's operation order).  Failure
    messages also give the largest ulp distance."""
    assert gpu.shape == ora.shape, (gpu.shape, ora.shape)
    g, o = to_f32(gpu, dtype).astype(np.float64), to_f32(ora, dtype).astype(np.float64)
    denom = np.maximum(np.abs(o), 2.0 ** -126)
    with np.errstate(invalid="ignore"):      # inf - inf where both sides are inf
        rel = np.abs(g - o) / denom
    rel[(g == o)] = 0.0
    max_rel = float(rel.max()) if rel.size else 0.0
    bits_g = gpu.view(np.uint16 if dtype == DTYPE_BF16 else np.uint32)
    bits_o = ora.view(np.uint16 if dtype == DTYPE_BF16 else np.uint32)
    mism = int(np.count_nonzero(bits_g != bits_o))
    if max_rel > TOL[dtype] or mism:
        ulp = max_ulp(gpu, ora, dtype)
        assert max_rel <= TOL[dtype], \
            f"{what}: max rel err {max_rel:.3e} > {TOL[dtype]} ({mism} bit mismatches, max {ulp} ulp)"
        assert mism == 0, f"{what}: {mism} bit mismatches (max rel err {max_rel:.3e}, max {ulp} ulp)"
    return max_rel, mism


def oracle_scheduler(w: wl.Workload):
    from oracle import sched as osd
    kw = dict(w.sched)
    mode = kw.pop("mode")
    return osd.Scheduler(w.n, mode, **kw)


def rip_scheduler(w: wl.Workload):
    import paper_1909_08029_amd as rip
    kw = dict(w.sched)
    mode = kw.pop("mode")
    return rip.Scheduler(w.n, mode, **kw)


class DeviceRun:
    """The HIP path on a workload: device state, one replicas handle per
    gradient-ring slot, the library's scheduler."""

    def __init__(self, w: wl.Workload, layout: str = "flat", fused: bool = True):
        import paper_1909_08029_amd as rip
        self.w, self.fused = w, fused
        self.state = wl.DeviceState(w, layout)
        self.state.fill()
        self.handles = [rip.Replicas(self.state.param, gs, self.state.mom)
                        for gs in self.state.grad_sets]
        self.sched = rip_scheduler(w)
        self.schedule: List[Tuple[List[int], List[Tuple[int, ...]]]] = []
        self.launches: List[int] = []   # kernels each step enqueued
        self.t = 0

    def step(self):
        import paper_1909_08029_amd as rip
        w = self.w
        active, groups = rip.rip_schedule_groups(self.sched, self.t, w.eligible(self.t))
        h = self.handles[w.grad_slot(self.t)]
        opt = dict(weight_decay=w.weight_decay, nesterov=w.nesterov)
        if self.fused:
            rip.rip_preduce(h, groups, active, lr=w.lr, momentum=w.momentum, **opt)
            kernels = rip.rip_last_launch_count()
        else:
            kernels = 0
            if active:
                rip.rip_local_step(h, active, w.lr, w.momentum, **opt)
                kernels = rip.rip_last_launch_count()
            rip.rip_preduce(h, groups)
            kernels += rip.rip_last_launch_count()
        self.schedule.append((active, groups))
        self.launches.append(kernels)
        self.t += 1

    def run(self, steps: int):
        for _ in range(steps):
            self.step()


def oracle_windows(w: wl.Workload, schedule, windows: Sequence[Tuple[int, int]],
                   fused: bool = True):
    """The oracle's state after ``schedule`` on each flat window [a, b)."""
    from oracle import preduce as op
    dt = op.BF16 if w.dtype == DTYPE_BF16 else op.F32
    out = []
    for a, b in windows:
        p, grad, v = wl.host_inputs(w, a, b)
        for t, (active, groups) in enumerate(schedule):
            p, v = op.step(p, grad(w.grad_slot(t)), v, groups, active, w.lr,
                           w.momentum if w.momentum else None, dt, fused,
                           w.weight_decay, w.nesterov)
        out.append((p, v))
    return out


def sample_windows(P: int, count: int, width: int, seed: int, must: Sequence[int] = ()):
    """Windows [a, a+width) covering the first and last elements, the given
    boundaries, and random positions."""
    rs = np.random.default_rng(seed)
    width = min(width, P)
    starts = {0, P - width}
    for m in must:
        starts.add(int(min(max(0, m - width // 2), P - width)))
    while len(starts) < count and len(starts) < P - width + 1:
        starts.add(int(rs.integers(0, P - width + 1)))
    return sorted((a, a + width) for a in starts)


def check_against_oracle(run: DeviceRun, windows, label: str):
    w = run.w
    ora = oracle_windows(w, run.schedule, windows, run.fused)
    worst = 0.0
    for (a, b), (p, v) in zip(windows, ora):
        for r in range(w.n):
            mr, _ = compare(run.state.window("param", r, a, b), p[r], w.dtype,
                            f"{label} param r={r} [{a},{b})")
            worst = max(worst, mr)
            if v is not None:
                mr, _ = compare(run.state.window("mom", r, a, b), v[r], w.dtype,
                                f"{label} mom r={r} [{a},{b})")
    return worst
