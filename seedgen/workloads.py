"""Synthetic workloads shaped like the paper's models (recipes only).

The paper trains VGG-16 and ResNet-50 (Sec. 7.1.2); its datasets and weights
are not needed to exercise the synchronization path, whose cost depends only
on the number of replicas, the parameter count, the storage type and the
schedule.  Each workload below is N replicas of a flat parameter buffer (or
a set of layer-sized segments) with seeded synthetic contents:

  parameters  ~ normal-like, sigma 1     key(seed, TAG_PARAM, replica, 0)
  gradients   ~ normal-like, sigma_g     key(seed, TAG_GRAD, replica, ring slot)
  momentum    zeros

Gradients come from a ring of ``grad_ring`` resident sets; step t reads set
t mod grad_ring, so consecutive steps see different gradients while every
input is in device memory before timing starts.

This module holds recipes and device/CPU fills; none of the method's
arithmetic.  Schedules are produced by each side's own scheduler.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import DTYPE_BF16, DTYPE_F32, TAG_GRAD, TAG_PARAM, normal, fill_normal_gpu

# VGG-16 (ImageNet, 224x224) trainable tensors per layer, weight + bias:
# 13 convolutions then 3 fully connected layers; 138,357,544 in total.
VGG16_SEGMENTS = [1792, 36928, 73856, 147584, 295168, 590080, 590080, 1180160,
                  2359808, 2359808, 2359808, 2359808, 2359808,
                  102764544, 16781312, 4097000]
RESNET50_PARAMS = 25_600_000

# scheduler modes (values of the C ABI; the oracle uses the same numbers)
TABLE, STATIC, RANDOM_GB, GD, SCRIPTED, RULE, INTER_INTRA, ADPSGD = range(8)


@dataclass
class Workload:
    name: str
    n: int
    seg_numel: List[int]
    dtype: int
    lr: float
    momentum: float
    grad_sigma: float
    sched: Dict
    steps: int
    seed: int
    straggler_every: Optional[int] = None   # worker 0 eligible once every k steps
    param_sigma: float = 1.0
    grad_ring: int = 2
    note: str = ""
    weight_decay: float = 0.0
    nesterov: bool = False

    @property
    def numel(self) -> int:
        return sum(self.seg_numel)

    @property
    def esize(self) -> int:
        return 2 if self.dtype == DTYPE_BF16 else 4

    def eligible(self, t: int) -> Optional[List[bool]]:
        if self.straggler_every is None:
            return None
        e = [True] * self.n
        e[0] = (t % self.straggler_every == 0)
        return e

    def grad_slot(self, t: int) -> int:
        return t % self.grad_ring

    def alg_bytes(self, active: Sequence[int], groups: Sequence[Sequence[int]]) -> int:
        """Minimum HBM bytes of one fused step: an active replica reads w, g
        (and v) and writes w (and v); a group member that did not update reads
        and writes w; everything else is untouched."""
        act = set(active)
        members = {m for g in groups for m in g}
        s, P = self.esize, self.numel
        per_active = 2 * s + s + (2 * s if self.momentum else 0)
        b = sum(per_active for r in act) + sum(2 * s for r in members - act)
        # an active worker in a singleton group or alone: same bytes; a
        # singleton group of a non-active worker is the identity (0 bytes)
        b -= sum(2 * s for g in groups if len(g) == 1 and g[0] not in act)
        return b * P

    def alg_bytes_unfused(self, active: Sequence[int], groups: Sequence[Sequence[int]]) -> int:
        """Minimum HBM bytes of the same step done as two passes: the local
        update of every active replica (read w, g [, v], write w [, v]), then
        a P-Reduce that reads and writes w of every member of a group of two
        or more."""
        s, P = self.esize, self.numel
        per_active = 2 * s + s + (2 * s if self.momentum else 0)
        b = per_active * len(set(active))
        b += sum(2 * s * len(g) for g in groups if len(g) > 1)
        return b * P


WORKLOADS: Dict[int, Workload] = {
    1: Workload("c1_n4_p1m_fp32_fixed", 4, [1_048_576], DTYPE_F32, 0.1, 0.0, 0.01,
                dict(mode=TABLE, table=[[(0, 1, 2)]]), 10, 1,
                note="fits the 256 MB Infinity Cache: not an HBM measurement"),
    2: Workload("c2_n16_p25.6m_fp32_static4x4", 16, [RESNET50_PARAMS], DTYPE_F32, 0.1, 0.0, 0.01,
                dict(mode=STATIC, seed=2, group_size=4, period=4), 100, 2),
    3: Workload("c3_n16_p138m_vgg16seg_fp32_mom_static2x8", 16, list(VGG16_SEGMENTS), DTYPE_F32,
                0.1, 0.9, 0.01, dict(mode=STATIC, seed=3, group_size=8, period=4), 50, 3),
    4: Workload("c4_n32_p25.6m_fp32_randomgb_k2to8_straggler", 32, [RESNET50_PARAMS], DTYPE_F32,
                0.1, 0.0, 0.01, dict(mode=RANDOM_GB, seed=4, kmin=2, kmax=8), 200, 4,
                straggler_every=4),
    5: Workload("c5_n8_p1.3b_bf16_static2x4", 8, [1_300_000_000], DTYPE_BF16, 0.01, 0.0, 1e-3,
                dict(mode=STATIC, seed=5, group_size=4, period=4), 20, 5),
}


# The scheduling policies the paper compares, as schedules of the same fused
# kernel on a workload's replicas: random groups with Group Buffers (Step 3 of
# Fig. 4), Global Division with and without the slowdown filter (Sec. 5.1,
# Sec. 5.3), Inter-Intra synchronization with 4 workers per node (Sec. 5.2),
# a seeded static schedule of groups of 4 (Sec. 4.2), AD-PSGD's random pairs
# (Fig. 3) and All-Reduce as one group of every worker.  Group sizes 2..8
# follow the heterogeneous workload; the filter threshold C_thres (a tunable
# constant in the paper) is 4, the straggler's update interval.
SCHEDULE_VARIANTS = ("random_gb", "gd", "gd_filter", "inter_intra", "static", "adpsgd",
                     "allreduce")


def with_schedule(w: Workload, name: str) -> Workload:
    """The workload with its schedule replaced by one of SCHEDULE_VARIANTS."""
    n, seed = w.n, w.seed
    sched = {
        "random_gb": dict(mode=RANDOM_GB, seed=seed, kmin=2, kmax=8),
        "gd": dict(mode=GD, seed=seed, kmin=2, kmax=8),
        "gd_filter": dict(mode=GD, seed=seed, kmin=2, kmax=8, c_thres=4),
        "inter_intra": dict(mode=INTER_INTRA, seed=seed, kmin=2, kmax=8, c_thres=4,
                            n_nodes=max(1, n // 4)),
        "static": dict(mode=STATIC, seed=seed, group_size=4 if n % 4 == 0 else 1, period=4),
        "adpsgd": dict(mode=ADPSGD, seed=seed),
        "allreduce": dict(mode=TABLE, table=[[tuple(range(n))]]),
    }
    if name not in sched:
        raise ValueError(f"unknown schedule {name!r}; choose from {SCHEDULE_VARIANTS}")
    return scaled(w, w.seg_numel, sched=sched[name], name=f"{w.name}_{name}")


def scaled(w: Workload, numel: Sequence[int], **kw) -> Workload:
    """Same recipe with other segment sizes (for small parity cases)."""
    d = dict(w.__dict__)
    d["seg_numel"] = list(numel)
    d.update(kw)
    return Workload(**d)


# ---------------------------------------------------------------------------
# device buffers (torch only allocates and hands out pointers)
# ---------------------------------------------------------------------------
class DeviceState:
    """All replicas of a workload in device memory.

    layout "flat": one buffer per replica and kind, segments are views into
    it back to back (the zero-copy form of flattening the model, Sec. 6.1).
    layout "separate": every segment is its own allocation.
    layout "arena": one allocation per kind holding every replica's flat
    buffer at a pitch of (P * element size rounded up to 256 bytes) + pad."""

    def __init__(self, w: Workload, layout: str = "flat", device: str = "cuda", pad: int = 0):
        import torch
        self.w, self.layout = w, layout
        tdt = torch.bfloat16 if w.dtype == DTYPE_BF16 else torch.float32
        P = w.numel
        offs = np.concatenate([[0], np.cumsum(w.seg_numel)]).astype(np.int64)
        self.seg_off = [int(o) for o in offs]
        nseg = len(w.seg_numel)
        pitch = ((P * w.esize + 255) // 256) * 256 + pad
        if layout == "arena" and pitch % 16:
            raise ValueError("arena pad must keep 16-byte alignment")

        def views(flat):
            return [flat[self.seg_off[s]:self.seg_off[s + 1]] for s in range(nseg)]

        def alloc_kind():
            """Returns per-replica (flat tensor or None, segment views)."""
            if layout == "arena":
                arena = torch.empty(w.n * pitch, dtype=torch.uint8, device=device)
                out = []
                for r in range(w.n):
                    flat = arena[r * pitch:r * pitch + P * w.esize].view(tdt)
                    out.append((flat, views(flat)))
                return out
            if layout == "flat":
                out = []
                for r in range(w.n):
                    flat = torch.empty(P, dtype=tdt, device=device)
                    out.append((flat, views(flat)))
                return out
            return [(None, [torch.empty(m, dtype=tdt, device=device) for m in w.seg_numel])
                    for r in range(w.n)]

        kind = alloc_kind()
        self.param_flat = [f for f, _ in kind]
        self.param = [segs for _, segs in kind]
        self.grad_sets = [[segs for _, segs in alloc_kind()] for _ in range(w.grad_ring)]
        self.mom = None
        if w.momentum:
            self.mom = [segs for _, segs in alloc_kind()]
            for segs in self.mom:
                for t in segs:
                    t.zero_()

    def fill(self):
        """Parameters and every gradient set from the seeded generator."""
        import torch
        w = self.w
        stream = torch.cuda.current_stream().cuda_stream
        for r in range(w.n):
            for s, t in enumerate(self.param[r]):
                fill_normal_gpu(t.data_ptr(), w.dtype, w.seed, TAG_PARAM, r, 0, self.seg_off[s],
                                t.numel(), w.param_sigma, stream)
        for slot, gs in enumerate(self.grad_sets):
            for r in range(w.n):
                for s, t in enumerate(gs[r]):
                    fill_normal_gpu(t.data_ptr(), w.dtype, w.seed, TAG_GRAD, r, slot,
                                    self.seg_off[s], t.numel(), w.grad_sigma, stream)

    def window(self, kind: str, r: int, a: int, b: int) -> np.ndarray:
        """Stored values of flat elements [a, b) of replica r, on the host
        (float32, or uint16 bf16 bit patterns)."""
        import torch
        segs = {"param": self.param, "mom": self.mom}[kind][r]
        parts = []
        for s, t in enumerate(segs):
            lo, hi = max(a, self.seg_off[s]), min(b, self.seg_off[s + 1])
            if lo < hi:
                parts.append(t[lo - self.seg_off[s]:hi - self.seg_off[s]])
        x = torch.cat(parts).cpu()
        if x.dtype == torch.bfloat16:
            return x.view(torch.int16).numpy().view(np.uint16)
        return x.numpy()


def host_inputs(w: Workload, a: int, b: int):
    """CPU copy of the workload's initial state on flat elements [a, b):
    (param[N, W], grad_fn(slot) -> [N, W], mom[N, W] or None)."""
    W = b - a
    param = np.stack([normal(w.seed, TAG_PARAM, r, 0, a, W, w.param_sigma, w.dtype)
                      for r in range(w.n)])
    cache = {}

    def grad(slot):
        if slot not in cache:
            cache[slot] = np.stack([normal(w.seed, TAG_GRAD, r, slot, a, W, w.grad_sigma, w.dtype)
                                    for r in range(w.n)])
        return cache[slot]

    mom = None
    if w.momentum:
        mom = np.zeros_like(param)
    return param, grad, mom
