"""Seeded random cases: the HIP path against the oracle on whole buffers.

Each case draws the replica count, ragged segment sizes (an empty one
included at times), the storage type, the optimizer (SGD or momentum, weight
decay, Nesterov), the fused or unfused form, flat or separately allocated
segments, and a two-row periodic table of random disjoint groups of any size
(lone workers, pairs, groups past the specialized sizes, everyone), with
worker 0 eligible one step in three so groups also hold members that do not
update.  Every element of every replica is compared after a few steps.
"""
import os

import numpy as np
import pytest

from seedgen import DTYPE_BF16, DTYPE_F32
from seedgen import workloads as wl

from gpu_util import DeviceRun, check_against_oracle, log

pytestmark = pytest.mark.gpu

# RIP_RANDOM_CASES raises the count for a longer one-off run; RIP_RANDOM_SCALE
# multiplies the segment sizes and RIP_RANDOM_MAX_N raises the replica count.
CASES = int(os.environ.get("RIP_RANDOM_CASES", "400"))
SCALE = int(os.environ.get("RIP_RANDOM_SCALE", "1"))
MAX_N = int(os.environ.get("RIP_RANDOM_MAX_N", "40"))


def _random_rows(rs, n, rows=2):
    table = []
    for _ in range(rows):
        order = [int(x) for x in rs.permutation(n)]
        keep = order[:int(rs.integers(1, n + 1))]
        groups, i = [], 0
        while i < len(keep):
            k = int(rs.integers(1, min(len(keep) - i, 20) + 1))
            if rs.random() < 0.1:
                k = len(keep) - i                       # the rest in one group
            groups.append(tuple(sorted(keep[i:i + k])))
            i += k
        table.append(groups)
    return table


def _case(case):
    rs = np.random.default_rng(7000 + case)
    n = int(rs.integers(1, MAX_N + 1))
    segs = [int(rs.integers(0, 9000)) * SCALE for _ in range(int(rs.integers(1, 4)))]
    if rs.random() < 0.3:
        segs.insert(int(rs.integers(0, len(segs) + 1)), 0)
    if sum(segs) == 0:
        segs[0] = int(rs.integers(1, 300))
    dtype = DTYPE_BF16 if rs.random() < 0.4 else DTYPE_F32
    mom = 0.9 if rs.random() < 0.5 else 0.0
    wd = 1e-3 if rs.random() < 0.3 else 0.0
    nesterov = bool(mom and rs.random() < 0.3)
    fused = bool(rs.random() < 0.8)
    layout = "separate" if rs.random() < 0.4 else "flat"
    w = wl.Workload(f"random{case}", n, segs, dtype, 0.1 if dtype == DTYPE_F32 else 20.0, mom,
                    0.01, dict(mode=wl.TABLE, table=_random_rows(rs, n)), 4, 100 + case,
                    straggler_every=3, param_sigma=1.0 if dtype == DTYPE_F32 else 0.05,
                    grad_ring=2, weight_decay=wd, nesterov=nesterov)
    return w, fused, layout


@pytest.mark.parametrize("case", range(CASES))
def test_random_case(case):
    import torch
    w, fused, layout = _case(case)
    log(f"case random {case}: N={w.n} segs={w.seg_numel} dtype={w.dtype} mom={w.momentum} "
        f"wd={w.weight_decay} nesterov={w.nesterov} fused={fused} layout={layout} "
        f"table={[[len(g) for g in row] for row in w.sched['table']]}")
    run = DeviceRun(w, layout, fused=fused)
    run.run(w.steps)
    torch.cuda.synchronize()
    check_against_oracle(run, [(0, w.numel)], f"random case {case}")
