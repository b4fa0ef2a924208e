"""Fused steps captured into a HIP graph replay exactly like eager launches.

Each rip_preduce call enqueues one kernel launch (two for steps that mix far
apart unit shapes) whose argument carries the whole step (schedule, optimizer scalars, the handle's pointer-table address)
and does no memset, copy or allocation, so a sequence of steps can be
captured once and replayed.  The graph is replayed several times with the
program's own eager work and synchronizations in between; after every replay
the buffers must equal both an eager run of the same steps and the oracle.
"""
import numpy as np
import pytest

from seedgen import DTYPE_BF16, DTYPE_F32
from seedgen import workloads as wl

from gpu_util import compare, log, oracle_windows

pytestmark = pytest.mark.gpu

# (active, groups) per captured step: grouped and lone updates, a group whose
# members do not all update, a pure P-Reduce of six, and a step that the
# library splits into two launches (a group of eight, which wants few
# resident waves, beside a pair and two lone updates, which want many)
STEPS = [
    ([0, 1, 2, 3, 4, 5], [(0, 1, 2), (3, 4)]),
    ([0, 2, 3], [(1, 5), (2, 3)]),
    ([], [(0, 1, 2, 3, 4, 5)]),
    (list(range(12)), [tuple(range(8)), (8, 9)]),
]


def _workload(dtype, momentum):
    return wl.Workload(f"graph_{'bf16' if dtype else 'fp32'}_{'mom' if momentum else 'sgd'}",
                       12, [3 * 4096 + 5], dtype, 0.1 if not dtype else 2.0, momentum,
                       0.01, dict(mode=wl.TABLE, table=[[(0, 1)]]), len(STEPS), 7,
                       param_sigma=1.0 if not dtype else 0.05, grad_ring=1)


def _launch_all(rip, h, w, stream):
    for active, groups in STEPS:
        rip.rip_preduce(h, groups, active, lr=w.lr, momentum=w.momentum, stream=stream)
        # the last step is the one the library splits into two launches
        assert rip.rip_last_launch_count() == (2 if len(groups[0]) == 8 else 1)


def _state(st, w):
    P = w.numel
    p = np.stack([st.window("param", r, 0, P) for r in range(w.n)])
    v = np.stack([st.window("mom", r, 0, P) for r in range(w.n)]) if w.momentum else None
    return p, v


@pytest.mark.parametrize("dtype,momentum", [(DTYPE_F32, 0.0), (DTYPE_BF16, 0.9)])
def test_graph_replays_match_eager_and_oracle(dtype, momentum):
    import torch
    import paper_1909_08029_amd as rip
    torch.cuda.set_device(0)
    w = _workload(dtype, momentum)
    log(f"case {w.name}: capture {len(STEPS)} steps, replay 3 times")
    eager = wl.DeviceState(w)
    eager.fill()
    graphed = wl.DeviceState(w)
    graphed.fill()
    he = rip.Replicas(eager.param, eager.grad_sets[0], eager.mom)
    hg = rip.Replicas(graphed.param, graphed.grad_sets[0], graphed.mom)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _launch_all(rip, hg, w, torch.cuda.current_stream())
    torch.cuda.synchronize()
    # capturing records the launches without running them
    p0, _ = _state(graphed, w)
    pe0, _ = _state(eager, w)
    assert np.array_equal(p0, pe0)

    noise = torch.empty(1 << 20, device="cuda")
    schedule = []
    for rep in range(3):
        g.replay()
        noise.normal_()                      # the program's own eager work
        _ = float(noise.sum())               # ... and a synchronization
        _launch_all(rip, he, w, torch.cuda.current_stream())
        torch.cuda.synchronize()
        schedule += STEPS
        pg, vg = _state(graphed, w)
        pe, ve = _state(eager, w)
        view = np.uint16 if dtype == DTYPE_BF16 else np.uint32
        assert np.array_equal(pg.view(view), pe.view(view)), f"replay {rep}: graph != eager"
        if momentum:
            assert np.array_equal(vg.view(view), ve.view(view)), f"replay {rep}: momentum"
        (po, vo), = oracle_windows(w, schedule, [(0, w.numel)])
        for r in range(w.n):
            compare(pg[r], po[r], dtype, f"{w.name} replay {rep} param r={r}")
            if momentum:
                compare(vg[r], vo[r], dtype, f"{w.name} replay {rep} mom r={r}")
    del g
    he.close()
    hg.close()
