"""rip_replicas_create_noalloc: the registration that allocates no device
memory gives the same steps as rip_replicas_create.

Two registrations in a row on one device (the second smaller: fewer
replicas, fewer elements, another storage type), each checked bit for bit
against a handle from rip_replicas_create running the same step on a copy of
the same inputs; the superseded handle is refused without touching memory;
tables above the fixed array's size are refused; and steps on such a handle
captured into a HIP graph replay like eager steps on an allocating handle.
"""
import numpy as np
import pytest

from seedgen import DTYPE_BF16, DTYPE_F32
from seedgen import workloads as wl

from gpu_util import compare, log

pytestmark = pytest.mark.gpu


def state(w):
    st = wl.DeviceState(w)
    st.fill()
    return st


def run_step(h, w, groups, active):
    import paper_1909_08029_amd as rip
    rip.rip_preduce(h, groups, active, lr=w.lr, momentum=w.momentum)


def check_same(a, b, w, label):
    for r in range(w.n):
        compare(b.window("param", r, 0, w.numel), a.window("param", r, 0, w.numel), w.dtype,
                f"{label} param r={r}")
        if w.momentum:
            compare(b.window("mom", r, 0, w.numel), a.window("mom", r, 0, w.numel), w.dtype,
                    f"{label} mom r={r}")


CALLS = [
    # (workload, groups, active)
    (wl.Workload("noalloc1", 8, [3 * 4096 + 5, 1000], DTYPE_F32, 0.1, 0.9, 0.01,
                 dict(mode=wl.TABLE, table=[[(0, 1, 2, 3)]]), 1, 81),
     [(0, 2, 5), (1, 3, 4, 6)], [0, 1, 2, 3, 5, 7]),
    (wl.Workload("noalloc2", 4, [2 * 1024 + 3], DTYPE_BF16, 30.0, 0.0, 0.01,
                 dict(mode=wl.TABLE, table=[[(0, 1)]]), 1, 82, param_sigma=0.05),
     [(1, 2)], [0, 1]),
]


def test_noalloc_registration_matches_allocating_one():
    import torch
    import paper_1909_08029_amd as rip
    torch.cuda.set_device(0)
    prev = None
    for i, (w, groups, active) in enumerate(CALLS):
        log(f"case noalloc call {i}: N={w.n} P={w.numel} dtype={w.dtype}")
        a, b = state(w), state(w)
        ha = rip.Replicas(a.param, a.grad_sets[0], a.mom)
        hb = rip.Replicas(b.param, b.grad_sets[0], b.mom, noalloc=True)
        for _ in range(2):
            run_step(ha, w, groups, active)
            run_step(hb, w, groups, active)
        torch.cuda.synchronize()
        check_same(a, b, w, f"call {i}")
        if prev is not None:
            # the first handle's tables were overwritten: it must refuse to launch
            pw, pst, pg, pa = prev
            before = [pst.window("param", r, 0, pw.numel).copy() for r in range(pw.n)]
            with pytest.raises(rip.RipError) as exc:
                run_step(pst_handle, pw, pg, pa)
            assert exc.value.code == rip.RIP_E_INVAL and "superseded" in str(exc.value)
            torch.cuda.synchronize()
            for r in range(pw.n):
                assert np.array_equal(pst.window("param", r, 0, pw.numel), before[r])
            pst_handle.close()
        prev = (w, b, groups, active)
        pst_handle = hb
        ha.close()
    pst_handle.close()


def test_noalloc_rejects_tables_above_its_size():
    import torch
    import paper_1909_08029_amd as rip
    torch.cuda.set_device(0)
    n, S = 200, 14            # 24*200*14 bytes of pointer table alone > 65536
    log(f"case noalloc oversize N={n} S={S}")
    param = [[torch.zeros(16, device="cuda") for _ in range(S)] for _ in range(n)]
    with pytest.raises(rip.RipError) as exc:
        rip.Replicas(param, None, None, noalloc=True)
    assert exc.value.code == rip.RIP_E_UNSUPPORTED
    # the same registration through the allocating entry point works
    rip.Replicas(param, None, None).close()


def test_noalloc_handle_launches_replay_from_a_graph():
    """The use it is for: register once without allocating, capture the
    steps into a HIP graph, replay; each replay equals eager steps on an
    allocating handle."""
    import torch
    import paper_1909_08029_amd as rip
    torch.cuda.set_device(0)
    w, groups, active = CALLS[0]
    log(f"case noalloc graph: N={w.n} P={w.numel}")
    a, b = state(w), state(w)
    ha = rip.Replicas(a.param, a.grad_sets[0], a.mom)
    hb = rip.Replicas(b.param, b.grad_sets[0], b.mom, noalloc=True)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        rip.rip_preduce(hb, groups, active, lr=w.lr, momentum=w.momentum,
                        stream=torch.cuda.current_stream())
    torch.cuda.synchronize()
    for rep in range(3):
        g.replay()
        run_step(ha, w, groups, active)
        torch.cuda.synchronize()
        check_same(a, b, w, f"graph replay {rep}")
    del g
    ha.close()
    hb.close()
