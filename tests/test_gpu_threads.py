"""Two host threads drive the library at once, each with its own scheduler,
replicas handle and stream (the header's rule: one handle per thread).  The
library keeps no shared mutable state besides the launch settings and a
per-thread error message, so both runs must equal the oracle exactly, and an
error raised on one thread must not show up in the other's last error."""
import threading

import numpy as np
import pytest

from seedgen import DTYPE_BF16, DTYPE_F32
from seedgen import workloads as wl

from gpu_util import compare, log, oracle_windows

pytestmark = pytest.mark.gpu


def _workload(i):
    if i == 0:
        return wl.Workload("threads_a", 8, [3 * 4096 + 11], DTYPE_F32, 0.1, 0.9, 0.01,
                           dict(mode=wl.STATIC, seed=21, group_size=4, period=4), 12, 81,
                           grad_ring=1)
    return wl.Workload("threads_b", 12, [5000, 2049], DTYPE_BF16, 20.0, 0.0, 0.01,
                       dict(mode=wl.RANDOM_GB, seed=22, kmin=2, kmax=5), 12, 82,
                       straggler_every=3, param_sigma=0.05, grad_ring=1)


def test_two_threads_two_handles():
    import torch
    import paper_1909_08029_amd as rip
    torch.cuda.set_device(0)
    works = [_workload(0), _workload(1)]
    states, handles, scheds, streams = [], [], [], []
    for w in works:
        st = wl.DeviceState(w)
        st.fill()
        states.append(st)
        handles.append(rip.Replicas(st.param, st.grad_sets[0], st.mom))
        kw = dict(w.sched)
        scheds.append(rip.Scheduler(w.n, kw.pop("mode"), **kw))
        streams.append(torch.cuda.Stream())
    torch.cuda.synchronize()
    schedules = [[], []]
    errors = [None, None]
    barrier = threading.Barrier(2)

    def worker(i):
        try:
            torch.cuda.set_device(0)
            w = works[i]
            barrier.wait()
            for t in range(w.steps):
                a, g = rip.rip_step(scheds[i], handles[i], t, w.lr, momentum=w.momentum,
                                    eligible=w.eligible(t), stream=streams[i])
                schedules[i].append((a, g))
                if i == 1 and t == 5:
                    # an argument error on this thread only
                    with pytest.raises(rip.RipError):
                        rip.rip_preduce(handles[i], [(0, 0)], [], stream=streams[i])
                    assert rip.lib.rip_last_error()
            streams[i].synchronize()
            if i == 0:
                assert rip.lib.rip_last_error() == b""
        except BaseException as e:  # reported by the main thread
            errors[i] = e

    log("case two threads: static fp32 momentum and random groups bf16")
    threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=120)
    assert not any(th.is_alive() for th in threads)
    for e in errors:
        if e is not None:
            raise e
    torch.cuda.synchronize()
    for i, w in enumerate(works):
        (po, vo), = oracle_windows(w, schedules[i], [(0, w.numel)])
        for r in range(w.n):
            compare(states[i].window("param", r, 0, w.numel), po[r], w.dtype,
                    f"thread {i} param r={r}")
            if w.momentum:
                compare(states[i].window("mom", r, 0, w.numel), vo[r], w.dtype,
                        f"thread {i} mom r={r}")
    for h in handles:
        h.close()
