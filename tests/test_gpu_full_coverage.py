"""Full-coverage parity at full size: every element of every replica after
several fused steps, compared bit for bit with the oracle.

The device state is streamed to the host in chunks of 2^22 elements.  The
initial inputs of each chunk come from the seeded generator's GPU twin (the
shared input module; `test_seedgen_gpu_matches_cpu` pins it bit-exact to its
numpy form), copied to the host, and the oracle runs the same schedule on the
chunk, which is exact in isolation because the method is element-wise.
Chunks run on a thread pool (numpy releases the GIL on whole-array work);
on a 16-core host the four workloads take about a minute together (the
1.3B-element bf16 one about half of it)."""
from __future__ import annotations

import concurrent.futures as cf
import time

import numpy as np
import pytest

import seedgen
from seedgen import DTYPE_BF16
from seedgen import workloads as wl

from gpu_util import DeviceRun, compare, log, oracle_scheduler

pytestmark = pytest.mark.gpu

CHUNK = 1 << 22
WORKERS = 8

# (config, fused steps before the comparison)
CASES = [(2, 6), (3, 4), (4, 24), (5, 4)]


def _gen(scratch, w: wl.Workload, tag: int, r: int, step: int, a: int, W: int, sigma: float):
    """Elements [a, a+W) of one seeded input stream, on the host."""
    import torch
    seedgen.fill_normal_gpu(scratch.data_ptr(), w.dtype, w.seed, tag, r, step, a, W, sigma,
                            torch.cuda.current_stream().cuda_stream)
    x = scratch[:W].cpu()
    return x.view(torch.int16).numpy().view(np.uint16) if w.dtype == DTYPE_BF16 else x.numpy()


def _oracle_chunk(w: wl.Workload, schedule, p, grads, v, got_p, got_v, label):
    from oracle import preduce as op
    dt = op.BF16 if w.dtype == DTYPE_BF16 else op.F32
    for t, (active, groups) in enumerate(schedule):
        p, v = op.step(p, grads[w.grad_slot(t)], v, groups, active, w.lr,
                       w.momentum if w.momentum else None, dt, True, w.weight_decay, w.nesterov)
    worst = 0.0
    for r in range(w.n):
        mr, _ = compare(got_p[r], p[r], w.dtype, f"{label} param r={r}")
        worst = max(worst, mr)
        if v is not None:
            compare(got_v[r], v[r], w.dtype, f"{label} mom r={r}")
    return worst


@pytest.mark.parametrize("cfg,steps", CASES)
def test_full_coverage(cfg, steps):
    import torch
    w = wl.WORKLOADS[cfg]
    log(f"case full coverage config {cfg} ({w.name}) steps={steps}")
    t0 = time.time()
    run = DeviceRun(w, "flat")
    run.run(steps)
    torch.cuda.synchronize()
    osch = oracle_scheduler(w)
    assert run.schedule == [osch.step(t, w.eligible(t)) for t in range(steps)]
    tdt = torch.bfloat16 if w.dtype == DTYPE_BF16 else torch.float32
    scratch = torch.empty(CHUNK, dtype=tdt, device="cuda")
    P, n = w.numel, w.n
    pending, worst, done = [], 0.0, 0
    with cf.ThreadPoolExecutor(max_workers=WORKERS) as pool:
        for a in range(0, P, CHUNK):
            b = min(P, a + CHUNK)
            W = b - a
            p = np.stack([_gen(scratch, w, seedgen.TAG_PARAM, r, 0, a, W, w.param_sigma)
                          for r in range(n)])
            grads = [np.stack([_gen(scratch, w, seedgen.TAG_GRAD, r, slot, a, W, w.grad_sigma)
                               for r in range(n)]) for slot in range(min(w.grad_ring, steps))]
            v = np.zeros_like(p) if w.momentum else None
            got_p = [run.state.window("param", r, a, b) for r in range(n)]
            got_v = [run.state.window("mom", r, a, b) for r in range(n)] if w.momentum else None
            pending.append(pool.submit(_oracle_chunk, w, run.schedule, p, grads, v, got_p, got_v,
                                       f"config{cfg} [{a},{b})"))
            while len(pending) >= WORKERS:
                worst = max(worst, pending.pop(0).result())
                done += 1
                if done % 16 == 0:
                    log(f"config {cfg}: {done} chunks checked ({time.time() - t0:.0f} s)")
        for f in pending:
            worst = max(worst, f.result())
    log(f"config {cfg}: all {P} elements x {n} replicas bit-exact after {steps} steps, "
        f"max rel err {worst:.2e}, {time.time() - t0:.0f} s")
    del run, scratch
    torch.cuda.empty_cache()
