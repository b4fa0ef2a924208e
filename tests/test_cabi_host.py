"""Host-side checks of librip (CPU only, no GPU needed).

* The library loads and exports every function include/rip.h declares.
* The C++ scheduler reproduces the oracle's schedules bit-for-bit over 10^4
  steps in every mode, with and without a straggler.
* Argument checks that run before any HIP call return the documented codes.
"""
import ctypes
import os
import re

import pytest

import paper_1909_08029_amd as rip
from oracle import sched as os_

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "rip.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rip_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = header_functions()
    assert {"rip_schedule_groups", "rip_local_step", "rip_preduce"} <= set(names)
    lib = ctypes.CDLL(rip.LIB_PATH)
    for name in names:
        assert hasattr(lib, name), f"{name} declared in rip.h but not exported"
    assert rip.abi_version() == 2


def _straggler(n, t, every):
    e = [True] * n
    e[0] = (t % every == 0)
    return e


CASES = [
    # (n, oracle kwargs, binding kwargs, straggler period or None)
    (4, dict(mode=os_.TABLE, table=[[(0, 1, 2)]]), dict(mode=rip.SCHED_TABLE, table=[[(0, 1, 2)]]), None),
    (16, dict(mode=os_.STATIC, seed=2, group_size=4, period=4),
     dict(mode=rip.SCHED_STATIC, seed=2, group_size=4, period=4), None),
    (16, dict(mode=os_.STATIC, seed=3, group_size=8, period=4),
     dict(mode=rip.SCHED_STATIC, seed=3, group_size=8, period=4), 4),
    (8, dict(mode=os_.STATIC, seed=5, group_size=4, period=4),
     dict(mode=rip.SCHED_STATIC, seed=5, group_size=4, period=4), None),
    (32, dict(mode=os_.RANDOM_GB, seed=4, kmin=2, kmax=8),
     dict(mode=rip.SCHED_RANDOM_GB, seed=4, kmin=2, kmax=8), 4),
    (32, dict(mode=os_.GD, seed=4, kmin=2, kmax=8),
     dict(mode=rip.SCHED_GD, seed=4, kmin=2, kmax=8), 4),
    (32, dict(mode=os_.GD, seed=9, kmin=3, kmax=3, c_thres=3),
     dict(mode=rip.SCHED_GD, seed=9, kmin=3, kmax=3, c_thres=3), 5),
    (16, dict(mode=os_.RULE, n_nodes=4), dict(mode=rip.SCHED_RULE, n_nodes=4), 3),
    (32, dict(mode=os_.ADPSGD, seed=10), dict(mode=rip.SCHED_ADPSGD, seed=10), 4),
    (5, dict(mode=os_.ADPSGD, seed=11), dict(mode=rip.SCHED_ADPSGD, seed=11), None),
    (1, dict(mode=os_.ADPSGD, seed=12), dict(mode=rip.SCHED_ADPSGD, seed=12), None),
    (32, dict(mode=os_.INTER_INTRA, seed=6, kmin=2, kmax=4, n_nodes=4),
     dict(mode=rip.SCHED_INTER_INTRA, seed=6, kmin=2, kmax=4, n_nodes=4), 4),
    (24, dict(mode=os_.INTER_INTRA, seed=7, kmin=1, kmax=3, c_thres=2, n_nodes=3),
     dict(mode=rip.SCHED_INTER_INTRA, seed=7, kmin=1, kmax=3, c_thres=2, n_nodes=3), 3),
    (7, dict(mode=os_.RANDOM_GB, seed=2 ** 64 - 1, kmin=1, kmax=9),
     dict(mode=rip.SCHED_RANDOM_GB, seed=2 ** 64 - 1, kmin=1, kmax=9), 2),
    (12, dict(mode=os_.TABLE, table=[[(0, 5), (1, 2, 3)], [], [(4, 6, 7, 8, 9, 10, 11)]]),
     dict(mode=rip.SCHED_TABLE, table=[[(0, 5), (1, 2, 3)], [], [(4, 6, 7, 8, 9, 10, 11)]]), 3),
    # rows not ordered by first member, singletons: output keeps the row's own order
    (10, dict(mode=os_.TABLE, table=[[(3, 9), (0, 7), (5,)], [(6, 8), (4,), (1, 2, 5)]]),
     dict(mode=rip.SCHED_TABLE, table=[[(3, 9), (0, 7), (5,)], [(6, 8), (4,), (1, 2, 5)]]), 3),
]


@pytest.mark.parametrize("n,okw,bkw,strag", CASES)
def test_scheduler_parity_with_oracle(n, okw, bkw, strag):
    steps = 10000
    o = os_.Scheduler(n, **okw)
    c = rip.Scheduler(n, **bkw)
    for t in range(steps):
        el = None if strag is None else _straggler(n, t, strag)
        assert rip.rip_schedule_groups(c, t, el) == o.step(t, el), f"step {t}"
    for i in range(n):
        ws = c.worker(i)
        depth = int(o.waiting[i]) if o.mode == os_.ADPSGD else len(o.gb[i])
        assert (ws.requests, ws.syncs, ws.skips, bool(ws.waiting), ws.gb_depth) == \
            (o.c[i], o.syncs[i], o.skips[i], o.waiting[i], depth)
        assert ws.requests == ws.syncs + ws.skips + ws.waiting


def test_scripted_walkthrough_matches_oracle():
    script = [(0, 4, 5), (4, 5, 7)]
    o = os_.Scheduler(8, os_.SCRIPTED, script=script)
    c = rip.Scheduler(8, rip.SCHED_SCRIPTED, script=script)
    only = lambda *ws: [i in ws for i in range(8)]
    for t, el in enumerate([only(0, 7), only(4, 5), only(4, 5)]):
        assert rip.rip_schedule_groups(c, t, el) == o.step(t, el)


def test_failed_step_leaves_state_unchanged():
    # W2 asks first but the script's next group (0, 1) does not contain it
    c2 = rip.Scheduler(4, rip.SCHED_SCRIPTED, script=[(0, 1)])
    with pytest.raises(rip.RipError) as e2:
        rip.rip_schedule_groups(c2, 0, [False, False, True, False])
    assert e2.value.code == rip.RIP_E_INVAL
    assert c2.worker(2).requests == 0
    # the same step can be retried after the failure
    assert rip.rip_schedule_groups(c2, 0, [True, True, False, False]) == ([0, 1], [(0, 1)])


def test_scheduler_argument_errors():
    with pytest.raises(rip.RipError) as e:
        rip.Scheduler(0, rip.SCHED_RANDOM_GB)
    assert e.value.code == rip.RIP_E_INVAL
    with pytest.raises(rip.RipError) as e:
        rip.Scheduler(257, rip.SCHED_RANDOM_GB)
    assert e.value.code == rip.RIP_E_UNSUPPORTED
    with pytest.raises(rip.RipError) as e:
        rip.Scheduler(10, rip.SCHED_STATIC, group_size=4)
    assert e.value.code == rip.RIP_E_INVAL
    with pytest.raises(rip.RipError) as e:
        rip.Scheduler(8, rip.SCHED_STATIC, group_size=1)      # never connected
    assert e.value.code == rip.RIP_E_INVAL
    with pytest.raises(rip.RipError) as e:
        rip.Scheduler(8, 99)
    assert e.value.code == rip.RIP_E_UNSUPPORTED
    with pytest.raises(rip.RipError) as e:
        rip.Scheduler(8, rip.SCHED_RANDOM_GB, kmin=3, kmax=2)
    assert e.value.code == rip.RIP_E_INVAL
    with pytest.raises(rip.RipError) as e:
        rip.Scheduler(4, rip.SCHED_TABLE, table=[[(0, 1), (1, 2)]])   # overlap in a row
    assert e.value.code == rip.RIP_E_INVAL
    with pytest.raises(rip.RipError) as e:
        rip.Scheduler(4, rip.SCHED_TABLE, table=[[(1, 0)]])           # not ascending
    assert e.value.code == rip.RIP_E_INVAL
    with pytest.raises(rip.RipError) as e:
        rip.Scheduler(12, rip.SCHED_RULE, n_nodes=3)                  # odd ring
    assert e.value.code == rip.RIP_E_INVAL
    s = rip.Scheduler(4, rip.SCHED_RANDOM_GB, kmin=2, kmax=2)
    rip.rip_schedule_groups(s, 0)
    with pytest.raises(rip.RipError) as e:
        rip.rip_schedule_groups(s, 5)
    assert e.value.code == rip.RIP_E_INVAL and "consecutive" in str(e.value)


def test_replicas_create_checks_before_any_device_call():
    lib = rip.lib
    out = ctypes.c_void_p()
    numel = (ctypes.c_int64 * 1)(1024)
    good = (ctypes.c_void_p * 2)(0x10000, 0x20000)
    bad_align = (ctypes.c_void_p * 2)(0x10000, 0x20008)
    null = (ctypes.c_void_p * 2)(0x10000, None)
    assert lib.rip_replicas_create(2, 1, 7, numel, good, None, None, ctypes.byref(out)) == \
        rip.RIP_E_UNSUPPORTED
    assert lib.rip_replicas_create(0, 1, 0, numel, good, None, None, ctypes.byref(out)) == \
        rip.RIP_E_INVAL
    assert lib.rip_replicas_create(300, 1, 0, numel, good, None, None, ctypes.byref(out)) == \
        rip.RIP_E_UNSUPPORTED
    assert lib.rip_replicas_create(2, 1, 0, numel, bad_align, None, None, ctypes.byref(out)) == \
        rip.RIP_E_ALIGN
    assert lib.rip_replicas_create(2, 1, 0, numel, good, null, None, ctypes.byref(out)) == \
        rip.RIP_E_INVAL
    assert b"NULL" in lib.rip_last_error()
    assert lib.rip_preduce(None, None, None, 0, None, 0, None, None) == rip.RIP_E_INVAL
    assert rip.rip_last_launch_count() == 0
    sgd = rip.Sgd(0.1, 0.0, 0.0, 0)
    assert lib.rip_local_step(None, None, 0, ctypes.byref(sgd), None) == rip.RIP_E_INVAL
    assert rip.rip_last_launch_count() == 0


def test_step_rejects_null_handles_and_leaves_the_scheduler():
    lib = rip.lib
    s = rip.Scheduler(4, rip.SCHED_STATIC, seed=2, group_size=2, period=4)
    sgd = rip.Sgd(0.1, 0.0, 0.0, 0)
    assert lib.rip_step(s._h, None, 0, None, ctypes.byref(sgd), None,
                        None, None, None, None, None) == rip.RIP_E_INVAL
    assert lib.rip_step(None, None, 0, None, ctypes.byref(sgd), None,
                        None, None, None, None, None) == rip.RIP_E_INVAL
    assert lib.rip_step(s._h, None, 0, None, None, None,
                        None, None, None, None, None) == rip.RIP_E_INVAL
    # the scheduler did not move: step 0 is still the next step
    fresh = rip.Scheduler(4, rip.SCHED_STATIC, seed=2, group_size=2, period=4)
    assert rip.rip_schedule_groups(s, 0) == rip.rip_schedule_groups(fresh, 0)


def _random_sched_case(seed):
    """A random scheduler configuration (any mode) with random eligibility."""
    import numpy as np
    rs = np.random.default_rng(seed)
    mode = int(rs.choice([os_.TABLE, os_.STATIC, os_.RANDOM_GB, os_.GD, os_.RULE,
                          os_.INTER_INTRA, os_.ADPSGD]))
    kw = {}
    if mode == os_.RULE:
        nodes = int(rs.choice([1, 2, 4, 6]))
        n, kw = 4 * nodes, dict(n_nodes=nodes)
    elif mode == os_.INTER_INTRA:
        nodes = int(rs.integers(1, 6))
        n = nodes * int(rs.integers(1, 7))
        kmin = int(rs.integers(1, 5))
        kw = dict(seed=int(rs.integers(0, 2 ** 63)), kmin=kmin, kmax=kmin + int(rs.integers(0, 5)),
                  c_thres=int(rs.integers(0, 5)), n_nodes=nodes)
    elif mode == os_.STATIC:
        k = int(rs.integers(2, 6))
        n = k * int(rs.integers(1, 8))
        kw = dict(seed=int(rs.integers(0, 2 ** 63)), group_size=k, period=int(rs.integers(1, 6)))
    elif mode == os_.TABLE:
        n = int(rs.integers(1, 30))
        table = []
        for _ in range(int(rs.integers(1, 4))):
            order = [int(x) for x in rs.permutation(n)][:int(rs.integers(0, n + 1))]
            row, i = [], 0
            while i < len(order):
                k = int(rs.integers(1, len(order) - i + 1))
                row.append(tuple(sorted(order[i:i + k])))
                i += k
            table.append(row)
        kw = dict(table=table)
    else:
        n = int(rs.integers(1, 40))
        kmin = int(rs.integers(1, 6))
        kw = dict(seed=int(rs.integers(0, 2 ** 63)), kmin=kmin, kmax=kmin + int(rs.integers(0, 6)))
        if mode == os_.GD:
            kw["c_thres"] = int(rs.integers(0, 6))
        if mode == os_.ADPSGD:
            kw = dict(seed=kw["seed"])
    p_eligible = float(rs.choice([1.0, 0.9, 0.6, 0.3]))
    masks = [[bool(x) for x in rs.random(n) < p_eligible] for _ in range(300)]
    return n, mode, kw, masks


@pytest.mark.parametrize("seed", range(150))
def test_scheduler_parity_random_configurations(seed):
    """C++ scheduler = oracle scheduler on random configurations of every mode
    with random per-step eligibility, 300 steps, including the per-worker
    counters."""
    n, mode, kw, masks = _random_sched_case(seed)
    bkw = dict(kw)
    try:
        o = os_.Scheduler(n, mode, **kw)
    except ValueError:
        with pytest.raises(rip.RipError):
            rip.Scheduler(n, mode, **bkw)
        return
    c = rip.Scheduler(n, mode, **bkw)
    for t, el in enumerate(masks):
        assert rip.rip_schedule_groups(c, t, el) == o.step(t, el), f"mode {mode} step {t}"
    for i in range(n):
        ws = c.worker(i)
        depth = int(o.waiting[i]) if o.mode == os_.ADPSGD else len(o.gb[i])
        assert (ws.requests, ws.syncs, ws.skips, bool(ws.waiting), ws.gb_depth) == \
            (o.c[i], o.syncs[i], o.skips[i], o.waiting[i], depth)
