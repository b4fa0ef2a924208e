"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Small shapes are compared element by element over the whole buffers: sizes
that span several tiles and end in a ragged tail, every specialized group
size and the generic path, fp32 and bf16 storage, SGD and momentum, fused and
unfused forms, flat and separately allocated segments.  The five paper-shaped
workloads run at full size in the launch configuration the benchmark times,
and are checked on sampled windows (exact, because the method is
element-wise and the inputs are counter-based).
"""
import numpy as np
import pytest

from seedgen import DTYPE_BF16, DTYPE_F32
from seedgen import workloads as wl

from gpu_util import (DeviceRun, check_against_oracle, compare, log, oracle_scheduler,
                      sample_windows)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def full_windows(P):
    return [(0, P)]


def test_seedgen_gpu_matches_cpu():
    import torch
    import seedgen
    for dtype, tdt in ((DTYPE_F32, torch.float32), (DTYPE_BF16, torch.bfloat16)):
        for start, count in ((0, 1), (12345, 100003), ((1 << 33) + 7, 4099)):
            t = torch.empty(count, dtype=tdt, device="cuda")
            seedgen.fill_tensor(t, 11, seedgen.TAG_GRAD, 3, 5, 0.01, start=start)
            cpu = seedgen.normal(11, seedgen.TAG_GRAD, 3, 5, start, count, 0.01, dtype)
            g = t.cpu()
            g = g.view(torch.int16).numpy().view(np.uint16) if dtype else g.numpy()
            np.testing.assert_array_equal(g, cpu)


def test_config1_full_trajectory():
    """N=4 fp32 replicas of 1,048,576; SGD lr 0.1; group {0,1,2}; 10 steps."""
    w = wl.WORKLOADS[1]
    log(f"case {w.name}")
    run = DeviceRun(w)
    run.run(w.steps)
    osch = oracle_scheduler(w)
    assert run.schedule == [osch.step(t, w.eligible(t)) for t in range(w.steps)]
    assert all(g == [(0, 1, 2)] and a == [0, 1, 2, 3] for a, g in run.schedule)
    check_against_oracle(run, full_windows(w.numel), w.name)


SMALL_P = [1, 3, 4, 4097, 3 * 4096 + 5, 2 * 8192 + 13]


@pytest.mark.parametrize("dtype", [DTYPE_F32, DTYPE_BF16])
@pytest.mark.parametrize("P", SMALL_P)
def test_every_group_size_small(dtype, P):
    """One table row holding groups of sizes 1..9 (9 takes the generic path)
    over 45 replicas plus 3 ungrouped workers; some members inactive."""
    sizes = list(range(1, 10))
    groups, start = [], 0
    for k in sizes:
        groups.append(tuple(range(start, start + k)))
        start += k
    n = start + 3
    base = wl.Workload("small", n, [P], dtype, 0.1 if dtype == DTYPE_F32 else 50.0, 0.0,
                       0.01, dict(mode=wl.TABLE, table=[groups]), 3, 21,
                       straggler_every=2, param_sigma=1.0 if dtype == DTYPE_F32 else 0.05)
    log(f"case all-k dtype={dtype} P={P}")
    run = DeviceRun(base)
    run.run(base.steps)
    check_against_oracle(run, full_windows(P), f"allk P={P}")


@pytest.mark.parametrize("dtype", [DTYPE_F32, DTYPE_BF16])
@pytest.mark.parametrize("wd,nesterov,mom", [(0.0, False, 0.9), (1e-2, True, 0.9),
                                             (5e-3, False, 0.0)])
def test_large_groups_with_optimizers(dtype, wd, nesterov, mom):
    """Groups above the specialized sizes (9, 16 and 23 members: one, two and
    three chunks of eight, a ragged last chunk) with momentum, weight decay
    and Nesterov, some members not updating, over segments with ragged tails."""
    table = [[tuple(range(0, 9)), tuple(range(9, 25)), tuple(range(25, 48))],
             [tuple(range(1, 48, 2)), tuple(range(0, 48, 2))]]
    w = wl.Workload("wide", 48, [3 * 4096 + 11, 2048, 9], dtype,
                    0.1 if dtype == DTYPE_F32 else 20.0, mom, 0.01,
                    dict(mode=wl.TABLE, table=table), 6, 23, straggler_every=3,
                    param_sigma=1.0 if dtype == DTYPE_F32 else 0.05, grad_ring=3,
                    weight_decay=wd, nesterov=nesterov)
    for layout in ("flat", "separate"):
        log(f"case wide groups dtype={dtype} wd={wd} nesterov={nesterov} mom={mom} {layout}")
        run = DeviceRun(w, layout)
        run.run(w.steps)
        assert any(len(g) > 8 for _, gs in run.schedule for g in gs)
        check_against_oracle(run, full_windows(w.numel), f"wide {layout}")


@pytest.mark.parametrize("dtype", [DTYPE_F32, DTYPE_BF16])
@pytest.mark.parametrize("layout", ["flat", "separate"])
def test_segments_with_momentum(dtype, layout):
    """Layer-sized segments (the first VGG-16 tensors, a ragged one, an empty
    one), momentum 0.9, static groups of 8 over 16 replicas."""
    segs = [1792, 36928, 7, 0, 73856 + 3, 5000]
    w = wl.scaled(wl.WORKLOADS[3], segs, steps=5, grad_ring=3,
                  dtype=dtype, lr=0.1 if dtype == DTYPE_F32 else 20.0)
    log(f"case segments layout={layout} dtype={dtype}")
    run = DeviceRun(w, layout)
    run.run(w.steps)
    check_against_oracle(run, full_windows(w.numel), f"segments {layout}")


@pytest.mark.parametrize("dtype,mom", [(DTYPE_F32, 0.9), (DTYPE_BF16, 0.0)])
def test_many_small_separate_segments(dtype, mom):
    """Hundreds of separately allocated segments, most shorter than one tile
    (some empty, some a few elements, a few spanning several tiles): every
    launch searches a long segment table and most work runs through the
    element-wise tail path."""
    rs = np.random.default_rng(33)
    segs = [int(x) for x in rs.choice([0, 1, 3, 17, 255, 700, 1031, 2048, 9000], size=300)]
    w = wl.scaled(wl.WORKLOADS[4], segs, steps=5, n=7, dtype=dtype, momentum=mom,
                  lr=0.1 if dtype == DTYPE_F32 else 20.0,
                  sched=dict(mode=wl.RANDOM_GB, seed=12, kmin=2, kmax=5))
    log(f"case many segments: S={len(segs)} P={w.numel} dtype={dtype} mom={mom}")
    run = DeviceRun(w, "separate")
    run.run(w.steps)
    check_against_oracle(run, full_windows(w.numel), "many segments")


@pytest.mark.parametrize("dtype", [DTYPE_F32, DTYPE_BF16])
def test_unfused_local_step_then_preduce(dtype):
    """rip_local_step followed by a pure rip_preduce: two stores (for bf16,
    two roundings), as the oracle's unfused form."""
    w = wl.scaled(wl.WORKLOADS[4], [40_000 + 9], steps=12, n=12, dtype=dtype,
                  lr=0.1 if dtype == DTYPE_F32 else 30.0, momentum=0.9,
                  sched=dict(mode=wl.RANDOM_GB, seed=8, kmin=2, kmax=5))
    log(f"case unfused dtype={dtype}")
    run = DeviceRun(w, fused=False)
    run.run(w.steps)
    check_against_oracle(run, full_windows(w.numel), "unfused")


@pytest.mark.parametrize("dtype", [DTYPE_F32, DTYPE_BF16])
@pytest.mark.parametrize("wd,nesterov,mom,fused", [
    (1e-4, False, 0.9, True),      # the paper's ResNet-50 optimizer
    (1e-2, True, 0.9, True),
    (5e-3, False, 0.0, True),
    (0.0, True, 0.5, True),
    (1e-2, True, 0.9, False),
])
def test_optimizer_variants(dtype, wd, nesterov, mom, fused):
    """Weight decay and Nesterov momentum, fused and unfused, on random
    groups with a straggler (so groups also hold members that did not
    update this step)."""
    w = wl.scaled(wl.WORKLOADS[3], [3 * 4096 + 11, 777], steps=8, n=8, dtype=dtype,
                  lr=0.1 if dtype == DTYPE_F32 else 20.0, momentum=mom, weight_decay=wd,
                  nesterov=nesterov, sched=dict(mode=wl.RANDOM_GB, seed=9, kmin=2, kmax=8),
                  straggler_every=3, grad_ring=3)
    log(f"case optimizer dtype={dtype} wd={wd} nesterov={nesterov} mom={mom} fused={fused}")
    run = DeviceRun(w, "separate", fused=fused)
    run.run(w.steps)
    check_against_oracle(run, full_windows(w.numel), "optimizer")


def test_nesterov_without_momentum_is_rejected():
    import paper_1909_08029_amd as rip
    w = wl.Workload("nest", 2, [4096], DTYPE_F32, 0.1, 0.0, 0.01,
                    dict(mode=wl.TABLE, table=[[(0, 1)]]), 1, 71, grad_ring=1)
    st = wl.DeviceState(w)
    st.fill()
    h = rip.Replicas(st.param, st.grad_sets[0], None)
    with pytest.raises(rip.RipError) as e:
        rip.rip_preduce(h, [(0, 1)], [0, 1], lr=0.1, nesterov=True)
    assert e.value.code == rip.RIP_E_INVAL


def test_random_gb_straggler_small():
    w = wl.scaled(wl.WORKLOADS[4], [3 * 4096 + 17], steps=40)
    log("case random-gb small")
    run = DeviceRun(w)
    run.run(w.steps)
    osch = oracle_scheduler(w)
    assert run.schedule == [osch.step(t, w.eligible(t)) for t in range(w.steps)]
    check_against_oracle(run, full_windows(w.numel), "randomgb-small")


@pytest.mark.parametrize("mode,kw", [(wl.GD, dict(seed=6, kmin=2, kmax=4, c_thres=3)),
                                     (wl.RULE, dict(n_nodes=2)),
                                     (wl.INTER_INTRA, dict(seed=8, kmin=2, kmax=3, n_nodes=2)),
                                     (wl.ADPSGD, dict(seed=9))])
def test_other_schedulers_small(mode, kw):
    n = 8
    w = wl.scaled(wl.WORKLOADS[4], [8193], steps=20, n=n, sched=dict(mode=mode, **kw))
    log(f"case scheduler mode={mode}")
    run = DeviceRun(w)
    run.run(w.steps)
    check_against_oracle(run, full_windows(w.numel), f"mode{mode}")


@pytest.mark.parametrize("dtype,mom", [(DTYPE_F32, 0.9), (DTYPE_F32, 0.0), (DTYPE_BF16, 0.9)])
def test_split_launches_global_division(dtype, mom):
    """Global Division with groups of two to eight: steps whose units want
    residency caps far apart run as two launches (checked through the launch
    count the library reports); every element matches the oracle."""
    n = 16
    w = wl.scaled(wl.WORKLOADS[4], [3 * 4096 + 77], steps=16, n=n, dtype=dtype, momentum=mom,
                  lr=0.1 if dtype == DTYPE_F32 else 20.0,
                  param_sigma=1.0 if dtype == DTYPE_F32 else 0.05,
                  sched=dict(mode=wl.GD, seed=12, kmin=2, kmax=8))
    log(f"case split launches dtype={dtype} momentum={mom}")
    run = DeviceRun(w)
    run.run(w.steps)
    assert 2 in run.launches and 1 in run.launches, run.launches
    check_against_oracle(run, full_windows(w.numel), f"split dtype={dtype} mom={mom}")


def test_allreduce_and_max_replicas():
    """k = N = 256 (the largest handle): P-Reduce over every replica is the
    global mean; then pairs (AD-PSGD's k = 2)."""
    import paper_1909_08029_amd as rip
    n, P = 256, 4096 + 3
    table = [[tuple(range(n))], [tuple((2 * i, 2 * i + 1)) for i in range(n // 2)]]
    w = wl.Workload("maxn", n, [P], DTYPE_F32, 0.1, 0.0, 0.01, dict(mode=wl.TABLE, table=table),
                    2, 31, grad_ring=1)
    log("case k=N=256")
    run = DeviceRun(w)
    run.run(2)
    check_against_oracle(run, full_windows(P), "k=N")
    with pytest.raises(rip.RipError):
        rip.Scheduler(257, wl.TABLE, table=[[(0,)]])


@pytest.mark.parametrize("dtype,P", [(DTYPE_F32, 1_100_000_007), (DTYPE_BF16, 2_200_000_011)])
def test_buffers_beyond_4gib(dtype, P):
    """Replica buffers of 4.4 GB: byte offsets past 2^32 in the tiled paths
    and the ragged tail; windows straddle the 4 GiB offset and the end."""
    import torch
    w = wl.Workload("big", 3, [P], dtype, 0.1 if dtype == DTYPE_F32 else 20.0, 0.0, 0.01,
                    dict(mode=wl.TABLE, table=[[(0, 1)], [(1, 2)]]), 2, 81, grad_ring=1,
                    param_sigma=1.0 if dtype == DTYPE_F32 else 0.05)
    log(f"case buffers beyond 4 GiB dtype={dtype} P={P}")
    run = DeviceRun(w)
    run.run(w.steps)
    torch.cuda.synchronize()
    boundary = (1 << 32) // w.esize
    windows = sample_windows(P, 8, 1 << 15, seed=82, must=[boundary])
    assert any(a < boundary < b for a, b in windows) and windows[-1][1] == P
    check_against_oracle(run, windows, f"beyond 4 GiB dtype={dtype}")
    del run
    torch.cuda.empty_cache()


@pytest.mark.parametrize("dtype", [DTYPE_F32, DTYPE_BF16])
def test_single_replica(dtype):
    """N = 1: the local update alone (its own group of one), with momentum."""
    w = wl.Workload("one", 1, [3 * 4096 + 7], dtype, 0.1 if dtype == DTYPE_F32 else 20.0, 0.9,
                    0.01, dict(mode=wl.TABLE, table=[[(0,)], []]), 4, 83, grad_ring=2,
                    param_sigma=1.0 if dtype == DTYPE_F32 else 0.05)
    log(f"case single replica dtype={dtype}")
    run = DeviceRun(w)
    run.run(w.steps)
    assert [a for a, _ in run.schedule] == [[0]] * 4
    check_against_oracle(run, full_windows(w.numel), "N=1")


@pytest.fixture
def launch_defaults():
    """Restores the process-wide launch settings whatever the test does."""
    import paper_1909_08029_amd as rip
    yield rip
    rip.rip_set_max_blocks(0)
    rip.rip_set_blocks_per_cu(0)


@pytest.mark.parametrize("max_blocks,per_cu", [(1, 0), (7, 0), (1000, 0), (0, 1), (0, 3), (0, 32)])
def test_launch_settings_do_not_change_results(launch_defaults, max_blocks, per_cu):
    """Few workgroups looping over all tiles (the grid-stride path) and
    residency caps from 1 to 32 workgroups per CU: same bits as the oracle,
    on groups of many sizes, lone updates and momentum."""
    rip = launch_defaults
    rip.rip_set_max_blocks(max_blocks)
    rip.rip_set_blocks_per_cu(per_cu)
    table = [[(0, 1, 2), (3, 4), tuple(range(5, 15))], [(1, 3, 5, 7, 9, 11, 13), (0, 2)]]
    w = wl.Workload("launch", 16, [3 * 4096 + 13, 1000], DTYPE_F32, 0.1, 0.9, 0.01,
                    dict(mode=wl.TABLE, table=table), 4, 91, straggler_every=2, grad_ring=2)
    log(f"case launch settings max_blocks={max_blocks} blocks_per_cu={per_cu}")
    run = DeviceRun(w)
    run.run(w.steps)
    check_against_oracle(run, full_windows(w.numel), f"max_blocks={max_blocks} per_cu={per_cu}")


def test_pure_preduce_invariants_and_untouched():
    """Members end bit-identical, replicas outside every group keep their
    bytes, and the replica sum is preserved (doubly stochastic F^G)."""
    import torch
    import paper_1909_08029_amd as rip
    n, P = 10, 70001
    w = wl.Workload("inv", n, [P], DTYPE_F32, 0.1, 0.0, 0.01,
                    dict(mode=wl.TABLE, table=[[(0,)]]), 1, 41, grad_ring=1)
    st = wl.DeviceState(w)
    st.fill()
    h = rip.Replicas(st.param, None, None)
    before = [st.window("param", r, 0, P).copy() for r in range(n)]
    groups = [(1, 4, 7), (2, 3), (5, 6, 8, 9)]
    rip.rip_preduce(h, groups)
    torch.cuda.synchronize()
    after = [st.window("param", r, 0, P) for r in range(n)]
    np.testing.assert_array_equal(after[0].view(np.uint32), before[0].view(np.uint32))
    for g in groups:
        for m in g[1:]:
            np.testing.assert_array_equal(after[m].view(np.uint32), after[g[0]].view(np.uint32))
    s0 = np.sum([b.astype(np.float64) for b in before], axis=0)
    s1 = np.sum([a.astype(np.float64) for a in after], axis=0)
    bound = 8 * 2.0 ** -24 * np.sum([np.abs(b.astype(np.float64)) for b in before], axis=0)
    assert np.all(np.abs(s1 - s0) <= bound)
    # idempotent for pairs: a second P-Reduce changes nothing
    rip.rip_preduce(h, [(2, 3)])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(st.window("param", 2, 0, P).view(np.uint32),
                                  after[2].view(np.uint32))


def test_bf16_update_is_applied():
    """With lr*g below half a bf16 ulp the update rounds away; with a large
    lr it must show.  Guards against a kernel that drops the update."""
    import torch
    import paper_1909_08029_amd as rip
    n, P = 4, 8192 * 2 + 5
    w = wl.Workload("bf16upd", n, [P], DTYPE_BF16, 100.0, 0.0, 1e-3,
                    dict(mode=wl.TABLE, table=[[(0, 1)]]), 1, 51, grad_ring=1,
                    param_sigma=0.01)
    run = DeviceRun(w)
    before = run.state.window("param", 2, 0, P).copy()
    run.run(1)
    torch.cuda.synchronize()
    after = run.state.window("param", 2, 0, P)
    assert (after != before).mean() > 0.9
    check_against_oracle(run, full_windows(P), "bf16 update")


def test_error_paths_change_nothing():
    import torch
    import paper_1909_08029_amd as rip
    n, P = 6, 4100
    w = wl.Workload("err", n, [P], DTYPE_F32, 0.1, 0.0, 0.01,
                    dict(mode=wl.TABLE, table=[[(0,)]]), 1, 61, grad_ring=1)
    st = wl.DeviceState(w)
    st.fill()
    h = rip.Replicas(st.param, st.grad_sets[0], None)
    h_nograd = rip.Replicas(st.param, None, None)
    before = [st.window("param", r, 0, P).copy() for r in range(n)]
    cases = [
        (lambda: rip.rip_preduce(h, [(0, 1), (1, 2)], [], lr=0.1), rip.RIP_E_OVERLAP),
        (lambda: rip.rip_preduce(h, [(2, 1)], [], lr=0.1), rip.RIP_E_INVAL),
        (lambda: rip.rip_preduce(h, [(0, 6)], [], lr=0.1), rip.RIP_E_INVAL),
        (lambda: rip.rip_preduce(h, [(0, 1)], [0, 0], lr=0.1), rip.RIP_E_INVAL),
        (lambda: rip.rip_preduce(h, [(0, 1)], [0]), rip.RIP_E_INVAL),           # no sgd
        (lambda: rip.rip_preduce(h_nograd, [(0, 1)], [0], lr=0.1), rip.RIP_E_INVAL),
        (lambda: rip.rip_preduce(h, [(0, 1)], [0], lr=0.1, momentum=0.9), rip.RIP_E_INVAL),
        (lambda: rip.rip_local_step(h, [7], 0.1), rip.RIP_E_INVAL),
    ]
    for fn, code in cases:
        with pytest.raises(rip.RipError) as e:
            fn()
        assert e.value.code == code, str(e.value)
    # empty step is a no-op
    rip.rip_preduce(h, [], [], lr=0.1)
    rip.rip_preduce(h, [(3,)], [], lr=0.1)       # singleton, not active: identity
    torch.cuda.synchronize()
    for r in range(n):
        np.testing.assert_array_equal(st.window("param", r, 0, P).view(np.uint32),
                                      before[r].view(np.uint32))
    # a zero-length replica set registers and does nothing
    z = wl.Workload("zero", 2, [0], DTYPE_F32, 0.1, 0.0, 0.01,
                    dict(mode=wl.TABLE, table=[[(0,)]]), 1, 62, grad_ring=1)
    zs = wl.DeviceState(z)
    hz = rip.Replicas(zs.param, zs.grad_sets[0], None)
    rip.rip_preduce(hz, [(0, 1)], [0, 1], lr=0.1)
    torch.cuda.synchronize()


def _register(dtype, numel, param, grad=None, mom=None):
    """rip_replicas_create on raw pointers; returns its status (the handle,
    if any, is destroyed)."""
    import ctypes
    import paper_1909_08029_amd as rip
    S = len(numel)
    n = len(param) // S

    def arr(xs):
        return None if xs is None else (ctypes.c_void_p * len(xs))(*xs)

    h = ctypes.c_void_p()
    rc = rip.lib.rip_replicas_create(n, S, dtype, (ctypes.c_int64 * S)(*numel), arr(param),
                                     arr(grad), arr(mom), ctypes.byref(h))
    if rc == 0:
        rip.lib.rip_replicas_destroy(h)
    return rc


def test_registration_checks_buffers():
    """Registration rejects host memory, segments that run past their
    allocation and written buffers that alias another buffer; gradients may
    be shared.  None of the rejections leaves an error behind for torch."""
    import torch
    import paper_1909_08029_amd as rip
    P = 4096
    buf = torch.zeros(8 * P, device="cuda")
    b = buf.data_ptr()
    q = P * 4                                   # bytes of one segment
    pinned = torch.zeros(P, pin_memory=True)
    pageable = np.zeros(P, dtype=np.float32)
    cases = [
        ("disjoint params and grads", [P], [b, b + q], [b + 2 * q, b + 3 * q], None, rip.RIP_OK),
        ("shared gradient", [P], [b, b + q], [b + 2 * q, b + 2 * q], None, rip.RIP_OK),
        ("pinned host param", [P], [pinned.data_ptr()], None, None, rip.RIP_E_INVAL),
        ("pageable host grad", [P], [b], [pageable.ctypes.data], None, rip.RIP_E_INVAL),
        ("past the allocation", [1 << 36], [b], None, None, rip.RIP_E_INVAL),
        ("params overlap", [P], [b, b + q // 2], None, None, rip.RIP_E_OVERLAP),
        ("grad aliases a param", [P], [b, b + q], [b + 2 * q, b], None, rip.RIP_E_OVERLAP),
        ("param inside a grad", [P], [b + 16, b + 2 * q], [b, b + 3 * q], None, rip.RIP_E_OVERLAP),
        ("mom aliases a param", [P], [b, b + q], None, [b + 2 * q, b + q], rip.RIP_E_OVERLAP),
        ("empty segment is not checked", [P, 0], [b, pageable.ctypes.data], None, None,
         rip.RIP_OK),
        ("segments of one replica overlap", [P, P], [b, b + q // 2], None, None,
         rip.RIP_E_OVERLAP),
    ]
    for name, numel, param, grad, mom, code in cases:
        log(f"case registration: {name}")
        assert _register(DTYPE_F32, numel, param, grad, mom) == code, name
    # torch's own error check after a launch still sees a clean state
    assert float(torch.ones(1024, device="cuda").sum()) == 1024.0
    torch.cuda.synchronize()


@pytest.mark.parametrize("dtype", [DTYPE_F32, DTYPE_BF16])
def test_shared_gradient_equals_copies(dtype):
    """Replicas that share one gradient buffer step exactly like replicas
    holding copies of it."""
    import torch
    import paper_1909_08029_amd as rip
    n, P = 4, 3 * 4096 + 77
    tdt = torch.bfloat16 if dtype == DTYPE_BF16 else torch.float32
    gen = torch.Generator().manual_seed(91)
    p0 = [torch.randn(P, generator=gen).to(tdt).cuda() for _ in range(n)]
    g = torch.randn(P, generator=gen).to(tdt).cuda()
    p1 = [t.clone() for t in p0]
    shared = rip.Replicas([[t] for t in p0], [[g] for _ in range(n)], None)
    copies = rip.Replicas([[t] for t in p1], [[g.clone()] for _ in range(n)], None)
    for h in (shared, copies):
        rip.rip_preduce(h, [(0, 2, 3)], [0, 1, 3], lr=0.05)
        rip.rip_preduce(h, [(1, 2)], [1, 2], lr=0.05)
    torch.cuda.synchronize()
    view = torch.int16 if dtype == DTYPE_BF16 else torch.int32
    for a, c in zip(p0, p1):
        assert torch.equal(a.view(view), c.view(view))
    shared.close()
    copies.close()


# ---------------------------------------------------------------------------
# the five paper-shaped workloads at full size, sampled windows
# ---------------------------------------------------------------------------
FULL = [(2, 6, "flat"), (3, 4, "flat"), (3, 3, "separate"), (4, 24, "flat"), (5, 4, "flat")]


@pytest.mark.parametrize("cfg,steps,layout", FULL)
def test_full_size_config_windows(cfg, steps, layout):
    import torch
    w = wl.WORKLOADS[cfg]
    log(f"case full config {cfg} ({w.name}) steps={steps} layout={layout}")
    run = DeviceRun(w, layout)
    run.run(steps)
    torch.cuda.synchronize()
    osch = oracle_scheduler(w)
    assert run.schedule == [osch.step(t, w.eligible(t)) for t in range(steps)]
    bounds = np.cumsum(w.seg_numel)[:-1].tolist()
    windows = sample_windows(w.numel, 32, 1 << 16, seed=cfg, must=bounds)
    covered = len(set().union(*(range(a, b) for a, b in windows))) if w.numel < 1 << 24 else \
        sum(b - a for a, b in windows)
    worst = check_against_oracle(run, windows, f"config{cfg}")
    log(f"config {cfg}: {len(windows)} windows of up to 65536 x {w.n} replicas ok "
        f"({100.0 * covered / w.numel:.3f}% of each replica), max rel err {worst:.2e}")
    del run
    torch.cuda.empty_cache()


# ---------------------------------------------------------------------------
# the paper's scheduling policies on the heterogeneous workload's full shape
# (N = 32 fp32 replicas of 25.6M, worker 0 at a quarter of the others' rate)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("name", [n for n in wl.SCHEDULE_VARIANTS if n != "random_gb"])
def test_full_size_schedule_variants(name):
    import torch
    w = wl.with_schedule(wl.WORKLOADS[4], name)
    steps = 12
    log(f"case full heterogeneous workload schedule={name} steps={steps}")
    run = DeviceRun(w)
    run.run(steps)
    torch.cuda.synchronize()
    osch = oracle_scheduler(w)
    assert run.schedule == [osch.step(t, w.eligible(t)) for t in range(steps)]
    windows = sample_windows(w.numel, 8, 1 << 15, seed=40)
    worst = check_against_oracle(run, windows, f"config4 {name}")
    log(f"heterogeneous {name}: {len(windows)} windows x {w.n} replicas ok, max rel err {worst:.2e}")
    del run
    torch.cuda.empty_cache()


# ---------------------------------------------------------------------------
# rip_step: group generation and the fused launch in one call
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("dtype", [DTYPE_F32, DTYPE_BF16])
def test_step_equals_schedule_then_preduce(dtype):
    """rip_step on one copy, rip_schedule_groups + rip_preduce on another:
    same schedules, same bits after every step, and the oracle's result."""
    import torch
    import paper_1909_08029_amd as rip
    w = wl.scaled(wl.WORKLOADS[4], [3 * 4096 + 17], steps=12, n=12, dtype=dtype,
                  lr=0.1 if dtype == DTYPE_F32 else 20.0, momentum=0.9,
                  param_sigma=1.0 if dtype == DTYPE_F32 else 0.05,
                  sched=dict(mode=wl.GD, seed=12, kmin=2, kmax=9, c_thres=3))
    log(f"case rip_step dtype={dtype}")
    a, b = DeviceRun(w), DeviceRun(w)
    view = np.uint16 if dtype == DTYPE_BF16 else np.uint32
    for t in range(w.steps):
        h = a.handles[w.grad_slot(t)]
        got = rip.rip_step(a.sched, h, t, w.lr, w.momentum, eligible=w.eligible(t))
        a.schedule.append(got)
        b.step()
        assert got == b.schedule[-1], f"step {t}"
        torch.cuda.synchronize()
        for r in range(w.n):
            assert np.array_equal(a.state.window("param", r, 0, w.numel).view(view),
                                  b.state.window("param", r, 0, w.numel).view(view)), (t, r)
    check_against_oracle(a, full_windows(w.numel), "rip_step")


def test_step_failure_leaves_scheduler_and_memory():
    """Rejected rip_step calls (momentum without momentum buffers, handles of
    different sizes) launch nothing and leave the scheduler at the same step."""
    import torch
    import paper_1909_08029_amd as rip
    w = wl.scaled(wl.WORKLOADS[4], [4099], steps=2, n=6, momentum=0.0,
                  sched=dict(mode=wl.RANDOM_GB, seed=13, kmin=2, kmax=4))
    run = DeviceRun(w)
    before = [run.state.window("param", r, 0, w.numel).copy() for r in range(w.n)]
    h = run.handles[0]
    with pytest.raises(rip.RipError) as e:
        rip.rip_step(run.sched, h, 0, 0.1, momentum=0.9)       # no momentum buffers
    assert e.value.code == rip.RIP_E_INVAL
    other = wl.DeviceState(wl.scaled(w, [4099], n=5))
    other.fill()
    h5 = rip.Replicas(other.param, other.grad_sets[0], None)
    with pytest.raises(rip.RipError) as e:
        rip.rip_step(run.sched, h5, 0, 0.1)                    # 5 replicas, 6 workers
    assert e.value.code == rip.RIP_E_INVAL
    torch.cuda.synchronize()
    for r in range(w.n):
        assert np.array_equal(run.state.window("param", r, 0, w.numel).view(np.uint32),
                              before[r].view(np.uint32))
    osch = oracle_scheduler(w)
    assert rip.rip_step(run.sched, h, 0, w.lr) == osch.step(0, None)
