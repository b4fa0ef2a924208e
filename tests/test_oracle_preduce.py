"""Pins for the oracle's P-Reduce arithmetic (CPU only).

Every test checks the oracle against something other than itself: the paper's
matrix statement X F^G evaluated densely in float64, its worked conflict
example (exact fractions), library routines (numpy mean, torch's bf16
rounding), closed forms of the SGD and momentum recurrences, and the
invariants of Sec. 3.3 (doubly stochastic averaging, (F^G)^T F^G = F^G).
"""
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import preduce as op

U32 = 2.0 ** -24          # unit roundoff of fp32
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rng_f32(rs, shape, scale=1.0):
    return (rs.standard_normal(shape) * scale).astype(np.float32)


def dense_F(n, groups):
    """F^G of Sec. 3.2 for a set of disjoint groups, float64 (rows = source)."""
    F = np.eye(n)
    for g in groups:
        for i in g:
            F[i, i] = 0.0
        for i in g:
            for j in g:
                F[i, j] = 1.0 / len(g)
    return F


def random_groups(rs, n, max_groups=None):
    perm = list(rs.permutation(n))
    groups = []
    while perm and (max_groups is None or len(groups) < max_groups):
        k = int(rs.integers(1, min(len(perm), 5) + 1))
        groups.append(tuple(sorted(int(x) for x in perm[:k])))
        perm = perm[k:]
    return groups


# ---------------------------------------------------------------------------
# storage format
# ---------------------------------------------------------------------------
def test_bf16_rounding_matches_torch():
    rs = np.random.default_rng(0)
    x = np.concatenate([
        rs.standard_normal(100000).astype(np.float32),
        (rs.standard_normal(1000) * 1e-39).astype(np.float32),        # subnormals
        np.array([0.0, -0.0, 1.0, -1.0, 3.4e38, -3.4e38, np.inf, -np.inf], np.float32),
        # exact ties: low half 0x8000 with even and odd kept bit
        np.array([0x3F808000, 0x3F818000, 0x3F7F8000, 0x00008000], np.uint32).view(np.float32),
    ])
    ours = op.f32_to_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    back = op.bf16_to_f32(ours)
    ref_back = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(back.view(np.uint32), ref_back.view(np.uint32))
    nan = op.f32_to_bf16(np.array([np.nan], np.float32))
    assert np.isnan(op.bf16_to_f32(nan))[0]


# ---------------------------------------------------------------------------
# P-Reduce against the paper's matrix form
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(6))
def test_preduce_matches_dense_FG(seed):
    rs = np.random.default_rng(seed)
    n, p = int(rs.integers(2, 9)), int(rs.integers(1, 65))
    X = rng_f32(rs, (n, p))
    groups = random_groups(rs, n)
    got = op.preduce(X, groups)
    # X in the paper is weights x workers; x'_j = sum_i x_i F_ij.
    exact = (X.astype(np.float64).T @ dense_F(n, groups)).T
    absum = (np.abs(X).astype(np.float64).T @ np.abs(dense_F(n, groups))).T
    for g in groups:
        k = len(g)
        bound = (k + 2) * U32 * absum[list(g)]
        assert np.all(np.abs(got[list(g)] - exact[list(g)]) <= bound)


def test_allreduce_special_case_is_mean():
    # k = N: P-Reduce over all workers is All-Reduce (mean), Sec. 3.2.
    rs = np.random.default_rng(1)
    n, p = 7, 4099
    X = rng_f32(rs, (n, p))
    got = op.preduce(X, [tuple(range(n))])
    mean = np.mean(X.astype(np.float64), axis=0)
    bound = (n + 2) * U32 * np.mean(np.abs(X.astype(np.float64)), axis=0)
    for r in range(n):
        assert np.all(np.abs(got[r] - mean) <= bound)
        np.testing.assert_array_equal(got[r].view(np.uint32), got[0].view(np.uint32))


def test_pair_average_is_correctly_rounded():
    # k = 2 is the AD-PSGD pair average x_i, x_j <- (x_i + x_j)/2 (Fig. 3):
    # fp32 sum then *0.5 is the correctly rounded half-sum.
    rs = np.random.default_rng(2)
    X = rng_f32(rs, (4, 100000))
    got = op.preduce(X, [(0, 3), (1, 2)])
    for a, b in [(0, 3), (1, 2)]:
        ref = ((X[a].astype(np.float64) + X[b].astype(np.float64)) / 2).astype(np.float32)
        np.testing.assert_array_equal(got[a].view(np.uint32), ref.view(np.uint32))
        np.testing.assert_array_equal(got[b].view(np.uint32), ref.view(np.uint32))


def test_singleton_group_and_non_members_untouched():
    # F^G_uu = 1 for u outside G; a group of one is the identity.
    rs = np.random.default_rng(3)
    X = rng_f32(rs, (6, 1001))
    got = op.preduce(X, [(1,), (2, 4)])
    for r in (0, 1, 3, 5):
        np.testing.assert_array_equal(got[r].view(np.uint32), X[r].view(np.uint32))
    assert not np.array_equal(got[2], X[2])


def test_members_identical_and_mean_preserved():
    # Doubly stochastic F^G (Sec. 3.3): column sums 1 => sum over workers kept.
    rs = np.random.default_rng(4)
    n = 8
    X = rng_f32(rs, (n, 5000))
    groups = [(0, 2, 5), (1, 3, 4, 6, 7)]
    got = op.preduce(X, groups)
    for g in groups:
        for m in g[1:]:
            np.testing.assert_array_equal(got[m].view(np.uint32), got[g[0]].view(np.uint32))
    before = X.astype(np.float64).sum(axis=0)
    after = got.astype(np.float64).sum(axis=0)
    bound = 8 * U32 * np.abs(X.astype(np.float64)).sum(axis=0)
    assert np.all(np.abs(after - before) <= bound)


def test_idempotent():
    # (F^G)^T F^G = F^G (Sec. 3.3): applying P-Reduce twice equals once.
    # Exact in fp32 for k <= 2; within 2 ulp otherwise (sum of k equal values).
    rs = np.random.default_rng(5)
    X = rng_f32(rs, (8, 20000))
    groups = [(0,), (1, 6), (2, 3, 7), (4, 5)]
    once = op.preduce(X, groups)
    twice = op.preduce(once, groups)
    for g in groups:
        if len(g) <= 2:
            np.testing.assert_array_equal(twice[list(g)].view(np.uint32),
                                          once[list(g)].view(np.uint32))
        else:
            d = np.abs(twice[list(g)].view(np.int32).astype(np.int64) -
                       once[list(g)].view(np.int32).astype(np.int64))
            assert d.max() <= 2


def test_idempotence_of_F_exact():
    # The matrix identity itself, in exact rational arithmetic.
    for groups in ([(0, 1, 2)], [(0, 3), (1, 2, 4)], [(0, 1, 2, 3, 4)]):
        F = [[Fraction(int(i == j)) for j in range(5)] for i in range(5)]
        for g in groups:
            for i in g:
                for j in g:
                    F[i][j] = Fraction(1, len(g))
        FtF = [[sum(F[l][i] * F[l][j] for l in range(5)) for j in range(5)] for i in range(5)]
        assert FtF == F


def _read_matrices(path):
    mats, name, rows = {}, None, []
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        if "/" in line or line.replace(" ", "").isdigit():
            rows.append([Fraction(x) for x in line.split()])
            if len(rows) == 5:
                mats[name], rows = rows, []
        else:
            name = line
    return mats


def test_conflict_worked_example():
    """Sec. 3.1-3.2: two conflicting pair syncs (0,3) then (4,3) compose to
    W_fused; P-Reduce of {0,3,4} is the relaxed F^G.  Both doubly stochastic,
    and they differ."""
    m = _read_matrices(os.path.join(GOLDEN, "conflict_example.txt"))
    mul = lambda A, B: [[sum(A[i][l] * B[l][j] for l in range(5)) for j in range(5)]
                        for i in range(5)]
    assert mul(m["W_k"], m["W_k1"]) == m["W_fused"]
    for M in m.values():
        assert all(sum(r) == 1 for r in M)
        assert all(sum(M[i][j] for i in range(5)) == 1 for j in range(5))
    assert m["W_fused"] != m["F_034"]

    # The oracle reproduces both with inputs whose results are exact in fp32.
    rs = np.random.default_rng(6)
    X = (rs.integers(-1000, 1000, size=(5, 257)) * 4).astype(np.float32)
    seq = op.preduce(op.preduce(X, [(0, 3)]), [(3, 4)])
    Wf = np.array([[float(x) for x in r] for r in m["W_fused"]])
    np.testing.assert_array_equal(seq, (X.astype(np.float64).T @ Wf).T.astype(np.float32))
    X3 = (rs.integers(-1000, 1000, size=(5, 257)) * 3).astype(np.float32)
    got = op.preduce(X3, [(0, 3, 4)])
    F = np.array([[float(x) for x in r] for r in m["F_034"]])
    exact = (X3.astype(np.float64).T @ F).T
    assert np.all(np.abs(got - exact) <= 5 * U32 * np.abs(X3).sum(axis=0) / 3)


# ---------------------------------------------------------------------------
# local update (Step 2) against closed forms
# ---------------------------------------------------------------------------
def test_sgd_closed_form():
    rs = np.random.default_rng(7)
    n, p, T, lr = 3, 4096, 25, 0.1
    W0 = rng_f32(rs, (n, p))
    G = rng_f32(rs, (n, p), 0.01)
    W = W0
    for _ in range(T):
        W, _ = op.step(W, G, None, [], range(n), lr=lr)
    exact = W0.astype(np.float64) - T * np.float64(np.float32(lr)) * G.astype(np.float64)
    # each of the T steps rounds the product and the difference
    bound = T * 2 * U32 * (np.abs(W0).astype(np.float64) + T * lr * np.abs(G) + 1e-30)
    assert np.all(np.abs(W - exact) <= bound)
    # a sign slip moves by 2*T*lr*g, far outside the bound
    assert np.max(np.abs(W - exact)) < 1e-2 * T * lr * np.max(np.abs(G))


def test_momentum_closed_form():
    # v_t = mu v_{t-1} + g, v_0 = 0  =>  v_t = g (1 - mu^t)/(1 - mu);
    # w_T = w_0 - lr * g * sum_{t=1..T} (1 - mu^t)/(1 - mu).
    rs = np.random.default_rng(8)
    n, p, T, lr, mu = 2, 4096, 30, 0.1, 0.9
    W = rng_f32(rs, (n, p))
    W0 = W.copy()
    G = rng_f32(rs, (n, p), 0.01)
    V = np.zeros_like(W)
    for _ in range(T):
        W, V = op.step(W, G, V, [], range(n), lr=lr, momentum=mu)
    mu64, lr64 = np.float64(np.float32(mu)), np.float64(np.float32(lr))
    vT = G.astype(np.float64) * (1 - mu64 ** T) / (1 - mu64)
    coef = sum((1 - mu64 ** t) / (1 - mu64) for t in range(1, T + 1))
    wT = W0.astype(np.float64) - lr64 * G.astype(np.float64) * coef
    assert np.all(np.abs(V - vT) <= 4 * T * U32 * np.abs(G) / (1 - mu64))
    assert np.all(np.abs(W - wT) <= 4 * T * U32 * (np.abs(W0) + lr * coef * np.abs(G)))


def test_fused_equals_unfused_for_fp32():
    rs = np.random.default_rng(9)
    n = 6
    X, G = rng_f32(rs, (n, 3000)), rng_f32(rs, (n, 3000), 0.01)
    V = rng_f32(rs, (n, 3000), 0.01)
    groups, active = [(0, 2, 3), (4, 5)], [0, 1, 2, 5]
    a = op.step(X, G, V, groups, active, 0.1, 0.9, fused=True)
    b = op.step(X, G, V, groups, active, 0.1, 0.9, fused=False)
    np.testing.assert_array_equal(a[0].view(np.uint32), b[0].view(np.uint32))
    np.testing.assert_array_equal(a[1].view(np.uint32), b[1].view(np.uint32))


def test_step_against_float64_definition():
    """Fused step (update of active workers, then P-Reduce; members that did
    not update contribute their stored value) against the float64 statement
    X' = (X - lr G diag(1_A)) F^G."""
    rs = np.random.default_rng(10)
    n, p, lr = 8, 3001, 0.1
    X, G = rng_f32(rs, (n, p)), rng_f32(rs, (n, p), 0.01)
    groups, active = [(0, 3, 6), (1, 7), (2,)], [0, 2, 4, 6, 7]
    got, _ = op.step(X, G, None, groups, active, lr)
    D = np.zeros(n)
    D[active] = 1.0
    upd = X.astype(np.float64) - np.float64(np.float32(lr)) * G.astype(np.float64) * D[:, None]
    exact = (upd.T @ dense_F(n, groups)).T
    absum = (np.abs(upd).T @ np.abs(dense_F(n, groups))).T
    assert np.all(np.abs(got - exact) <= 12 * U32 * absum)
    # non-member, non-active replicas are bit-identical
    for r in (5,):
        np.testing.assert_array_equal(got[r].view(np.uint32), X[r].view(np.uint32))


def test_bf16_step_rounds_once():
    """bf16 storage: the fused step's stored value is the float64 result
    rounded to bf16, up to the fp32 arithmetic error (one bf16 ulp at most)."""
    rs = np.random.default_rng(11)
    n, p = 8, 20000
    Xf = rng_f32(rs, (n, p), 1e-2)
    Gf = rng_f32(rs, (n, p), 1e-3)
    X, G = op.f32_to_bf16(Xf), op.f32_to_bf16(Gf)
    lr = 100.0      # large enough that the update survives bf16 rounding
    groups, active = [(0, 1, 2, 3), (4, 6)], list(range(n))
    got, _ = op.step(X, G, None, groups, active, lr, dtype=op.BF16)
    Xw, Gw = op.bf16_to_f32(X).astype(np.float64), op.bf16_to_f32(G).astype(np.float64)
    exact = ((Xw - np.float64(np.float32(lr)) * Gw).T @ dense_F(n, groups)).T
    ref = op.f32_to_bf16(exact.astype(np.float32))
    d = np.abs(got.view(np.int16).astype(np.int32) - ref.view(np.int16).astype(np.int32))
    assert d.max() <= 1
    assert (d == 0).mean() > 0.99
    # the update is visible: dropping it changes most elements
    no_upd, _ = op.step(X, G, None, groups, [], lr, dtype=op.BF16)
    assert (no_upd != got).mean() > 0.5


def test_schedule_validation():
    X = np.zeros((4, 8), np.float32)
    with pytest.raises(ValueError):
        op.preduce(X, [(0, 1), (1, 2)])
    with pytest.raises(ValueError):
        op.preduce(X, [(2, 1)])
    with pytest.raises(ValueError):
        op.preduce(X, [(0, 4)])


def test_weight_decay_closed_form():
    # SGD with weight decay and constant g: w_{t+1} = (1 - lr*wd) w_t - lr*g,
    # so w_T = (w_0 + g/wd) (1 - lr*wd)^T - g/wd.
    rs = np.random.default_rng(12)
    n, p, T, lr, wd = 2, 4096, 40, 0.1, 1e-2
    W = rng_f32(rs, (n, p))
    W0 = W.copy()
    G = rng_f32(rs, (n, p), 0.01)
    for _ in range(T):
        W, _ = op.step(W, G, None, [], range(n), lr=lr, weight_decay=wd)
    lr64, wd64 = np.float64(np.float32(lr)), np.float64(np.float32(wd))
    a = 1 - lr64 * wd64
    G64 = G.astype(np.float64)
    exact = (W0.astype(np.float64) + G64 / wd64) * a ** T - G64 / wd64
    assert np.all(np.abs(W - exact) <= 4 * T * U32 * (np.abs(W0) + T * lr * np.abs(G)))
    # dropping the decay term moves w by about T*lr*wd*|w|, far outside the bound
    W_nodecay = W0 - np.float32(T * lr) * G
    assert np.max(np.abs(W_nodecay - exact)) > 100 * np.max(4 * T * U32 * np.abs(W0))


def test_nesterov_closed_form():
    # v_t = g (1 - mu^t)/(1 - mu); Nesterov step d_t = g + mu v_t;
    # w_T = w_0 - lr * sum_{t=1..T} d_t.
    rs = np.random.default_rng(13)
    n, p, T, lr, mu = 2, 4096, 30, 0.1, 0.9
    W = rng_f32(rs, (n, p))
    W0 = W.copy()
    G = rng_f32(rs, (n, p), 0.01)
    V = np.zeros_like(W)
    for _ in range(T):
        W, V = op.step(W, G, V, [], range(n), lr=lr, momentum=mu, nesterov=True)
    mu64, lr64 = np.float64(np.float32(mu)), np.float64(np.float32(lr))
    G64 = G.astype(np.float64)
    coef = sum(1 + mu64 * (1 - mu64 ** t) / (1 - mu64) for t in range(1, T + 1))
    exact = W0.astype(np.float64) - lr64 * G64 * coef
    assert np.all(np.abs(W - exact) <= 6 * T * U32 * (np.abs(W0) + lr * coef * np.abs(G)))
    # heavy-ball (no look-ahead) ends elsewhere: sum of v_t differs from sum of d_t
    coef_hb = sum((1 - mu64 ** t) / (1 - mu64) for t in range(1, T + 1))
    assert abs(coef - coef_hb) > 1.0
