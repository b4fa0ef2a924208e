"""The oracle's pins catch plausible mistakes (CPU only).

Each case plants one mistake in the oracle (on the CPU, by patching a
function for the duration of the check) and requires that at least one pin
test of tests/test_oracle_preduce.py or tests/test_oracle_sched.py fails.
"""
import contextlib
from collections import deque

import numpy as np
import pytest

import test_oracle_draws as td
import test_oracle_preduce as tp
import test_oracle_sched as ts
from oracle import preduce as op
from oracle import sched as osd
from oracle import splitmix as osm

PRE_PINS = [
    *[(tp.test_preduce_matches_dense_FG, (s,)) for s in range(6)],
    (tp.test_allreduce_special_case_is_mean, ()),
    (tp.test_pair_average_is_correctly_rounded, ()),
    (tp.test_singleton_group_and_non_members_untouched, ()),
    (tp.test_members_identical_and_mean_preserved, ()),
    (tp.test_idempotent, ()),
    (tp.test_conflict_worked_example, ()),
    (tp.test_sgd_closed_form, ()),
    (tp.test_momentum_closed_form, ()),
    (tp.test_weight_decay_closed_form, ()),
    (tp.test_nesterov_closed_form, ()),
    (tp.test_step_against_float64_definition, ()),
    (tp.test_bf16_step_rounds_once, ()),
    (tp.test_bf16_rounding_matches_torch, ()),
]

SCHED_PINS = [
    (ts.test_group_generator_walkthrough, ()),
    (ts.test_global_division_example, ()),
    (ts.test_rule_table_matches_fig8_and_fig9, ()),
    *[(ts.test_static_table_partitions_and_connects, a)
      for a in [(16, 4, 2), (16, 8, 3), (8, 4, 5), (12, 3, 11)]],
    (ts.test_table_mode_straggler_waits_for_same_iteration, ()),
    *[(ts.test_group_buffer_invariants, a)
      for a in [(osd.RANDOM_GB, 0), (osd.GD, 0), (osd.GD, 3)]],
    (ts.test_random_group_contains_requester, ()),
    (ts.test_slowdown_filter_rule, ()),
]


def static_row_pin(n, k):
    with pytest.MonkeyPatch.context() as mp:
        td.test_static_row_is_a_uniform_partition(n, k, mp)


DRAW_PINS = [
    (td.test_bounded_power_of_two_is_the_top_bits, ()),
    *[(td.test_bounded_depends_on_the_high_word_only, (n,)) for n in (3, 7, 100)],
    *[(td.test_shuffle_gives_every_permutation_once, (n,)) for n in (3, 4, 5)],
    *[(td.test_partial_shuffle_gives_every_ordered_selection_once, a)
      for a in [(4, 2), (5, 3), (5, 5)]],
    *[(td.test_random_group_draws_every_subset, a) for a in [(4, 0), (5, 2)]],
    *[(td.test_global_division_order_is_every_permutation, (n,)) for n in (3, 4)],
    (td.test_global_division_pairs_are_uniform, ()),
    *[(td.test_chunks_order_is_every_permutation, (n,)) for n in (3, 4)],
    *[(static_row_pin, a) for a in [(4, 2), (6, 3)]],
    *[(td.test_adpsgd_partner_is_every_other_worker_once, a) for a in [(4, 0), (5, 3)]],
    (td.test_inter_intra_heads_and_their_order, ()),
]


@contextlib.contextmanager
def patched(obj, name, value):
    old = getattr(obj, name)
    setattr(obj, name, value)
    try:
        yield
    finally:
        setattr(obj, name, old)


def failures(pins):
    n = 0
    for fn, args in pins:
        try:
            fn(*args)
        except (AssertionError, ValueError, IndexError, ZeroDivisionError, KeyError):
            n += 1
    return n


# --- mistakes in the arithmetic ---------------------------------------------
def mean_drops_last(values):
    k = len(values)
    s = np.array(values[0], dtype=np.float32, copy=True)
    for x in values[1:-1]:
        s = s + x
    return s * op.inv_k(k)


def mean_of_first_two(values):
    return op.inv_k(2) * (values[0] + values[1 % len(values)])


def mean_wrong_divisor(values):
    k = len(values)
    s = np.array(values[0], dtype=np.float32, copy=True)
    for x in values[1:]:
        s = s + x
    return s * op.inv_k(k + 1)


def update_sign_flip(w, g, v, lr, momentum, wd=0.0, nesterov=False):
    u, v2 = ORIG_UPDATE(w, g, v, lr, momentum, wd, nesterov)
    return w + (w - u), v2


def update_lr_inside_momentum(w, g, v, lr, momentum, wd=0.0, nesterov=False):
    if momentum is None:
        return ORIG_UPDATE(w, g, v, lr, momentum, wd, nesterov)
    v_new = np.float32(momentum) * v + np.float32(lr) * g
    return w - v_new, v_new


def update_uses_old_velocity(w, g, v, lr, momentum, wd=0.0, nesterov=False):
    if momentum is None:
        return ORIG_UPDATE(w, g, v, lr, momentum, wd, nesterov)
    v_new = np.float32(momentum) * v + g
    return w - np.float32(lr) * v, v_new


def update_decay_sign_flipped(w, g, v, lr, momentum, wd=0.0, nesterov=False):
    return ORIG_UPDATE(w, g, v, lr, momentum, -wd, nesterov)


def update_ignores_nesterov(w, g, v, lr, momentum, wd=0.0, nesterov=False):
    return ORIG_UPDATE(w, g, v, lr, momentum, wd, False)


def bf16_truncate(x):
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return (b >> np.uint32(16)).astype(np.uint16)


def bf16_ties_away(x):
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return ((b + np.uint32(0x8000)) >> np.uint32(16)).astype(np.uint16)


ORIG_UPDATE = op.local_update
ORIG_STEP = op.step


def step_updates_every_member(param, grad, mom, groups, active, lr=0.0, momentum=None,
                              dtype=op.F32, fused=True, weight_decay=0.0, nesterov=False):
    if grad is not None:
        active = sorted(set(active) | {m for g in groups for m in g})
    return ORIG_STEP(param, grad, mom, groups, active, lr, momentum, dtype, fused,
                     weight_decay, nesterov)


ARITH = [
    ("sum drops the last member", "group_mean", mean_drops_last),
    ("mean of the first two members only", "group_mean", mean_of_first_two),
    ("divides by k+1", "group_mean", mean_wrong_divisor),
    ("update sign flipped", "local_update", update_sign_flip),
    ("lr folded into the velocity", "local_update", update_lr_inside_momentum),
    ("update uses the old velocity", "local_update", update_uses_old_velocity),
    ("weight decay sign flipped", "local_update", update_decay_sign_flipped),
    ("Nesterov look-ahead ignored", "local_update", update_ignores_nesterov),
    ("bf16 truncates", "f32_to_bf16", bf16_truncate),
    ("bf16 rounds ties away from zero", "f32_to_bf16", bf16_ties_away),
    ("update applied to every group member", "step", step_updates_every_member),
]


@pytest.mark.parametrize("label,name,fn", ARITH, ids=[a[0] for a in ARITH])
def test_arithmetic_mistake_is_caught(label, name, fn):
    assert failures(PRE_PINS) == 0
    with patched(op, name, fn):
        assert failures(PRE_PINS) > 0, f"no pin caught: {label}"


# --- mistakes in the scheduler ----------------------------------------------
def random_group_without_requester(self, i):
    n = self.n
    k = min(self.kmin + self.rng.bounded(self.kmax - self.kmin + 1), n)
    others = [j for j in range(n) if j != i]
    for j in range(k):
        x = j + self.rng.bounded(max(1, n - 1 - j)) if j < n - 1 else j
        others[j], others[min(x, n - 2)] = others[min(x, n - 2)], others[j]
    self._new_group(others[:k])


def step_ignores_buffer_order(self, t, eligible=None):
    # runs every group whose members are all waiting, heads or not
    if t != self.t:
        raise ValueError("steps must be consecutive")
    self.t += 1
    n = self.n
    elig = [True] * n if eligible is None else [bool(e) for e in eligible]
    active = [i for i in range(n) if elig[i] and not self.waiting[i]]
    for i in active:
        self._request(i)
    executed = []
    for h in sorted(self.groups):
        g = self.groups[h]
        if all(self.waiting[m] for m in g):
            executed.append((h, g))
    out = []
    for h, g in executed:
        for m in g:
            if h in self.gb[m]:
                self.gb[m].remove(h)
            self.waiting[m] = bool(self.gb[m]) and False
            self.syncs[m] += 1
        out.append(g)
        del self.groups[h]
    return active, out


def division_filter_reversed(self, i):
    idle = [w for w in range(self.n) if not self.gb[w] and
            (self.c_thres <= 0 or self.c[w] - self.c[i] < self.c_thres)]
    for a in range(len(idle) - 1, 0, -1):
        b = self.rng.bounded(a + 1)
        idle[a], idle[b] = idle[b], idle[a]
    pos, made = 0, []
    while pos < len(idle):
        k = self.kmin + self.rng.bounded(self.kmax - self.kmin + 1)
        made.append(self.groups[self._new_group(idle[pos:pos + k])])
        pos += k
    self.divisions.append((i, list(self.c), made))


def rule_table_no_ring(n_nodes):
    rows = ORIG_RULE(n_nodes)
    rows[2] = [g for g in rows[2] if not (len(g) == 2 and g[0] % 4 == 1)]
    return rows


ORIG_RULE = osd.rule_table

SCHED = [
    ("random group leaves out its requester", osd.Scheduler, "_random_group",
     random_group_without_requester),
    ("groups run without waiting for their turn in the buffer", osd.Scheduler, "step",
     step_ignores_buffer_order),
    ("slowdown filter reversed", osd.Scheduler, "_global_division", division_filter_reversed),
    ("ring pairs of phase 2 missing", osd, "rule_table", rule_table_no_ring),
]


@pytest.mark.parametrize("label,obj,name,fn", SCHED, ids=[a[0] for a in SCHED])
def test_scheduler_mistake_is_caught(label, obj, name, fn):
    assert failures(SCHED_PINS) == 0
    with patched(obj, name, fn):
        assert failures(SCHED_PINS) > 0, f"no pin caught: {label}"


# --- mistakes in the seeded draws -------------------------------------------
def bounded_modulo(self, n):
    return self.next() % n


def bounded_low_bits(self, n):
    return ((self.next() & 0xFFFFFFFF) * n) >> 32


def shuffle_sattolo(items, rng):
    for a in range(len(items) - 1, 0, -1):
        b = rng.bounded(a)
        items[a], items[b] = items[b], items[a]
    return items


def shuffle_stops_early(items, rng):
    for a in range(len(items) - 1, 1, -1):
        b = rng.bounded(a + 1)
        items[a], items[b] = items[b], items[a]
    return items


def shuffle_range_too_wide(items, rng):
    for a in range(len(items) - 1, 0, -1):
        b = min(rng.bounded(a + 2), a)
        items[a], items[b] = items[b], items[a]
    return items


def partial_shuffle_without_offset(items, m, rng):
    for j in range(m):
        x = rng.bounded(len(items) - j)
        items[j], items[x] = items[x], items[j]
    return items


ORIG_ADPSGD = osd.Scheduler._adpsgd_step
ORIG_INTER_INTRA = osd.Scheduler._inter_intra_division


def adpsgd_partner_may_be_self(self, active):
    # draws the partner over all n workers instead of the n-1 others
    for i in active:
        self.c[i] += 1
        if self.n == 1:
            self.skips[i] += 1
            continue
        self.partner[i] = self.rng.bounded(self.n - 1)
        self.seq[i] = self.next_id
        self.next_id += 1
        self.waiting[i] = True
    locked, executed = set(), []
    for i in sorted((w for w in range(self.n) if self.waiting[w]), key=lambda w: self.seq[w]):
        j = self.partner[i]
        if i in locked or j in locked:
            continue
        locked |= {i, j}
        self.waiting[i] = False
        self.syncs[i] += 1
        executed.append(tuple(sorted({i, j})))
    return executed


def inter_intra_first_worker_heads(self, i):
    # the head of each node is always its first idle worker, not a draw
    # (the division draws the heads first, one per node)
    rng = self.rng
    idle = [w for w in range(self.n) if not self.gb[w]]
    nodes = len({w // self.per_node for w in idle})
    calls = {"n": 0}

    class Wrapped:
        def bounded(self, n):
            calls["n"] += 1
            if calls["n"] <= nodes:
                return 0
            return rng.bounded(n)
    self.rng = Wrapped()
    try:
        ORIG_INTER_INTRA(self, i)
    finally:
        self.rng = rng


DRAWS = [
    ("bounded takes the output modulo n", osm.Stream, "bounded", bounded_modulo),
    ("bounded maps the low 32 bits", osm.Stream, "bounded", bounded_low_bits),
    ("Sattolo's cyclic shuffle instead of Fisher-Yates", osd, "shuffle", shuffle_sattolo),
    ("Fisher-Yates stops one position early", osd, "shuffle", shuffle_stops_early),
    ("Fisher-Yates draws from one slot too many", osd, "shuffle", shuffle_range_too_wide),
    ("partial shuffle forgets the +j offset", osd, "partial_shuffle",
     partial_shuffle_without_offset),
    ("AD-PSGD partner drawn without skipping the requester", osd.Scheduler, "_adpsgd_step",
     adpsgd_partner_may_be_self),
    ("Inter-Intra head is always the node's first idle worker", osd.Scheduler,
     "_inter_intra_division", inter_intra_first_worker_heads),
]


@pytest.mark.parametrize("label,obj,name,fn", DRAWS, ids=[a[0] for a in DRAWS])
def test_draw_mistake_is_caught(label, obj, name, fn):
    assert failures(DRAW_PINS) == 0
    with patched(obj, name, fn):
        assert failures(DRAW_PINS) > 0, f"no pin caught: {label}"
