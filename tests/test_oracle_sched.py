"""Pins for the oracle's group scheduler (CPU only).

Checked against the paper's worked examples (the Group Generator walk-through
of Sec. 4.1, the Global Division example of Sec. 5.1, the static schedule
facts of Fig. 8 and the rule table of Fig. 9), the published SplitMix64
reference outputs, and the invariants the protocol fixes: groups of one step
are disjoint, every request is served by exactly one group, nobody waits
forever, and each period of a static schedule connects all workers.
"""
import os
import random

import pytest

from oracle import sched as os_
from oracle.splitmix import Stream

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_splitmix_reference_outputs():
    lines = [l.split() for l in open(os.path.join(GOLDEN, "splitmix64_seed1234567.txt"))
             if l.strip() and not l.startswith("#")]
    seed = int(lines[0][1])
    want = [int(l[0]) for l in lines[1:]]
    s = Stream(seed)
    assert [s.next() for _ in want] == want


def test_bounded_range_and_spread():
    s = Stream(42)
    xs = [s.bounded(7) for _ in range(70000)]
    assert min(xs) == 0 and max(xs) == 6
    for v in range(7):
        assert abs(xs.count(v) - 10000) < 500


def check_step_invariants(sch, active, groups, n):
    seen = set()
    for g in groups:
        assert list(g) == sorted(set(g))
        assert not (seen & set(g)), "groups of one step overlap"
        seen |= set(g)
    assert active == sorted(set(active))
    for i in range(n):
        assert sch.syncs[i] + sch.skips[i] + int(sch.waiting[i]) == sch.c[i]


def test_group_generator_walkthrough():
    """Sec. 4.1: of 8 workers, W0 and W7 request first; the generator forms
    [0,4,5] for W0, then [4,5,7] for W7, which conflicts (W4, W5) and stays
    pending until [0,4,5] has run and released its locks."""
    s = os_.Scheduler(8, os_.SCRIPTED, script=[(0, 4, 5), (4, 5, 7)])
    only = lambda *ws: [i in ws for i in range(8)]
    act, groups = s.step(0, only(0, 7))
    assert act == [0, 7] and groups == []
    assert list(s.gb[4]) == [0, 1] and list(s.gb[7]) == [1]
    act, groups = s.step(1, only(4, 5))       # W4, W5 reach their sync
    assert act == [4, 5] and groups == [(0, 4, 5)]
    assert s.waiting[7] and not s.waiting[4]
    act, groups = s.step(2, only(4, 5))       # next iteration: the pending group
    assert act == [4, 5] and groups == [(4, 5, 7)]
    assert not any(s.waiting)
    assert s.syncs == [1, 0, 0, 0, 2, 2, 0, 1]


def test_scripted_group_must_contain_requester():
    s = os_.Scheduler(4, os_.SCRIPTED, script=[(1, 2)])
    with pytest.raises(ValueError):
        s.step(0, [True, False, False, False])


def test_global_division_example():
    """Sec. 5.1, Fig. 10: with 4 idle workers, W0's request divides all of
    them into two disjoint pairs; W3's later request gets its pair from the
    buffer without generating anything."""
    s = os_.Scheduler(4, os_.GD, seed=7, kmin=2, kmax=2)
    only = lambda *ws: [i in ws for i in range(4)]
    act, groups = s.step(0, only(0))
    assert s.next_id == 2
    made = sorted(s.groups.values())
    assert sorted(m for g in made for m in g) == [0, 1, 2, 3]
    assert all(len(g) == 2 for g in made)
    w0 = [g for g in made if 0 in g][0]
    w3 = [g for g in made if 3 in g][0]
    if w0 == w3:
        return  # same pair: nothing more to show
    act, groups = s.step(1, only(3))
    assert s.next_id == 2          # no new group for W3
    others = [m for m in w3 if m != 3]
    act, groups = s.step(2, only(*others))
    assert groups == [w3]


def test_rule_table_matches_fig8_and_fig9():
    rows = os_.rule_table(4)           # 16 workers on 4 nodes
    assert len(rows) == 4
    # Fig. 8: W0, W4, W8, W12 form one group in iteration 4k
    assert (0, 4, 8, 12) in rows[0]
    # Fig. 8: W2, W6, W10, W14 do not synchronize in iteration 4k+2
    in_row2 = {m for g in rows[2] for m in g}
    assert {2, 6, 10, 14}.isdisjoint(in_row2)
    # Fig. 9 phase 0: LW1 idle, LW2 with LW3; phase 2: LW1 with the opposite node's LW1
    assert {1, 5, 9, 13}.isdisjoint({m for g in rows[0] for m in g})
    assert (2, 3) in rows[0] and (14, 15) in rows[0]
    assert (1, 9) in rows[2] and (5, 13) in rows[2] and (0, 3) in rows[2]
    assert rows[1] == rows[3] == [(0, 1, 2, 3), (4, 5, 6, 7), (8, 9, 10, 11), (12, 13, 14, 15)]
    assert os_.union_connected(16, rows)
    s = os_.Scheduler(16, os_.RULE, n_nodes=4)
    for t in range(12):
        act, groups = s.step(t)
        assert act == list(range(16))
        assert groups == rows[t % 4]
        check_step_invariants(s, act, groups, 16)


@pytest.mark.parametrize("n,k,seed", [(16, 4, 2), (16, 8, 3), (8, 4, 5), (12, 3, 11)])
def test_static_table_partitions_and_connects(n, k, seed):
    rows = os_.static_table(n, k, 4, seed)
    for row in rows:
        assert sorted(m for g in row for m in g) == list(range(n))
        assert all(len(g) == k for g in row)
        assert [g[0] for g in row] == sorted(g[0] for g in row)
    assert os_.union_connected(n, rows)
    s = os_.Scheduler(n, os_.STATIC, seed=seed, group_size=k, period=4)
    for t in range(9):
        act, groups = s.step(t)
        assert act == list(range(n)) and groups == rows[t % 4]


def test_static_rejects_disconnected_and_bad_sizes():
    with pytest.raises(ValueError):
        os_.static_table(10, 4, 4, 0)
    with pytest.raises(ValueError):
        os_.static_table(8, 1, 4, 0)      # singletons never connect


def test_table_mode_straggler_waits_for_same_iteration():
    """A static schedule cannot route around a slow worker (Sec. 4.3): its
    groups only run when every member is at the same iteration."""
    rows = os_.static_table(8, 2, 4, 9)
    s = os_.Scheduler(8, os_.STATIC, seed=9, group_size=2, period=4)
    for t in range(200):
        elig = [True] * 8
        elig[0] = (t % 4 == 0)
        act, groups = s.step(t, elig)
        check_step_invariants(s, act, groups, 8)
        for g in groups:
            its = {s.c[m] for m in g}
            assert len(its) == 1
            it = its.pop() - 1
            assert g in rows[it % 4]
    # worker 0 ran 50 iterations; everyone is within a period-bounded lead
    assert s.c[0] == 50
    assert max(s.c) <= s.c[0] + 8


@pytest.mark.parametrize("mode,c_thres", [(os_.RANDOM_GB, 0), (os_.GD, 0), (os_.GD, 3)])
def test_group_buffer_invariants(mode, c_thres):
    n = 32
    s = os_.Scheduler(n, mode, seed=4, kmin=2, kmax=8, c_thres=c_thres)
    last_served = [0] * n
    for t in range(600):
        elig = [True] * n
        elig[0] = (t % 4 == 0)
        act, groups = s.step(t, elig)
        check_step_invariants(s, act, groups, n)
        for g in groups:
            if mode == os_.RANDOM_GB:
                assert 2 <= len(g) <= 8
            for m in g:
                last_served[m] = t
        for i in range(n):
            if s.waiting[i]:
                assert t - last_served[i] < 120, "worker starved"
    assert all(c > 0 for c in s.syncs)


def test_random_group_contains_requester():
    s = os_.Scheduler(10, os_.RANDOM_GB, seed=1, kmin=3, kmax=5)
    only = lambda *ws: [i in ws for i in range(10)]
    s.step(0, only(6))
    g = s.groups[0]
    assert 6 in g and 3 <= len(g) <= 5


def test_slowdown_filter_rule():
    """Sec. 5.3: a division started by worker i only admits workers w with
    c_i - c_w < C_thres; with the filter, most workers stop depending on the
    slow one."""
    n, steps = 8, 400

    def run(c_thres):
        s = os_.Scheduler(n, os_.GD, seed=3, kmin=2, kmax=2, c_thres=c_thres)
        for t in range(steps):
            elig = [True] * n
            elig[0] = (t % 8 == 0)
            s.step(t, elig)
        return s

    s = run(2)
    assert s.divisions
    for i, c, made in s.divisions:
        members = {m for g in made for m in g}
        assert i in members
        assert all(c[i] - c[w] < 2 for w in members)
        idle_ok = [w for w in range(n) if c[i] - c[w] < 2]
        assert members <= set(idle_ok)
    nofilter = run(0)
    assert any(c[i] - c[w] >= 2 for i, c, made in nofilter.divisions
               for g in made for w in g)
    full = lambda sch: sum(1 for c in sch.c if c >= 0.95 * steps)
    assert full(s) >= n - 2 > full(nofilter)


@pytest.mark.parametrize("n,nodes,kmin,kmax", [(16, 4, 2, 3), (32, 4, 2, 8), (12, 3, 1, 2)])
def test_inter_intra_division(n, nodes, kmin, kmax):
    """Sec. 5.2: a division gives every idle worker two buffered groups.  The
    inter-phase group is either a group of head workers (at most one per
    node, one head per node in all) or a group of one node's non-head
    workers; the intra-phase group is every idle worker of the node."""
    per = n // nodes
    s = os_.Scheduler(n, os_.INTER_INTRA, seed=5, kmin=kmin, kmax=kmax, n_nodes=nodes)
    s.step(0, [i == 0 for i in range(n)])          # only worker 0 asks: all others idle
    i, c, made = s.divisions[0]
    node = lambda w: w // per
    intra = made[-nodes:]
    inter = made[:-nodes]
    assert sorted(intra) == [tuple(range(nd * per, nd * per + per)) for nd in range(nodes)]
    assert sorted(m for g in inter for m in g) == list(range(n))
    heads = set()
    for g in inter:
        if len({node(m) for m in g}) > 1:
            heads |= set(g)
    # each multi-node group holds at most one worker per node
    for g in inter:
        nds = [node(m) for m in g]
        assert len(nds) == len(set(nds)) or len(set(nds)) == 1
    assert len({node(h) for h in heads}) == len(heads)
    for w in range(n):
        # worker 0's inter group may already have run (if it was alone)
        assert len(s.gb[w]) == (2 if w != 0 else len(s.gb[w]))
        assert s.groups[s.gb[w][-1]] == tuple(range(node(w) * per, node(w) * per + per))
    # run on: every worker alternates inter and intra phases; all stay served
    for t in range(1, 200):
        act, groups = s.step(t)
        check_step_invariants(s, act, groups, n)
    assert min(s.syncs) > 50


def test_adpsgd_pairs():
    """Fig. 3: every executed group is a pair holding its requester; pairs of
    one step are disjoint; the partner is uniform over the other workers; the
    oldest waiting request always runs (no starvation)."""
    n = 8
    s = os_.Scheduler(n, os_.ADPSGD, seed=13)
    partner_counts = [[0] * n for _ in range(n)]
    for t in range(3000):
        elig = [True] * n
        elig[0] = (t % 4 == 0)
        waiting_before = {w for w in range(n) if s.waiting[w]}
        act, groups = s.step(t, elig)
        check_step_invariants(s, act, groups, n)
        requesters = set(act) | waiting_before
        oldest = min((w for w in requesters if w in act or w in waiting_before),
                     key=lambda w: s.seq[w], default=None)
        for g in groups:
            assert len(g) == 2
            assert g[0] in requesters or g[1] in requesters
        if requesters:
            assert any(oldest in g for g in groups)
        for i in act:
            if s.waiting[i] or any(i in g for g in groups):
                partner_counts[i][s.partner[i]] += 1
    for i in range(1, n):
        row = [partner_counts[i][j] for j in range(n) if j != i]
        assert partner_counts[i][i] == 0
        assert max(row) < 1.4 * min(row)
    one = os_.Scheduler(1, os_.ADPSGD, seed=1)
    assert one.step(0) == ([0], []) and one.skips == [1]


def test_inter_intra_rejects_uneven_nodes():
    with pytest.raises(ValueError):
        os_.Scheduler(10, os_.INTER_INTRA, kmin=2, kmax=2, n_nodes=4)


def test_steps_must_be_consecutive():
    s = os_.Scheduler(4, os_.RANDOM_GB, seed=0, kmin=2, kmax=2)
    s.step(0)
    with pytest.raises(ValueError):
        s.step(2)
