"""Pins for the oracle's seeded draws (CPU only).

The group generator's random choices -- static rows (Sec. 4.2), random groups
(Step 3 of Fig. 4), Global Division (Sec. 5.1), the Inter-Intra division
(Sec. 5.2) and AD-PSGD's partners (Fig. 3) -- come from three pieces:

  bounded(n)        Lemire's multiply-shift map of a SplitMix64 output onto
                    [0, n): it uses the high 32 bits of the output;
  shuffle           Fisher-Yates from the last position down;
  partial_shuffle   the first m steps of Fisher-Yates from the front.

They are pinned here by what the mathematics fixes, not by re-running their
formulas: bounded(2^j) is the top j bits of the published SplitMix64 outputs,
and a shuffle driven through *every* possible draw sequence produces every
permutation (every ordered selection) exactly once -- the bijection that makes
Fisher-Yates uniform, which Sattolo's variant, off-by-one ranges and a
partial shuffle that forgets its offset all break.  The scheduler's uses of
them (static rows, random groups, divisions, chunks, Inter-Intra heads,
AD-PSGD partners) are enumerated the same way end to end.
"""
import itertools
import math
import os
from collections import Counter

import pytest

from oracle import sched as osd
from oracle.splitmix import Stream

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def golden_stream():
    lines = [l.split() for l in open(os.path.join(GOLDEN, "splitmix64_seed1234567.txt"))
             if l.strip() and not l.startswith("#")]
    return int(lines[0][1]), [int(l[0]) for l in lines[1:]]


# --- bounded(n) ---------------------------------------------------------------
def test_bounded_power_of_two_is_the_top_bits():
    """bounded(2^j) over the published seed-1234567 stream equals the top j
    bits of each output (a modulo or low-bits map gives the low bits)."""
    seed, outs = golden_stream()
    for j in range(1, 9):
        s = Stream(seed)
        assert [s.bounded(1 << j) for _ in outs] == [x >> (64 - j) for x in outs], j


class Fixed(Stream):
    """A stream whose outputs are given."""

    def __init__(self, outputs):
        super().__init__(0)
        self.outs = list(outputs)

    def next(self):
        return self.outs.pop(0)


@pytest.mark.parametrize("n", [1, 2, 3, 5, 7, 100, 1000003, (1 << 31) + 1])
def test_bounded_depends_on_the_high_word_only(n):
    """Outputs whose high 32 bits are all zero map to 0 and all ones to n-1,
    whatever the low bits; raising the high word never lowers the result."""
    lows = [0, 1, 0x7FFFFFFF, 0xFFFFFFFF, 0x9E3779B9]
    s = Fixed([lo for lo in lows] + [(0xFFFFFFFF << 32) | lo for lo in lows])
    assert [s.bounded(n) for _ in lows] == [0] * len(lows)
    assert [s.bounded(n) for _ in lows] == [n - 1] * len(lows)
    his = sorted({0, 1, 12345, 1 << 31, 0xDEADBEEF, 0xFFFFFFFE, 0xFFFFFFFF})
    s = Fixed([h << 32 | 0xFFFFFFFF for h in his])
    got = [s.bounded(n) for _ in his]
    assert got == sorted(got) and all(0 <= v < n for v in got)


# --- enumeration of every draw sequence --------------------------------------
class Scripted(Stream):
    """Answers bounded(n) from a prefix of chosen values, then 0; records the
    range of every draw so the caller can advance to the next sequence."""

    def __init__(self, prefix):
        super().__init__(0)
        self.prefix = list(prefix)
        self.values, self.ranges = [], []

    def bounded(self, n):
        assert n >= 1
        i = len(self.values)
        v = self.prefix[i] if i < len(self.prefix) else 0
        assert 0 <= v < n, "a replayed draw left its range"
        self.values.append(v)
        self.ranges.append(n)
        return v


def every_draw_sequence(run):
    """Runs `run(stream)` once per possible sequence of bounded() results
    (an odometer over the draw tree; later ranges may depend on earlier
    values) and returns the results in order."""
    out, prefix = [], []
    while True:
        s = Scripted(prefix)
        out.append(run(s))
        i = len(s.values) - 1
        while i >= 0 and s.values[i] + 1 >= s.ranges[i]:
            i -= 1
        if i < 0:
            return out
        prefix = s.values[:i] + [s.values[i] + 1]


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5])
def test_shuffle_gives_every_permutation_once(n):
    runs = every_draw_sequence(lambda s: tuple(osd.shuffle(list(range(n)), s)))
    assert len(runs) == math.factorial(n)
    assert sorted(runs) == sorted(itertools.permutations(range(n)))


@pytest.mark.parametrize("L,m", [(L, m) for L in range(1, 6) for m in range(0, L + 1)])
def test_partial_shuffle_gives_every_ordered_selection_once(L, m):
    items = [10 * x for x in range(L)]
    runs = every_draw_sequence(lambda s: tuple(osd.partial_shuffle(list(items), m, s)[:m]))
    assert len(runs) == math.perm(L, m)
    assert sorted(runs) == sorted(itertools.permutations(items, m))


def with_stream(sch, s):
    sch.rng = s
    return sch


@pytest.mark.parametrize("n,i", [(2, 0), (3, 1), (4, 0), (5, 2), (5, 4)])
def test_random_group_draws_every_subset(n, i):
    """A random group of size k (Step 3 of Fig. 4) holds its requester and a
    uniform (k-1)-subset of the others: over every draw sequence each size in
    [kmin, kmax] is drawn once, and each subset comes out (k-1)! times."""
    kmin, kmax = 1, n

    def run(s):
        sch = with_stream(osd.Scheduler(n, osd.RANDOM_GB, kmin=kmin, kmax=kmax), s)
        sch._random_group(i)
        (g,) = sch.groups.values()
        return g

    runs = Counter(every_draw_sequence(run))
    others = [j for j in range(n) if j != i]
    want = Counter()
    for k in range(kmin, kmax + 1):
        for sub in itertools.combinations(others, k - 1):
            want[tuple(sorted((i,) + sub))] += math.factorial(k - 1)
    assert runs == want


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5])
def test_global_division_order_is_every_permutation(n):
    """Global Division (Sec. 5.1) with groups of one: the groups come out in
    the shuffled order of the idle workers, so over every draw sequence each
    order of the n workers appears exactly once."""
    def run(s):
        sch = with_stream(osd.Scheduler(n, osd.GD, kmin=1, kmax=1), s)
        sch._global_division(0)
        return tuple(g[0] for _, g in sorted(sch.groups.items()))

    runs = every_draw_sequence(run)
    assert sorted(runs) == sorted(itertools.permutations(range(n)))


def test_global_division_pairs_are_uniform():
    """Pairs of 4 idle workers: every ordered pairing (which pair is made
    first) from 4! draw sequences, each exactly 4 times (2 orders within each
    of the 2 pairs)."""
    def run(s):
        sch = with_stream(osd.Scheduler(4, osd.GD, kmin=2, kmax=2), s)
        sch._global_division(0)
        return tuple(g for _, g in sorted(sch.groups.items()))

    runs = Counter(every_draw_sequence(run))
    assert sum(runs.values()) == 24 and len(runs) == 6
    assert set(runs.values()) == {4}


@pytest.mark.parametrize("n", [2, 3, 4, 5])
def test_chunks_order_is_every_permutation(n):
    """The division helper of Inter-Intra (Sec. 5.2): chunks of one are the
    shuffled order, every permutation once."""
    members = [3 * x + 1 for x in range(n)]

    def run(s):
        sch = with_stream(osd.Scheduler(n, osd.INTER_INTRA, kmin=1, kmax=1, n_nodes=1), s)
        return tuple(c[0] for c in sch._chunks(members))

    runs = every_draw_sequence(run)
    assert sorted(runs) == sorted(itertools.permutations(members))


def all_partitions(items, k):
    """Every partition of `items` into blocks of k (as sorted tuples)."""
    if not items:
        return [()]
    first, rest = items[0], items[1:]
    out = []
    for mates in itertools.combinations(rest, k - 1):
        left = [x for x in rest if x not in mates]
        for p in all_partitions(left, k):
            out.append(tuple(sorted(((first,) + mates,) + p)))
    return out


@pytest.mark.parametrize("n,k", [(2, 1), (3, 3), (4, 2), (6, 2), (6, 3)])
def test_static_row_is_a_uniform_partition(n, k, monkeypatch):
    """A row of the seeded static schedule (Sec. 4.2) is the shuffle cut into
    groups of k: over every draw sequence of one row, each partition into
    groups of k appears n! / (number of partitions) times."""
    monkeypatch.setattr(osd, "union_connected", lambda n_, rows: True)

    def run(s):
        monkeypatch.setattr(osd, "Stream", lambda key: s)
        (row,) = osd.static_table(n, k, 1, seed=0)
        return tuple(sorted(row))

    runs = Counter(every_draw_sequence(run))
    parts = all_partitions(list(range(n)), k)
    assert sum(runs.values()) == math.factorial(n)
    assert set(runs) == set(parts)
    assert set(runs.values()) == {math.factorial(n) // len(parts)}


@pytest.mark.parametrize("n,i", [(2, 1), (4, 0), (5, 3)])
def test_adpsgd_partner_is_every_other_worker_once(n, i):
    """AD-PSGD (Fig. 3): the requester's passive partner is a uniform draw
    over the other workers -- each exactly once over every draw sequence."""
    def run(s):
        sch = with_stream(osd.Scheduler(n, osd.ADPSGD), s)
        (g,) = sch._adpsgd_step([i])
        return g

    runs = every_draw_sequence(run)
    assert sorted(runs) == sorted(tuple(sorted((i, j))) for j in range(n) if j != i)


def test_inter_intra_heads_and_their_order():
    """Inter-Intra (Sec. 5.2), 2 nodes of 2 workers, groups of one: each node's
    head is either of its idle workers and the two heads come in either
    order -- each of the 2 x 2 x 2 outcomes from exactly one draw sequence;
    each node's intra-phase group is the whole node."""
    def run(s):
        sch = with_stream(osd.Scheduler(4, osd.INTER_INTRA, kmin=1, kmax=1, n_nodes=2), s)
        sch._inter_intra_division(0)
        made = [g for _, g in sorted(sch.groups.items())]
        assert made[-2:] == [(0, 1), (2, 3)]
        return made[0][0], made[1][0]

    runs = every_draw_sequence(run)
    want = [(a, b) for h0 in (0, 1) for h1 in (2, 3) for a, b in ((h0, h1), (h1, h0))]
    assert sorted(runs) == sorted(want)
