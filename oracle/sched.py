"""Oracle group scheduler (Step 3 of Fig. 4) -- test infrastructure only.

A plain Python statement of how groups are generated and serialized, in a
stepped model of the paper's asynchronous protocol.  Each call ``step(t,
eligible)`` answers: which workers run their local update this step, and which
(disjoint) groups run their P-Reduce this step.

Worker state (Sec. 4.1 and Sec. 5.1):
  c[i]        requests made so far (the per-worker counter of Sec. 5.3);
  gb[i]       the Group Buffer: ordered list of groups that include i (Sec. 5.1);
  waiting[i]  i has finished its local update and is blocked in P-Reduce,
              which is a collective: it completes only when every member of
              the group has asked for it (Sec. 5.1).

One step t:
  1. Active workers A_t: eligible this step and not waiting, ascending.  They
     run Step 2 (local update) in this step's launch.
  2. Each active worker, in ascending order (the Group Generator serves
     requests one at a time, Sec. 4.1), requests a group:
       * table modes (static schedule of Sec. 4.2, Fig. 8; the rule table of
         Fig. 9): the group of row (iteration mod period) containing i, where
         the iteration is the request's index c[i]-1; a worker with no group
         in that row skips synchronization and does not wait;
       * group-buffer modes: if gb[i] is non-empty its head is i's group;
         otherwise new groups are generated and appended to the buffer of
         every member -- one random group containing i (RANDOM_GB, Step 3 of
         Fig. 4 with the buffer of Sec. 5.1), or a random partition of every
         idle worker (empty buffer) into groups (Global Division, Sec. 5.1),
         optionally keeping only workers whose counter is within C_thres of
         the initiator's (Sec. 5.3), the two-phase Inter-Intra division of
         Sec. 5.2, or the next group of a fixed script.
  3. A group executes when it is the head of every member's buffer and every
     member is waiting (the lock-vector rule of Sec. 4.1: overlapping groups
     run one after the other, in creation order).  Executed groups are
     therefore disjoint.  Members pop it and stop waiting.

Table modes keep at most one entry per buffer, keyed by (iteration, group of
the row); members of one row group reach it at the same iteration.

Random draws come from one sequential SplitMix64 stream keyed
fold(seed, SCHED=3) (group-buffer modes), or one stream per (attempt, row)
keyed fold(seed, 3, attempt, row) for seeded static tables.
"""
from __future__ import annotations

from collections import deque
from typing import List, Optional, Sequence, Tuple

from .splitmix import Stream, fold

TABLE = 0
STATIC = 1
RANDOM_GB = 2
GD = 3
SCRIPTED = 4
RULE = 5
INTER_INTRA = 6
ADPSGD = 7

SCHED_TAG = 3
MAX_STATIC_ATTEMPTS = 1000


# ---------------------------------------------------------------------------
# seeded draws
# ---------------------------------------------------------------------------
def shuffle(items: list, rng: Stream) -> list:
    """Fisher-Yates (Knuth's Algorithm P, drawn from the last position down):
    position a = L-1 .. 1 swaps with position rng.bounded(a + 1) in [0, a].
    Every permutation comes from exactly one draw sequence.  In place;
    returns the list."""
    for a in range(len(items) - 1, 0, -1):
        b = rng.bounded(a + 1)
        items[a], items[b] = items[b], items[a]
    return items


def partial_shuffle(items: list, m: int, rng: Stream) -> list:
    """The first m steps of Fisher-Yates drawn from the front: position
    j = 0 .. m-1 swaps with position j + rng.bounded(L - j) in [j, L).  The
    first m items are then a uniform ordered selection; every ordered
    selection comes from exactly one draw sequence.  In place; returns the
    list."""
    for j in range(m):
        x = j + rng.bounded(len(items) - j)
        items[j], items[x] = items[x], items[j]
    return items


# ---------------------------------------------------------------------------
# periodic tables
# ---------------------------------------------------------------------------
def union_connected(n: int, rows: Sequence[Sequence[Sequence[int]]]) -> bool:
    """Is the graph joining the members of every group of every row connected?
    (The spectral-gap condition of Sec. 3.3 asks for this.)"""
    parent = list(range(n))

    def find(a):
        while parent[a] != a:
            parent[a] = parent[parent[a]]
            a = parent[a]
        return a

    for row in rows:
        for g in row:
            for m in g[1:]:
                ra, rb = find(g[0]), find(m)
                if ra != rb:
                    parent[ra] = rb
    return len({find(i) for i in range(n)}) == 1


def static_table(n: int, k: int, period: int, seed: int) -> List[List[Tuple[int, ...]]]:
    """Seeded conflict-free periodic schedule (Sec. 4.2): every row is a random
    partition of the n workers into groups of k.  A period whose union graph
    is not connected is redrawn with the next attempt number."""
    if n < 1 or k < 1 or period < 1 or n % k != 0:
        raise ValueError("static schedule needs n % k == 0 and positive sizes")
    for attempt in range(MAX_STATIC_ATTEMPTS):
        rows = []
        for rho in range(period):
            a = shuffle(list(range(n)), Stream(fold(seed, SCHED_TAG, attempt, rho)))
            groups = [tuple(sorted(a[c:c + k])) for c in range(0, n, k)]
            groups.sort(key=lambda g: g[0])
            rows.append(groups)
        if union_connected(n, rows):
            return rows
    raise ValueError("no connected static schedule found")


def rule_table(n_nodes: int) -> List[List[Tuple[int, ...]]]:
    """The rule-based static function S of Fig. 9: four local workers per node,
    worker rank = node*4 + local index, period 4.

      phase 0: local worker 0 of every node in one group; 1 alone (no sync);
               2 with 3
      phase 1: local workers 0-3 of each node
      phase 2: 0 with 3; 1 with local worker 1 of the node opposite on the
               ring of nodes (node + n_nodes/2); 2 alone (no sync)
      phase 3: local workers 0-3 of each node
    """
    if n_nodes < 1 or (n_nodes > 1 and n_nodes % 2 != 0):
        raise ValueError("the ring rule needs one node or an even number of nodes")
    m = n_nodes
    rows = []
    rows.append([tuple(4 * nd for nd in range(m))] +
                [(4 * nd + 2, 4 * nd + 3) for nd in range(m)])
    rows.append([tuple(range(4 * nd, 4 * nd + 4)) for nd in range(m)])
    r2 = [(4 * nd, 4 * nd + 3) for nd in range(m)]
    if m > 1:
        r2 += [tuple(sorted((4 * nd + 1, 4 * ((nd + m // 2) % m) + 1)))
               for nd in range(m // 2)]
    rows.append(r2)
    rows.append([tuple(range(4 * nd, 4 * nd + 4)) for nd in range(m)])
    return [sorted(r, key=lambda g: g[0]) for r in rows]


# ---------------------------------------------------------------------------
# the scheduler
# ---------------------------------------------------------------------------
class Scheduler:
    def __init__(self, n: int, mode: int, seed: int = 0, group_size: int = 0,
                 period: int = 4, kmin: int = 2, kmax: int = 2, c_thres: int = 0,
                 table: Optional[Sequence[Sequence[Sequence[int]]]] = None,
                 script: Optional[Sequence[Sequence[int]]] = None, n_nodes: int = 0):
        if n < 1:
            raise ValueError("need at least one worker")
        self.n, self.mode = n, mode
        self.t = 0
        self.c = [0] * n
        self.syncs = [0] * n
        self.skips = [0] * n
        self.waiting = [False] * n
        self.gb = [deque() for _ in range(n)]
        self.groups = {}            # id -> members (ascending tuple)
        self.next_id = 0
        self.kmin, self.kmax, self.c_thres = kmin, kmax, c_thres
        self.rows = None
        self.divisions = []         # (initiator, counters at the time, groups made)
        if mode == TABLE:
            self.rows = [[tuple(g) for g in row] for row in table]
        elif mode == STATIC:
            self.rows = static_table(n, group_size, period, seed)
        elif mode == RULE:
            if n != 4 * n_nodes:
                raise ValueError("rule table needs n == 4 * n_nodes")
            self.rows = rule_table(n_nodes)
        elif mode == ADPSGD:
            self.rng = Stream(fold(seed, SCHED_TAG))
            self.partner = [-1] * n
            self.seq = [0] * n
        elif mode in (RANDOM_GB, GD, INTER_INTRA):
            if not 1 <= kmin <= kmax:
                raise ValueError("need 1 <= kmin <= kmax")
            if mode == INTER_INTRA and (n_nodes < 1 or n % n_nodes != 0):
                raise ValueError("inter-intra needs n % n_nodes == 0")
            self.per_node = n // n_nodes if n_nodes else 0
            self.rng = Stream(fold(seed, SCHED_TAG))
        elif mode == SCRIPTED:
            self.script = [tuple(g) for g in script]
            self.script_pos = 0
        else:
            raise ValueError(f"unknown mode {mode}")
        if self.rows is not None:
            for row in self.rows:
                seen = set()
                for g in row:
                    if list(g) != sorted(set(g)) or any(not 0 <= m < n for m in g):
                        raise ValueError("bad table group")
                    if seen & set(g):
                        raise ValueError("table row has overlapping groups")
                    seen |= set(g)

    # -- group creation (group-buffer modes) --------------------------------
    def _new_group(self, members) -> int:
        gid = self.next_id
        self.next_id += 1
        self.groups[gid] = tuple(sorted(members))
        for m in self.groups[gid]:
            self.gb[m].append(gid)
        return gid

    def _random_group(self, i: int):
        n = self.n
        k = min(self.kmin + self.rng.bounded(self.kmax - self.kmin + 1), n)
        others = partial_shuffle([j for j in range(n) if j != i], k - 1, self.rng)
        self._new_group([i] + others[:k - 1])

    def _global_division(self, i: int):
        idle = [w for w in range(self.n) if not self.gb[w] and
                (self.c_thres <= 0 or self.c[i] - self.c[w] < self.c_thres)]
        shuffle(idle, self.rng)
        pos, made = 0, []
        while pos < len(idle):
            k = self.kmin + self.rng.bounded(self.kmax - self.kmin + 1)
            made.append(self.groups[self._new_group(idle[pos:pos + k])])
            pos += k
        self.divisions.append((i, list(self.c), made))

    def _chunks(self, members):
        """Fisher-Yates shuffle, then consecutive chunks of drawn sizes."""
        members = shuffle(list(members), self.rng)
        pos, out = 0, []
        while pos < len(members):
            k = self.kmin + self.rng.bounded(self.kmax - self.kmin + 1)
            out.append(members[pos:pos + k])
            pos += k
        return out

    def _inter_intra_division(self, i: int):
        """Inter-Intra synchronization (Sec. 5.2) as a division of the idle
        workers: each gets two buffer entries, an inter-phase group (one head
        per node, chosen at random among the node's idle workers, heads
        grouped across nodes; the other idle workers grouped within their
        node), then an intra-phase group (every idle worker of its node)."""
        idle = [w for w in range(self.n) if not self.gb[w] and
                (self.c_thres <= 0 or self.c[i] - self.c[w] < self.c_thres)]
        nodes = {}
        for w in idle:
            nodes.setdefault(w // self.per_node, []).append(w)
        heads, locals_ = [], {}
        for nd in sorted(nodes):
            ws = nodes[nd]
            h = ws[self.rng.bounded(len(ws))]
            heads.append(h)
            locals_[nd] = [w for w in ws if w != h]
        made = [self.groups[self._new_group(g)] for g in self._chunks(heads)]
        for nd in sorted(nodes):
            made += [self.groups[self._new_group(g)] for g in self._chunks(locals_[nd])]
        for nd in sorted(nodes):
            made.append(self.groups[self._new_group(nodes[nd])])
        self.divisions.append((i, list(self.c), made))

    def _scripted_group(self, i: int):
        if self.script_pos >= len(self.script):
            raise ValueError("script exhausted")
        g = self.script[self.script_pos]
        self.script_pos += 1
        if i not in g:
            raise ValueError(f"scripted group {g} does not contain requester {i}")
        self._new_group(g)

    # -- AD-PSGD (the baseline of Fig. 3) ------------------------------------
    def _adpsgd_step(self, active):
        """Each requester picks a random other worker j (Step 3 of Fig. 3)
        and averages with it atomically (Step 4); j is passive and need not
        be waiting.  Pairs whose workers are already locked this step wait;
        the oldest request is served first."""
        for i in active:
            self.c[i] += 1
            if self.n == 1:
                self.skips[i] += 1
                continue
            x = self.rng.bounded(self.n - 1)
            self.partner[i] = x if x < i else x + 1
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
            executed.append(tuple(sorted((i, j))))
        return executed

    # -- one request --------------------------------------------------------
    def _request(self, i: int):
        self.c[i] += 1
        if self.rows is not None:
            it = self.c[i] - 1
            rho = it % len(self.rows)
            for gi, g in enumerate(self.rows[rho]):
                if i in g:
                    key = (it, gi)
                    self.groups[key] = g
                    self.gb[i].append(key)
                    self.waiting[i] = True
                    return
            self.skips[i] += 1
            return
        if not self.gb[i]:
            if self.mode == RANDOM_GB:
                self._random_group(i)
            elif self.mode == GD:
                self._global_division(i)
            elif self.mode == INTER_INTRA:
                self._inter_intra_division(i)
            else:
                self._scripted_group(i)
        self.waiting[i] = True

    # -- one step -----------------------------------------------------------
    def step(self, t: int, eligible: Optional[Sequence[bool]] = None):
        """Returns (active, groups) for step t; groups are ascending tuples."""
        if t != self.t:
            raise ValueError(f"steps must be consecutive: expected {self.t}, got {t}")
        self.t += 1
        n = self.n
        elig = [True] * n if eligible is None else [bool(e) for e in eligible]
        active = [i for i in range(n) if elig[i] and not self.waiting[i]]
        if self.mode == ADPSGD:
            return active, self._adpsgd_step(active)
        for i in active:
            self._request(i)
        ready = set()
        for i in range(n):
            if self.waiting[i]:
                h = self.gb[i][0]
                if all(self.waiting[m] and self.gb[m][0] == h for m in self.groups[h]):
                    ready.add(h)
        order = sorted(ready)
        executed = []
        for h in order:
            g = self.groups[h]
            for m in g:
                self.gb[m].popleft()
                self.waiting[m] = False
                self.syncs[m] += 1
            executed.append(g)
            del self.groups[h]
        return active, executed
