// Group generation for P-Reduce (Step 3 of the algorithm of Fig. 4):
// static periodic schedules (Sec. 4.2, Fig. 8), the rule table of Fig. 9,
// and the centralized Group Generator with per-worker Group Buffers
// (Sec. 4.1, Sec. 5.1), Global Division and the slowdown filter (Sec. 5.1,
// Sec. 5.3), in a stepped model of the asynchronous protocol.  The contract
// of every entry point is in include/rip.h.
//
// The whole state lives on the host and is tiny (N <= RIP_MAX_REPLICAS
// workers, at most one pending group per request); a step costs O(N * k).

#include <algorithm>
#include <cstring>
#include <deque>
#include <functional>
#include <map>
#include <new>
#include <vector>

#include "rip_internal.h"

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ULL;
constexpr int kSchedTag = 3;
constexpr int kMaxStaticAttempts = 1000;

// SplitMix64 output function (Steele, Lea & Flood, OOPSLA 2014).
inline uint64_t mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

inline uint64_t fold(uint64_t k, std::initializer_list<uint64_t> comps) {
  for (uint64_t c : comps) k = mix(k + kGamma * (c + 1));
  return k;
}

struct Stream {
  uint64_t state;
  uint64_t next() {
    state += kGamma;
    return mix(state);
  }
  // Lemire's multiply-shift map to [0, n), without rejection.
  int32_t bounded(uint32_t n) { return (int32_t)(((next() >> 32) * (uint64_t)n) >> 32); }
};

using Group = std::vector<int32_t>;
using Row = std::vector<Group>;

bool union_connected(int n, const std::vector<Row>& rows) {
  std::vector<int> parent(n);
  for (int i = 0; i < n; ++i) parent[i] = i;
  auto find = [&](int a) {
    while (parent[a] != a) a = parent[a] = parent[parent[a]];
    return a;
  };
  int comps = n;
  for (const Row& row : rows)
    for (const Group& g : row)
      for (size_t j = 1; j < g.size(); ++j) {
        int a = find(g[0]), b = find(g[j]);
        if (a != b) {
          parent[a] = b;
          --comps;
        }
      }
  return comps == 1;
}

void sort_row(Row& row) {
  std::sort(row.begin(), row.end(), [](const Group& a, const Group& b) { return a[0] < b[0]; });
}

// Seeded periodic table: each row a random partition into groups of k;
// redraw the whole period until its union graph is connected.
bool make_static_table(int n, int k, int period, uint64_t seed, std::vector<Row>& rows) {
  for (int attempt = 0; attempt < kMaxStaticAttempts; ++attempt) {
    rows.assign(period, Row());
    for (int rho = 0; rho < period; ++rho) {
      Stream s{fold(seed, {(uint64_t)kSchedTag, (uint64_t)attempt, (uint64_t)rho})};
      std::vector<int32_t> a(n);
      for (int i = 0; i < n; ++i) a[i] = i;
      for (int i = n - 1; i >= 1; --i) std::swap(a[i], a[s.bounded((uint32_t)i + 1)]);
      for (int c = 0; c < n; c += k) {
        Group g(a.begin() + c, a.begin() + c + k);
        std::sort(g.begin(), g.end());
        rows[rho].push_back(std::move(g));
      }
      sort_row(rows[rho]);
    }
    if (union_connected(n, rows)) return true;
  }
  return false;
}

// Fig. 9: four local workers per node (rank = node*4 + local), period 4.
void make_rule_table(int nodes, std::vector<Row>& rows) {
  rows.assign(4, Row());
  Group lw0;
  for (int nd = 0; nd < nodes; ++nd) lw0.push_back(4 * nd);
  rows[0].push_back(lw0);                                                  // LW0 on all nodes
  for (int nd = 0; nd < nodes; ++nd) rows[0].push_back({4 * nd + 2, 4 * nd + 3});  // LW2-LW3
  for (int ph : {1, 3})
    for (int nd = 0; nd < nodes; ++nd)
      rows[ph].push_back({4 * nd, 4 * nd + 1, 4 * nd + 2, 4 * nd + 3});      // all local
  for (int nd = 0; nd < nodes; ++nd) rows[2].push_back({4 * nd, 4 * nd + 3});  // LW0-LW3
  if (nodes > 1)
    for (int nd = 0; nd < nodes / 2; ++nd)                                  // LW1 across the ring
      rows[2].push_back({4 * nd + 1, 4 * (nd + nodes / 2) + 1});
  for (Row& r : rows) sort_row(r);
}

bool valid_group(const int32_t* m, int32_t len, int n) {
  if (len < 1) return false;
  for (int32_t j = 0; j < len; ++j) {
    if (m[j] < 0 || m[j] >= n) return false;
    if (j > 0 && m[j] <= m[j - 1]) return false;
  }
  return true;
}

}  // namespace

struct rip_sched {
  int n = 0, mode = 0;
  int kmin = 0, kmax = 0, c_thres = 0;
  int per_node = 1;  // INTER_INTRA: workers per node
  // evolving state (copied as a whole to make a failed step a no-op)
  struct State {
    int64_t t = 0;
    std::vector<int64_t> c, syncs, skips;
    std::vector<uint8_t> waiting;
    std::vector<std::deque<int64_t>> gb;
    std::map<int64_t, Group> groups;  // live groups by id (ordered = creation)
    int64_t next_id = 0;
    Stream rng{0};
    size_t script_pos = 0;
    std::vector<int32_t> partner;  // ADPSGD: chosen neighbour of a waiting requester
    std::vector<int64_t> seq;      // ADPSGD: request order of a waiting requester
  } st;
  // The state before the step in progress, kept between steps so that saving
  // it reuses its allocations instead of making new ones every step.
  State saved;
  std::vector<int64_t> ready;  // scratch of schedule_step, kept for its capacity
  std::vector<Row> rows;       // table modes
  std::vector<Group> script;   // SCRIPTED

  bool table_mode() const { return !rows.empty(); }

  int64_t new_group(Group g) {
    std::sort(g.begin(), g.end());
    int64_t id = st.next_id++;
    for (int32_t m : g) st.gb[m].push_back(id);
    st.groups.emplace(id, std::move(g));
    return id;
  }

  void random_group(int i) {
    int k = std::min(kmin + st.rng.bounded((uint32_t)(kmax - kmin + 1)), n);
    std::vector<int32_t> others;
    others.reserve(n - 1);
    for (int j = 0; j < n; ++j)
      if (j != i) others.push_back(j);
    for (int j = 0; j < k - 1; ++j) {
      int x = j + st.rng.bounded((uint32_t)(n - 1 - j));
      std::swap(others[j], others[x]);
    }
    Group g(others.begin(), others.begin() + (k - 1));
    g.push_back(i);
    new_group(std::move(g));
  }

  void global_division(int i) {
    std::vector<int32_t> idle;
    for (int w = 0; w < n; ++w)
      if (st.gb[w].empty() && (c_thres <= 0 || st.c[i] - st.c[w] < c_thres)) idle.push_back(w);
    for (int a = (int)idle.size() - 1; a >= 1; --a)
      std::swap(idle[a], idle[st.rng.bounded((uint32_t)a + 1)]);
    size_t pos = 0;
    while (pos < idle.size()) {
      size_t k = (size_t)(kmin + st.rng.bounded((uint32_t)(kmax - kmin + 1)));
      size_t end = std::min(idle.size(), pos + k);
      new_group(Group(idle.begin() + pos, idle.begin() + end));
      pos = end;
    }
  }

  // Fisher-Yates shuffle of `m`, then consecutive chunks of drawn sizes.
  std::vector<Group> chunks(std::vector<int32_t> m) {
    for (int a = (int)m.size() - 1; a >= 1; --a) std::swap(m[a], m[st.rng.bounded((uint32_t)a + 1)]);
    std::vector<Group> out;
    size_t pos = 0;
    while (pos < m.size()) {
      const size_t k = (size_t)(kmin + st.rng.bounded((uint32_t)(kmax - kmin + 1)));
      const size_t end = std::min(m.size(), pos + k);
      out.emplace_back(m.begin() + pos, m.begin() + end);
      pos = end;
    }
    return out;
  }

  // Inter-Intra synchronization (Sec. 5.2) as one division of the idle
  // workers: an inter-phase group for each (a random head per node, heads
  // grouped across nodes; the rest grouped within their node), then an
  // intra-phase group of every idle worker of the node.
  void inter_intra_division(int i) {
    std::map<int, std::vector<int32_t>> nodes;  // ascending node id
    for (int w = 0; w < n; ++w)
      if (st.gb[w].empty() && (c_thres <= 0 || st.c[i] - st.c[w] < c_thres))
        nodes[w / per_node].push_back(w);
    std::vector<int32_t> heads;
    std::map<int, std::vector<int32_t>> rest;
    for (auto& [nd, ws] : nodes) {
      const int32_t h = ws[st.rng.bounded((uint32_t)ws.size())];
      heads.push_back(h);
      for (int32_t w : ws)
        if (w != h) rest[nd].push_back(w);
      rest[nd];  // a node whose only idle worker is its head has no local groups
    }
    for (Group& g : chunks(heads)) new_group(std::move(g));
    for (auto& [nd, ws] : rest)
      for (Group& g : chunks(ws)) new_group(std::move(g));
    for (auto& [nd, ws] : nodes) new_group(ws);
  }

  // AD-PSGD (Fig. 3): each requester picks a uniformly random other worker
  // and averages with it atomically; the partner is passive.  Pairs whose
  // workers are already locked in this step wait, oldest request first.
  int32_t adpsgd_step(const int32_t* active, int32_t na, int32_t* group_offsets,
                      int32_t* members, int32_t* n_groups) {
    for (int32_t a = 0; a < na; ++a) {
      const int i = active[a];
      st.c[i] += 1;
      if (n == 1) {
        st.skips[i] += 1;
        continue;
      }
      const int x = st.rng.bounded((uint32_t)(n - 1));
      st.partner[i] = x < i ? x : x + 1;
      st.seq[i] = st.next_id++;
      st.waiting[i] = 1;
    }
    std::vector<int32_t> order;
    for (int w = 0; w < n; ++w)
      if (st.waiting[w]) order.push_back(w);
    std::sort(order.begin(), order.end(),
              [&](int32_t p, int32_t q) { return st.seq[p] < st.seq[q]; });
    std::vector<uint8_t> locked(n, 0);
    int32_t ng = 0, pos = 0;
    group_offsets[0] = 0;
    for (int32_t i : order) {
      const int32_t j = st.partner[i];
      if (locked[i] || locked[j]) continue;
      locked[i] = locked[j] = 1;
      st.waiting[i] = 0;
      st.syncs[i] += 1;
      members[pos++] = std::min(i, j);
      members[pos++] = std::max(i, j);
      group_offsets[++ng] = pos;
    }
    *n_groups = ng;
    return RIP_OK;
  }

  int32_t request(int i) {
    st.c[i] += 1;
    if (table_mode()) {
      int64_t it = st.c[i] - 1;
      const Row& row = rows[(size_t)(it % (int64_t)rows.size())];
      for (size_t gi = 0; gi < row.size(); ++gi) {
        if (std::binary_search(row[gi].begin(), row[gi].end(), i)) {
          int64_t key = it * (int64_t)(n + 1) + (int64_t)gi;  // orders as (iteration, gi)
          st.groups.try_emplace(key, row[gi]);  // once per group and iteration
          st.gb[i].push_back(key);
          st.waiting[i] = 1;
          return RIP_OK;
        }
      }
      st.skips[i] += 1;
      return RIP_OK;
    }
    if (st.gb[i].empty()) {
      if (mode == RIP_SCHED_RANDOM_GB) {
        random_group(i);
      } else if (mode == RIP_SCHED_GD) {
        global_division(i);
      } else if (mode == RIP_SCHED_INTER_INTRA) {
        inter_intra_division(i);
      } else {
        if (st.script_pos >= script.size())
          return rip::fail(RIP_E_INVAL, "scripted group list exhausted at worker %d", i);
        const Group& g = script[st.script_pos++];
        if (!std::binary_search(g.begin(), g.end(), i))
          return rip::fail(RIP_E_INVAL, "scripted group %zu does not contain requester %d",
                           st.script_pos - 1, i);
        new_group(g);
      }
    }
    st.waiting[i] = 1;
    return RIP_OK;
  }
};

extern "C" int32_t rip_sched_create(const rip_sched_cfg* cfg, rip_sched** out) {
  rip::clear_error();
  if (!cfg || !out) return rip::fail(RIP_E_INVAL, "rip_sched_create: null argument");
  *out = nullptr;
  const int n = cfg->n_workers;
  if (n < 1 || n > RIP_MAX_REPLICAS)
    return rip::fail(n < 1 ? RIP_E_INVAL : RIP_E_UNSUPPORTED, "n_workers %d not in [1, %d]", n,
                     RIP_MAX_REPLICAS);
  rip_sched* s = new (std::nothrow) rip_sched();
  if (!s) return rip::fail(RIP_E_NOMEM, "out of host memory");
  s->n = n;
  s->mode = cfg->mode;
  s->st.c.assign(n, 0);
  s->st.syncs.assign(n, 0);
  s->st.skips.assign(n, 0);
  s->st.waiting.assign(n, 0);
  s->st.gb.assign(n, {});
  int32_t rc = RIP_OK;
  switch (cfg->mode) {
    case RIP_SCHED_TABLE: {
      if (cfg->period < 1 || !cfg->row_offsets || !cfg->group_offsets || !cfg->members ||
          cfg->n_groups < 0 || cfg->row_offsets[0] != 0 ||
          cfg->row_offsets[cfg->period] != cfg->n_groups) {
        rc = rip::fail(RIP_E_INVAL, "TABLE needs period >= 1 and consistent row/group offsets");
        break;
      }
      s->rows.assign(cfg->period, Row());
      for (int r = 0; r < cfg->period && rc == RIP_OK; ++r) {
        if (cfg->row_offsets[r + 1] < cfg->row_offsets[r]) {
          rc = rip::fail(RIP_E_INVAL, "row_offsets not monotone at row %d", r);
          break;
        }
        std::vector<uint8_t> used(n, 0);
        for (int g = cfg->row_offsets[r]; g < cfg->row_offsets[r + 1]; ++g) {
          const int32_t a = cfg->group_offsets[g], b = cfg->group_offsets[g + 1];
          if (b < a || !valid_group(cfg->members + a, b - a, n)) {
            rc = rip::fail(RIP_E_INVAL, "table group %d is empty, out of range or not ascending", g);
            break;
          }
          Group grp(cfg->members + a, cfg->members + b);
          for (int32_t m : grp) {
            if (used[m]) {
              rc = rip::fail(RIP_E_INVAL, "table row %d has worker %d in two groups", r, m);
              break;
            }
            used[m] = 1;
          }
          if (rc != RIP_OK) break;
          s->rows[r].push_back(std::move(grp));
        }
        // The caller's order within a row is kept: groups of a step come out
        // by (iteration, position in the row as given).
      }
      // A period without any group is a table of pure local steps.
      if (rc == RIP_OK && cfg->n_groups == 0) s->rows.assign(cfg->period, Row{});
      break;
    }
    case RIP_SCHED_STATIC: {
      const int k = cfg->group_size;
      if (k < 1 || cfg->period < 1 || n % k != 0) {
        rc = rip::fail(RIP_E_INVAL, "STATIC needs group_size >= 1, period >= 1, N %% k == 0");
        break;
      }
      if (!make_static_table(n, k, cfg->period, cfg->seed, s->rows))
        rc = rip::fail(RIP_E_INVAL, "STATIC: no period with a connected union graph in %d attempts",
                       kMaxStaticAttempts);
      break;
    }
    case RIP_SCHED_RULE: {
      const int nodes = cfg->n_nodes;
      if (nodes < 1 || n != 4 * nodes || (nodes > 1 && nodes % 2 != 0)) {
        rc = rip::fail(RIP_E_INVAL, "RULE needs N == 4*n_nodes with n_nodes 1 or even");
        break;
      }
      make_rule_table(nodes, s->rows);
      break;
    }
    case RIP_SCHED_RANDOM_GB:
    case RIP_SCHED_GD:
    case RIP_SCHED_INTER_INTRA: {
      if (cfg->kmin < 1 || cfg->kmax < cfg->kmin) {
        rc = rip::fail(RIP_E_INVAL, "need 1 <= kmin <= kmax");
        break;
      }
      if (cfg->mode == RIP_SCHED_INTER_INTRA) {
        if (cfg->n_nodes < 1 || n % cfg->n_nodes != 0) {
          rc = rip::fail(RIP_E_INVAL, "INTER_INTRA needs N %% n_nodes == 0");
          break;
        }
        s->per_node = n / cfg->n_nodes;
      }
      s->kmin = cfg->kmin;
      s->kmax = cfg->kmax;
      s->c_thres = cfg->c_thres;
      s->st.rng.state = fold(cfg->seed, {(uint64_t)kSchedTag});
      break;
    }
    case RIP_SCHED_ADPSGD: {
      s->st.rng.state = fold(cfg->seed, {(uint64_t)kSchedTag});
      s->st.partner.assign(n, -1);
      s->st.seq.assign(n, 0);
      break;
    }
    case RIP_SCHED_SCRIPTED: {
      if (cfg->n_groups < 0 || (cfg->n_groups > 0 && (!cfg->group_offsets || !cfg->members))) {
        rc = rip::fail(RIP_E_INVAL, "SCRIPTED needs group_offsets and members");
        break;
      }
      for (int g = 0; g < cfg->n_groups; ++g) {
        const int32_t a = cfg->group_offsets[g], b = cfg->group_offsets[g + 1];
        if (b < a || !valid_group(cfg->members + a, b - a, n)) {
          rc = rip::fail(RIP_E_INVAL, "scripted group %d is empty, out of range or not ascending", g);
          break;
        }
        s->script.emplace_back(cfg->members + a, cfg->members + b);
      }
      break;
    }
    default:
      rc = rip::fail(RIP_E_UNSUPPORTED, "unknown scheduler mode %d", cfg->mode);
  }
  if (rc != RIP_OK) {
    delete s;
    return rc;
  }
  // A table whose rows carry no group at all still works (every worker skips).
  if ((cfg->mode == RIP_SCHED_TABLE) && s->rows.empty()) s->rows.assign(1, Row{});
  *out = s;
  return RIP_OK;
}

extern "C" void rip_sched_destroy(rip_sched* s) { delete s; }

namespace {

// One step of group generation on s->st (the caller restores it on error).
int32_t schedule_step(rip_sched* s, const uint8_t* eligible, int32_t* active, int32_t* n_active,
                      int32_t* group_offsets, int32_t* members, int32_t* n_groups) {
  const int n = s->n;
  s->st.t += 1;

  int32_t na = 0;
  for (int i = 0; i < n; ++i)
    if ((!eligible || eligible[i]) && !s->st.waiting[i]) active[na++] = i;
  if (s->mode == RIP_SCHED_ADPSGD) {
    *n_active = na;
    return s->adpsgd_step(active, na, group_offsets, members, n_groups);
  }
  for (int32_t a = 0; a < na; ++a) {
    int32_t rc = s->request(active[a]);
    if (rc != RIP_OK) return rc;
  }
  // Groups whose every member is blocked on them, in id order.
  std::vector<int64_t>& ready = s->ready;
  ready.clear();
  for (int i = 0; i < n; ++i) {
    if (!s->st.waiting[i]) continue;
    const int64_t h = s->st.gb[i].front();
    bool ok = true;
    for (int32_t m : s->st.groups.at(h))
      if (!s->st.waiting[m] || s->st.gb[m].front() != h) {
        ok = false;
        break;
      }
    if (ok) ready.push_back(h);
  }
  std::sort(ready.begin(), ready.end());
  ready.erase(std::unique(ready.begin(), ready.end()), ready.end());
  int32_t ng = 0, pos = 0;
  group_offsets[0] = 0;
  for (int64_t h : ready) {
    auto it = s->st.groups.find(h);
    for (int32_t m : it->second) {
      s->st.gb[m].pop_front();
      s->st.waiting[m] = 0;
      s->st.syncs[m] += 1;
      members[pos++] = m;
    }
    group_offsets[++ng] = pos;
    s->st.groups.erase(it);
  }
  *n_active = na;
  *n_groups = ng;
  return RIP_OK;
}

}  // namespace

namespace rip {

int32_t sched_workers(const rip_sched* s) { return s->n; }

int32_t schedule_then(rip_sched* s, int64_t step, const uint8_t* eligible, int32_t* active,
                      int32_t* n_active, int32_t* group_offsets, int32_t* members,
                      int32_t* n_groups, const std::function<int32_t()>& then) {
  if (step != s->st.t)
    return fail(RIP_E_INVAL, "steps must be consecutive: expected %lld, got %lld",
                (long long)s->st.t, (long long)step);
  // A failed step leaves no trace.  Group generation itself can fail only in
  // the scripted mode (an exhausted or inconsistent script); otherwise only
  // `then` can, so the state is saved only when one of the two is present.
  const bool may_fail = then || s->mode == RIP_SCHED_SCRIPTED;
  if (may_fail) s->saved = s->st;
  int32_t rc = schedule_step(s, eligible, active, n_active, group_offsets, members, n_groups);
  if (rc == RIP_OK && then) rc = then();
  if (rc != RIP_OK && may_fail) s->st = s->saved;
  return rc;
}

}  // namespace rip

extern "C" int32_t rip_schedule_groups(rip_sched* s, int64_t step, const uint8_t* eligible,
                                       int32_t* active, int32_t* n_active, int32_t* group_offsets,
                                       int32_t* members, int32_t* n_groups) {
  rip::clear_error();
  if (!s || !active || !n_active || !group_offsets || !members || !n_groups)
    return rip::fail(RIP_E_INVAL, "rip_schedule_groups: null argument");
  return rip::schedule_then(s, step, eligible, active, n_active, group_offsets, members, n_groups,
                            nullptr);
}

extern "C" int32_t rip_sched_worker(const rip_sched* s, int32_t worker, rip_worker_state* out) {
  rip::clear_error();
  if (!s || !out) return rip::fail(RIP_E_INVAL, "rip_sched_worker: null argument");
  if (worker < 0 || worker >= s->n) return rip::fail(RIP_E_INVAL, "worker %d out of range", worker);
  out->requests = s->st.c[worker];
  out->syncs = s->st.syncs[worker];
  out->skips = s->st.skips[worker];
  out->waiting = s->st.waiting[worker];
  out->gb_depth = s->mode == RIP_SCHED_ADPSGD ? (int32_t)s->st.waiting[worker]
                                              : (int32_t)s->st.gb[worker].size();
  return RIP_OK;
}
