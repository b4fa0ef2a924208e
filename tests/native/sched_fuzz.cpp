// Host-only fuzz driver for librip's group scheduler (rip_sched.cpp), built
// with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_sched_sanitized.py.  It links the scheduler alone (no HIP): the
// two error-reporting helpers the scheduler calls are defined below.
//
// For many random configurations of every mode it runs steps with random
// eligibility through the C ABI and checks what every schedule must satisfy:
// active ids ascending and distinct, eligible and not blocked; groups
// non-empty, ascending, in range and pairwise disjoint; the groups' members
// unblocked afterwards; per worker requests == syncs + skips + waiting; a
// failed step changes nothing.  Invalid configurations must be rejected with
// an error code.  Prints "sched fuzz ok" and exits 0 when every check held.
#include <algorithm>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

#include "rip.h"
#include "rip_internal.h"

namespace rip {
namespace {
thread_local std::string g_error;
}
int32_t fail(int32_t code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_error = buf;
  return code;
}
void clear_error() { g_error.clear(); }
}  // namespace rip

namespace {

uint64_t g_state = 0x1234567ULL;
uint64_t next_u64() {  // SplitMix64 (Steele, Lea & Flood 2014)
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ULL);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}
int uniform(int lo, int hi) {  // [lo, hi]
  return lo + (int)(next_u64() % (uint64_t)(hi - lo + 1));
}

int g_failures = 0;
int g_accepted[8] = {}, g_rejected = 0;
long long g_steps = 0;
#define CHECK(cond, ...)                                          \
  do {                                                            \
    if (!(cond)) {                                                \
      std::fprintf(stderr, "check failed: %s: ", #cond);          \
      std::fprintf(stderr, __VA_ARGS__);                          \
      std::fprintf(stderr, "\n");                                 \
      if (++g_failures > 20) std::exit(1);                        \
    }                                                             \
  } while (0)

struct Table {
  std::vector<int32_t> rows, offsets, members;
  int n_groups = 0;
};

Table random_table(int n, int period) {
  Table t;
  t.rows.push_back(0);
  t.offsets.push_back(0);
  for (int r = 0; r < period; ++r) {
    std::vector<int32_t> ids(n);
    for (int i = 0; i < n; ++i) ids[i] = i;
    for (int i = n - 1; i > 0; --i) std::swap(ids[i], ids[uniform(0, i)]);
    int used = uniform(0, n), pos = 0;
    while (pos < used) {
      int k = uniform(1, used - pos);
      std::vector<int32_t> g(ids.begin() + pos, ids.begin() + pos + k);
      std::sort(g.begin(), g.end());
      t.members.insert(t.members.end(), g.begin(), g.end());
      t.offsets.push_back((int32_t)t.members.size());
      ++t.n_groups;
      pos += k;
    }
    t.rows.push_back(t.n_groups);
  }
  return t;
}

void run_case(int c) {
  rip_sched_cfg cfg{};
  Table table;
  const int mode = uniform(0, 7);
  int n = uniform(1, 48);
  cfg.mode = mode;
  cfg.seed = next_u64();
  cfg.kmin = uniform(1, 6);
  cfg.kmax = cfg.kmin + uniform(0, 6);
  cfg.c_thres = uniform(0, 5);
  cfg.period = uniform(1, 5);
  if (mode == RIP_SCHED_STATIC) {
    cfg.group_size = uniform(1, 6);
    n = cfg.group_size * uniform(1, 8);
  } else if (mode == RIP_SCHED_RULE) {
    cfg.n_nodes = uniform(0, 4) * 2;
    if (cfg.n_nodes == 0) cfg.n_nodes = 1;
    n = 4 * cfg.n_nodes;
  } else if (mode == RIP_SCHED_INTER_INTRA) {
    cfg.n_nodes = uniform(1, 6);
    n = cfg.n_nodes * uniform(1, 6);
  } else if (mode == RIP_SCHED_TABLE || mode == RIP_SCHED_SCRIPTED) {
    table = random_table(n, mode == RIP_SCHED_TABLE ? cfg.period : uniform(1, 40));
    cfg.row_offsets = table.rows.data();
    cfg.group_offsets = table.offsets.data();
    cfg.members = table.members.data();
    cfg.n_groups = table.n_groups;
    if (mode == RIP_SCHED_SCRIPTED) cfg.period = 0;
  }
  if (uniform(0, 9) == 0) n = uniform(-1, 0);                  // invalid sizes
  if (uniform(0, 19) == 0) cfg.kmax = cfg.kmin - 1;            // invalid range
  cfg.n_workers = n;

  rip_sched* s = nullptr;
  const int32_t rc = rip_sched_create(&cfg, &s);
  const bool bad_n = n < 1 || n > RIP_MAX_REPLICAS;
  if (bad_n) CHECK(rc != RIP_OK, "case %d: N = %d accepted", c, n);
  if (rc != RIP_OK) {
    CHECK(s == nullptr, "case %d: handle returned on error", c);
    ++g_rejected;
    return;
  }
  ++g_accepted[mode];
  std::vector<int32_t> active(n), offsets(n + 1), members(n);
  std::vector<uint8_t> eligible(n), was_waiting(n);
  const int steps = uniform(1, 400);
  const int p_eligible = uniform(1, 10);
  for (int64_t t = 0; t < steps; ++t) {
    for (int i = 0; i < n; ++i) eligible[i] = uniform(1, 10) <= p_eligible;
    for (int i = 0; i < n; ++i) {
      rip_worker_state ws{};
      CHECK(rip_sched_worker(s, i, &ws) == RIP_OK, "case %d", c);
      was_waiting[i] = (uint8_t)ws.waiting;
    }
    int32_t na = -1, ng = -1;
    const int32_t r = rip_schedule_groups(s, t, eligible.data(), active.data(), &na,
                                          offsets.data(), members.data(), &ng);
    if (r != RIP_OK) {
      // only a scripted schedule can fail a step (exhausted or a group
      // without its requester); the same step must then be rejected again
      CHECK(mode == RIP_SCHED_SCRIPTED, "case %d mode %d step %lld: error %d", c, mode,
            (long long)t, r);
      CHECK(rip_schedule_groups(s, t, eligible.data(), active.data(), &na, offsets.data(),
                                members.data(), &ng) == r,
            "case %d: a failed step changed the state", c);
      break;
    }
    ++g_steps;
    CHECK(na >= 0 && na <= n && ng >= 0 && ng <= n, "case %d: counts %d %d", c, na, ng);
    for (int a = 0; a < na; ++a) {
      CHECK(active[a] >= 0 && active[a] < n, "case %d: active id %d", c, active[a]);
      if (a > 0) CHECK(active[a] > active[a - 1], "case %d: active not ascending", c);
      CHECK(eligible[active[a]] && !was_waiting[active[a]], "case %d: active %d", c, active[a]);
    }
    std::vector<uint8_t> seen(n, 0);
    CHECK(offsets[0] == 0, "case %d: offsets[0]", c);
    for (int g = 0; g < ng; ++g) {
      CHECK(offsets[g + 1] > offsets[g] && offsets[g + 1] <= n, "case %d: group %d", c, g);
      for (int j = offsets[g]; j < offsets[g + 1] && j < n; ++j) {
        const int m = members[j];
        CHECK(m >= 0 && m < n, "case %d: member %d", c, m);
        if (m < 0 || m >= n) continue;
        if (j > offsets[g]) CHECK(m > members[j - 1], "case %d: group not ascending", c);
        CHECK(!seen[m], "case %d step %lld: worker %d in two groups", c, (long long)t, m);
        seen[m] = 1;
      }
    }
    for (int i = 0; i < n; ++i) {
      rip_worker_state ws{};
      CHECK(rip_sched_worker(s, i, &ws) == RIP_OK, "case %d", c);
      CHECK(ws.requests == ws.syncs + ws.skips + ws.waiting, "case %d: worker %d counters", c, i);
      if (seen[i] && mode != RIP_SCHED_ADPSGD) CHECK(!ws.waiting, "case %d: member %d blocked", c, i);
    }
  }
  rip_worker_state ws{};
  CHECK(rip_sched_worker(s, n, &ws) != RIP_OK, "case %d: worker N accepted", c);
  rip_sched_destroy(s);
}

}  // namespace

int main(int argc, char** argv) {
  const int cases = argc > 1 ? std::atoi(argv[1]) : 2000;
  for (int c = 0; c < cases; ++c) run_case(c);
  rip_sched_destroy(nullptr);
  if (g_failures) {
    std::printf("sched fuzz: %d failed checks\n", g_failures);
    return 1;
  }
  std::printf("sched fuzz ok: %d configurations (%d rejected), %lld steps; accepted per mode:", cases,
              g_rejected, g_steps);
  for (int m = 0; m < 8; ++m) std::printf(" %d", g_accepted[m]);
  std::printf("\n");
  return 0;
}
