// Host-only checks of the launch residency policy (rip_launch_policy.h),
// built and run by tests/test_launch_policy.py.  Prints "launch policy ok"
// and exits 0 when every check held.
#include <cstdio>
#include <vector>

#include "rip_launch_policy.h"

namespace {
int g_failures = 0;
#define CHECK_EQ(got, want, what)                                                   \
  do {                                                                              \
    const int g_ = (got), w_ = (want);                                              \
    if (g_ != w_) {                                                                 \
      std::fprintf(stderr, "check failed: %s: got %d, want %d\n", what, g_, w_);    \
      ++g_failures;                                                                 \
    }                                                                               \
  } while (0)

int waves(const std::vector<int32_t>& k, const std::vector<int32_t>& act, bool mom) {
  return rip::policy::launch_waves(k.data(), act.data(), (int32_t)k.size(), mom);
}
}  // namespace

int main() {
  using namespace rip::policy;
  char what[128];
  // Launches of one unit shape take that shape's table entry.
  for (int k = 1; k <= kMaxK; ++k) {
    std::snprintf(what, sizeof what, "SGD group of %d", k);
    CHECK_EQ(waves({k, k}, {k, k}, false), kWavesSgd[k], what);
    std::snprintf(what, sizeof what, "momentum group of %d", k);
    CHECK_EQ(waves({k}, {k}, true), kWavesMom[k], what);
    if (k > 1) {
      std::snprintf(what, sizeof what, "averaging-only group of %d", k);
      CHECK_EQ(waves({k, k, k}, {0, 0, 0}, false), kWavesAvg[k], what);
    }
  }
  // Groups above kMaxK use entry 0 (the chunked path).
  CHECK_EQ(waves({32}, {32}, false), kWavesSgd[0], "SGD group of 32");
  CHECK_EQ(waves({9}, {9}, true), kWavesMom[0], "momentum group of 9");
  CHECK_EQ(waves({256}, {0}, false), kWavesAvg[0], "averaging-only group of 256");
  // A pair with one updating member: halfway between the two shapes.
  const double pair = 0.5 * kWavesSgd[2] + 0.5 * kWavesAvg[2];
  CHECK_EQ(waves({2}, {1}, false), 2 * (int)((pair + 1.999) / 2), "pair, one member updating");
  // Mixed launch: byte-weighted mean rounded up to an even cap.  A group of
  // four (12 byte units, preference kWavesSgd[4]) with a group of eight (24,
  // kWavesSgd[8]).
  {
    const double mean = (12.0 * kWavesSgd[4] + 24.0 * kWavesSgd[8]) / 36.0;
    int want = 2;
    while (want < mean - 1e-9) want += 2;
    CHECK_EQ(waves({4, 8}, {4, 8}, false), want, "groups of four and eight");
  }
  // A mean between two even caps goes up: a group of five (15 byte units,
  // kWavesSgd[5]) with a group of four (12, kWavesSgd[4]).
  {
    const double mean = (15.0 * kWavesSgd[5] + 12.0 * kWavesSgd[4]) / 27.0;
    int want = 2;
    while (want < mean - 1e-9) want += 2;
    CHECK_EQ(waves({5, 4}, {5, 4}, false), want, "groups of five and four (rounded up)");
    CHECK_EQ(want, 10, "the mean of that launch lies between 8 and 10");
  }
  // Every result is even and within the tables' range.
  for (int k1 = 1; k1 <= 12; ++k1)
    for (int a1 = 0; a1 <= k1; ++a1)
      for (int k2 = 1; k2 <= 12; ++k2)
        for (int mom = 0; mom < 2; ++mom) {
          const int w = waves({k1, k2}, {a1, k2}, mom != 0);
          if (w % 2 != 0 || w < 4 || w > 14) {
            std::fprintf(stderr, "check failed: k %d/%d act %d/%d mom %d -> %d\n", k1, k2, a1,
                         k2, mom, w);
            ++g_failures;
          }
        }
  // Splitting a launch in two.
  {
    uint8_t part[16];
    int w0 = 0, w1 = 0;
    // one shape: never split
    std::vector<int32_t> k{4, 4, 4, 4}, a{4, 4, 4, 4};
    CHECK_EQ(split_units(k.data(), a.data(), 4, false, part, &w0, &w1), 0, "one shape");
    // too few units
    k = {2, 8};
    a = {2, 8};
    CHECK_EQ(split_units(k.data(), a.data(), 2, true, part, &w0, &w1), 0, "two units");
    // a Global Division step with momentum: pairs and triples (prefer 10)
    // against groups of 6-8 (prefer 4-6): split, small groups first
    k = {2, 3, 8, 6, 2, 7};
    a = {2, 3, 8, 6, 2, 7};
    CHECK_EQ(split_units(k.data(), a.data(), 6, true, part, &w0, &w1), 1, "GD with momentum");
    const int want_part[6] = {0, 0, 1, 1, 0, 1};
    for (int u = 0; u < 6; ++u) CHECK_EQ(part[u], want_part[u], "GD with momentum: part");
    {
      std::vector<int32_t> k0{2, 3, 2}, k1{8, 6, 7};
      CHECK_EQ(w0, waves(k0, k0, true), "GD with momentum: first cap");
      CHECK_EQ(w1, waves(k1, k1, true), "GD with momentum: second cap");
      CHECK_EQ(w0 - w1 >= kSplitMinGap, 1, "GD with momentum: caps far apart");
    }
    // one small part below the byte share: no split (a pair beside five groups of eight)
    k = {2, 8, 8, 8, 8, 8};
    a = {2, 8, 8, 8, 8, 8};
    CHECK_EQ(split_units(k.data(), a.data(), 6, true, part, &w0, &w1), 0, "small share");
    // the split step of tests/test_gpu_graph.py: a group of eight beside a
    // pair and two lone updates, SGD and momentum
    k = {8, 2, 1, 1};
    a = {8, 2, 1, 1};
    for (int mom = 0; mom < 2; ++mom) {
      CHECK_EQ(split_units(k.data(), a.data(), 4, mom != 0, part, &w0, &w1), 1,
               "group of eight, pair, two lone updates");
      CHECK_EQ(part[0], 1, "the group of eight goes second");
    }
    // caps too close: SGD groups of 5 (pref 8) with groups of 7 (8) never split
    k = {5, 7, 5, 7};
    a = {5, 7, 5, 7};
    CHECK_EQ(split_units(k.data(), a.data(), 4, false, part, &w0, &w1), 0, "caps equal");
  }
  // No units: the default.
  CHECK_EQ(waves({}, {}, false), kWavesDefault, "no units");
  if (g_failures) {
    std::printf("launch policy: %d failed checks\n", g_failures);
    return 1;
  }
  std::printf("launch policy ok\n");
  return 0;
}
