// Residency cap of one fused-kernel launch (resident waves per CU, enforced
// by the host with an LDS reservation), chosen from the units the launch
// runs.  Plain host code with no HIP dependency, so it is tested on its own.
#pragma once

#include <cmath>
#include <cstdint>

namespace rip {
namespace policy {

constexpr int kMaxK = 8;  // largest group size with a specialized kernel path

// Resident waves per CU at which each unit shape sustained the most HBM
// bandwidth on MI355X, by group size k (entry 0: groups above kMaxK, which
// stream their members in chunks of kMaxK), for units whose members all
// update (plain SGD, momentum) and for units that only average.  Measured
// with bench.py --sweep-caps (32 fp32 replicas of 25.6M parameters, every
// unit of one size, even caps of 2-16 waves/CU, one process per shape; two
// sessions on different machines agreed).  A lane keeps one 16-byte load in
// flight per slot of every stream it reads (w, plus g and v when the member
// updates), so units that read more streams peak with fewer resident waves;
// beyond that, more waves add outstanding requests without adding bandwidth
// (GB/s, plain SGD group of eight at 6 / 8 / 10 waves: 6246 / 5937 / 5892;
// momentum group of three at 4 / 6 / 8: 4697 / 5154 / 6028).  Where two caps
// measured within 1%, the table takes the one that also suited the mixed
// launches of the paper's schedules.  Odd caps measured the same as the even
// cap below them (the LDS reservation appears to be granted per half of a
// CU's LDS), so only even caps are used.  bf16 units (8 replicas of 1.3G
// parameters) peaked at the same caps within 2%, except averaging-only groups
// of eight, which ran 5% faster at 6 than at 8 (fp32: equal).
constexpr int kWavesSgd[kMaxK + 1] = {4, 12, 10, 8, 10, 8, 8, 8, 6};
constexpr int kWavesMom[kMaxK + 1] = {4, 12, 10, 10, 8, 6, 6, 6, 4};
constexpr int kWavesAvg[kMaxK + 1] = {6, 12, 14, 10, 12, 10, 8, 8, 6};

// The cap used when a launch has no units (nothing is launched then).
constexpr int kWavesDefault = 8;

// Preferred cap of one unit of k members of which `act` update this step:
// the averaging-only and all-updating preferences, interpolated by the share
// of updating members.
inline double unit_waves(int32_t k, int32_t act, bool mom) {
  const int idx = k <= kMaxK ? k : 0;
  const double f = (double)act / (double)k;
  return f * (mom ? kWavesMom[idx] : kWavesSgd[idx]) + (1.0 - f) * kWavesAvg[idx];
}

// Cap of a launch running `units` units (unit u: k[u] members, act[u] of them
// updating; mom: the launch applies momentum).  The units' preferences are
// averaged, weighted by the bytes each moves (an updating member moves w, g
// and v; an averaging one w), and the mean is rounded up to an even cap: a cap
// below a shape's preference cost more (SGD groups of 2-4 at 8 waves: -3%)
// than one above it (groups of 5-8 at 10: -1%).
inline int launch_waves(const int32_t* k, const int32_t* act, int32_t units, bool mom) {
  double num = 0.0, den = 0.0;
  for (int32_t u = 0; u < units; ++u) {
    const double bytes = act[u] * (mom ? 5.0 : 3.0) + (k[u] - act[u]) * 2.0;
    num += unit_waves(k[u], act[u], mom) * bytes;
    den += bytes;
  }
  if (den == 0.0) return kWavesDefault;
  return 2 * (int)std::ceil(num / den / 2.0 - 1e-6);
}

// A step whose units prefer caps far apart (Global Division and Inter-Intra
// steps mix groups of two to eight, and lone updates, in one launch) runs
// as two launches, each at the cap of its own units: the units preferring
// at least kSplitCap waves per CU, then the others.  Only when the step has
// at least kSplitMinUnits units, each part carries at least kSplitMinShare
// of the step's bytes, and the parts' caps differ by at least kSplitMinGap;
// otherwise the second launch's ramp and tail cost more than the better
// caps gain (steps of one or two random groups).
constexpr int kSplitCap = 8;
constexpr int kSplitMinUnits = 3;
constexpr double kSplitMinShare = 0.15;
constexpr int kSplitMinGap = 4;
constexpr int kMaxUnits = 256;  // a launch's units are disjoint, so at most the replicas

// Decides the split of a launch's units.  Returns true and fills part[u]
// (0: the first launch, preferring >= kSplitCap waves; 1: the second) and
// the two launches' caps, or returns false (one launch at launch_waves).
inline bool split_units(const int32_t* k, const int32_t* act, int32_t units, bool mom,
                        uint8_t* part, int* waves0, int* waves1) {
  if (units < kSplitMinUnits || units > kMaxUnits) return false;
  int32_t k0[kMaxUnits], a0[kMaxUnits], k1[kMaxUnits], a1[kMaxUnits];
  int32_t n0 = 0, n1 = 0;
  double b0 = 0.0, b1 = 0.0;
  for (int32_t u = 0; u < units; ++u) {
    const double bytes = act[u] * (mom ? 5.0 : 3.0) + (k[u] - act[u]) * 2.0;
    if (unit_waves(k[u], act[u], mom) >= kSplitCap - 1e-9) {
      part[u] = 0;
      k0[n0] = k[u];
      a0[n0++] = act[u];
      b0 += bytes;
    } else {
      part[u] = 1;
      k1[n1] = k[u];
      a1[n1++] = act[u];
      b1 += bytes;
    }
  }
  if (n0 == 0 || n1 == 0) return false;
  if (b0 < kSplitMinShare * (b0 + b1) || b1 < kSplitMinShare * (b0 + b1)) return false;
  *waves0 = launch_waves(k0, a0, n0, mom);
  *waves1 = launch_waves(k1, a1, n1, mom);
  return *waves0 - *waves1 >= kSplitMinGap;
}

}  // namespace policy
}  // namespace rip
