// A plain C++ consumer of librip's C ABI (no Python, no torch): registers
// replicas allocated with hipMalloc, schedules one step from a table, runs
// the fused local update + P-Reduce, and checks every element against values
// computed here in closed form.  Inputs are small integers and multiples of
// 1/8, so every fp32 operation of the step is exact and the expected values
// are exact too.  Exit status 0 on success.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "rip.h"

#define CHECK_HIP(x)                                                               \
  do {                                                                             \
    hipError_t e_ = (x);                                                           \
    if (e_ != hipSuccess) {                                                        \
      std::printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__);  \
      return 1;                                                                    \
    }                                                                              \
  } while (0)
#define CHECK_RIP(x)                                                                        \
  do {                                                                                      \
    int32_t r_ = (x);                                                                       \
    if (r_ != RIP_OK) {                                                                     \
      std::printf("rip error %d (%s) at line %d\n", (int)r_, rip_last_error(), __LINE__);  \
      return 1;                                                                             \
    }                                                                                       \
  } while (0)

int main() {
  const int N = 8;
  const int64_t P = 3 * 4096 * 4 + 7;  // several tiles and a ragged tail
  std::printf("cabi smoke: N=%d P=%lld abi=%d\n", N, (long long)P, (int)rip_abi_version());
  if (rip_abi_version() != RIP_ABI_VERSION) return 1;

  std::vector<std::vector<float>> w(N, std::vector<float>(P)), g(N, std::vector<float>(P));
  for (int r = 0; r < N; ++r)
    for (int64_t e = 0; e < P; ++e) {
      w[r][e] = (float)(r * 4 + (int)(e % 16));   // small integers
      g[r][e] = 0.25f * (float)((e + r) % 8);      // multiples of 1/4
    }
  std::vector<void*> dw(N), dg(N);
  for (int r = 0; r < N; ++r) {
    CHECK_HIP(hipMalloc(&dw[r], P * sizeof(float)));
    CHECK_HIP(hipMalloc(&dg[r], P * sizeof(float)));
    CHECK_HIP(hipMemcpy(dw[r], w[r].data(), P * sizeof(float), hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(dg[r], g[r].data(), P * sizeof(float), hipMemcpyHostToDevice));
  }
  rip_replicas* rep = nullptr;
  CHECK_RIP(rip_replicas_create(N, 1, RIP_FP32, &P, dw.data(), dg.data(), nullptr, &rep));

  // One table row: {0,1,2,3}, {4,5}; worker 6 has no group; worker 7 is not eligible.
  const int32_t rows[2] = {0, 2};
  const int32_t goff[3] = {0, 4, 6};
  const int32_t mem[6] = {0, 1, 2, 3, 4, 5};
  rip_sched_cfg cfg;
  std::memset(&cfg, 0, sizeof cfg);
  cfg.n_workers = N;
  cfg.mode = RIP_SCHED_TABLE;
  cfg.period = 1;
  cfg.row_offsets = rows;
  cfg.group_offsets = goff;
  cfg.members = mem;
  cfg.n_groups = 2;
  rip_sched* sched = nullptr;
  CHECK_RIP(rip_sched_create(&cfg, &sched));
  const uint8_t eligible[N] = {1, 1, 1, 1, 1, 1, 1, 0};
  int32_t active[N], n_active = 0, off[N + 1], members[N], n_groups = 0;
  CHECK_RIP(rip_schedule_groups(sched, 0, eligible, active, &n_active, off, members, &n_groups));
  if (n_active != 7 || n_groups != 2 || off[1] != 4 || off[2] != 6) {
    std::printf("unexpected schedule: %d active, %d groups\n", (int)n_active, (int)n_groups);
    return 1;
  }

  // An overlapping pair of groups is refused before any launch.
  const int32_t bad_off[3] = {0, 2, 4};
  const int32_t bad_mem[4] = {0, 1, 1, 2};
  rip_sgd sgd = {0.5f, 0.0f, 0.0f, 0};
  if (rip_preduce(rep, bad_off, bad_mem, 2, active, n_active, &sgd, nullptr) != RIP_E_OVERLAP ||
      std::strlen(rip_last_error()) == 0) {
    std::printf("overlap not reported\n");
    return 1;
  }

  CHECK_RIP(rip_preduce(rep, off, members, n_groups, active, n_active, &sgd, nullptr));
  CHECK_HIP(hipDeviceSynchronize());

  std::vector<float> got(P);
  int64_t bad = 0;
  for (int r = 0; r < N; ++r) {
    CHECK_HIP(hipMemcpy(got.data(), dw[r], P * sizeof(float), hipMemcpyDeviceToHost));
    for (int64_t e = 0; e < P; ++e) {
      auto u = [&](int q) { return w[q][e] - 0.5f * g[q][e]; };
      float want;
      if (r < 4) want = (u(0) + u(1) + u(2) + u(3)) * 0.25f;
      else if (r < 6) want = (u(4) + u(5)) * 0.5f;
      else if (r == 6) want = u(6);
      else want = w[7][e];
      if (got[e] != want) ++bad;
    }
  }
  rip_sched_destroy(sched);
  rip_replicas_destroy(rep);
  for (int r = 0; r < N; ++r) {
    CHECK_HIP(hipFree(dw[r]));
    CHECK_HIP(hipFree(dg[r]));
  }
  if (bad) {
    std::printf("%lld elements differ from the closed form\n", (long long)bad);
    return 1;
  }
  std::printf("cabi smoke ok\n");
  return 0;
}
