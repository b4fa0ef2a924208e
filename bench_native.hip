// Native throughput of the fused step through the C ABI alone: no Python,
// no torch.  Registers N flat replicas (parameters, gradients, momentum when
// asked for) and runs rip_step -- group generation for the step, then the
// fused local update and P-Reduce in one launch -- for a number of steps,
// the way a C or C++ training loop would call the library.  A measurement
// program beside bench.py (`bench.py --native` builds and runs it), not part
// of the library.
//
//   bench_native [--replicas N] [--params P] [--group K | --fixed a,b,...]
//                    [--momentum M] [--bf16] [--steps S] [--warmup W]
//
// --group K: the seeded static schedule (period 4) of groups of K, every
// worker updating every step.  --fixed: one table row holding one group
// (the listed workers); the other workers update alone.  Prints one JSON
// line: wall-clock and HIP-event GB/s over the algorithmic bytes of the
// timed steps, and the host time spent per rip_step call.
#include <hip/hip_runtime.h>

#include <chrono>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "rip.h"

namespace {

// Uniform values in [-scale, scale) from a SplitMix64-style hash of the index.
__global__ void fill_f32(float* p, int64_t n, uint64_t seed, float scale) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    uint64_t z = seed + 0x9E3779B97F4A7C15ull * (uint64_t)(i + 1);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    p[i] = scale * ((float)(int32_t)(uint32_t)z * (1.0f / 2147483648.0f));
  }
}
__global__ void fill_bf16(uint16_t* p, int64_t n, uint64_t seed, float scale) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    uint64_t z = seed + 0x9E3779B97F4A7C15ull * (uint64_t)(i + 1);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    const float f = scale * ((float)(int32_t)(uint32_t)z * (1.0f / 2147483648.0f));
    p[i] = (uint16_t)(__float_as_uint(f) >> 16);  // truncation is fine for inputs
  }
}

int die(const char* what) {
  std::fprintf(stderr, "bench_native: %s\n", what);
  return 1;
}
int die_rip(const char* what, int32_t rc) {
  std::fprintf(stderr, "bench_native: %s failed (%d): %s\n", what, rc, rip_last_error());
  return 1;
}
int die_hip(const char* what, hipError_t e) {
  std::fprintf(stderr, "bench_native: %s: %s\n", what, hipGetErrorString(e));
  return 1;
}

}  // namespace

int main(int argc, char** argv) {
  int n = 16, group = 4, steps = 100, warmup = 10;
  int64_t params = 25600000;
  float momentum = 0.0f;
  bool bf16 = false;
  std::vector<int32_t> fixed;
  for (int i = 1; i < argc; ++i) {
    const std::string a = argv[i];
    const bool has = i + 1 < argc;
    if (a == "--replicas" && has) n = std::atoi(argv[++i]);
    else if (a == "--params" && has) params = std::atoll(argv[++i]);
    else if (a == "--group" && has) group = std::atoi(argv[++i]);
    else if (a == "--momentum" && has) momentum = (float)std::atof(argv[++i]);
    else if (a == "--steps" && has) steps = std::atoi(argv[++i]);
    else if (a == "--warmup" && has) warmup = std::atoi(argv[++i]);
    else if (a == "--bf16") bf16 = true;
    else if (a == "--fixed" && has) {
      for (const char* p = argv[++i]; *p;) {
        fixed.push_back((int32_t)std::strtol(p, const_cast<char**>(&p), 10));
        if (*p == ',') ++p;
        else if (*p) return die("--fixed takes comma-separated worker ids");
      }
    } else {
      return die("unknown or incomplete argument (see the header of bench_native.hip)");
    }
  }
  if (n < 1 || n > RIP_MAX_REPLICAS || params < 1 || steps < 1 || warmup < 0)
    return die("bad sizes");

  // Schedule.
  rip_sched_cfg cfg{};
  cfg.n_workers = n;
  cfg.seed = 2;
  int32_t rows[2] = {0, 1}, offsets[2] = {0, 0};
  if (!fixed.empty()) {
    cfg.mode = RIP_SCHED_TABLE;
    offsets[1] = (int32_t)fixed.size();
    cfg.row_offsets = rows;
    cfg.group_offsets = offsets;
    cfg.members = fixed.data();
    cfg.n_groups = 1;
    cfg.period = 1;
  } else {
    cfg.mode = RIP_SCHED_STATIC;
    cfg.group_size = group;
    cfg.period = 4;
  }
  rip_sched* sched = nullptr;
  int32_t rc = rip_sched_create(&cfg, &sched);
  if (rc != RIP_OK) return die_rip("rip_sched_create", rc);

  // Replicas: one flat buffer per replica and kind.
  const int esize = bf16 ? 2 : 4;
  const size_t bytes = (size_t)params * esize;
  std::vector<void*> param(n), grad(n), mom(momentum != 0.0f ? n : 0);
  auto fill = [&](void* p, uint64_t seed, float scale) {
    if (bf16)
      hipLaunchKernelGGL(fill_bf16, dim3(4096), dim3(256), 0, 0, static_cast<uint16_t*>(p),
                         params, seed, scale);
    else
      hipLaunchKernelGGL(fill_f32, dim3(4096), dim3(256), 0, 0, static_cast<float*>(p), params,
                         seed, scale);
  };
  for (int r = 0; r < n; ++r) {
    hipError_t e = hipMalloc(&param[r], bytes);
    if (e == hipSuccess) e = hipMalloc(&grad[r], bytes);
    if (e == hipSuccess && !mom.empty()) e = hipMalloc(&mom[r], bytes);
    if (e != hipSuccess) return die_hip("hipMalloc", e);
    fill(param[r], 1000 + r, 1.0f);
    fill(grad[r], 2000 + r, 0.01f);
    if (!mom.empty() && (e = hipMemset(mom[r], 0, bytes)) != hipSuccess)
      return die_hip("hipMemset", e);
  }
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return die_hip("fill", e);
  const int64_t numel = params;
  rip_replicas* reps = nullptr;
  rc = rip_replicas_create(n, 1, bf16 ? RIP_BF16 : RIP_FP32, &numel, param.data(), grad.data(),
                           mom.empty() ? nullptr : mom.data(), &reps);
  if (rc != RIP_OK) return die_rip("rip_replicas_create", rc);

  hipStream_t stream = nullptr;
  if ((e = hipStreamCreate(&stream)) != hipSuccess) return die_hip("hipStreamCreate", e);
  const rip_sgd sgd{bf16 ? 0.01f : 0.1f, momentum, 0.0f, 0};
  std::vector<int32_t> act(n), off(n + 1), mem(n);
  int32_t na = 0, ng = 0;
  // Algorithmic bytes of one step: every updating replica reads w, g (and v)
  // and writes w (and v); a group member that did not update reads and
  // writes w; every worker in these schedules updates every step.
  auto step_bytes = [&]() {
    std::vector<uint8_t> touched(n, 0);
    double b = 0.0;
    for (int i = 0; i < na; ++i) {
      touched[act[i]] = 1;
      b += (double)params * esize * (momentum != 0.0f ? 5 : 3);
    }
    for (int j = 0; j < off[ng]; ++j)
      if (!touched[mem[j]]) b += (double)params * esize * 2;
    return b;
  };
  int64_t t = 0;
  for (; t < warmup; ++t) {
    rc = rip_step(sched, reps, t, nullptr, &sgd, stream, act.data(), &na, off.data(), mem.data(),
                  &ng);
    if (rc != RIP_OK) return die_rip("rip_step", rc);
  }
  if ((e = hipStreamSynchronize(stream)) != hipSuccess) return die_hip("warmup", e);

  hipEvent_t e0, e1;
  if ((e = hipEventCreate(&e0)) != hipSuccess || (e = hipEventCreate(&e1)) != hipSuccess)
    return die_hip("hipEventCreate", e);
  double total = 0.0;
  const auto w0 = std::chrono::steady_clock::now();
  (void)hipEventRecord(e0, stream);
  for (int i = 0; i < steps; ++i, ++t) {
    rc = rip_step(sched, reps, t, nullptr, &sgd, stream, act.data(), &na, off.data(), mem.data(),
                  &ng);
    if (rc != RIP_OK) return die_rip("rip_step", rc);
    total += step_bytes();
  }
  const auto w_enq = std::chrono::steady_clock::now();
  (void)hipEventRecord(e1, stream);
  if ((e = hipStreamSynchronize(stream)) != hipSuccess) return die_hip("timed steps", e);
  const auto w1 = std::chrono::steady_clock::now();
  float ms = 0.0f;
  (void)hipEventElapsedTime(&ms, e0, e1);
  const double wall = std::chrono::duration<double>(w1 - w0).count();
  const double enq_us = std::chrono::duration<double, std::micro>(w_enq - w0).count() / steps;
  std::printf(
      "{\"native\": \"rip_step\", \"replicas\": %d, \"params\": %lld, \"storage\": \"%s\", "
      "\"schedule\": \"%s\", \"momentum\": %g, \"steps\": %d, \"warmup\": %d, "
      "\"ms_per_step\": %.4f, \"value_gbps\": %.1f, \"events_gbps\": %.1f, "
      "\"host_us_per_call\": %.2f}\n",
      n, (long long)params, bf16 ? "bf16" : "fp32", fixed.empty() ? "static" : "fixed",
      (double)momentum, steps, warmup, wall * 1e3 / steps, total / wall / 1e9,
      total / (ms * 1e-3) / 1e9, enq_us);

  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  rip_replicas_destroy(reps);
  rip_sched_destroy(sched);
  (void)hipStreamDestroy(stream);
  for (int r = 0; r < n; ++r) {
    (void)hipFree(param[r]);
    (void)hipFree(grad[r]);
    if (!mom.empty()) (void)hipFree(mom[r]);
  }
  return 0;
}
