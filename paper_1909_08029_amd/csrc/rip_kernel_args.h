// Launch descriptor shared by the host code and the fused kernel of librip.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

#include "rip.h"

namespace rip {

#ifndef RIP_BLOCK
#define RIP_BLOCK 64
#endif
#ifndef RIP_LOADS_IN_FLIGHT
#define RIP_LOADS_IN_FLIGHT 12
#endif
constexpr int kBlock = RIP_BLOCK;  // threads per workgroup: one wave64
constexpr int kMaxK = 8;           // largest group size with a specialized path
constexpr int kTileOptions = 4;    // tiles of 1, 2, 4 or 8 slots per thread

// A tile of a unit is kBlock threads x 2^slot_log2 slots x 16 bytes of each
// member stream.  The slot count keeps about RIP_LOADS_IN_FLIGHT 16-byte
// loads outstanding per thread (k members x w, g and, with momentum, v), so
// small groups and lone updates still have enough bytes in flight while a
// workgroup moves a similar number of bytes whatever the group size.  Groups
// above kMaxK take the element-wise path with one slot.
constexpr int slot_log2(int k, bool mom) {
  if (k > kMaxK) return 0;
  const int s = RIP_LOADS_IN_FLIGHT / (k * (mom ? 3 : 2));
  int l = 0;
  while (l < kTileOptions - 1 && (2 << l) <= s) ++l;
  return l;
}

// Passed by value as the kernel argument (about 2.2 KiB), so each launch
// carries its own schedule and no device staging buffer is needed.
struct StepArgs {
  const uint64_t* ptab;       // device [3][S][N]: param, grad, mom pointers
  const int64_t* seg_numel;   // device [S]
  const int64_t* seg_tile0;   // device [kTileOptions][S + 1]: first tile of each
                              // segment, for tiles of 1, 2, 4, 8 slots
  int32_t n_seg, n_rep, n_units;
  uint32_t work;              // work items (tiles) of all units
  uint32_t uniform_tiles;     // tiles per unit when all units have the same count, else 0
  int64_t flat_numel;         // elements of the only segment when n_seg == 1
  float lr, mu, wd;
  int32_t nesterov;
  uint32_t unit_work0[RIP_MAX_REPLICAS + 1];  // first work item of each unit
  // 16-bit tables start 4-byte aligned: the kernel reads them as dwords
  alignas(4) uint16_t unit_off[RIP_MAX_REPLICAS + 1];  // unit u = member[unit_off[u] .. unit_off[u+1])
  alignas(4) uint16_t member[RIP_MAX_REPLICAS];        // replica ids, ascending within a unit
  uint32_t active_bits[RIP_MAX_REPLICAS / 32];  // replicas doing their local update
};

hipError_t launch_fused_step(const StepArgs& a, bool bf16, bool mom, int blocks,
                             size_t lds_bytes, hipStream_t stream);

}  // namespace rip
