// Launch descriptor shared by the host code and the fused kernel of librip.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

#include "rip.h"

namespace rip {

#ifndef RIP_BLOCK
#define RIP_BLOCK 256
#endif
#ifndef RIP_SLOTS
#define RIP_SLOTS 4
#endif
constexpr int kBlock = RIP_BLOCK;  // threads per workgroup (wave64)
constexpr int kSlots = RIP_SLOTS;  // 16-byte slots per thread per tile
constexpr int kMaxK = 8;     // largest group size with a specialized path

// Passed by value as the kernel argument (about 1.1 KiB), so each launch
// carries its own schedule and no device staging buffer is needed.
struct StepArgs {
  const uint64_t* ptab;       // device [3][S][N]: param, grad, mom pointers
  const int64_t* seg_numel;   // device [S]
  const int64_t* seg_tile0;   // device [S + 1]: first tile of each segment
  int64_t tiles;              // tiles per unit (seg_tile0[S])
  int64_t work;               // units * tiles
  int32_t n_seg, n_rep, n_units, reserved;
  float lr, mu;
  uint16_t unit_off[RIP_MAX_REPLICAS + 1];  // unit u = member[unit_off[u] .. unit_off[u+1])
  uint16_t member[RIP_MAX_REPLICAS];        // replica ids, ascending within a unit
  uint32_t active_bits[RIP_MAX_REPLICAS / 32];  // replicas doing their local update
};

hipError_t launch_fused_step(const StepArgs& a, bool bf16, bool mom, int blocks,
                             hipStream_t stream);

}  // namespace rip
