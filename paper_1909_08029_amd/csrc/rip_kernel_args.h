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
// above kMaxK use one slot and stream their members in chunks of kMaxK.
constexpr int slot_log2(int k, bool mom) {
  if (k > kMaxK) return 0;
  const int s = RIP_LOADS_IN_FLIGHT / (k * (mom ? 3 : 2));
  int l = 0;
  while (l < kTileOptions - 1 && (2 << l) <= s) ++l;
  return l;
}

// Passed by value as the kernel argument (about 2.4 KiB), so each launch
// carries its own schedule and no device staging buffer is needed.
struct StepArgs {
  const uint64_t* ptab;       // device [3][S][N]: param, grad, mom pointers
  const int64_t* seg_numel;   // device [S]
  const int64_t* seg_tile0;   // device [kTileOptions][S + 1]: first tile of each
                              // segment, for tiles of 1, 2, 4, 8 slots
  int32_t n_seg, n_rep, n_units;
  uint32_t work;              // work items (tiles) of all units
  uint32_t uniform_tiles;     // tiles per unit when all units have the same count, else 0
  uint32_t uniform_k;         // members per unit when all units have the same size, else 0
  int64_t flat_numel;         // elements of the only segment when n_seg == 1
  float lr, mu, wd;
  int32_t nesterov;
  uint32_t unit_work0[RIP_MAX_REPLICAS + 1];  // first work item of each unit
  uint32_t unit_info[RIP_MAX_REPLICAS];       // see unit_info_pack
  // Replica ids, ascending within a unit; unit u = member[base_u .. base_u + k_u).
  // The kernel reads the 16 bytes from the dword holding member[base_u], so
  // the table is padded to keep that read inside it.
  alignas(16) uint8_t member[RIP_MAX_REPLICAS + 16];
  uint32_t active_bits[RIP_MAX_REPLICAS / 32];  // replicas doing their local update
};

// One dword per unit: first member index (8 bits), member count k (9 bits),
// and the update flags of its first eight members (bit j = member j is
// active), so a workgroup learns its unit from a single scalar load.
constexpr uint32_t unit_info_pack(uint32_t base, uint32_t k, uint32_t act8) {
  return base | (k << 8) | (act8 << 17);
}
constexpr uint32_t unit_info_base(uint32_t info) { return info & 0xFFu; }
constexpr uint32_t unit_info_k(uint32_t info) { return (info >> 8) & 0x1FFu; }
constexpr uint32_t unit_info_act8(uint32_t info) { return info >> 17; }
static_assert(RIP_MAX_REPLICAS <= 256, "unit_info packs member indices into 8 bits");

// ext: weight decay or Nesterov momentum is on (the kernel variant that
// handles them; the plain variant leaves them out of the arithmetic).
hipError_t launch_fused_step(const StepArgs& a, bool bf16, bool mom, bool ext, int blocks,
                             size_t lds_bytes, hipStream_t stream);

}  // namespace rip
