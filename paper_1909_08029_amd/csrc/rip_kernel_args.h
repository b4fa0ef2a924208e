// Launch descriptor shared by the host code and the fused kernel of librip.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

#include "rip.h"

namespace rip {

#ifndef RIP_BLOCK
#define RIP_BLOCK 64
#endif
constexpr int kBlock = RIP_BLOCK;  // threads per workgroup: one wave64
constexpr int kMaxK = 8;           // largest group size with a specialized path
constexpr int kTileOptions = 4;    // tiles of 1, 2, 4 or 8 slots per thread

// A tile of a unit is kBlock threads x 2^slot_log2(k, mom) slots x 16 bytes
// of each member stream, and a lane keeps one 16-byte load in flight per
// slot of every stream it reads (w, plus g and v for a member that updates),
// so small units take several slots: lone updates four, pairs two, groups of
// three two without momentum and one with it; larger units take one slot,
// and the host's residency cap sets the depth of outstanding requests.
// (A group of three without momentum at one slot streamed 2% faster alone,
// at 14 waves per CU, but the higher cap it needs slowed the mixed-size
// launches of Global Division by 1%.)  Groups above kMaxK use one slot and
// stream their members in chunks of kMaxK.
constexpr int kSlotLog2Sgd[kMaxK + 1] = {0, 2, 1, 1, 0, 0, 0, 0, 0};
constexpr int kSlotLog2Mom[kMaxK + 1] = {0, 2, 1, 0, 0, 0, 0, 0, 0};
constexpr int slot_log2(int k, bool mom) {
  return k > kMaxK ? 0 : (mom ? kSlotLog2Mom[k] : kSlotLog2Sgd[k]);
}

// Passed by value as the kernel argument (about 2.6 KiB), so each launch
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
