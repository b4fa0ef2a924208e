// Host side of librip: replica registration, argument checking, building the
// per-step launch descriptor, and error reporting.  The contract of every
// entry point is in include/rip.h.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "rip_internal.h"
#include "rip_kernel_args.h"
#include "rip_launch_policy.h"

namespace rip {

namespace {
thread_local std::string g_last_error;
thread_local int32_t g_last_launches = 0;  // kernels the last step call enqueued
std::atomic<int> g_max_blocks{0};
std::atomic<int> g_blocks_per_cu{0};
// One workgroup per tile up to 2^25 workgroups (2^31 work-items, within the
// dispatch's 32-bit grid size); beyond that workgroups loop over tiles.  A
// workgroup that loops ran the bf16 workload 4% slower than one tile each.
constexpr int kDefaultMaxBlocks = 1 << 25;
}  // namespace

int32_t fail(int32_t code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

void clear_error() { g_last_error.clear(); }

}  // namespace rip

struct rip_replicas {
  int32_t n = 0, n_seg = 0, dtype = 0, device = 0;
  int32_t lds_per_cu = 0;  // bytes of LDS per compute unit on `device`
  int64_t numel0 = 0;      // elements of segment 0 (the whole range when flat)
  bool has_grad = false, has_mom = false;
  int64_t tiles[rip::kTileOptions] = {};  // tiles per unit, by slot option
  void* dmem = nullptr;  // ptab [3][S][N] u64 | seg_numel [S] i64 | seg_tile0 [4][S+1] i64
  // Handles from rip_replicas_create_noalloc keep their tables in the
  // device's fixed table array instead of dmem; `generation` tells whether
  // a later such handle on the same device has overwritten them.
  bool in_fixed_array = false;
  uint64_t generation = 0;
  const uint64_t* d_ptab = nullptr;
  const int64_t* d_numel = nullptr;
  const int64_t* d_tile0 = nullptr;
};

// The device tables of the handle made by rip_replicas_create_noalloc.  In
// host code this name is a host-side stand-in, not a device address: host
// code uses only the per-device address from hipGetSymbolAddress below.
static __device__ __align__(256) uint8_t scratch[RIP_NOALLOC_TABLE_BYTES];

namespace rip {
namespace {
constexpr int kMaxDevices = 64;
std::mutex g_fixed_mu;
void* g_fixed_ptr[kMaxDevices] = {};      // address of `scratch` on each device
uint64_t g_fixed_gen[kMaxDevices] = {};   // generation of the handle owning it

// Address of the fixed table array on `device` (the current device), looked
// up once per device.  Caller holds g_fixed_mu.
int32_t fixed_array(int device, void** out) {
  if (device < 0 || device >= kMaxDevices)
    return fail(RIP_E_UNSUPPORTED, "device %d above the %d the library supports", device,
                kMaxDevices);
  if (!g_fixed_ptr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(RIP_E_HIP, "hipGetSymbolAddress(table array): %s", hipGetErrorString(e));
    g_fixed_ptr[device] = p;
  }
  *out = g_fixed_ptr[device];
  return RIP_OK;
}
}  // namespace
}  // namespace rip

extern "C" const char* rip_last_error(void) { return rip::g_last_error.c_str(); }
extern "C" int32_t rip_last_launch_count(void) { return rip::g_last_launches; }
extern "C" int32_t rip_abi_version(void) { return RIP_ABI_VERSION; }

extern "C" int32_t rip_set_blocks_per_cu(int32_t blocks_per_cu) {
  if (blocks_per_cu < 0) return rip::fail(RIP_E_INVAL, "blocks_per_cu must be >= 0");
  rip::g_blocks_per_cu.store(blocks_per_cu);
  return RIP_OK;
}

extern "C" int32_t rip_set_max_blocks(int32_t max_blocks) {
  if (max_blocks < 0) return rip::fail(RIP_E_INVAL, "max_blocks must be >= 0");
  rip::g_max_blocks.store(max_blocks);
  return RIP_OK;
}

namespace {

static_assert(rip::policy::kMaxK == rip::kMaxK, "launch policy and kernel disagree on kMaxK");

int elems_per_16b(int32_t dtype) { return dtype == RIP_BF16 ? 8 : 4; }
int elem_size(int32_t dtype) { return dtype == RIP_BF16 ? 2 : 4; }

// True when, for every replica, each non-empty segment starts right where
// the previous non-empty one ends (for one pointer kind).
bool back_to_back(void* const* p, int32_t n, int32_t S, const int64_t* numel, int esize) {
  for (int32_t r = 0; r < n; ++r) {
    const char* end = nullptr;
    for (int32_t s = 0; s < S; ++s) {
      if (numel[s] == 0) continue;
      const char* a = static_cast<const char*>(p[(size_t)r * S + s]);
      if (end && a != end) return false;
      end = a + numel[s] * esize;
    }
  }
  return true;
}

int32_t check_nonnull(void* const* p, const char* what, int32_t n, int32_t S,
                      const int64_t* numel) {
  for (int32_t r = 0; r < n; ++r)
    for (int32_t s = 0; s < S; ++s)
      if (numel[s] != 0 && !p[(size_t)r * S + s])
        return rip::fail(RIP_E_INVAL, "%s[%d*S+%d] is NULL", what, r, s);
  return RIP_OK;
}

// Every address the kernel uses as a base must be 16-byte aligned: each
// non-empty segment, or only the first one when the segments are coalesced.
int32_t check_align(void* const* p, const char* what, int32_t n, int32_t S, const int64_t* numel,
                    bool flat) {
  for (int32_t r = 0; r < n; ++r)
    for (int32_t s = 0; s < S; ++s) {
      if (numel[s] == 0) continue;
      const void* q = p[(size_t)r * S + s];
      if (reinterpret_cast<uintptr_t>(q) % 16 != 0)
        return rip::fail(RIP_E_ALIGN, "%s[%d*S+%d] = %p is not 16-byte aligned", what, r, s, q);
      if (flat) break;
    }
  return RIP_OK;
}

// A registered range of one buffer kind.
struct Range {
  uintptr_t begin, end;
  bool written;  // param and mom are written by a step; grad only read
  const char* what;
  int32_t r, s;
};

// Every non-empty segment must be memory of `device` that the kernel can
// address (device or managed memory, not a host pointer), must lie inside
// the allocation that holds its first byte, and the buffers a step writes
// must overlap no other registered buffer.  Gradient buffers may overlap
// each other (several replicas may read one gradient).  A kernel that
// touches memory outside an allocation faults the GPU, and aliasing makes a
// step's result depend on the order of its memory accesses, so both are
// rejected here, once, instead of being left to the launches.
int32_t check_buffers(void* const* param, void* const* grad, void* const* mom, int32_t n,
                      int32_t S, const int64_t* numel, int esize, int device) {
  std::vector<Range> ranges;
  const struct {
    void* const* p;
    const char* what;
    bool written;
  } kinds[3] = {{param, "param", true}, {grad, "grad", false}, {mom, "mom", true}};
  for (const auto& k : kinds) {
    if (!k.p) continue;
    for (int32_t r = 0; r < n; ++r)
      for (int32_t s = 0; s < S; ++s) {
        if (numel[s] == 0) continue;
        void* q = k.p[(size_t)r * S + s];
        hipPointerAttribute_t attr{};
        hipError_t e = hipPointerGetAttributes(&attr, q);
        if (e != hipSuccess) {
          (void)hipGetLastError();  // leave no sticky error for the caller's next check
          return rip::fail(RIP_E_INVAL, "%s[%d*S+%d] = %p is not device memory (%s)", k.what, r,
                           s, q, hipGetErrorString(e));
        }
        if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged)
          return rip::fail(RIP_E_INVAL, "%s[%d*S+%d] = %p is not device memory (type %d)",
                           k.what, r, s, q, (int)attr.type);
        if (attr.type == hipMemoryTypeDevice && attr.device != device)
          return rip::fail(RIP_E_INVAL, "%s[%d*S+%d] is on device %d, the current device is %d",
                           k.what, r, s, attr.device, device);
        const uintptr_t b = reinterpret_cast<uintptr_t>(q);
        const uintptr_t len = (uintptr_t)numel[s] * (uintptr_t)esize;
        hipDeviceptr_t base = nullptr;
        size_t size = 0;
        e = hipMemGetAddressRange(&base, &size, q);
        if (e != hipSuccess) {
          (void)hipGetLastError();
          return rip::fail(RIP_E_INVAL, "%s[%d*S+%d] = %p: allocation not found (%s)", k.what, r,
                           s, q, hipGetErrorString(e));
        }
        const uintptr_t a0 = reinterpret_cast<uintptr_t>(base);
        if (b < a0 || b - a0 >= size || len > size - (b - a0))
          return rip::fail(RIP_E_INVAL,
                           "%s[%d*S+%d]: %lld elements run past the end of its allocation "
                           "(%zu bytes from %p)",
                           k.what, r, s, (long long)numel[s], size, base);
        ranges.push_back({b, b + len, k.written, k.what, r, s});
      }
  }
  std::sort(ranges.begin(), ranges.end(),
            [](const Range& x, const Range& y) { return x.begin < y.begin; });
  // Sweep in address order, remembering the furthest-reaching range seen so
  // far and the furthest-reaching written one.
  const Range* far_all = nullptr;
  const Range* far_written = nullptr;
  for (const Range& x : ranges) {
    const Range* hit = x.written ? far_all : far_written;
    if (hit && x.begin < hit->end)
      return rip::fail(RIP_E_OVERLAP, "%s[%d*S+%d] overlaps %s[%d*S+%d]", x.what, x.r, x.s,
                       hit->what, hit->r, hit->s);
    if (!far_all || x.end > far_all->end) far_all = &x;
    if (x.written && (!far_written || x.end > far_written->end)) far_written = &x;
  }
  return RIP_OK;
}

}  // namespace

namespace {

int32_t create_replicas(int32_t n_replicas, int32_t n_segments, int32_t dtype,
                        const int64_t* seg_numel, void* const* param, void* const* grad,
                        void* const* mom, rip_replicas** out, bool noalloc) {
  rip::clear_error();
  if (!out) return rip::fail(RIP_E_INVAL, "rip_replicas_create: out is NULL");
  *out = nullptr;
  if (dtype != RIP_FP32 && dtype != RIP_BF16)
    return rip::fail(RIP_E_UNSUPPORTED, "unknown dtype %d", dtype);
  if (n_replicas < 1) return rip::fail(RIP_E_INVAL, "n_replicas %d < 1", n_replicas);
  if (n_replicas > RIP_MAX_REPLICAS)
    return rip::fail(RIP_E_UNSUPPORTED, "n_replicas %d > %d", n_replicas, RIP_MAX_REPLICAS);
  if (n_segments < 1 || !seg_numel || !param)
    return rip::fail(RIP_E_INVAL, "need n_segments >= 1, seg_numel and param");
  for (int32_t s = 0; s < n_segments; ++s)
    if (seg_numel[s] < 0) return rip::fail(RIP_E_INVAL, "seg_numel[%d] < 0", s);
  int32_t rc;
  if ((rc = check_nonnull(param, "param", n_replicas, n_segments, seg_numel)) != RIP_OK) return rc;
  if (grad && (rc = check_nonnull(grad, "grad", n_replicas, n_segments, seg_numel)) != RIP_OK)
    return rc;
  if (mom && (rc = check_nonnull(mom, "mom", n_replicas, n_segments, seg_numel)) != RIP_OK)
    return rc;

  // Collapse back-to-back segments into one flat range per replica.
  const int esize = elem_size(dtype);
  int64_t total = 0;
  for (int32_t s = 0; s < n_segments; ++s) total += seg_numel[s];
  const bool flat = back_to_back(param, n_replicas, n_segments, seg_numel, esize) &&
                    (!grad || back_to_back(grad, n_replicas, n_segments, seg_numel, esize)) &&
                    (!mom || back_to_back(mom, n_replicas, n_segments, seg_numel, esize));
  if ((rc = check_align(param, "param", n_replicas, n_segments, seg_numel, flat)) != RIP_OK)
    return rc;
  if (grad && (rc = check_align(grad, "grad", n_replicas, n_segments, seg_numel, flat)) != RIP_OK)
    return rc;
  if (mom && (rc = check_align(mom, "mom", n_replicas, n_segments, seg_numel, flat)) != RIP_OK)
    return rc;
  int device = 0;
  hipError_t e = hipGetDevice(&device);
  if (e != hipSuccess) return rip::fail(RIP_E_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if ((rc = check_buffers(param, grad, mom, n_replicas, n_segments, seg_numel, esize, device)) !=
      RIP_OK)
    return rc;
  const int32_t S = flat ? 1 : n_segments;
  const int32_t N = n_replicas;
  std::vector<uint64_t> ptab((size_t)3 * S * N, 0);
  std::vector<int64_t> numel(S), tile0((size_t)rip::kTileOptions * (S + 1));
  for (int32_t s = 0; s < S; ++s) {
    numel[s] = flat ? total : seg_numel[s];
    for (int32_t r = 0; r < N; ++r) {
      size_t src = (size_t)r * n_segments + s;
      if (flat) {  // the flat range starts at the first non-empty segment
        int32_t s0 = 0;
        while (s0 + 1 < n_segments && seg_numel[s0] == 0) ++s0;
        src = (size_t)r * n_segments + s0;
      }
      const size_t dst = (size_t)s * N + r;
      ptab[dst] = reinterpret_cast<uint64_t>(param[src]);
      ptab[(size_t)S * N + dst] = grad ? reinterpret_cast<uint64_t>(grad[src]) : 0;
      ptab[(size_t)2 * S * N + dst] = mom ? reinterpret_cast<uint64_t>(mom[src]) : 0;
    }
  }
  // First tile of every segment, for each tile size (1, 2, 4, 8 slots).
  for (int o = 0; o < rip::kTileOptions; ++o) {
    const int64_t tile_elems = ((int64_t)rip::kBlock * elems_per_16b(dtype)) << o;
    int64_t* t0 = tile0.data() + (size_t)o * (S + 1);
    t0[0] = 0;
    for (int32_t s = 0; s < S; ++s) t0[s + 1] = t0[s] + (numel[s] + tile_elems - 1) / tile_elems;
  }

  const size_t bytes_ptab = ptab.size() * sizeof(uint64_t);
  const size_t bytes = bytes_ptab + (size_t)S * 8 + tile0.size() * 8;
  if (noalloc && bytes > (size_t)RIP_NOALLOC_TABLE_BYTES)
    return rip::fail(RIP_E_UNSUPPORTED,
                     "rip_replicas_create_noalloc: the tables of %d replicas x %d segments "
                     "take %zu bytes, above the fixed array's %d",
                     N, S, bytes, RIP_NOALLOC_TABLE_BYTES);
  rip_replicas* h = new (std::nothrow) rip_replicas();
  if (!h) return rip::fail(RIP_E_NOMEM, "out of host memory");
  h->n = N;
  h->n_seg = S;
  h->dtype = dtype;
  h->has_grad = grad != nullptr;
  h->has_mom = mom != nullptr;
  for (int o = 0; o < rip::kTileOptions; ++o) h->tiles[o] = tile0[(size_t)o * (S + 1) + S];
  h->numel0 = numel[0];
  h->device = device;
  e = hipDeviceGetAttribute(&h->lds_per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor,
                            h->device);
  if (e != hipSuccess) {
    delete h;
    return rip::fail(RIP_E_HIP, "rip_replicas_create: %s", hipGetErrorString(e));
  }
  std::vector<char> staging(bytes);
  std::memcpy(staging.data(), ptab.data(), bytes_ptab);
  std::memcpy(staging.data() + bytes_ptab, numel.data(), (size_t)S * 8);
  std::memcpy(staging.data() + bytes_ptab + (size_t)S * 8, tile0.data(), tile0.size() * 8);
  char* d = nullptr;
  if (noalloc) {
    // Stage into the device's fixed array.  The handle that owned it is
    // superseded before the copy starts, so that a failed copy cannot leave
    // it pointing at half-written tables.
    std::lock_guard<std::mutex> lock(rip::g_fixed_mu);
    void* fixed = nullptr;
    const int32_t rc2 = rip::fixed_array(device, &fixed);
    if (rc2 != RIP_OK) {
      delete h;
      return rc2;
    }
    const uint64_t generation = ++rip::g_fixed_gen[device];
    e = hipMemcpy(fixed, staging.data(), bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      delete h;
      return rip::fail(RIP_E_HIP, "rip_replicas_create_noalloc: %s", hipGetErrorString(e));
    }
    h->in_fixed_array = true;
    h->generation = generation;
    d = static_cast<char*>(fixed);
  } else {
    e = hipMalloc(&h->dmem, bytes);
    if (e != hipSuccess) {
      delete h;
      return rip::fail(e == hipErrorOutOfMemory ? RIP_E_NOMEM : RIP_E_HIP,
                       "rip_replicas_create: %s", hipGetErrorString(e));
    }
    d = static_cast<char*>(h->dmem);
    e = hipMemcpy(d, staging.data(), bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      (void)hipFree(h->dmem);
      delete h;
      return rip::fail(RIP_E_HIP, "rip_replicas_create: %s", hipGetErrorString(e));
    }
  }
  h->d_ptab = reinterpret_cast<const uint64_t*>(d);
  h->d_numel = reinterpret_cast<const int64_t*>(d + bytes_ptab);
  h->d_tile0 = reinterpret_cast<const int64_t*>(d + bytes_ptab + (size_t)S * 8);
  *out = h;
  return RIP_OK;
}

// A handle whose tables a later rip_replicas_create_noalloc call on its
// device has overwritten must not launch.
int32_t check_current(const rip_replicas* r) {
  if (!r->in_fixed_array) return RIP_OK;
  std::lock_guard<std::mutex> lock(rip::g_fixed_mu);
  if (rip::g_fixed_gen[r->device] != r->generation)
    return rip::fail(RIP_E_INVAL,
                     "this rip_replicas_create_noalloc handle was superseded by a later one on "
                     "device %d (they share one table array)",
                     r->device);
  return RIP_OK;
}

}  // namespace

extern "C" int32_t rip_replicas_create(int32_t n_replicas, int32_t n_segments, int32_t dtype,
                                       const int64_t* seg_numel, void* const* param,
                                       void* const* grad, void* const* mom, rip_replicas** out) {
  return create_replicas(n_replicas, n_segments, dtype, seg_numel, param, grad, mom, out, false);
}

extern "C" int32_t rip_replicas_create_noalloc(int32_t n_replicas, int32_t n_segments,
                                               int32_t dtype, const int64_t* seg_numel,
                                               void* const* param, void* const* grad,
                                               void* const* mom, rip_replicas** out) {
  return create_replicas(n_replicas, n_segments, dtype, seg_numel, param, grad, mom, out, true);
}

extern "C" void rip_replicas_destroy(rip_replicas* r) {
  if (!r) return;
  if (r->dmem) (void)hipFree(r->dmem);
  delete r;
}

namespace {

// The units' sizes and updating members (for the launch policy).
struct UnitShapes {
  int32_t n = 0;
  int32_t k[RIP_MAX_REPLICAS], act[RIP_MAX_REPLICAS];
};

// Checks one step's schedule and turns it into units (groups first, in the
// order given, then active workers outside every group, ascending).
int32_t build_step(const rip_replicas* r, const int32_t* group_offsets, const int32_t* members,
                   int32_t n_groups, const int32_t* active, int32_t n_active, const rip_sgd* sgd,
                   rip::StepArgs& a, bool& mom, UnitShapes& shapes) {
  const int32_t N = r->n;
  if (n_groups < 0 || n_active < 0) return rip::fail(RIP_E_INVAL, "negative count");
  if (n_groups > 0 && (!group_offsets || !members))
    return rip::fail(RIP_E_INVAL, "groups given without group_offsets/members");
  if (n_active > 0 && !active) return rip::fail(RIP_E_INVAL, "active is NULL");
  if (!sgd && n_active > 0) return rip::fail(RIP_E_INVAL, "active workers need an sgd step");
  if (n_active > N) return rip::fail(RIP_E_INVAL, "n_active %d > n_replicas %d", n_active, N);
  if (sgd && n_active > 0) {
    if (!r->has_grad) return rip::fail(RIP_E_INVAL, "local update without gradient buffers");
    if (sgd->momentum != 0.0f && !r->has_mom)
      return rip::fail(RIP_E_INVAL, "momentum %g without momentum buffers", (double)sgd->momentum);
  }
  if (sgd && sgd->nesterov && sgd->momentum == 0.0f)
    return rip::fail(RIP_E_INVAL, "Nesterov momentum needs a nonzero momentum");
  std::vector<uint8_t> in_group(N, 0), is_active(N, 0);
  for (int32_t i = 0; i < n_active; ++i) {
    const int32_t id = active[i];
    if (id < 0 || id >= N) return rip::fail(RIP_E_INVAL, "active id %d out of range", id);
    if (is_active[id]) return rip::fail(RIP_E_INVAL, "active id %d listed twice", id);
    is_active[id] = 1;
  }
  if (n_groups > 0 && group_offsets[0] != 0)
    return rip::fail(RIP_E_INVAL, "group_offsets[0] must be 0");
  for (int32_t g = 0; g < n_groups; ++g) {
    const int32_t b = group_offsets[g], e = group_offsets[g + 1];
    if (e <= b) return rip::fail(RIP_E_INVAL, "group %d is empty or offsets decrease", g);
    if (e > N) return rip::fail(RIP_E_OVERLAP, "groups list more than %d members", N);
    for (int32_t j = b; j < e; ++j) {
      const int32_t m = members[j];
      if (m < 0 || m >= N) return rip::fail(RIP_E_INVAL, "member %d of group %d out of range", m, g);
      if (j > b && m <= members[j - 1])
        return rip::fail(RIP_E_INVAL, "group %d is not strictly ascending", g);
      if (in_group[m]) return rip::fail(RIP_E_OVERLAP, "replica %d is in two groups", m);
      in_group[m] = 1;
    }
  }

  std::memset(&a, 0, sizeof a);
  int32_t units = 0, pos = 0;
  std::vector<int32_t> unit_off(1, 0);
  for (int32_t g = 0; g < n_groups; ++g) {
    const int32_t b = group_offsets[g], e = group_offsets[g + 1];
    if (e - b == 1 && !is_active[members[b]]) continue;  // identity: nothing to do
    for (int32_t j = b; j < e; ++j) a.member[pos++] = (uint8_t)members[j];
    unit_off.push_back(pos);
    ++units;
  }
  for (int32_t id = 0; id < N; ++id)
    if (is_active[id] && !in_group[id]) {
      a.member[pos++] = (uint8_t)id;
      unit_off.push_back(pos);
      ++units;
    }
  for (int32_t id = 0; id < N; ++id)
    if (is_active[id]) a.active_bits[id >> 5] |= 1u << (id & 31);
  for (int32_t u = 0; u < units; ++u) {
    const int32_t b = unit_off[u], k = unit_off[u + 1] - b;
    uint32_t act8 = 0;
    for (int32_t j = 0; j < k && j < 8; ++j) act8 |= (uint32_t)is_active[a.member[b + j]] << j;
    a.unit_info[u] = rip::unit_info_pack((uint32_t)b, (uint32_t)k, act8);
  }
  a.uniform_k = units > 0 ? (uint32_t)(unit_off[1] - unit_off[0]) : 0;
  for (int32_t u = 1; u < units && a.uniform_k; ++u)
    if ((uint32_t)(unit_off[u + 1] - unit_off[u]) != a.uniform_k) a.uniform_k = 0;
  a.ptab = r->d_ptab;
  a.seg_numel = r->d_numel;
  a.seg_tile0 = r->d_tile0;
  a.n_seg = r->n_seg;
  a.n_rep = N;
  a.n_units = units;
  a.lr = sgd ? sgd->lr : 0.0f;
  a.mu = sgd ? sgd->momentum : 0.0f;
  a.wd = sgd ? sgd->weight_decay : 0.0f;
  a.nesterov = sgd && sgd->nesterov ? 1 : 0;
  mom = sgd && sgd->momentum != 0.0f && n_active > 0;
  int64_t work = 0;
  a.unit_work0[0] = 0;
  for (int32_t u = 0; u < units; ++u) {
    const int k = unit_off[u + 1] - unit_off[u];
    work += r->tiles[rip::slot_log2(k, mom)];
    if (work >= (int64_t)1 << 31)
      return rip::fail(RIP_E_UNSUPPORTED, "more than 2^31 tiles in one step (replicas too large)");
    a.unit_work0[u + 1] = (uint32_t)work;
  }
  a.work = (uint32_t)work;
  a.uniform_tiles = units > 0 ? a.unit_work0[1] : 0;
  for (int32_t u = 1; u < units && a.uniform_tiles; ++u)
    if (a.unit_work0[u + 1] - a.unit_work0[u] != a.uniform_tiles) a.uniform_tiles = 0;
  a.flat_numel = r->n_seg == 1 ? r->numel0 : 0;
  shapes.n = units;
  for (int32_t u = 0; u < units; ++u) {
    const int32_t b = unit_off[u];
    shapes.k[u] = unit_off[u + 1] - b;
    shapes.act[u] = 0;
    for (int32_t j = 0; j < shapes.k[u]; ++j) shapes.act[u] += is_active[a.member[b + j]];
  }
  return RIP_OK;
}

// The launch of the units u with part[u] == which, in their order: the
// same member table, active bits and scalars, with the unit tables rebuilt.
void subset_step(const rip::StepArgs& a, const uint8_t* part, int which, rip::StepArgs& out) {
  std::memcpy(&out, &a, sizeof a);
  int32_t n = 0;
  uint32_t work = 0;
  out.unit_work0[0] = 0;
  for (int32_t u = 0; u < a.n_units; ++u) {
    if (part[u] != which) continue;
    out.unit_info[n] = a.unit_info[u];
    work += a.unit_work0[u + 1] - a.unit_work0[u];
    out.unit_work0[++n] = work;
  }
  out.n_units = n;
  out.work = work;
  out.uniform_k = 0;  // the units no longer sit at base = unit * k
  out.uniform_tiles = n > 0 ? out.unit_work0[1] : 0;
  for (int32_t u = 1; u < n && out.uniform_tiles; ++u)
    if (out.unit_work0[u + 1] - out.unit_work0[u] != out.uniform_tiles) out.uniform_tiles = 0;
}

}  // namespace

extern "C" int32_t rip_preduce(const rip_replicas* r, const int32_t* group_offsets,
                               const int32_t* members, int32_t n_groups, const int32_t* active,
                               int32_t n_active, const rip_sgd* sgd, void* stream) {
  rip::clear_error();
  rip::g_last_launches = 0;
  if (!r) return rip::fail(RIP_E_INVAL, "rip_preduce: replicas handle is NULL");
  rip::StepArgs a;
  bool mom = false;
  UnitShapes shapes;
  int32_t rc =
      build_step(r, group_offsets, members, n_groups, active, n_active, sgd, a, mom, shapes);
  if (rc != RIP_OK) return rc;
  if (a.work == 0) return RIP_OK;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return rip::fail(RIP_E_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev != r->device)
    return rip::fail(RIP_E_INVAL, "current device %d differs from the handle's device %d", dev,
                     r->device);
  if ((rc = check_current(r)) != RIP_OK) return rc;
  const int max_blocks =
      rip::g_max_blocks.load() > 0 ? rip::g_max_blocks.load() : rip::kDefaultMaxBlocks;
  const int forced_bpc = rip::g_blocks_per_cu.load();
  const bool ext = a.wd != 0.0f || a.nesterov != 0;
  auto launch = [&](const rip::StepArgs& x, int waves) -> int32_t {
    if (x.work == 0) return RIP_OK;
    const int blocks = (int)(x.work < (uint32_t)max_blocks ? x.work : (uint32_t)max_blocks);
    const int bpc = forced_bpc > 0 ? forced_bpc : waves * 64 / rip::kBlock;
    size_t lds = 0;
    if (bpc > 0 && r->lds_per_cu > 0) lds = (size_t)(r->lds_per_cu / bpc) & ~(size_t)255;
    const hipError_t le = rip::launch_fused_step(x, r->dtype == RIP_BF16, mom, ext, blocks, lds,
                                                 static_cast<hipStream_t>(stream));
    if (le != hipSuccess) return rip::fail(RIP_E_HIP, "kernel launch: %s", hipGetErrorString(le));
    ++rip::g_last_launches;
    return RIP_OK;
  };
  // One launch, or two when the units want residency caps far apart (and
  // no cap is forced).
  uint8_t part[RIP_MAX_REPLICAS];
  int w0 = 0, w1 = 0;
  if (forced_bpc == 0 &&
      rip::policy::split_units(shapes.k, shapes.act, shapes.n, mom, part, &w0, &w1)) {
    rip::StepArgs a0, a1;
    subset_step(a, part, 0, a0);
    subset_step(a, part, 1, a1);
    if ((rc = launch(a0, w0)) != RIP_OK) return rc;
    return launch(a1, w1);
  }
  return launch(a, rip::policy::launch_waves(shapes.k, shapes.act, shapes.n, mom));
}

extern "C" int32_t rip_step(rip_sched* s, const rip_replicas* r, int64_t step,
                            const uint8_t* eligible, const rip_sgd* sgd, void* stream,
                            int32_t* active, int32_t* n_active, int32_t* group_offsets,
                            int32_t* members, int32_t* n_groups) {
  rip::clear_error();
  rip::g_last_launches = 0;
  if (!s || !r || !sgd) return rip::fail(RIP_E_INVAL, "rip_step: null scheduler, replicas or sgd");
  if (rip::sched_workers(s) != r->n)
    return rip::fail(RIP_E_INVAL, "scheduler has %d workers, replicas handle %d",
                     rip::sched_workers(s), r->n);
  // Everything the launch could reject for any schedule is checked before
  // the scheduler moves.
  if (!r->has_grad) return rip::fail(RIP_E_INVAL, "rip_step: replicas have no gradient buffers");
  if (sgd->momentum != 0.0f && !r->has_mom)
    return rip::fail(RIP_E_INVAL, "momentum %g without momentum buffers", (double)sgd->momentum);
  if (sgd->nesterov && sgd->momentum == 0.0f)
    return rip::fail(RIP_E_INVAL, "Nesterov momentum needs a nonzero momentum");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return rip::fail(RIP_E_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev != r->device)
    return rip::fail(RIP_E_INVAL, "current device %d differs from the handle's device %d", dev,
                     r->device);
  if (const int32_t rc0 = check_current(r); rc0 != RIP_OK) return rc0;
  int32_t act_buf[RIP_MAX_REPLICAS], off_buf[RIP_MAX_REPLICAS + 1], mem_buf[RIP_MAX_REPLICAS];
  int32_t na = 0, ng = 0;
  int32_t* act = active ? active : act_buf;
  int32_t* off = group_offsets ? group_offsets : off_buf;
  int32_t* mem = members ? members : mem_buf;
  const int32_t rc = rip::schedule_then(s, step, eligible, act, &na, off, mem, &ng, [&] {
    return rip_preduce(r, off, mem, ng, act, na, sgd, stream);
  });
  if (rc == RIP_OK) {
    if (n_active) *n_active = na;
    if (n_groups) *n_groups = ng;
  }
  return rc;
}

extern "C" int32_t rip_local_step(const rip_replicas* r, const int32_t* active, int32_t n_active,
                                  const rip_sgd* sgd, void* stream) {
  if (!sgd) {
    rip::clear_error();
    rip::g_last_launches = 0;
    return rip::fail(RIP_E_INVAL, "rip_local_step: sgd is NULL");
  }
  return rip_preduce(r, nullptr, nullptr, 0, active, n_active, sgd, stream);
}
