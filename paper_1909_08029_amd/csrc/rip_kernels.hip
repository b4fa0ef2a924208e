// Fused local update + P-Reduce for CDNA4 (gfx950).
//
// One launch runs one step of the algorithm of Fig. 4 for every scheduled
// unit of work: a group G (Step 4, the F^G of Sec. 3.2, with the Step 2
// update of its members that compute this step folded in) or a worker that
// updates without synchronizing.  Disjoint groups run concurrently (Sec. 3.2).
//
// Work decomposition.  Every unit touches the same element range of its
// members' buffers, so the launch is a list of (unit, tile) work items, one
// per single-wave workgroup, unit after unit.  A tile is 64 lanes x 1-8
// slots x 16 bytes of each member stream; the slot count shrinks as the
// unit's number of streams grows (see slot_log2), so every lane keeps 8-16
// 16-byte loads in flight (24 for a group of eight with momentum).  The host caps residency per launch at 4-14 waves per CU
// (an LDS reservation), fewer when the units read more streams: HBM3E
// delivered its best rate at a bounded depth of outstanding requests, not at
// full occupancy.
// A workgroup handles one unit, so the unit's size k, its member ids and their active
// flags are wave-uniform: they sit in scalar registers and every branch on
// them is a scalar branch.  Each thread issues the loads of all members
// (and their gradients / momenta) for all its slots before any arithmetic,
// then writes the mean back to every member.
//
// The operation is a stream over HBM with no data reuse and about one flop
// per 4 bytes, so there is no LDS tiling and no matrix-core work: the design
// aims at full-width (dwordx4) coalesced accesses and enough bytes in flight
// per CU.
//
// Arithmetic follows the exact fp32 order documented in include/rip.h (no
// contraction into FMA, sequential sum in ascending member order, product
// with (float)(1.0/k)); bf16 values widen exactly and round to nearest-even
// once when stored.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "rip_kernel_args.h"

#pragma clang fp contract(off)

namespace rip {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Replica buffers are plain device memory: the element-wise path (ragged
// tails) accesses them through the global address space so the compiler
// emits global_* (not flat_*) instructions.
#define RIP_GLOBAL __attribute__((address_space(1)))

// Full tiles are accessed through buffer instructions, non-temporal (every
// byte is touched once per step): a descriptor per member stream whose base
// is the tile's first byte and whose size is the tile's bytes, and a
// per-lane offset of at most a few KB.  On gfx950 this form streamed 3-4%
// faster than the same non-temporal accesses as global instructions (with a
// 64-bit per-lane address or an SGPR base and 32-bit offset alike), and
// faster than a buffer descriptor over the whole stream with the tile offset
// folded into the per-lane offset.  The descriptor's size also bounds every
// access in hardware.
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr int kRsrcWord3 = 0x00020000;  // raw (untyped) buffer, 32-bit data format
constexpr int kNonTemporal = 2;         // cache-policy operand: nt

__device__ __forceinline__ Rsrc tile_rsrc(const char* base, int64_t tile_byte, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base) + tile_byte, 0, bytes,
                                           kRsrcWord3);
}
__device__ __forceinline__ u32x4 bld16(Rsrc r, int off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kNonTemporal);
}
__device__ __forceinline__ void bst16(Rsrc r, int off, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, kNonTemporal);
}

// The launch tables -- the kernel argument's own arrays (unit tables, member
// ids, active bits) and the registered pointer and segment tables -- are
// never written while a launch runs.  Reading them through the constant
// address space lets the compiler fetch these wave-uniform values with
// scalar loads, also inside divergent code; read as ordinary global memory
// they become vector loads that wait behind the streaming traffic (the
// kernel's own stores could alias them, as far as the compiler can tell).
// The argument's arrays are read where the argument lives, in the kernel-
// argument segment (the only explicit argument, at its start), never through
// the address of a by-value copy, which is private memory in an unoptimized
// build.
#define RIP_CONST __attribute__((address_space(4)))

typedef const RIP_CONST StepArgs KArgs;
__device__ __forceinline__ KArgs& kargs() {
  return *(KArgs*)__builtin_amdgcn_kernarg_segment_ptr();
}

template <typename T>
__device__ __forceinline__ T cld(const T* p, int64_t i) {
  return ((const RIP_CONST T*)p)[i];
}
template <typename T>
__device__ __forceinline__ T cld(const RIP_CONST T* p, int64_t i) {
  return p[i];
}
// Byte i of the member table, read as its containing dword.
__device__ __forceinline__ int cld8(const RIP_CONST uint8_t* p, int i) {
  const uint32_t word = ((const RIP_CONST uint32_t*)p)[i >> 2];
  return (int)((word >> ((i & 3) * 8)) & 0xFFu);
}
// Bytes i .. i+7 of the (16-byte aligned, padded) member table as one 64-bit
// value, byte j in bits 8j..8j+7: one 16-byte scalar load of the aligned
// dwords that hold them, then a funnel shift.
typedef uint32_t u32x4c __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint64_t cld8x8(const RIP_CONST uint8_t* p, int i) {
  const u32x4c d = ((const RIP_CONST u32x4c*)p)[i >> 4];
  const u32x4c e = ((const RIP_CONST u32x4c*)p)[(i >> 4) + 1];
  // 32 bytes d|e hold bytes (i & ~15) .. (i & ~15) + 31, which cover i .. i+7
  const int sh = (i & 15) * 8;  // 0..120
  const uint64_t q0 = d.x | ((uint64_t)d.y << 32), q1 = d.z | ((uint64_t)d.w << 32);
  const uint64_t q2 = e.x | ((uint64_t)e.y << 32);
  if (sh == 0) return q0;
  if (sh < 64) return (q0 >> sh) | (q1 << (64 - sh));
  if (sh == 64) return q1;
  return (q1 >> (sh - 64)) | (q2 << (128 - sh));
}

__device__ __forceinline__ float bf16_lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t x) { return __uint_as_float(x & 0xFFFF0000u); }

// fp32 -> bf16, round to nearest even, NaN kept quiet: gfx950's
// v_cvt_pk_bf16_f32 (what clang emits for a conversion to __bf16), two values
// per instruction.  Its results equal the round-to-nearest-even definition
// for all 2^32 fp32 inputs (tests/test_gpu_ieee_edges.py runs every one).
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t bf16_pack2(float lo, float hi) {
  const f32x2 f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}
__device__ __forceinline__ uint16_t bf16_round(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

template <bool BF16>
struct Vec;

// 16 bytes = 4 fp32
template <>
struct Vec<false> {
  static constexpr int N = 4;
  static __device__ __forceinline__ void unpack(u32x4 x, float (&f)[N]) {
    f[0] = __uint_as_float(x.x);
    f[1] = __uint_as_float(x.y);
    f[2] = __uint_as_float(x.z);
    f[3] = __uint_as_float(x.w);
  }
  static __device__ __forceinline__ u32x4 pack(const float (&f)[N]) {
    u32x4 x;
    x.x = __float_as_uint(f[0]);
    x.y = __float_as_uint(f[1]);
    x.z = __float_as_uint(f[2]);
    x.w = __float_as_uint(f[3]);
    return x;
  }
};

// 16 bytes = 8 bf16; element 2i is the low half of word i
template <>
struct Vec<true> {
  static constexpr int N = 8;
  static __device__ __forceinline__ void unpack(u32x4 x, float (&f)[N]) {
    f[0] = bf16_lo(x.x); f[1] = bf16_hi(x.x);
    f[2] = bf16_lo(x.y); f[3] = bf16_hi(x.y);
    f[4] = bf16_lo(x.z); f[5] = bf16_hi(x.z);
    f[6] = bf16_lo(x.w); f[7] = bf16_hi(x.w);
  }
  static __device__ __forceinline__ u32x4 pack(const float (&f)[N]) {
    u32x4 x;
    x.x = bf16_pack2(f[0], f[1]);
    x.y = bf16_pack2(f[2], f[3]);
    x.z = bf16_pack2(f[4], f[5]);
    x.w = bf16_pack2(f[6], f[7]);
    return x;
  }
};

// Scalar element access for tails and the generic (k > 8) path.
template <bool BF16>
__device__ __forceinline__ float ld1(const char* base, int64_t e) {
  if constexpr (BF16)
    return __uint_as_float(uint32_t(((const RIP_GLOBAL uint16_t*)base)[e]) << 16);
  else
    return ((const RIP_GLOBAL float*)base)[e];
}
template <bool BF16>
__device__ __forceinline__ void st1(char* base, int64_t e, float v) {
  if constexpr (BF16)
    ((RIP_GLOBAL uint16_t*)base)[e] = bf16_round(v);
  else
    ((RIP_GLOBAL float*)base)[e] = v;
}

// (float)(1.0/k) for every group size, evaluated at compile time.
struct InvTable {
  float v[RIP_MAX_REPLICAS + 1];
};
constexpr InvTable make_inv_table() {
  InvTable t{};
  for (int k = 1; k <= RIP_MAX_REPLICAS; ++k) t.v[k] = (float)(1.0 / k);
  return t;
}
__constant__ InvTable kInv = make_inv_table();

// Step 2 for one element (fp32, this order, no contraction):
//   g' = g + wd*w                       (only when weight decay is on)
//   SGD:       u = w - lr*g'
//   momentum:  v = mu*v + g';  u = w - lr*v,  or with Nesterov u = w - lr*(g' + mu*v)
// EXT selects the kernel variant that handles weight decay and Nesterov.
// Their flags are wave-uniform, but the compiler turns the tests into
// per-element selects, computing both sides: that more than doubles the
// arithmetic per element, which costs bandwidth when few waves share a CU.
// Plain SGD and heavy-ball momentum therefore get a variant without them;
// with wd == 0 and no Nesterov both variants compute the same values.
struct Opt {
  float lr, mu, wd;
  bool nesterov;
};

template <bool MOM, bool EXT>
__device__ __forceinline__ float update(float w, float g, float& v, const Opt& o) {
  if constexpr (EXT) {
    if (o.wd != 0.0f) g = g + o.wd * w;
  }
  if constexpr (MOM) {
    v = o.mu * v + g;
    if constexpr (EXT) return w - o.lr * (o.nesterov ? g + o.mu * v : v);
    return w - o.lr * v;
  } else {
    return w - o.lr * g;
  }
}

struct Members {
  char* w[kMaxK];
  const char* g[kMaxK];
  char* v[kMaxK];
  bool act[kMaxK];
};

// The unit's member ids (one per byte of `ids`) came with the unit; their
// pointers are 3K independent scalar loads, all issued before one wait.
template <int K, bool MOM>
__device__ __forceinline__ void load_members(const StepArgs& a, uint64_t ids, uint32_t act8,
                                             int seg, Members& m) {
  const int plane = a.n_seg * a.n_rep;
#pragma unroll
  for (int j = 0; j < K; ++j) {
    const int id = (int)((ids >> (8 * j)) & 0xFFu);
    const int idx = seg * a.n_rep + id;
    m.w[j] = reinterpret_cast<char*>(cld(a.ptab, idx));
    m.g[j] = reinterpret_cast<const char*>(cld(a.ptab, plane + idx));
    m.v[j] = reinterpret_cast<char*>(cld(a.ptab, 2 * plane + idx));
    m.act[j] = (act8 >> j) & 1u;
  }
  // Materialize every member's pointers and flag here, so one wait covers
  // all of these scalar loads.  Left alone, the compiler sinks each pointer
  // load next to its use, and every vector load then waits for its own
  // scalar round trip: the wave's loads go out one at a time.
#pragma unroll
  for (int j = 0; j < K; ++j) {
    asm volatile("" ::"s"(m.w[j]), "s"(m.g[j]), "s"((int)m.act[j]));
    if constexpr (MOM) asm volatile("" ::"s"(m.v[j]));
  }
}

// U consecutive 16-byte slots of a full tile for a unit of K members; the
// tile starts `tile_byte` bytes into every member stream.
template <int K, int U, bool BF16, bool MOM, bool EXT>
__device__ __forceinline__ void tile_slots(const Members& m, int64_t tile_byte, const Opt& o) {
  using V = Vec<BF16>;
  constexpr int N = V::N;
  constexpr float inv_k = (float)(1.0 / K);
  constexpr int kTileBytes = U * kBlock * 16;
  int off[U];  // this lane's byte offset of each slot within the tile
#pragma unroll
  for (int u = 0; u < U; ++u) off[u] = (u * kBlock + (int)threadIdx.x) * 16;
  Rsrc rw[K], rg[K], rv[K];
#pragma unroll
  for (int j = 0; j < K; ++j) {
    rw[j] = tile_rsrc(m.w[j], tile_byte, kTileBytes);
    rg[j] = tile_rsrc(m.g[j], tile_byte, kTileBytes);
    if constexpr (MOM) rv[j] = tile_rsrc(m.v[j], tile_byte, kTileBytes);
  }
  u32x4 wv[U][K], gv[U][K], vv[U][K];
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int j = 0; j < K; ++j) {
      wv[u][j] = bld16(rw[j], off[u]);
      if (m.act[j]) {
        gv[u][j] = bld16(rg[j], off[u]);
        if constexpr (MOM) vv[u][j] = bld16(rv[j], off[u]);
      }
    }
  // All arithmetic comes before the first store.  Stores count against the
  // same vmcnt as loads, and because the gradient and momentum loads are
  // conditional (active members only) the compiler's waits before each
  // member's arithmetic are conservative: a momentum store issued between two
  // members would make the next wait cover that store's completion, a full
  // write round trip.  (A straight-line variant for groups whose members all
  // update, with exact waits, measured no faster and slowed bf16 by 2%.)
  u32x4 out[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    float s[N];
#pragma unroll
    for (int j = 0; j < K; ++j) {
      float x[N];
      V::unpack(wv[u][j], x);
      if (m.act[j]) {
        float g[N], v[N];
        V::unpack(gv[u][j], g);
        if constexpr (MOM) V::unpack(vv[u][j], v);
#pragma unroll
        for (int i = 0; i < N; ++i) x[i] = update<MOM, EXT>(x[i], g[i], v[i], o);
        if constexpr (MOM) vv[u][j] = V::pack(v);
      }
#pragma unroll
      for (int i = 0; i < N; ++i) s[i] = (j == 0) ? x[i] : s[i] + x[i];
    }
    if constexpr (K > 1) {
#pragma unroll
      for (int i = 0; i < N; ++i) s[i] = s[i] * inv_k;
    }
    out[u] = V::pack(s);
  }
  // Keep the instruction scheduler from sinking arithmetic below the stores.
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (MOM) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < K; ++j)
        if (m.act[j]) bst16(rv[j], off[u], vv[u][j]);
  }
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int j = 0; j < K; ++j) bst16(rw[j], off[u], out[u]);
}

// Element-wise path for a partial tile (any k): each thread walks elements
// e0 + i*stride below `end`.
template <bool BF16, bool MOM, bool EXT>
__device__ void elementwise(const StepArgs& a, int base, int k, int seg, int64_t begin,
                            int64_t end) {
  const int plane = a.n_seg * a.n_rep;
  const float inv_k = kInv.v[k];
  const Opt o{a.lr, a.mu, a.wd, a.nesterov != 0};
  for (int64_t e = begin + threadIdx.x; e < end; e += kBlock) {
    float s = 0.0f;
    for (int j = 0; j < k; ++j) {
      const int id = cld8(kargs().member, base + j);
      const int idx = seg * a.n_rep + id;
      char* w = reinterpret_cast<char*>(cld(a.ptab, idx));
      float x = ld1<BF16>(w, e);
      if ((cld(kargs().active_bits, id >> 5) >> (id & 31)) & 1u) {
        const float g = ld1<BF16>(reinterpret_cast<const char*>(cld(a.ptab, plane + idx)), e);
        if constexpr (MOM) {
          char* vp = reinterpret_cast<char*>(cld(a.ptab, 2 * plane + idx));
          float v = ld1<BF16>(vp, e);
          x = update<true, EXT>(x, g, v, o);
          st1<BF16>(vp, e, v);
        } else {
          float unused = 0.0f;
          x = update<false, EXT>(x, g, unused, o);
        }
      }
      s = (j == 0) ? x : s + x;
    }
    if (k > 1) s = s * inv_k;
    for (int j = 0; j < k; ++j) {
      const int id = cld8(kargs().member, base + j);
      st1<BF16>(reinterpret_cast<char*>(cld(a.ptab, seg * a.n_rep + id)), e, s);
    }
  }
}

// A full tile of a group larger than kMaxK (All-Reduce as one group of every
// worker, large divisions): the members stream through in chunks of eight,
// 16-byte accesses as in tile_slots, their updated values summed into one
// running fp32 sum in ascending member order; the mean then goes to every
// member.  Each member's w, g and v are read once and written once, as in
// the specialized paths; only the member pointers are fetched twice.
template <bool BF16, bool MOM, bool EXT>
__device__ __forceinline__ void wide_tile(const StepArgs& a, int base, int k, int seg,
                                          int64_t e_tile) {
  using V = Vec<BF16>;
  constexpr int N = V::N;
  constexpr int C = kMaxK;  // members per chunk
  const int plane = a.n_seg * a.n_rep;
  const Opt o{a.lr, a.mu, a.wd, a.nesterov != 0};
  const int64_t tile_byte = e_tile * (BF16 ? 2 : 4);
  constexpr int kTileBytes = kBlock * 16;
  const int off = (int)threadIdx.x * 16;
  float s[N];
  for (int j0 = 0; j0 < k; j0 += C) {
    const uint64_t ids = cld8x8(kargs().member, base + j0);  // bytes past the unit are unused
    char* w[C];
    const char* g[C];
    char* v[C];
    bool act[C];
#pragma unroll
    for (int jj = 0; jj < C; ++jj) {
      const int id = (int)((ids >> (8 * jj)) & 0xFFu);
      const int idx = seg * a.n_rep + id;
      const bool in = j0 + jj < k;
      w[jj] = in ? reinterpret_cast<char*>(cld(a.ptab, idx)) : nullptr;
      g[jj] = in ? reinterpret_cast<const char*>(cld(a.ptab, plane + idx)) : nullptr;
      v[jj] = in && MOM ? reinterpret_cast<char*>(cld(a.ptab, 2 * plane + idx)) : nullptr;
      act[jj] = in && ((cld(kargs().active_bits, id >> 5) >> (id & 31)) & 1u);
    }
#pragma unroll
    for (int jj = 0; jj < C; ++jj) {
      asm volatile("" ::"s"(w[jj]), "s"(g[jj]), "s"((int)act[jj]));
      if constexpr (MOM) asm volatile("" ::"s"(v[jj]));
    }
    Rsrc rw[C], rg[C], rv[C];
#pragma unroll
    for (int jj = 0; jj < C; ++jj) {
      rw[jj] = tile_rsrc(w[jj], tile_byte, kTileBytes);
      rg[jj] = tile_rsrc(g[jj], tile_byte, kTileBytes);
      if constexpr (MOM) rv[jj] = tile_rsrc(v[jj], tile_byte, kTileBytes);
    }
    u32x4 wv[C], gv[C], vv[C];
#pragma unroll
    for (int jj = 0; jj < C; ++jj) {
      if (j0 + jj < k) {
        wv[jj] = bld16(rw[jj], off);
        if (act[jj]) {
          gv[jj] = bld16(rg[jj], off);
          if constexpr (MOM) vv[jj] = bld16(rv[jj], off);
        }
      }
    }
#pragma unroll
    for (int jj = 0; jj < C; ++jj) {
      if (j0 + jj < k) {
        float x[N];
        V::unpack(wv[jj], x);
        if (act[jj]) {
          float gf[N], vf[N];
          V::unpack(gv[jj], gf);
          if constexpr (MOM) V::unpack(vv[jj], vf);
#pragma unroll
          for (int i = 0; i < N; ++i) x[i] = update<MOM, EXT>(x[i], gf[i], vf[i], o);
          if constexpr (MOM) vv[jj] = V::pack(vf);
        }
#pragma unroll
        for (int i = 0; i < N; ++i) s[i] = (j0 + jj == 0) ? x[i] : s[i] + x[i];
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (MOM) {
#pragma unroll
      for (int jj = 0; jj < C; ++jj)
        if (act[jj]) bst16(rv[jj], off, vv[jj]);
    }
  }
  const float inv_k = kInv.v[k];
#pragma unroll
  for (int i = 0; i < N; ++i) s[i] = s[i] * inv_k;
  const u32x4 out = V::pack(s);
  for (int j0 = 0; j0 < k; j0 += C) {
    const uint64_t ids = cld8x8(kargs().member, base + j0);
    char* w[C];
#pragma unroll
    for (int jj = 0; jj < C; ++jj) {
      const int id = (int)((ids >> (8 * jj)) & 0xFFu);
      w[jj] = j0 + jj < k ? reinterpret_cast<char*>(cld(a.ptab, seg * a.n_rep + id)) : nullptr;
    }
#pragma unroll
    for (int jj = 0; jj < C; ++jj) asm volatile("" ::"s"(w[jj]));
#pragma unroll
    for (int jj = 0; jj < C; ++jj)
      if (j0 + jj < k) bst16(tile_rsrc(w[jj], tile_byte, kTileBytes), off, out);
  }
}

// Last index i in [0, n) with v[i] <= x (v ascending, v[0] <= x).
template <typename P, typename X>
__device__ __forceinline__ int last_le(P v, int n, X x) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if ((X)cld(v, mid) <= x) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// The unit a workgroup works on, as the main loop decoded it.
struct Unit {
  int base, k;    // member[base .. base + k)
  uint32_t act8;  // update flags of members 0..7
  uint64_t ids;   // member ids 0..7, one per byte
};

// Launch-wide values, read once per workgroup before anything else.
struct Header {
  uint32_t work, uniform_tiles, uniform_k;
  int n_seg;
  int64_t flat_numel;
};

// One tile of a unit of K members (K <= kMaxK, or 0 for the element-wise path
// with any k).  The tile geometry is a compile-time constant here, so a
// workgroup reaches its first vector load after a handful of scalar
// instructions: a flat handle needs no segment search at all.
template <int K, bool BF16, bool MOM, bool EXT>
__device__ __forceinline__ void unit_tile(const StepArgs& a, const Header& h, const Unit& u,
                                          int64_t tile) {
  constexpr int O = slot_log2(K == 0 ? kMaxK + 1 : K, MOM);
  constexpr int SL = 1 << O;
  constexpr int N = Vec<BF16>::N;
  constexpr int64_t TE = (int64_t)kBlock * N * SL;  // elements per tile
  int seg = 0;
  int64_t e_tile, numel;
  if (h.n_seg == 1) {
    e_tile = tile * TE;
    numel = h.flat_numel;
  } else {
    const int64_t* tile0 = a.seg_tile0 + O * (h.n_seg + 1);
    seg = last_le(tile0, h.n_seg, tile);
    e_tile = (tile - cld(tile0, seg)) * TE;
    numel = cld(a.seg_numel, seg);
  }
  if constexpr (K > 0) {
    if (e_tile + TE <= numel) {
      constexpr int esize = BF16 ? 2 : 4;
      Members m;
      load_members<K, MOM>(a, u.ids, u.act8, seg, m);
      tile_slots<K, SL, BF16, MOM, EXT>(m, e_tile * esize, Opt{a.lr, a.mu, a.wd, a.nesterov != 0});
      return;
    }
  } else {
    if (e_tile + TE <= numel) {
      wide_tile<BF16, MOM, EXT>(a, u.base, u.k, seg, e_tile);
      return;
    }
  }
  const int64_t end = (e_tile + TE < numel) ? e_tile + TE : numel;
  elementwise<BF16, MOM, EXT>(a, u.base, u.k, seg, e_tile, end);
}

template <bool BF16, bool MOM, bool EXT>
__global__ __launch_bounds__(kBlock) void fused_step_kernel(StepArgs a) {
  // Load the whole header into scalar registers in one batch up front: left
  // to itself the compiler spreads it over several batches (and loads
  // flat_numel late, through a select of addresses), and every extra batch is
  // one more dependent scalar round trip before the workgroup's first vector
  // load.
  const Header h{a.work, a.uniform_tiles, a.uniform_k, a.n_seg, a.flat_numel};
  asm volatile("" ::"s"(h.work), "s"(h.uniform_tiles), "s"(h.uniform_k), "s"(h.n_seg),
               "s"(h.flat_numel), "s"(a.ptab), "s"(a.n_rep), "s"(a.lr), "s"(a.mu), "s"(a.wd),
               "s"(a.nesterov), "s"(a.n_units), "s"(a.seg_numel), "s"(a.seg_tile0));
  for (uint32_t w = blockIdx.x; w < h.work; w += gridDim.x) {
    int unit;
    int64_t tile;
    if (h.uniform_tiles) {  // every unit has the same tile count
      unit = (int)(w / h.uniform_tiles);
      tile = (int64_t)(w - (uint32_t)unit * h.uniform_tiles);
    } else {
      unit = last_le(kargs().unit_work0, a.n_units, w);
      tile = (int64_t)(w - cld(kargs().unit_work0, unit));
    }
    // With equal-sized units the member window's address needs no load, so
    // it is fetched together with the unit's info word: the unit costs one
    // scalar round trip, its members' pointers a second.
    const uint32_t info = cld(kargs().unit_info, unit);
    Unit u;
    if (h.uniform_k) {
      u.k = (int)h.uniform_k;
      u.base = unit * u.k;
    } else {
      u.k = (int)unit_info_k(info);
      u.base = (int)unit_info_base(info);
    }
    u.act8 = unit_info_act8(info);
    u.ids = cld8x8(kargs().member, u.base);
    switch (u.k) {
      case 1: unit_tile<1, BF16, MOM, EXT>(a, h, u, tile); break;
      case 2: unit_tile<2, BF16, MOM, EXT>(a, h, u, tile); break;
      case 3: unit_tile<3, BF16, MOM, EXT>(a, h, u, tile); break;
      case 4: unit_tile<4, BF16, MOM, EXT>(a, h, u, tile); break;
      case 5: unit_tile<5, BF16, MOM, EXT>(a, h, u, tile); break;
      case 6: unit_tile<6, BF16, MOM, EXT>(a, h, u, tile); break;
      case 7: unit_tile<7, BF16, MOM, EXT>(a, h, u, tile); break;
      case 8: unit_tile<8, BF16, MOM, EXT>(a, h, u, tile); break;
      default: unit_tile<0, BF16, MOM, EXT>(a, h, u, tile); break;
    }
  }
}

}  // namespace

namespace {
template <bool BF16, bool MOM>
const void* kernel_for(bool ext) {
  return ext ? reinterpret_cast<const void*>(&fused_step_kernel<BF16, MOM, true>)
             : reinterpret_cast<const void*>(&fused_step_kernel<BF16, MOM, false>);
}
}  // namespace

hipError_t launch_fused_step(const StepArgs& a, bool bf16, bool mom, bool ext, int blocks,
                             size_t lds_bytes, hipStream_t stream) {
  const void* fn = bf16 ? (mom ? kernel_for<true, true>(ext) : kernel_for<true, false>(ext))
                        : (mom ? kernel_for<false, true>(ext) : kernel_for<false, false>(ext));
  void* args[] = {const_cast<StepArgs*>(&a)};
  // hipLaunchKernel reports this launch's own status (not an earlier sticky error).
  // lds_bytes is a reservation only (the kernel uses no LDS): it caps how
  // many workgroups share a CU.
  return hipLaunchKernel(fn, dim3(blocks), dim3(kBlock), args, lds_bytes, stream);
}

}  // namespace rip
