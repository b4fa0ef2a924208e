// Practical HBM stream ceilings on this GPU, for the roofline of the fused
// step kernel (a measurement program beside bench.py: `bench.py --ceiling`
// builds and runs it; not part of the library).  Each kernel is a bare stream with the fused step's access
// shape and launch style (single-wave workgroups, one 1 KB-per-stream tile
// each, non-temporal 16-byte accesses, resident waves per CU capped with a
// dynamic LDS reservation):
//
//   read     one stream read (4 vectors per lane, so loads stay in flight)
//   copy     one stream read, one written
//   2R1W     w <- w - lr * g on one replica (the lone local update)
//   group4   four replicas averaged after their update (8 reads, 4 writes),
//            the shape of a P-Reduce group of four
//   group8m  eight replicas with momentum averaged after their update
//            (24 reads, 16 writes), the shape of a group of eight with
//            momentum
//
// group4 and group8m use the fused kernel's own access form for full tiles
// (buffer instructions, a descriptor per stream and tile); group4-global is
// the same shape through global instructions, and read, copy and 2R1W use
// global instructions too.
//
// Every stream is 1 GiB.  The buffers are measured twice: filled with
// random values (as the workloads are) and zero-filled, because the
// sustained bandwidth depends on the data moved.  Standalone program; prints
// one line per (data, waves/CU) with GB/s counted as bytes the stream moves
// divided by kernel time (5 back-to-back launches after one warm-up).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
#define GLOBAL __attribute__((address_space(1)))

__device__ __forceinline__ f32x4 load_nt(const char* p) {
  return __builtin_nontemporal_load((const GLOBAL f32x4*)p);
}
__device__ __forceinline__ void store_nt(char* p, f32x4 v) {
  __builtin_nontemporal_store(v, (GLOBAL f32x4*)p);
}

constexpr int kLanes = 64;
constexpr int kStreams = 24;

struct Streams {
  char* p[kStreams];
  uint32_t tiles;  // workgroups; each covers kLanes x 16 bytes of every stream it touches
  float lr;
};

enum Kind { kRead = 0, kCopy = 1, k2R1W = 2, kGroup4 = 3, kGroup8Mom = 4, kGroup4Buf = 5,
            kGroup8MomBuf = 6 };

// The buffer form of the fused kernel's full tiles: a descriptor per stream
// whose base is the tile's first byte and whose size is the tile, lanes
// addressing it with a small offset; non-temporal.
typedef __amdgpu_buffer_rsrc_t Rsrc;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ Rsrc tile_rsrc(char* base, uint32_t t) {
  return __builtin_amdgcn_make_buffer_rsrc(base + (int64_t)t * kLanes * 16, 0, kLanes * 16,
                                           0x00020000);
}
__device__ __forceinline__ f32x4 bload(Rsrc r) {
  return __builtin_bit_cast(
      f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)threadIdx.x * 16, 0, 2));
}
__device__ __forceinline__ void bstore(Rsrc r, f32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, (int)threadIdx.x * 16,
                                         0, 2);
}

template <int KIND>
__global__ __launch_bounds__(kLanes) void stream_kernel(Streams s) {
  const uint32_t grid = KIND == kRead ? s.tiles / 4 : s.tiles;
  const uint32_t t = blockIdx.x;
  if (t >= grid) return;
  if constexpr (KIND == kRead) {
    // 4 tiles per workgroup so each lane keeps 4 loads in flight
    f32x4 acc = {0, 0, 0, 0};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t off = (((int64_t)t * 4 + u) * kLanes + threadIdx.x) * 16;
      acc += load_nt(s.p[0] + off);
    }
    // never true for the fills used here; keeps the loads live
    if (acc.x == 1234.5f && acc.y == -1234.5f) store_nt(s.p[1] + threadIdx.x * 16, acc);
  } else if constexpr (KIND == kGroup4Buf) {
    Rsrc r[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) r[j] = tile_rsrc(s.p[j], t);
    f32x4 w[4], g[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      w[j] = bload(r[j]);
      g[j] = bload(r[4 + j]);
    }
    f32x4 sum = w[0] - s.lr * g[0];
#pragma unroll
    for (int j = 1; j < 4; ++j) sum = sum + (w[j] - s.lr * g[j]);
    sum = sum * 0.25f;
#pragma unroll
    for (int j = 0; j < 4; ++j) bstore(r[j], sum);
  } else if constexpr (KIND == kGroup8MomBuf) {
    Rsrc r[24];
#pragma unroll
    for (int j = 0; j < 24; ++j) r[j] = tile_rsrc(s.p[j], t);
    f32x4 w[8], g[8], v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      w[j] = bload(r[j]);
      g[j] = bload(r[8 + j]);
      v[j] = bload(r[16 + j]);
    }
    f32x4 sum = {0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      v[j] = 0.9f * v[j] + g[j];
      sum = sum + (w[j] - s.lr * v[j]);
    }
    sum = sum * 0.125f;
#pragma unroll
    for (int j = 0; j < 8; ++j) bstore(r[16 + j], v[j]);
#pragma unroll
    for (int j = 0; j < 8; ++j) bstore(r[j], sum);
  } else {
    const int64_t off = ((int64_t)t * kLanes + threadIdx.x) * 16;
    if constexpr (KIND == kCopy) {
      store_nt(s.p[1] + off, load_nt(s.p[0] + off));
    } else if constexpr (KIND == k2R1W) {
      const f32x4 w = load_nt(s.p[0] + off), g = load_nt(s.p[1] + off);
      store_nt(s.p[0] + off, w - s.lr * g);
    } else if constexpr (KIND == kGroup8Mom) {
      f32x4 w[8], g[8], v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        w[j] = load_nt(s.p[j] + off);
        g[j] = load_nt(s.p[8 + j] + off);
        v[j] = load_nt(s.p[16 + j] + off);
      }
      f32x4 sum = {0, 0, 0, 0};
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        v[j] = 0.9f * v[j] + g[j];
        store_nt(s.p[16 + j] + off, v[j]);
        sum = sum + (w[j] - s.lr * v[j]);
      }
      sum = sum * 0.125f;
#pragma unroll
      for (int j = 0; j < 8; ++j) store_nt(s.p[j] + off, sum);
    } else {
      f32x4 w[4], g[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        w[j] = load_nt(s.p[j] + off);
        g[j] = load_nt(s.p[4 + j] + off);
      }
      f32x4 sum = w[0] - s.lr * g[0];
#pragma unroll
      for (int j = 1; j < 4; ++j) sum = sum + (w[j] - s.lr * g[j]);
      sum = sum * 0.25f;
#pragma unroll
      for (int j = 0; j < 4; ++j) store_nt(s.p[j] + off, sum);
    }
  }
}

// Uniform values in [-scale, scale) from a SplitMix64-style hash of the index.
__global__ void fill_random(float* p, int64_t n, uint64_t seed, float scale) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    uint64_t z = seed + 0x9E3779B97F4A7C15ull * (uint64_t)(i + 1);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    p[i] = scale * ((float)(int32_t)(uint32_t)z * (1.0f / 2147483648.0f));
  }
}

#define CHECK(x)                                                                        \
  do {                                                                                  \
    hipError_t e_ = (x);                                                                \
    if (e_ != hipSuccess) {                                                             \
      std::fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); \
      return -1.0;                                                                      \
    }                                                                                   \
  } while (0)

template <int KIND>
double time_ms(const Streams& s, size_t lds_bytes) {
  const uint32_t grid = KIND == kRead ? s.tiles / 4 : s.tiles;
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  hipLaunchKernelGGL(stream_kernel<KIND>, dim3(grid), dim3(kLanes), lds_bytes, 0, s);
  CHECK(hipGetLastError());
  CHECK(hipDeviceSynchronize());
  CHECK(hipEventRecord(e0));
  for (int i = 0; i < 5; ++i)
    hipLaunchKernelGGL(stream_kernel<KIND>, dim3(grid), dim3(kLanes), lds_bytes, 0, s);
  CHECK(hipEventRecord(e1));
  CHECK(hipEventSynchronize(e1));
  float ms = 0;
  CHECK(hipEventElapsedTime(&ms, e0, e1));
  CHECK(hipEventDestroy(e0));
  CHECK(hipEventDestroy(e1));
  return ms / 5.0;
}

}  // namespace

int main() {
  const int64_t bytes = 1ll << 30;  // per stream
  Streams s{};
  for (int j = 0; j < kStreams; ++j)
    if (hipMalloc(&s.p[j], bytes) != hipSuccess) {
      std::fprintf(stderr, "hipMalloc of stream %d failed\n", j);
      return 1;
    }
  s.tiles = (uint32_t)(bytes / (kLanes * 16));  // 1 GiB / 1 KB; a multiple of 4
  s.lr = 0.1f;
  int lds_per_cu = 0, cus = 0;
  if (hipDeviceGetAttribute(&lds_per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, 0) ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0))
    return 1;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, 0) != hipSuccess) return 1;
  std::printf("stream ceilings on %s, %d CUs, 1 GiB per stream, non-temporal 16-byte accesses\n",
              prop.gcnArchName, cus);
  const double gb = (double)bytes / 1e9;
  for (int random = 1; random >= 0; --random) {
    for (int j = 0; j < kStreams; ++j) {
      if (random) {
        // p[0..3] ~U[-1,1) and every other stream ~U[-0.01,0.01): random
        // mantissas and signs everywhere (group4 reads weights p[0..3] and
        // gradients p[4..7]; group8m weights p[0..7], gradients p[8..15],
        // momenta p[16..23])
        hipLaunchKernelGGL(fill_random, dim3(8192), dim3(256), 0, 0, reinterpret_cast<float*>(s.p[j]),
                           bytes / 4, (uint64_t)(1000 + j), j < 4 ? 1.0f : 0.01f);
      } else if (hipMemset(s.p[j], 0, bytes) != hipSuccess) {
        return 1;
      }
    }
    if (hipDeviceSynchronize() != hipSuccess) return 1;
    for (int waves : {4, 5, 6, 8, 10, 12, 16, 0}) {
      const size_t lds = waves ? ((size_t)(lds_per_cu / waves) & ~(size_t)255) : 0;
      const double t_read = time_ms<kRead>(s, lds), t_copy = time_ms<kCopy>(s, lds);
      const double t_2r1w = time_ms<k2R1W>(s, lds), t_g4 = time_ms<kGroup4>(s, lds);
      const double t_g4b = time_ms<kGroup4Buf>(s, lds);
      const double t_g8m = time_ms<kGroup8MomBuf>(s, lds);
      if (t_read < 0 || t_copy < 0 || t_2r1w < 0 || t_g4 < 0 || t_g4b < 0 || t_g8m < 0) return 1;
      char cap[16];
      std::snprintf(cap, sizeof cap, "%d", waves);
      std::printf("data=%-6s waves/CU=%-4s read %7.1f  copy %7.1f  2R1W %7.1f  group4-global %7.1f  "
                  "group4 %7.1f  group8m %7.1f GB/s\n",
                  random ? "random" : "zero", waves ? cap : "max", gb / t_read * 1e3,
                  2 * gb / t_copy * 1e3, 3 * gb / t_2r1w * 1e3, 12 * gb / t_g4 * 1e3,
                  12 * gb / t_g4b * 1e3, 40 * gb / t_g8m * 1e3);
      std::fflush(stdout);
    }
  }
  for (int j = 0; j < kStreams; ++j) (void)hipFree(s.p[j]);
  return 0;
}
