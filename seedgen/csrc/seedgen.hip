// GPU twin of the seedgen input generator (see seedgen/__init__.py for the
// definition).  Writes elements [start, start+count) of a keyed counter-based
// stream to device memory: h = SplitMix64-mix(key + GAMMA*(e+1)), an
// Irwin-Hall(4) integer from its four 16-bit lanes, times an fp32 scale;
// fp32 or bf16 (round to nearest even) storage.  Input generation only: it
// carries none of the P-Reduce arithmetic.

#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

__device__ __forceinline__ float value(uint64_t key, int64_t e, float scale) {
  const uint64_t h = mix64(key + 0x9E3779B97F4A7C15ULL * (uint64_t)(e + 1));
  const int32_t d = (int32_t)((h & 0xFFFF) + ((h >> 16) & 0xFFFF) + ((h >> 32) & 0xFFFF) +
                              (h >> 48)) - 131070;
  return (float)d * scale;
}

__device__ __forceinline__ uint16_t to_bf16(float f) {
  const uint32_t b = __float_as_uint(f);
  if ((b & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((b >> 16) | 0x40u);
  return (uint16_t)((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

__global__ __launch_bounds__(256) void fill_f32(float* dst, uint64_t key, int64_t start,
                                               int64_t count, float scale) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * 256)
    dst[i] = value(key, start + i, scale);
}

__global__ __launch_bounds__(256) void fill_bf16(uint16_t* dst, uint64_t key, int64_t start,
                                                int64_t count, float scale) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * 256)
    dst[i] = to_bf16(value(key, start + i, scale));
}

}  // namespace

// dtype 0 = fp32, 1 = bf16.  Returns 0, -1 on a bad argument, -5 on a HIP error.
extern "C" int32_t seedgen_fill_normal(void* dst, int32_t dtype, uint64_t key, int64_t start,
                                       int64_t count, float scale, void* stream) {
  if (count < 0 || start < 0 || (count > 0 && !dst) || (dtype != 0 && dtype != 1)) return -1;
  if (count == 0) return 0;
  int64_t blocks = (count + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const void* fn = dtype == 0 ? reinterpret_cast<const void*>(&fill_f32)
                              : reinterpret_cast<const void*>(&fill_bf16);
  void* args[] = {&dst, &key, &start, &count, &scale};
  return hipLaunchKernel(fn, dim3((unsigned)blocks), dim3(256), args, 0, s) == hipSuccess ? 0 : -5;
}
