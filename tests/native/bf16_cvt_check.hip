// Test helper (not part of librip): checks the fp32 -> bf16 conversion that
// the fused kernel uses to store bf16 results -- gfx950's v_cvt_pk_bf16_f32,
// which clang emits for __builtin_convertvector of two floats to two __bf16 --
// against the definition of round-to-nearest-even on the bit patterns, for
// every one of the 2^32 fp32 inputs.
//
// Definition (per 32-bit pattern b): if b is a NaN, the bf16 is its top half
// with the quiet bit (0x0040) set; otherwise (b + 0x7FFF + ((b >> 16) & 1))
// >> 16, which rounds the dropped 16 bits to nearest with ties to the even
// result, carrying into the exponent (and up to infinity) as needed.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t rne_definition(uint32_t b) {
  if ((b & 0x7FFFFFFFu) > 0x7F800000u) return (b >> 16) | 0x0040u;
  return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ uint32_t convert_pair(uint32_t b0, uint32_t b1) {
  const f32x2 f = {__uint_as_float(b0), __uint_as_float(b1)};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

constexpr int kThreads = 256;
constexpr int kPairsPerThread = 64;
constexpr uint32_t kBlocks = (1u << 31) / (kThreads * kPairsPerThread);  // 131072
constexpr int kKeep = 16;

// Thread t handles pairs p = t*64 + i (i < 64) of inputs (2p, 2p + 1); the
// grid's 2^25 threads cover p < 2^31, so every 32-bit pattern once.
__global__ __launch_bounds__(kThreads) void check_all(unsigned long long* mismatches,
                                                       uint32_t* first, uint32_t* n_first) {
  const uint64_t t = (uint64_t)blockIdx.x * kThreads + threadIdx.x;
  for (int i = 0; i < kPairsPerThread; ++i) {
    const uint32_t p = (uint32_t)(t * kPairsPerThread + i);
    const uint32_t b0 = 2u * p, b1 = 2u * p + 1u;
    const uint32_t got = convert_pair(b0, b1);
    const uint32_t want = rne_definition(b0) | (rne_definition(b1) << 16);
    if (got != want) {
      const uint32_t bad = (got & 0xFFFFu) != (want & 0xFFFFu) ? b0 : b1;
      atomicAdd(mismatches, 1ull);
      const uint32_t slot = atomicAdd(n_first, 1u);
      if (slot < (uint32_t)kKeep) first[slot] = bad;
    }
  }
}

__global__ void convert_array(const uint32_t* in, uint16_t* out, uint64_t n) {
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (2 * i + 1 < n) {
    const uint32_t v = convert_pair(in[2 * i], in[2 * i + 1]);
    out[2 * i] = (uint16_t)(v & 0xFFFFu);
    out[2 * i + 1] = (uint16_t)(v >> 16);
  } else if (2 * i < n) {
    out[2 * i] = (uint16_t)(convert_pair(in[2 * i], 0u) & 0xFFFFu);
  }
}

}  // namespace

// Pairs counted as mismatching (a pair with both halves wrong counts once)
// go to *mismatches; the first (up to 16) offending inputs to first[].
// Returns a hipError_t value (0 = success).
extern "C" int bf16_cvt_check_all(unsigned long long* mismatches, uint32_t* first) {
  struct Dev {
    unsigned long long count;
    uint32_t n_first;
    uint32_t first[kKeep];
  };
  Dev* d = nullptr;
  hipError_t e = hipMalloc(&d, sizeof(Dev));
  if (e != hipSuccess) return (int)e;
  e = hipMemset(d, 0, sizeof(Dev));
  if (e == hipSuccess) {
    hipLaunchKernelGGL(check_all, dim3(kBlocks), dim3(kThreads), 0, 0, &d->count, d->first,
                       &d->n_first);
    e = hipGetLastError();
  }
  Dev h{};
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipMemcpy(&h, d, sizeof(Dev), hipMemcpyDeviceToHost);
  (void)hipFree(d);
  if (e != hipSuccess) return (int)e;
  *mismatches = h.count;
  for (int i = 0; i < kKeep; ++i) first[i] = h.first[i];
  return 0;
}

// Converts n fp32 bit patterns (host array) on the GPU; host output.
extern "C" int bf16_cvt_apply(const uint32_t* in, uint16_t* out, uint64_t n) {
  if (n == 0) return 0;
  uint32_t* din = nullptr;
  uint16_t* dout = nullptr;
  hipError_t e = hipMalloc(&din, n * 4);
  if (e == hipSuccess) e = hipMalloc(&dout, n * 2);
  if (e == hipSuccess) e = hipMemcpy(din, in, n * 4, hipMemcpyHostToDevice);
  if (e == hipSuccess) {
    const uint64_t pairs = (n + 1) / 2;
    hipLaunchKernelGGL(convert_array, dim3((unsigned)((pairs + 255) / 256)), dim3(256), 0, 0, din,
                       dout, n);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipMemcpy(out, dout, n * 2, hipMemcpyDeviceToHost);
  (void)hipFree(din);
  (void)hipFree(dout);
  return (int)e;
}
