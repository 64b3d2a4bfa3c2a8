// Device side of the seeded input generator.  Produces exactly the bits that
// synth/gen.py produces on the host (same counter-based SplitMix64 stream,
// same quantile table, one fp32 multiply, integer round-to-nearest-even to
// bf16).  This library holds input generation only, none of the method.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z ^= z >> 30;
  z *= 0xBF58476D1CE4E5B9ull;
  z ^= z >> 27;
  z *= 0x94D049BB133111EBull;
  z ^= z >> 31;
  return z;
}

__global__ void fill_normal_kernel(void* __restrict__ out, int64_t n, int as_bf16,
                                   uint64_t key, uint64_t i0,
                                   const float* __restrict__ table, float sigma) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const uint64_t u = mix64(key + (i0 + (uint64_t)i + 1ull) * kGamma);
    const float v = __fmul_rn(table[u >> 48], sigma);
    if (as_bf16) {
      const uint32_t b = __float_as_uint(v);
      const uint32_t r = (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
      static_cast<uint16_t*>(out)[i] = (uint16_t)r;
    } else {
      static_cast<float*>(out)[i] = v;
    }
  }
}

}  // namespace

extern "C" {

// Fill out[0..n) with elements i0 .. i0+n-1 of the normal stream `key`.
// dtype 0: fp32 output, 1: bf16 output (stored as uint16 bit patterns).
// table: device pointer to the 65536-entry fp32 quantile table.
// Returns 0 on success or the hipError_t of the launch.
int synth_fill_normal(void* out, int64_t n, int dtype, uint64_t key, uint64_t i0,
                      const float* table, float sigma, void* stream) {
  if (n <= 0) return 0;
  if (out == nullptr || table == nullptr || (dtype != 0 && dtype != 1)) return (int)hipErrorInvalidValue;
  const int block = 256;
  int64_t blocks = (n + block - 1) / block;
  if (blocks > 1 << 16) blocks = 1 << 16;
  hipLaunchKernelGGL(fill_normal_kernel, dim3((unsigned)blocks), dim3(block), 0,
                     (hipStream_t)stream, out, n, dtype, key, i0, table, sigma);
  return (int)hipGetLastError();
}

}  // extern "C"
