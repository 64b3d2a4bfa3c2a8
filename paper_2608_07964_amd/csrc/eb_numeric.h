// Device numeric helpers of the library: bf16 <-> fp32 and typed row access.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace eb {

typedef uint16_t bf16_t;  // raw bfloat16 bit pattern

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}

// Round-to-nearest-even fp32 -> bf16; NaN stays a (quiet) NaN.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40u);
  return (bf16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ static __forceinline__ float round(float v) { return v; }
  __device__ static __forceinline__ float load(const float* p, size_t i) { return p[i]; }
  __device__ static __forceinline__ void store(float* p, size_t i, float v) { p[i] = v; }
};
template <> struct Elem<bf16_t> {
  // the value that storing v and loading it back gives
  __device__ static __forceinline__ float round(float v) { return bf16_to_f32(f32_to_bf16(v)); }
  __device__ static __forceinline__ float load(const bf16_t* p, size_t i) { return bf16_to_f32(p[i]); }
  __device__ static __forceinline__ void store(bf16_t* p, size_t i, float v) { p[i] = f32_to_bf16(v); }
};

// SiLU(g) * u in fp32: g / (1 + e^-g) * u with the hardware base-2
// exponential (e^-g = 2^(-g log2 e)) and reciprocal, each within about one
// ulp, far below the bf16 rounding of the result.
__device__ __forceinline__ float swiglu(float g, float u) {
  const float e = __builtin_amdgcn_exp2f(-g * 1.44269504088896341f);
  return g * __builtin_amdgcn_rcpf(1.0f + e) * u;
}

}  // namespace eb
