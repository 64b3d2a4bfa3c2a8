// Weighted unpermute-combine: the gather half of MoECompute_Combine.
// For every token of every micro-batch in the step (Eq. 1 plus the residual
// of Section 2.1):
//   x[t] += sum_{r<k} w[t][r] * o[inv[q(t,r)]] + sum_{s<S} o[inv[q(t,k+s)]]
// One wavefront per token, 4 consecutive elements per lane per pass, the sum
// formed in fp32 in slot order (routed ascending, then shared) before the
// residual add, so each token's result is independent of the schedule.
#include "eb_internal.h"
#include "eb_numeric.h"

namespace eb {
namespace {

template <typename TO>
struct Load4;
template <>
struct Load4<float> {
  __device__ static __forceinline__ float4 at(const float* p) {
    return *reinterpret_cast<const float4*>(p);
  }
};
template <>
struct Load4<bf16_t> {
  __device__ static __forceinline__ float4 at(const bf16_t* p) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                       __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
  }
};

template <typename TO>
__global__ __launch_bounds__(256) void combine_kernel(RunTable rt, int total, const TO* __restrict__ o,
                                                      const int32_t* __restrict__ inv) {
  const int lane = threadIdx.x & 63;
  const int g = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (g >= total) return;
  const int rho = find_entry(rt.tok_base, rt.n, g);
  const int t = g - rt.tok_base[rho];
  const int k = rt.k, slots = rt.k + rt.S, H = rt.H;
  const size_t q0 = (size_t)g * slots;
  const int P = total * slots;  // grouped rows; inv is clamped into [0, P)
  float* x = rt.x[rho] + (size_t)t * H;
  const float* w = rt.w[rho] + (size_t)t * k;
  for (int c = lane * 4; c < H; c += 256) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int r = 0; r < k; ++r) {
      const float wr = w[r];
      const float4 v = Load4<TO>::at(o + (size_t)min(max(inv[q0 + r], 0), P - 1) * H + c);
      acc.x = fmaf(wr, v.x, acc.x);
      acc.y = fmaf(wr, v.y, acc.y);
      acc.z = fmaf(wr, v.z, acc.z);
      acc.w = fmaf(wr, v.w, acc.w);
    }
    for (int r = k; r < slots; ++r) {
      const float4 v = Load4<TO>::at(o + (size_t)min(max(inv[q0 + r], 0), P - 1) * H + c);
      acc.x += v.x;
      acc.y += v.y;
      acc.z += v.z;
      acc.w += v.w;
    }
    float4 xv = *reinterpret_cast<float4*>(x + c);
    xv.x += acc.x;
    xv.y += acc.y;
    xv.z += acc.z;
    xv.w += acc.w;
    *reinterpret_cast<float4*>(x + c) = xv;
  }
}

}  // namespace

hipError_t launch_combine(const RunTable& rt, int total_tokens, int dtype, const void* o,
                          const int32_t* inv, hipStream_t s) {
  prof_start(EB_K_COMBINE, s);
  if (dtype == EB_DTYPE_BF16)
    hipLaunchKernelGGL(combine_kernel<bf16_t>, dim3((total_tokens + 3) / 4), dim3(256), 0, s, rt,
                       total_tokens, static_cast<const bf16_t*>(o), inv);
  else
    hipLaunchKernelGGL(combine_kernel<float>, dim3((total_tokens + 3) / 4), dim3(256), 0, s, rt,
                       total_tokens, static_cast<const float*>(o), inv);
  prof_stop(EB_K_COMBINE, s);
  return hipGetLastError();
}

}  // namespace eb
