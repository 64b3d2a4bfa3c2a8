// Weighted unpermute-combine: the gather half of MoECompute_Combine.
// For every token of every micro-batch in the step (Eq. 1 plus the residual
// of Section 2.1):
//   x[t] += sum_{r<k} w[t][r] * o[inv[q(t,r)]] + sum_{s<S} o[inv[q(t,k+s)]]
// One workgroup per token; each thread owns 8 consecutive elements per pass
// of 2048 and issues the loads of all k+S rows of a pass at once (the
// residual slice is read one pass ahead).  The sum is
// formed in fp32 in slot order (routed ascending, then shared) before the
// residual add, so each token's result is independent of the schedule.
#include "eb_internal.h"
#include "eb_numeric.h"

namespace eb {
namespace {

constexpr int kCombThreads = 256;

// 8 consecutive elements of an o row, as fp32.
template <typename TO>
struct Row8;
template <>
struct Row8<float> {
  float4 a, b;
  __device__ __forceinline__ void load(const float* p) {
    a = reinterpret_cast<const float4*>(p)[0];
    b = reinterpret_cast<const float4*>(p)[1];
  }
  __device__ __forceinline__ float at(int i) const {
    const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    return v[i];
  }
};
template <>
struct Row8<bf16_t> {
  uint4 u;
  __device__ __forceinline__ void load(const bf16_t* p) { u = *reinterpret_cast<const uint4*>(p); }
  // the row as a split-K down GEMM's sum would store it: bf16(p0 + p1),
  // the halves `stride` floats apart
  __device__ __forceinline__ void load_split(const float* p, long long stride) {
    const float4 a0 = reinterpret_cast<const float4*>(p)[0], a1 = reinterpret_cast<const float4*>(p)[1];
    const float4 b0 = reinterpret_cast<const float4*>(p + stride)[0];
    const float4 b1 = reinterpret_cast<const float4*>(p + stride)[1];
    u.x = (uint32_t)f32_to_bf16(a0.x + b0.x) | ((uint32_t)f32_to_bf16(a0.y + b0.y) << 16);
    u.y = (uint32_t)f32_to_bf16(a0.z + b0.z) | ((uint32_t)f32_to_bf16(a0.w + b0.w) << 16);
    u.z = (uint32_t)f32_to_bf16(a1.x + b1.x) | ((uint32_t)f32_to_bf16(a1.y + b1.y) << 16);
    u.w = (uint32_t)f32_to_bf16(a1.z + b1.z) | ((uint32_t)f32_to_bf16(a1.w + b1.w) << 16);
  }
  __device__ __forceinline__ float at(int i) const {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
    const uint32_t x = w[i >> 1];
    return __uint_as_float((i & 1) ? (x & 0xffff0000u) : (x << 16));
  }
};

// SPLIT (bf16 only): o is not stored; its rows are formed from the two fp32
// K halves of the down GEMM at part and part + stride, rounded as the
// split-K sum rounds them, so the result is the same bit for bit.
// NS: slots the kernel holds rows for (k + S <= NS); sized to the stack so
// that small k + S keeps few registers and many wavefronts per SIMD.
template <typename TO, class RTA, bool SPLIT, int NS>
__global__ __launch_bounds__(kCombThreads) void combine_kernel(RTA rta, const TO* __restrict__ o,
                                                               const int32_t* __restrict__ inv,
                                                               const float* __restrict__ part = nullptr,
                                                               long long stride = 0) {
  __shared__ int s_row[kMaxSlots];
  __shared__ float s_w[kMaxSlots];
  const RunTable& rt = rta.get();
  const int g = blockIdx.x;
  const int total = rt.tok_base[rt.n];
  if (g >= total) return;  // past the live tokens (grid sized for the largest step)
  const int rho = find_entry(rt.tok_base, rt.n, g);
  const int t = g - rt.tok_base[rho];
  const int k = rt.k, slots = rt.k + rt.S, H = rt.H;
  const int P = total * slots;  // grouped rows; inv is clamped into [0, P)
  if (threadIdx.x < slots) {
    s_row[threadIdx.x] = min(max(inv[(size_t)g * slots + threadIdx.x], 0), P - 1);
    s_w[threadIdx.x] = threadIdx.x < k ? in_global(rt.w[rho])[(size_t)t * k + threadIdx.x] : 1.f;
  }
  float* x = in_global(rt.x[rho]) + (size_t)t * H;
  // the residual slice of the first pass is read while inv is on its way,
  // that of each next pass during the current one
  float4 xn0 = make_float4(0.f, 0.f, 0.f, 0.f), xn1 = xn0;
  if (threadIdx.x * 8 < H) {
    xn0 = reinterpret_cast<float4*>(x + threadIdx.x * 8)[0];
    xn1 = reinterpret_cast<float4*>(x + threadIdx.x * 8)[1];
  }
  __syncthreads();
  for (int c = threadIdx.x * 8; c < H; c += kCombThreads * 8) {
    Row8<TO> v[NS];
#pragma unroll
    for (int r = 0; r < NS; ++r)
      if (r < slots) {
        if constexpr (SPLIT)
          v[r].load_split(part + (size_t)s_row[r] * H + c, stride);
        else
          v[r].load(o + (size_t)s_row[r] * H + c);
      }
    float4 x0 = xn0, x1 = xn1;
    if (c + kCombThreads * 8 < H) {
      xn0 = reinterpret_cast<float4*>(x + c + kCombThreads * 8)[0];
      xn1 = reinterpret_cast<float4*>(x + c + kCombThreads * 8)[1];
    }
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < NS; ++r) {
      if (r < k) {
        const float wr = s_w[r];
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = fmaf(wr, v[r].at(i), acc[i]);
      } else if (r < slots) {
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] += v[r].at(i);
      }
    }
    x0.x += acc[0]; x0.y += acc[1]; x0.z += acc[2]; x0.w += acc[3];
    x1.x += acc[4]; x1.y += acc[5]; x1.z += acc[6]; x1.w += acc[7];
    reinterpret_cast<float4*>(x + c)[0] = x0;
    reinterpret_cast<float4*>(x + c)[1] = x1;
  }
}

}  // namespace

namespace {

// Launch with the smallest slot capacity that holds k + S.
template <typename TO, class RTA, bool SPLIT>
void combine_launch(int slots, int grid_tokens, RTA a, const TO* o, const int32_t* inv, const float* part,
                    long long stride, hipStream_t s) {
  const dim3 grid(grid_tokens), block(kCombThreads);
  if (slots <= 2)
    hipLaunchKernelGGL((combine_kernel<TO, RTA, SPLIT, 2>), grid, block, 0, s, a, o, inv, part, stride);
  else if (slots <= 4)
    hipLaunchKernelGGL((combine_kernel<TO, RTA, SPLIT, 4>), grid, block, 0, s, a, o, inv, part, stride);
  else if (slots <= 8)
    hipLaunchKernelGGL((combine_kernel<TO, RTA, SPLIT, 8>), grid, block, 0, s, a, o, inv, part, stride);
  else
    hipLaunchKernelGGL((combine_kernel<TO, RTA, SPLIT, kMaxSlots>), grid, block, 0, s, a, o, inv, part, stride);
}

template <class RTA>
void combine_impl(RTA a, int slots, int grid_tokens, int dtype, const void* o, const int32_t* inv,
                  hipStream_t s) {
  prof_start(EB_K_COMBINE, s);
  if (grid_tokens > 0) {
    if (dtype == EB_DTYPE_BF16)
      combine_launch<bf16_t, RTA, false>(slots, grid_tokens, a, static_cast<const bf16_t*>(o), inv, nullptr, 0,
                                         s);
    else
      combine_launch<float, RTA, false>(slots, grid_tokens, a, static_cast<const float*>(o), inv, nullptr, 0, s);
  }
  prof_stop(EB_K_COMBINE, s);
}

}  // namespace

hipError_t launch_combine(const RunTable& rt, int dtype, const void* o, const int32_t* inv,
                          hipStream_t s) {
  combine_impl(ByValue<RunTable>{rt}, rt.k + rt.S, rt.tok_base[rt.n], dtype, o, inv, s);
  return hipGetLastError();
}

hipError_t launch_combine_dev(const RunTable* rt, int slots, int max_tokens, int dtype, const void* o,
                              const int32_t* inv, hipStream_t s) {
  combine_impl(InMemory<RunTable>{rt}, slots, max_tokens, dtype, o, inv, s);
  return hipGetLastError();
}

hipError_t launch_combine_split_dev(const RunTable* rt, int slots, int max_tokens, const float* part,
                                    long long stride, const int32_t* inv, hipStream_t s) {
  prof_start(EB_K_COMBINE, s);
  if (max_tokens > 0)
    combine_launch<bf16_t, InMemory<RunTable>, true>(slots, max_tokens, InMemory<RunTable>{rt}, nullptr, inv, part,
                                                     stride, s);
  prof_stop(EB_K_COMBINE, s);
  return hipGetLastError();
}

}  // namespace eb
