// Routing of one micro-batch at one layer (Section 2.1: W, I = topk(G(h'))):
//   norm_router_kernel  E <= 8 (bf16) / E <= 64 (fp32): one wavefront per token computes
//                       a = dtype(x * r * gain) and z = a Wg^T + bias in one pass
//                       (Wg stays in L2; lane partial sums, butterfly reductions)
//   rmsnorm_kernel +    bf16 stacks with E > 8: RMSNorm, then the router GEMM on
//   router_mfma_kernel  the matrix cores (split-K over the 4 wavefronts)
//   rmsnorm_kernel +    fp32 stacks with E > 64: RMSNorm, then an LDS-tiled fp32
//   logits_kernel       VALU GEMM for z
//   topk_kernel         top-k by wavefront argmax, softmax weights, expert counts
#include <math.h>

#include "eb_internal.h"
#include "eb_numeric.h"

namespace eb {
namespace {

// ---------------------------------------------------------------------------
// RMSNorm + cast.  Each lane sums its strided float4 slices in a fixed order;
// the butterfly reduction leaves the bit-identical total in every lane.
template <typename TA>
__global__ __launch_bounds__(256) void rmsnorm_kernel(int T, int H, const float* __restrict__ x,
                                                      const float* __restrict__ gain,
                                                      TA* __restrict__ a, float eps) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const float4* xr = reinterpret_cast<const float4*>(x + (size_t)t * H);
  const float4* g4 = reinterpret_cast<const float4*>(gain);
  const int n4 = H >> 2;
  float ss = 0.f;
  for (int i = lane; i < n4; i += 64) {
    const float4 v = xr[i];
    ss = fmaf(v.x, v.x, ss);
    ss = fmaf(v.y, v.y, ss);
    ss = fmaf(v.z, v.z, ss);
    ss = fmaf(v.w, v.w, ss);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
  const float r = 1.0f / sqrtf(ss / (float)H + eps);
  TA* ar = a + (size_t)t * H;
  for (int i = lane; i < n4; i += 64) {
    const float4 v = xr[i];
    const float4 g = g4[i];
    Elem<TA>::store(ar, 4 * i + 0, v.x * r * g.x);
    Elem<TA>::store(ar, 4 * i + 1, v.y * r * g.y);
    Elem<TA>::store(ar, 4 * i + 2, v.z * r * g.z);
    Elem<TA>::store(ar, 4 * i + 3, v.w * r * g.w);
  }
}

// ---------------------------------------------------------------------------
// Router logits z[T][E] = a Wg^T + bias.  Tile 32 tokens x 64 experts, K step
// 32, 256 threads with 2 x 4 outputs each; every output accumulates over h in
// ascending order.
constexpr int LG_BT = 32, LG_BE = 64, LG_BK = 32;

template <typename TA>
__global__ __launch_bounds__(256) void logits_kernel(int T, int H, int E, const TA* __restrict__ a,
                                                     const TA* __restrict__ Wg,
                                                     const float* __restrict__ bias,
                                                     float* __restrict__ z) {
  __shared__ float As[LG_BK][LG_BT + 1];
  __shared__ float Bs[LG_BK][LG_BE + 1];
  const int tid = threadIdx.x;
  const int ty = tid >> 4, tx = tid & 15;
  const int t0 = blockIdx.x * LG_BT, e0 = blockIdx.y * LG_BE;
  float acc[2][4] = {};
  for (int k0 = 0; k0 < H; k0 += LG_BK) {
    {  // A tile: 32 rows x 32 k, 4 elements per thread
      const int row = tid >> 3, kk = (tid & 7) * 4;
      const int t = min(t0 + row, T - 1);
#pragma unroll
      for (int i = 0; i < 4; ++i) As[kk + i][row] = Elem<TA>::load(a, (size_t)t * H + k0 + kk + i);
    }
    {  // B tile: 64 experts x 32 k, 8 elements per thread
      const int er = tid >> 2, kk = (tid & 3) * 8;
      const int e = e0 + er;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        Bs[kk + i][er] = e < E ? Elem<TA>::load(Wg, (size_t)e * H + k0 + kk + i) : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < LG_BK; ++kk) {
      const float a0 = As[kk][ty], a1 = As[kk][ty + 16];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float b = Bs[kk][tx + 16 * j];
        acc[0][j] = fmaf(a0, b, acc[0][j]);
        acc[1][j] = fmaf(a1, b, acc[1][j]);
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int t = t0 + ty + 16 * i;
    if (t >= T) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = e0 + tx + 16 * j;
      if (e < E) z[(size_t)t * E + e] = acc[i][j] + bias[e];
    }
  }
}

// ---------------------------------------------------------------------------
// Fused RMSNorm + router logits for E <= EMAX.  Lane l owns the 8-element
// chunks starting at h = 8 (l + 64 i); per chunk it forms the stored a values and adds
// their products with every router row into one accumulator per expert; each
// expert's lane partial sums are then reduced by a butterfly (bit-identical
// total in every lane) and lane e writes z[t][e].
template <typename TA, int EMAX>
__global__ __launch_bounds__(256) void norm_router_kernel(int T, int H, int E, const float* __restrict__ x,
                                                          const float* __restrict__ gain,
                                                          const TA* __restrict__ Wg,
                                                          const float* __restrict__ bias,
                                                          TA* __restrict__ a, float* __restrict__ z,
                                                          float eps) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const float* xr = x + (size_t)t * H;
  const int nchunk = H >> 3;  // 8-element chunks; lane l takes chunks l, l + 64, ...
  float ss = 0.f;
  for (int c = lane; c < nchunk; c += 64) {
    const float4* p4 = reinterpret_cast<const float4*>(xr + 8 * c);
    const float4 u = p4[0], v = p4[1];
    ss = fmaf(u.x, u.x, ss); ss = fmaf(u.y, u.y, ss); ss = fmaf(u.z, u.z, ss); ss = fmaf(u.w, u.w, ss);
    ss = fmaf(v.x, v.x, ss); ss = fmaf(v.y, v.y, ss); ss = fmaf(v.z, v.z, ss); ss = fmaf(v.w, v.w, ss);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
  const float r = 1.0f / sqrtf(ss / (float)H + eps);
  float acc[EMAX];
#pragma unroll
  for (int e = 0; e < EMAX; ++e) acc[e] = 0.f;
  TA* ar = a + (size_t)t * H;
  for (int c = lane; c < nchunk; c += 64) {
    const int h = 8 * c;
    const float4* p4 = reinterpret_cast<const float4*>(xr + h);
    const float4* g4 = reinterpret_cast<const float4*>(gain + h);
    const float4 u = p4[0], v = p4[1], gu = g4[0], gv = g4[1];
    float av[8] = {u.x * r * gu.x, u.y * r * gu.y, u.z * r * gu.z, u.w * r * gu.w,
                   v.x * r * gv.x, v.y * r * gv.y, v.z * r * gv.z, v.w * r * gv.w};
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      Elem<TA>::store(ar, h + q, av[q]);
      av[q] = Elem<TA>::round(av[q]);  // the stored (rounded) value feeds the router
    }
#pragma unroll
    for (int e = 0; e < EMAX; ++e) {
      if (e < E) {
        const TA* wr = Wg + (size_t)e * H + h;
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[e] = fmaf(av[q], Elem<TA>::load(wr, q), acc[e]);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < EMAX; ++e) {
    if (e < E) {
      float v = acc[e];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
      if (lane == e) z[(size_t)t * E + e] = v + bias[e];
    }
  }
}

// ---------------------------------------------------------------------------
// Router logits on the matrix cores (bf16 stacks, 8 < E <= 256):
// z[T][E] = a Wg^T + bias.  A workgroup takes 32 tokens and all experts
// (padded to NB blocks of 32); its 4 wavefronts split K into quarters, each
// accumulating a 32 x 32 NB partial with v_mfma_f32_32x32x16_bf16 from
// operands loaded straight from L2 into registers (one 32-wide K chunk
// prefetched).  Waves 1..3 leave their partials in LDS and wave 0 adds them in
// that order, then adds the bias: a fixed summation order, so the logits of a
// micro-batch do not depend on anything but its inputs.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx16_t __attribute__((ext_vector_type(16)));

template <int NB>
__global__ __launch_bounds__(256) void router_mfma_kernel(int T, int H, int E,
                                                          const bf16_t* __restrict__ a,
                                                          const bf16_t* __restrict__ Wg,
                                                          const float* __restrict__ bias,
                                                          float* __restrict__ z) {
  __shared__ float part[3][NB][16][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lrow = lane & 31, khalf = lane >> 5;
  const int t0 = blockIdx.x * 32;
  const int kq = H / 4, kbeg = wave * kq;
  // this lane's A row (token) and B rows (experts), clamped into range
  const bf16_t* arow = a + (size_t)min(t0 + lrow, T - 1) * H + kbeg + 8 * khalf;
  const bf16_t* brow[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
    brow[nb] = Wg + (size_t)min(nb * 32 + lrow, E - 1) * H + kbeg + 8 * khalf;
  floatx16_t acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[nb][v] = 0.f;
  // a 32-wide K chunk = two MFMA k-steps of 16
  bf16x8_t ac[2][2], bc[2][NB][2];
  auto load = [&](int buf, int k) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      ac[buf][s] = *reinterpret_cast<const bf16x8_t*>(arow + k + 16 * s);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        bc[buf][nb][s] = *reinterpret_cast<const bf16x8_t*>(brow[nb] + k + 16 * s);
    }
  };
  auto mma = [&](int buf) {
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ac[buf][s], bc[buf][nb][s], acc[nb], 0, 0, 0);
  };
  load(0, 0);
  for (int k = 0; k < kq; k += 64) {
    if (k + 32 < kq) load(1, k + 32);
    mma(0);
    if (k + 64 < kq) load(0, k + 64);
    if (k + 32 < kq) mma(1);
  }
  if (wave > 0) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int v = 0; v < 16; ++v) part[wave - 1][nb][v][lane] = acc[nb][v];
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      float sum = acc[nb][v];
#pragma unroll
      for (int w = 0; w < 3; ++w) sum += part[w][nb][v][lane];
      // C[row][col]: col = lane % 32 of block nb (expert), row = 8 (v/4) + 4 (lane/32) + v%4 (token)
      const int t = t0 + 8 * (v >> 2) + 4 * khalf + (v & 3);
      const int e = nb * 32 + lrow;
      if (t < T && e < E) z[(size_t)t * E + e] = sum + bias[e];
    }
  }
}

// ---------------------------------------------------------------------------
// Top-k, softmax weights and expert counts.  One wavefront per token; lane l
// holds logits e = l + 64 s.  Each pick is a wavefront argmax under the total
// order (larger z first, then lower expert id), so every lane agrees.
constexpr int TK_MAX_PER_LANE = 16;  // E <= 1024

__device__ __forceinline__ bool better(float v1, int e1, float v2, int e2) {
  return v1 > v2 || (v1 == v2 && e1 < e2);
}

__global__ __launch_bounds__(256) void topk_kernel(int T, int E, int k, int norm_topk,
                                                   const float* __restrict__ z,
                                                   int32_t* __restrict__ idx,
                                                   float* __restrict__ w,
                                                   int32_t* __restrict__ counts) {
  __shared__ int hist[1024];
  for (int e = threadIdx.x; e < E; e += blockDim.x) hist[e] = 0;
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t < T) {
    const int per = (E + 63) >> 6;
    float v[TK_MAX_PER_LANE];
    uint32_t taken = 0;
    float mx = -INFINITY;
#pragma unroll
    for (int s = 0; s < TK_MAX_PER_LANE; ++s) {
      const int e = lane + 64 * s;
      if (s < per && e < E) {
        v[s] = z[(size_t)t * E + e];
        mx = fmaxf(mx, v[s]);
      } else {
        v[s] = -INFINITY;
        taken |= 1u << s;
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
    float se = 0.f;
#pragma unroll
    for (int s = 0; s < TK_MAX_PER_LANE; ++s)
      if (!(taken & (1u << s))) se += expf(v[s] - mx);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) se += __shfl_xor(se, off, 64);
    // picks and unnormalised weights go straight to the outputs (lane 0);
    // the weights are divided by the softmax denominator afterwards
    float esum = 0.f;
    for (int r = 0; r < k; ++r) {
      float bv = -INFINITY;
      int be = E;  // sentinel: nothing selectable in this lane
#pragma unroll
      for (int s = 0; s < TK_MAX_PER_LANE; ++s) {
        const int e = lane + 64 * s;
        if (!(taken & (1u << s)) && better(v[s], e, bv, be)) {
          bv = v[s];
          be = e;
        }
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const float ov = __shfl_xor(bv, off, 64);
        const int oe = __shfl_xor(be, off, 64);
        if (better(ov, oe, bv, be)) {
          bv = ov;
          be = oe;
        }
      }
      if (be >= E) be = E - 1;  // only when every remaining logit is NaN
      if ((be & 63) == lane) taken |= 1u << (be >> 6);
      const float ev = expf(bv - mx);
      esum += ev;
      if (lane == 0) {
        idx[(size_t)t * k + r] = be;
        w[(size_t)t * k + r] = ev;
        atomicAdd(&hist[be], 1);
      }
    }
    if (lane == 0) {
      const float denom = norm_topk ? esum : se;
      for (int r = 0; r < k; ++r) w[(size_t)t * k + r] = w[(size_t)t * k + r] / denom;
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x)
    if (hist[e]) atomicAdd(&counts[e], hist[e]);
}

__global__ void zero_i32_kernel(int32_t* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

template <typename TA>
hipError_t route_typed(const eb_model_desc& d, int T, const float* x, const float* gain,
                       const void* Wg, const float* bias, void* a_out, float* logits,
                       int32_t* idx, float* w, int32_t* counts, hipStream_t s) {
  hipLaunchKernelGGL(zero_i32_kernel, dim3((d.E + 255) / 256), dim3(256), 0, s, counts, d.E);
  if (T == 0) return hipGetLastError();
  if (sizeof(TA) == 2 && d.E > 8) {
    // RMSNorm, then the router GEMM on the matrix cores
    prof_start(EB_K_ROUTE_NORM, s);
    hipLaunchKernelGGL(rmsnorm_kernel<TA>, dim3((T + 3) / 4), dim3(256), 0, s, T, d.H, x, gain,
                       static_cast<TA*>(a_out), d.rms_eps);
    prof_stop(EB_K_ROUTE_NORM, s);
    prof_start(EB_K_ROUTE_LOGITS, s);
    const dim3 grid((T + 31) / 32);
    const bf16_t* ab = static_cast<const bf16_t*>(a_out);
    const bf16_t* wb = static_cast<const bf16_t*>(Wg);
    const int nb = (d.E + 31) / 32;
    if (nb <= 2)
      hipLaunchKernelGGL(router_mfma_kernel<2>, grid, dim3(256), 0, s, T, d.H, d.E, ab, wb, bias, logits);
    else if (nb <= 4)
      hipLaunchKernelGGL(router_mfma_kernel<4>, grid, dim3(256), 0, s, T, d.H, d.E, ab, wb, bias, logits);
    else
      hipLaunchKernelGGL(router_mfma_kernel<8>, grid, dim3(256), 0, s, T, d.H, d.E, ab, wb, bias, logits);
    prof_stop(EB_K_ROUTE_LOGITS, s);
  } else if (d.E <= 64) {
    prof_start(EB_K_ROUTE_LOGITS, s);
    if (d.E <= 8)
      hipLaunchKernelGGL((norm_router_kernel<TA, 8>), dim3((T + 3) / 4), dim3(256), 0, s, T, d.H, d.E,
                         x, gain, static_cast<const TA*>(Wg), bias, static_cast<TA*>(a_out), logits,
                         d.rms_eps);
    else
      hipLaunchKernelGGL((norm_router_kernel<TA, 64>), dim3((T + 3) / 4), dim3(256), 0, s, T, d.H,
                         d.E, x, gain, static_cast<const TA*>(Wg), bias, static_cast<TA*>(a_out),
                         logits, d.rms_eps);
    prof_stop(EB_K_ROUTE_LOGITS, s);
  } else {
    prof_start(EB_K_ROUTE_NORM, s);
    hipLaunchKernelGGL(rmsnorm_kernel<TA>, dim3((T + 3) / 4), dim3(256), 0, s, T, d.H, x, gain,
                       static_cast<TA*>(a_out), d.rms_eps);
    prof_stop(EB_K_ROUTE_NORM, s);
    prof_start(EB_K_ROUTE_LOGITS, s);
    hipLaunchKernelGGL(logits_kernel<TA>, dim3((T + LG_BT - 1) / LG_BT, (d.E + LG_BE - 1) / LG_BE),
                       dim3(256), 0, s, T, d.H, d.E, static_cast<const TA*>(a_out),
                       static_cast<const TA*>(Wg), bias, logits);
    prof_stop(EB_K_ROUTE_LOGITS, s);
  }
  prof_start(EB_K_ROUTE_TOPK, s);
  hipLaunchKernelGGL(topk_kernel, dim3((T + 3) / 4), dim3(256), 0, s, T, d.E, d.k, d.norm_topk,
                     logits, idx, w, counts);
  prof_stop(EB_K_ROUTE_TOPK, s);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_route(const eb_model_desc& d, int T, const float* x, const float* gain,
                        const void* Wg, const float* bias, void* a_out, float* logits,
                        int32_t* idx, float* w, int32_t* counts, hipStream_t s) {
  if (d.dtype == EB_DTYPE_BF16)
    return route_typed<bf16_t>(d, T, x, gain, Wg, bias, a_out, logits, idx, w, counts, s);
  return route_typed<float>(d, T, x, gain, Wg, bias, a_out, logits, idx, w, counts, s);
}

}  // namespace eb
