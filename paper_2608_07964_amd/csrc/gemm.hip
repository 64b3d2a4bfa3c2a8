// Grouped expert GEMMs of one step: every (layer, expert) group of the step,
// from whatever layer, in one launch per GEMM (cross-layer workload
// combination, Section 4.1).  Groups are the contiguous row ranges
// offsets[key] .. offsets[key+1] of the grouped activations; the tile list
// (key, first row) comes from the permutation scan.
//
//   gate/up:  h = dtype( SiLU(A Wgate^T) * (A Wup^T) )   A [P][H], W_gu[l][e] [2F][H]
//   down:     o = dtype( h Wdown^T )                     h [P][F], W_dn[l][e] [H][F]
//
// bf16 path: MFMA v_mfma_f32_32x32x16_bf16, 128x128 output tile per
// workgroup of 4 wavefronts (2x2, 64x64 each), K step 64 staged through LDS
// with an XOR swizzle of 16-byte chunks, global loads for the next K step in
// flight while the current one is multiplied.  The gate/up B tile interleaves
// 32 gate rows and the 32 matching up rows per wavefront column, so each lane
// holds gate and up of the same (row, f) and SwiGLU runs in registers.
//
// Every output accumulates its K dimension in 16-wide MFMA steps in ascending
// order, whatever tile or group its row sits in: rows give the same bits
// whichever step (and schedule) they are computed in.
//
// fp32 path (fp32 stacks): LDS-tiled VALU GEMM, 64x64 tiles, 4x4 per thread,
// same K-order guarantee.
#include "eb_internal.h"
#include "eb_numeric.h"

namespace eb {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int kThreads = 256;
constexpr int kChunks = BK / 8;  // 16-byte chunks per LDS row

enum { MODE_GATEUP = 0, MODE_DOWN = 1 };

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ (row & 7); }

template <int MODE>
__global__ __launch_bounds__(kThreads) void grouped_gemm_bf16(GroupedProblem p, WeightTable wt,
                                                              const bf16_t* __restrict__ A,
                                                              bf16_t* __restrict__ C) {
  __shared__ __attribute__((aligned(16))) bf16_t As[BM * BK];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[BN * BK];

  const int tile = blockIdx.x;
  if (tile >= *p.n_tiles) return;
  const int2 td = p.tiles[tile];
  const int key = td.x, row0 = td.y;
  const int ES = p.E + p.S;
  const int layer = key / ES, e = key - layer * ES;
  const int row_end = p.offsets[key + 1];
  const int nt = blockIdx.y;
  const int K = MODE == MODE_GATEUP ? p.H : p.F;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  const bf16_t* Bbase;
  if (MODE == MODE_GATEUP)
    Bbase = static_cast<const bf16_t*>(wt.gu[layer]) + (size_t)e * 2 * p.F * p.H;
  else
    Bbase = static_cast<const bf16_t*>(wt.dn[layer]) + (size_t)e * p.H * p.F;

  // per-thread load slots: 4 chunks of A and 4 of B per K step
  const bf16_t* a_src[4];
  const bf16_t* b_src[4];
  int s_off[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int cid = tid + kThreads * i;
    const int r = cid / kChunks, c = cid % kChunks;
    const int grow = min(row0 + r, p.P - 1);  // ragged tail: in-bounds row, result discarded
    a_src[i] = A + (size_t)grow * K + c * 8;
    int brow;
    if (MODE == MODE_GATEUP) {
      const int wcol = r >> 6, within = r & 63;
      const int f = nt * 64 + wcol * 32 + (within & 31);
      brow = within < 32 ? f : p.F + f;
    } else {
      brow = nt * BN + r;
    }
    b_src[i] = Bbase + (size_t)brow * K + c * 8;
    s_off[i] = r * BK + swz(r, c) * 8;
  }

  floatx16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  uint4 ra[4], rb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ra[i] = *reinterpret_cast<const uint4*>(a_src[i]);
    rb[i] = *reinterpret_cast<const uint4*>(b_src[i]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    *reinterpret_cast<uint4*>(&As[s_off[i]]) = ra[i];
    *reinterpret_cast<uint4*>(&Bs[s_off[i]]) = rb[i];
  }
  __syncthreads();

  const int lrow = lane & 31, khalf = lane >> 5;
  for (int k0 = 0; k0 < K; k0 += BK) {
    const bool more = k0 + BK < K;
    if (more) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ra[i] = *reinterpret_cast<const uint4*>(a_src[i] + k0 + BK);
        rb[i] = *reinterpret_cast<const uint4*>(b_src[i] + k0 + BK);
      }
    }
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int c = ks * 2 + khalf;
      bf16x8 av[2], bv[2];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        const int r = wm * 64 + mb * 32 + lrow;
        av[mb] = *reinterpret_cast<const bf16x8*>(&As[r * BK + swz(r, c) * 8]);
      }
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const int r = wn * 64 + nb * 32 + lrow;
        bv[nb] = *reinterpret_cast<const bf16x8*>(&Bs[r * BK + swz(r, c) * 8]);
      }
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[mb], bv[nb], acc[mb][nb], 0, 0, 0);
    }
    __syncthreads();
    if (more) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        *reinterpret_cast<uint4*>(&As[s_off[i]]) = ra[i];
        *reinterpret_cast<uint4*>(&Bs[s_off[i]]) = rb[i];
      }
      __syncthreads();
    }
  }

  // epilogue: acc[mb][nb][v] is C[row][col] with col = lane%32 of the 32x32
  // block and row = 8*(v/4) + 4*(lane/32) + v%4
#pragma unroll
  for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int row = row0 + wm * 64 + mb * 32 + 8 * (v >> 2) + 4 * khalf + (v & 3);
      if (row >= row_end) continue;
      if (MODE == MODE_GATEUP) {
        const int f = nt * 64 + wn * 32 + lrow;
        C[(size_t)row * p.F + f] = f32_to_bf16(swiglu(acc[mb][0][v], acc[mb][1][v]));
      } else {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          const int n = nt * BN + wn * 64 + nb * 32 + lrow;
          C[(size_t)row * p.H + n] = f32_to_bf16(acc[mb][nb][v]);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// fp32 path
constexpr int FBM = 64, FBN = 64, FBK = 16;

template <int MODE>
__global__ __launch_bounds__(256) void grouped_gemm_f32(GroupedProblem p, WeightTable wt,
                                                        const float* __restrict__ A,
                                                        float* __restrict__ C) {
  __shared__ float As[FBK][FBM + 4];
  __shared__ float Bs[FBK][FBN + 4];
  const int tile = blockIdx.x;
  if (tile >= *p.n_tiles) return;
  const int2 td = p.tiles[tile];
  const int key = td.x, row0 = td.y;
  const int ES = p.E + p.S;
  const int layer = key / ES, e = key - layer * ES;
  const int row_end = p.offsets[key + 1];
  const int nt = blockIdx.y;
  const int K = MODE == MODE_GATEUP ? p.H : p.F;
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  const float* Bbase = MODE == MODE_GATEUP
                           ? static_cast<const float*>(wt.gu[layer]) + (size_t)e * 2 * p.F * p.H
                           : static_cast<const float*>(wt.dn[layer]) + (size_t)e * p.H * p.F;
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  const int arow = min(row0 + lr, p.P - 1);
  int brow;
  if (MODE == MODE_GATEUP) {
    const int f = nt * 32 + (lr & 31);
    brow = lr < 32 ? f : p.F + f;
  } else {
    brow = nt * FBN + lr;
  }
  const float* ap = A + (size_t)arow * K + lk;
  const float* bp = Bbase + (size_t)brow * K + lk;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += FBK) {
    const float4 av = *reinterpret_cast<const float4*>(ap + k0);
    const float4 bv = *reinterpret_cast<const float4*>(bp + k0);
    As[lk + 0][lr] = av.x; As[lk + 1][lr] = av.y; As[lk + 2][lr] = av.z; As[lk + 3][lr] = av.w;
    Bs[lk + 0][lr] = bv.x; Bs[lk + 1][lr] = bv.y; Bs[lk + 2][lr] = bv.z; Bs[lk + 3][lr] = bv.w;
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < FBK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = row0 + ty * 4 + i;
    if (row >= row_end) continue;
    if (MODE == MODE_GATEUP) {
#pragma unroll
      for (int jj = 0; jj < 2; ++jj)
        C[(size_t)row * p.F + nt * 32 + tx + 16 * jj] = swiglu(acc[i][jj], acc[i][jj + 2]);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) C[(size_t)row * p.H + nt * FBN + tx + 16 * j] = acc[i][j];
    }
  }
}

}  // namespace

int gemm_bm(int dtype) { return dtype == EB_DTYPE_BF16 ? BM : FBM; }

hipError_t launch_gateup(int dtype, const GroupedProblem& p, const WeightTable& wt,
                         const void* a_perm, void* h, hipStream_t s) {
  prof_start(EB_K_GATEUP, s);
  if (dtype == EB_DTYPE_BF16) {
    hipLaunchKernelGGL(grouped_gemm_bf16<MODE_GATEUP>, dim3(p.max_tiles, p.F / 64), dim3(kThreads),
                       0, s, p, wt, static_cast<const bf16_t*>(a_perm), static_cast<bf16_t*>(h));
  } else {
    hipLaunchKernelGGL(grouped_gemm_f32<MODE_GATEUP>, dim3(p.max_tiles, p.F / 32), dim3(256), 0,
                       s, p, wt, static_cast<const float*>(a_perm), static_cast<float*>(h));
  }
  prof_stop(EB_K_GATEUP, s);
  return hipGetLastError();
}

hipError_t launch_down(int dtype, const GroupedProblem& p, const WeightTable& wt, const void* h,
                       void* o, hipStream_t s) {
  prof_start(EB_K_DOWN, s);
  if (dtype == EB_DTYPE_BF16) {
    hipLaunchKernelGGL(grouped_gemm_bf16<MODE_DOWN>, dim3(p.max_tiles, p.H / BN), dim3(kThreads), 0,
                       s, p, wt, static_cast<const bf16_t*>(h), static_cast<bf16_t*>(o));
  } else {
    hipLaunchKernelGGL(grouped_gemm_f32<MODE_DOWN>, dim3(p.max_tiles, p.H / FBN), dim3(256), 0, s,
                       p, wt, static_cast<const float*>(h), static_cast<float*>(o));
  }
  prof_stop(EB_K_DOWN, s);
  return hipGetLastError();
}

}  // namespace eb
