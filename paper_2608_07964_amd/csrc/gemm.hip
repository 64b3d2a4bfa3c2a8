// Grouped expert GEMMs of one step: every (layer, expert) group of the step,
// from whatever layer, in one launch per GEMM (cross-layer workload
// combination, Section 4.1).  Groups are the contiguous row ranges
// offsets[key] .. offsets[key+1] of the grouped activations; the tile list
// (key, first row) comes from the permutation scan.
//
//   gate/up:  h = dtype( SiLU(A Wgate^T) * (A Wup^T) )   A [P][H], W_gu[l][e] [2F][H]
//   down:     o = dtype( h Wdown^T )                     h [P][F], W_dn[l][e] [H][F]
//
// bf16 path: MFMA v_mfma_f32_32x32x16_bf16, 256x256 output tile per
// workgroup of 8 wavefronts, K step 64 double-buffered in LDS with an XOR
// swizzle of 16-byte chunks, global loads of the next K step in flight while
// the current one is multiplied; persistent, XCD-aware work distribution.
// The gate/up B tile interleaves 32 gate rows and the 32 matching up rows per
// wavefront column, so each lane holds gate and up of the same (row, f) and
// SwiGLU runs in registers.
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

enum { MODE_GATEUP = 0, MODE_DOWN = 1 };

// bf16 tiles: 256 x 256 output per workgroup, K step 64, 8 wavefronts in a
// 2 (M) x 4 (N) grid of 128 x 64 wave tiles (4 x 2 MFMA 32x32 blocks each),
// two waves per SIMD.  LDS holds two K stages of A and B: 2 x 64 KB.
constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kThreads = 512;
constexpr int kChunks = BK / 8;              // 16-byte chunks per LDS row
constexpr int kTileElems = BM * BK;          // one operand tile in LDS
constexpr int kXcds = 8;

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ (row & 7); }

// Persistent grouped GEMM.  Work item = (group, n-tile, m-tile), enumerated
// group by group, n-tile-major, m-tile fastest, so consecutive items share
// the weight tile.  Workgroup b runs on XCD b % 8 (round-robin dispatch); XCD
// x walks its own contiguous eighth of the items with its 32 workgroups side
// by side, so items running together on one L2 share weight and activation
// tiles.
template <int MODE>
__global__ __launch_bounds__(kThreads, 1) void grouped_gemm_bf16(GroupedProblem p, WeightTable wt,
                                                                 const bf16_t* __restrict__ A,
                                                                 bf16_t* __restrict__ C,
                                                                 int n_ntiles) {
  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * 2 * kTileElems];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int lrow = lane & 31, khalf = lane >> 5;
  const int xcd = blockIdx.x % kXcds, slot = blockIdx.x / kXcds, nslots = gridDim.x / kXcds;
  const int G = *p.n_groups;
  const long long total = (long long)(*p.n_tiles) * n_ntiles;
  const int lo = (int)((xcd * total) / kXcds), hi = (int)(((xcd + 1) * total) / kXcds);
  const int K = MODE == MODE_GATEUP ? p.H : p.F;
  const int nk = K / BK;
  const int ES = p.E + p.S;

  for (int it = lo + slot; it < hi; it += nslots) {
    // group of this item: the last g with cum_mt[g] * n_ntiles <= it
    int glo = 0, ghi = G - 1;
    while (glo < ghi) {
      const int mid = (glo + ghi + 1) >> 1;
      if ((long long)p.groups[mid].w * n_ntiles <= it) glo = mid; else ghi = mid - 1;
    }
    const int4 gd = p.groups[glo];  // key, first row, rows, first m-tile
    const int mt = (gd.z + BM - 1) / BM;
    const int local = it - gd.w * n_ntiles;
    const int ni = local / mt, mi = local - ni * mt;
    const int row0 = gd.y + mi * BM, row_end = gd.y + gd.z;
    const int layer = gd.x / ES, e = gd.x - layer * ES;
    const bf16_t* Bbase = MODE == MODE_GATEUP
        ? static_cast<const bf16_t*>(wt.gu[layer]) + (size_t)e * 2 * p.F * p.H
        : static_cast<const bf16_t*>(wt.dn[layer]) + (size_t)e * p.H * p.F;

    // Thread tid moves 16-byte chunk c = tid % 8 of tile rows r_i = tid / 8 + 64 i
    // (i < 4) of both operands.  Offsets are 32-bit element offsets from the
    // tile's base pointers; staging lives in plain registers.
    const int c0 = tid % kChunks, r0 = tid / kChunks;
    const bf16_t* Atile = A + (size_t)row0 * K + c0 * 8;
    const int a_last = p.P - 1 - row0;  // ragged tail: clamp to an in-bounds row, result discarded
    const int ao0 = min(r0, a_last) * K, ao1 = min(r0 + 64, a_last) * K;
    const int ao2 = min(r0 + 128, a_last) * K, ao3 = min(r0 + 192, a_last) * K;
    int bo0, bo1, bo2, bo3;
    if (MODE == MODE_GATEUP) {
      // wave column wn owns 32 gate rows and the 32 matching up rows:
      // tile row r -> f = ni*128 + (r/64)*32 + r%32, gate row f or up row F+f
      const int within = r0 & 63;  // r0 < 64, rows r0 + 64 i share it
      const int fb = ni * (BN / 2) + (within & 31);
      const int up = within < 32 ? 0 : p.F;
      bo0 = (up + fb + 0) * K;
      bo1 = (up + fb + 32) * K;
      bo2 = (up + fb + 64) * K;
      bo3 = (up + fb + 96) * K;
    } else {
      bo0 = (ni * BN + r0) * K;
      bo1 = bo0 + 64 * K;
      bo2 = bo0 + 128 * K;
      bo3 = bo0 + 192 * K;
    }
    const bf16_t* Btile = Bbase + c0 * 8;
    const int s0 = r0 * BK + swz(r0, c0) * 8;  // LDS slot of row r0; rows r0 + 64 i: + 64 i BK

    floatx16 acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    uint4 ra0, ra1, ra2, ra3, rb0, rb1, rb2, rb3;
    auto gload = [&](int k) {
      ra0 = *reinterpret_cast<const uint4*>(Atile + ao0 + k);
      ra1 = *reinterpret_cast<const uint4*>(Atile + ao1 + k);
      ra2 = *reinterpret_cast<const uint4*>(Atile + ao2 + k);
      ra3 = *reinterpret_cast<const uint4*>(Atile + ao3 + k);
      rb0 = *reinterpret_cast<const uint4*>(Btile + bo0 + k);
      rb1 = *reinterpret_cast<const uint4*>(Btile + bo1 + k);
      rb2 = *reinterpret_cast<const uint4*>(Btile + bo2 + k);
      rb3 = *reinterpret_cast<const uint4*>(Btile + bo3 + k);
    };
    auto sstore = [&](bf16_t* As) {
      bf16_t* Bs = As + kTileElems;
      *reinterpret_cast<uint4*>(As + s0) = ra0;
      *reinterpret_cast<uint4*>(As + s0 + 64 * BK) = ra1;
      *reinterpret_cast<uint4*>(As + s0 + 128 * BK) = ra2;
      *reinterpret_cast<uint4*>(As + s0 + 192 * BK) = ra3;
      *reinterpret_cast<uint4*>(Bs + s0) = rb0;
      *reinterpret_cast<uint4*>(Bs + s0 + 64 * BK) = rb1;
      *reinterpret_cast<uint4*>(Bs + s0 + 128 * BK) = rb2;
      *reinterpret_cast<uint4*>(Bs + s0 + 192 * BK) = rb3;
    };

    gload(0);
    sstore(smem);
    __syncthreads();

    for (int kt = 0; kt < nk; ++kt) {
      const bf16_t* As = smem + (kt & 1) * 2 * kTileElems;
      const bf16_t* Bs = As + kTileElems;
      const bool more = kt + 1 < nk;
      if (more) gload((kt + 1) * BK);
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const int c = ks * 2 + khalf;
        bf16x8 av[4], bv[2];
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) {
          const int r = wm * 128 + mb * 32 + lrow;
          av[mb] = *reinterpret_cast<const bf16x8*>(&As[r * BK + swz(r, c) * 8]);
        }
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          const int r = wn * 64 + nb * 32 + lrow;
          bv[nb] = *reinterpret_cast<const bf16x8*>(&Bs[r * BK + swz(r, c) * 8]);
        }
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
#pragma unroll
          for (int nb = 0; nb < 2; ++nb)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[mb], bv[nb], acc[mb][nb], 0, 0, 0);
      }
      if (more) sstore(smem + ((kt + 1) & 1) * 2 * kTileElems);
      __syncthreads();
    }

    // epilogue: acc[mb][nb][v] is C[row][col] with col = lane%32 of the 32x32
    // block and row = 8*(v/4) + 4*(lane/32) + v%4
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = row0 + wm * 128 + mb * 32 + 8 * (v >> 2) + 4 * khalf + (v & 3);
        if (row >= row_end) continue;
        if (MODE == MODE_GATEUP) {
          const int f = ni * (BN / 2) + wn * 32 + lrow;
          C[(size_t)row * p.F + f] = f32_to_bf16(swiglu(acc[mb][0][v], acc[mb][1][v]));
        } else {
#pragma unroll
          for (int nb = 0; nb < 2; ++nb) {
            const int n = ni * BN + wn * 64 + nb * 32 + lrow;
            C[(size_t)row * p.H + n] = f32_to_bf16(acc[mb][nb][v]);
          }
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

static int persistent_grid() {
  static int grid = 0;
  if (grid == 0) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
      cus = 256;
    grid = (cus + kXcds - 1) / kXcds * kXcds;
  }
  return grid;
}

hipError_t launch_gateup(int dtype, const GroupedProblem& p, const WeightTable& wt,
                         const void* a_perm, void* h, hipStream_t s) {
  prof_start(EB_K_GATEUP, s);
  if (dtype == EB_DTYPE_BF16) {
    hipLaunchKernelGGL(grouped_gemm_bf16<MODE_GATEUP>, dim3(persistent_grid()), dim3(kThreads), 0, s,
                       p, wt, static_cast<const bf16_t*>(a_perm), static_cast<bf16_t*>(h),
                       p.F / (BN / 2));
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
    hipLaunchKernelGGL(grouped_gemm_bf16<MODE_DOWN>, dim3(persistent_grid()), dim3(kThreads), 0, s,
                       p, wt, static_cast<const bf16_t*>(h), static_cast<bf16_t*>(o), p.H / BN);
  } else {
    hipLaunchKernelGGL(grouped_gemm_f32<MODE_DOWN>, dim3(p.max_tiles, p.H / FBN), dim3(256), 0, s,
                       p, wt, static_cast<const float*>(h), static_cast<float*>(o));
  }
  prof_stop(EB_K_DOWN, s);
  return hipGetLastError();
}

}  // namespace eb
