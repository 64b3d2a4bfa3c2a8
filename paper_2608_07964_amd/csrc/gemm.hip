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
// workgroup of 4 wavefronts (128x128 each), K step 64 double-buffered in LDS,
// filled by buffer loads straight into LDS (XOR-swizzled 16-byte chunks) one
// stage ahead of the MFMAs; persistent, XCD-aware work distribution.  The gate/up B tile
// interleaves 64 gate rows and the 64 matching up rows per wavefront column,
// so each lane holds gate and up of the same (row, f) and SwiGLU runs in
// registers.
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

// bf16 tiles: 256 x 256 output per workgroup of 4 wavefronts (one per SIMD),
// each owning a 128 x 128 quarter as 4 x 4 MFMA 32x32 blocks (accumulators in
// AGPRs): 8 fragment reads per 16 MFMAs.  K advances 64 at a time, so every
// 128-byte line of A and B is consumed whole by one stage; two LDS stages of
// 64 KB (A and B tiles of 256 rows x 128 bytes) are filled by buffer loads
// straight into LDS one stage ahead.  Fragments of the next k-step are read
// while the MFMAs of the current one run, and the per-stage barrier sits
// before the last k-step's MFMAs, so neither the barrier nor LDS latency
// stalls the matrix cores.
constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kStages = 2;
constexpr int kThreads = 256;
constexpr int kKsteps = BK / 16;                 // MFMA k-steps per stage
constexpr int kTileElems = BM * BK;              // one operand tile of a stage
constexpr int kStageElems = 2 * kTileElems;      // A then B
constexpr int kRowBlocks = 8;                    // 8-row blocks per wave per operand
constexpr int kXcds = 8;

// 128-byte LDS rows hold eight 16-byte chunks; logical chunk c of row r sits
// at c ^ ((r >> 1) & 7).  A ds_read_b128 phase of 16 lanes reads 16
// consecutive rows at one logical chunk: two rows share each 256-byte bank
// window, and the XOR spreads the 8 rows of each parity over 8 chunks, so the
// 16 reads hit 16 distinct 16-byte groups of the 64 banks.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// s_waitcnt immediates (gfx9 encoding: vmcnt bits 3:0 and 15:14, expcnt
// 6:4, lgkmcnt 11:8).  Issued through the builtin so that the compiler's own
// wait insertion sees them and does not add conservative waits of its own.
constexpr int kWaitVm0 = (7 << 4) | (15 << 8);
constexpr int kWaitVm16 = (16 >> 4) << 14 | (7 << 4) | (15 << 8);
constexpr int kWaitLgkm0 = 15 | (3 << 14) | (7 << 4);

// Bare workgroup barrier: this wave's outstanding buffer->LDS loads stay in
// flight across it (a fenced __syncthreads would drain them).
__device__ __forceinline__ void bar() {
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Raw buffer descriptor over [base, base + bytes) (bytes < 2^32); offsets
// past the end read zeros.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// Load slots: wave w fills LDS rows 64 w + 8 j .. +7 of each operand tile
// (j < 8); lane l supplies row r_j = 64 w + 8 j + l / 8 at physical chunk
// l % 8, i.e. logical chunk c_j = (l % 8) ^ ((r_j >> 1) & 7), which is c_0 for
// even j and c_0 ^ 4 for odd j.  A row r_j and B row brow0 + 8 j (see the item
// setup) are affine in j, so a load's byte offset is a per-lane part that
// depends only on the parity of j plus a wave-uniform part (soffset).  A rows
// past the group's end lie outside the A descriptor's range and read zeros.
struct KLoop {
  bf16_t* smem;
  __amdgpu_buffer_rsrc_t ra, rb;   // buffer descriptors of the A tile and the expert's B
  int a_lane[2], b_lane[2];        // per-lane byte offsets for even / odd j
  int row_bytes;                   // K * 2
  int lds_load;                    // LDS element offset of the wave's first load row
  int lds_a, lds_b;                // LDS element offsets of this lane's fragment rows (chunk-free)
  int sw;                          // this lane's fragment swizzle ((row >> 1) & 7)
  int nk, khalf;
};

struct Frags {
  bf16x8 a[4], b[4];
};

// Fragment rows of one lane: A rows wm*128 + mb*32 + lrow, B rows
// wn*128 + nb*32 + lrow; (row >> 1) & 7 = (lrow >> 1) & 7 for all of them, so
// one chunk term per k-step serves every block and the block offsets are
// immediates.
template <int NACT>
__device__ __forceinline__ void read_frags(const KLoop& L, int stage, int ks, Frags& f) {
  const bf16_t* base = L.smem + (stage % kStages) * kStageElems + ((ks * 2 + L.khalf) ^ L.sw) * 8;
#pragma unroll
  for (int mb = 0; mb < NACT; ++mb)
    f.a[mb] = *reinterpret_cast<const bf16x8*>(base + L.lds_a + mb * 32 * BK);
#pragma unroll
  for (int nb = 0; nb < 4; ++nb)
    f.b[nb] = *reinterpret_cast<const bf16x8*>(base + kTileElems + L.lds_b + nb * 32 * BK);
}

template <int NACT>
__device__ __forceinline__ void mfmas(const Frags& f, floatx16 (&acc)[4][4]) {
#pragma unroll
  for (int mb = 0; mb < NACT; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
      acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[mb], f.b[nb], acc[mb][nb], 0, 0, 0);
}

// One item's K loop.  Stage s (K columns 64 s .. 64 s + 63) lives in LDS slot
// s % 2.  In step kt the four k-steps of stage kt run with the next k-step's
// fragments read ahead; before the MFMAs of the last k-step the wave waits for
// its loads of stage kt+1 and its reads of stage kt, the barrier publishes
// stage kt+1 and frees slot kt % 2, stage kt+2 is issued into it and the
// first fragments of stage kt+1 are read.  NACT = active 32-row blocks of the
// wave's 128 rows (inactive blocks of a ragged tile get neither LDS reads nor
// MFMAs).
template <int NACT>
__device__ __forceinline__ void k_loop(const KLoop& L, floatx16 (&acc)[4][4]) {
  // buffer (MUBUF) loads straight into LDS: lane l's 16 bytes land at the
  // wave-uniform LDS address + 16 l
  auto issue = [&](int s) {
    bf16_t* sa = L.smem + (s % kStages) * kStageElems + L.lds_load;
    bf16_t* sb = sa + kTileElems;
#pragma unroll
    for (int j = 0; j < kRowBlocks; ++j) {
      const int so = j * 8 * L.row_bytes + s * BK * 2;  // wave-uniform
      __builtin_amdgcn_raw_ptr_buffer_load_lds(L.ra, sa + j * 8 * BK, 16, L.a_lane[j & 1], so, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(L.rb, sb + j * 8 * BK, 16, L.b_lane[j & 1], so, 0, 0);
    }
  };
  const int nk = L.nk;
  issue(0);
  if (nk > 1) {
    issue(1);
    __builtin_amdgcn_s_waitcnt(kWaitVm16);
  } else {
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
  }
  bar();
  Frags f[2];
  if (NACT > 0) read_frags<NACT>(L, 0, 0, f[0]);
  for (int kt = 0; kt < nk; ++kt) {
#pragma unroll
    for (int ks = 0; ks < kKsteps - 1; ++ks) {
      if (NACT > 0) {
        read_frags<NACT>(L, kt, ks + 1, f[(ks + 1) & 1]);
        mfmas<NACT>(f[ks & 1], acc);
        // keep the next k-step's fragment reads spread between this k-step's
        // MFMAs (the machine scheduler would otherwise move reads next to
        // their consumers and expose LDS latency)
#pragma unroll
        for (int i = 0; i < NACT + 4; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one DS read
          __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // two MFMAs
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 4 * NACT - 2 * (NACT + 4) > 0 ? 4 * NACT - 2 * (NACT + 4) : 0, 0);
      }
    }
    // every fragment of stage kt is in registers, stage kt+1 has landed
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
    bar();
    if (kt + 2 < nk) issue(kt + 2);
    if (NACT > 0) {
      if (kt + 1 < nk) read_frags<NACT>(L, kt + 1, 0, f[0]);
      mfmas<NACT>(f[(kKsteps - 1) & 1], acc);
    }
  }
}

// Persistent grouped GEMM.  Work item = (group, n-tile, m-tile), enumerated
// group by group, n-tile-major, m-tile fastest, so consecutive items share
// the weight tile.  Workgroup b runs on XCD b % 8 (round-robin dispatch); XCD
// x walks its own contiguous eighth of the items with its workgroups side by
// side, so items running together on one L2 share weight and activation
// tiles.
template <int MODE>
__global__ __launch_bounds__(kThreads, 1) void grouped_gemm_bf16(GroupedProblem p, WeightTable wt,
                                                                 const bf16_t* __restrict__ A,
                                                                 bf16_t* __restrict__ C,
                                                                 int n_ntiles) {
  __shared__ __attribute__((aligned(1024))) bf16_t smem[kStages * kStageElems];
  // the LDS ring is written by global->LDS loads the compiler does not see
  asm volatile("" ::"v"(smem) : "memory");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int lrow = lane & 31, khalf = lane >> 5;
  const int xcd = blockIdx.x % kXcds, slot = blockIdx.x / kXcds, nslots = gridDim.x / kXcds;
  const int G = *p.n_groups;
  const long long total = (long long)(*p.n_tiles) * n_ntiles;
  const int lo = (int)((xcd * total) / kXcds), hi = (int)(((xcd + 1) * total) / kXcds);
  const int K = MODE == MODE_GATEUP ? p.H : p.F;
  const int nk = K / BK;
  const int ES = p.E + p.S;

  const int lr = lane >> 3, lp = lane & 7;  // load slot of this lane (see KLoop)

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
    const bf16_t* Atile = A + (size_t)row0 * K;
    const int a_last = min(BM, p.P - row0) - 1;  // rows past it read zeros; their results are discarded

    KLoop kl;
    kl.smem = smem;
    kl.ra = buffer_rsrc(Atile, (uint32_t)((a_last + 1) * K * 2));
    kl.rb = buffer_rsrc(Bbase, (uint32_t)((MODE == MODE_GATEUP ? 2 * p.F : p.H) * K * 2));
    kl.row_bytes = K * 2;
    {
      const int r0 = 64 * wave + lr;
      const int c0 = lp ^ ((r0 >> 1) & 7);
      int brow0;
      if (MODE == MODE_GATEUP) {
        // wave column wc = r / 128 owns 64 gate rows and the 64 matching up
        // rows: tile row r -> f = ni*128 + wc*64 + r%64, gate row f or up row
        // F+f.  For r = 64 w + 8 j + l/8: r/128 = w/2 and r%128 >= 64 iff w is odd.
        brow0 = ni * (BN / 2) + (wave >> 1) * 64 + lr + ((wave & 1) ? p.F : 0);
      } else {
        brow0 = ni * BN + r0;
      }
      kl.a_lane[0] = r0 * K * 2 + c0 * 16;
      kl.a_lane[1] = r0 * K * 2 + (c0 ^ 4) * 16;
      kl.b_lane[0] = brow0 * K * 2 + c0 * 16;
      kl.b_lane[1] = brow0 * K * 2 + (c0 ^ 4) * 16;
    }
    kl.lds_load = 64 * wave * BK;
    kl.lds_a = (wm * 128 + lrow) * BK;
    kl.lds_b = (wn * 128 + lrow) * BK;
    kl.sw = (lrow >> 1) & 7;
    kl.nk = nk;
    kl.khalf = khalf;

    floatx16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    // 32-row blocks of this wave's 128 rows that hold rows of the group
    const int nact = min(4, max(0, (row_end - (row0 + wm * 128) + 31) / 32));
    switch (nact) {
      case 4: k_loop<4>(kl, acc); break;
      case 3: k_loop<3>(kl, acc); break;
      case 2: k_loop<2>(kl, acc); break;
      case 1: k_loop<1>(kl, acc); break;
      default: k_loop<0>(kl, acc); break;
    }
    __syncthreads();  // every wave is done with the ring before the next item refills it

    // epilogue: acc[mb][nb][v] is C[row][col] with col = lane%32 of the 32x32
    // block and row = 8*(v/4) + 4*(lane/32) + v%4
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = row0 + wm * 128 + mb * 32 + 8 * (v >> 2) + 4 * khalf + (v & 3);
        if (row >= row_end) continue;
        if (MODE == MODE_GATEUP) {
#pragma unroll
          for (int nb = 0; nb < 2; ++nb) {
            const int f = ni * (BN / 2) + wn * 64 + nb * 32 + lrow;
            C[(size_t)row * p.F + f] = f32_to_bf16(swiglu(acc[mb][nb][v], acc[mb][nb + 2][v]));
          }
        } else {
#pragma unroll
          for (int nb = 0; nb < 4; ++nb) {
            const int n = ni * BN + wn * 128 + nb * 32 + lrow;
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
