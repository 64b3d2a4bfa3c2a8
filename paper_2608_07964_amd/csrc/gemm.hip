// Grouped expert GEMMs of one step: every (layer, expert) group of the step,
// from whatever layer, in one launch per GEMM (cross-layer workload
// combination, Section 4.1).  Groups are the contiguous row ranges
// offsets[key] .. offsets[key+1] of the grouped activations; the tile list
// (the group record of every row block) comes from the permutation scan.
//
//   gate/up:  h = dtype( SiLU(A Wgate^T) * (A Wup^T) )   A [P][H], W_gu[l][e] [2F][H]
//   down:     o = dtype( h Wdown^T )                     h [P][F], W_dn[l][e] [H][F]
//
// bf16 path: MFMA v_mfma_f32_32x32x16_bf16, up to 256x256 outputs per
// workgroup of 8 wavefronts, K stages of 64 in LDS rings filled by buffer
// loads straight into LDS (XOR-swizzled 16-byte chunks) several stages ahead
// of the MFMAs; persistent, XCD-aware work distribution.  The gate/up B tile
// interleaves the gate rows and the matching up rows per wavefront column,
// so each lane holds gate and up of the same (row, f) and SwiGLU runs in
// registers.  The expert weights are read in the packed layout that
// pack_bf16_kernel writes once (see there): every B stage of a tile is one
// contiguous 32 KB block holding exactly the bytes its LDS slot receives,
// and the blocks of one K stage of all of an expert's column tiles are
// adjacent, so concurrent items stream neighbouring blocks.
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

// bf16 tiles.  Every tile is BM x 256 outputs on a workgroup of 8 wavefronts
// (two per SIMD) and K advances 64 at a time, so every 128-byte line of A and
// B is consumed whole by one stage; stages are filled by buffer loads straight
// into LDS.  The B tile (256 weight rows x 64 k) is the same in every shape;
// the shape of an m-tile follows the rows it holds:
//
//   BM 256 (> 128 rows): 2 x 4 wavefronts of 128 x 64 (4 x 2 MFMA blocks),
//          A ring of 2 stages (32 KB each), B ring of 3 stages (32 KB each);
//   BM 128 (65..128 rows): 2 x 4 wavefronts of 64 x 64, 3 stages of A and B;
//   BM 64  (<= 64 rows): 2 x 4 wavefronts of 32 x 64, 4 stages of A and B.
//
// Two wavefronts per SIMD keep each matrix core fed while the other one
// waits on a barrier or on LDS.  Groups that run few m-tiles are bound by
// streaming their expert's weights from HBM, which needs many bytes in flight
// per CU: every shape keeps at least two B stages in flight.  Fragments of the
// next k-step are read while the MFMAs of the current one run (every
// instruction's place in the k-step is fixed, see kstep), and the per-stage
// barrier sits before the last k-step's MFMAs.
constexpr int BN = 256, BK = 64;
constexpr int kWaves = 8;                        // two wavefronts per SIMD
constexpr int kThreads = 64 * kWaves;
constexpr int kKsteps = BK / 16;                 // MFMA k-steps per stage
constexpr int kBLoads = BN / (8 * kWaves);       // 8-row B blocks per wave per stage
constexpr int kBPart = kBLoads / (BK / 16);      // B loads issued per k-step
static_assert(kBPart * (BK / 16) == kBLoads, "B loads split evenly over the k-steps");
constexpr int kXcds = 8;

template <int BM_, int WM_, int SA_, int SB_>
struct TileCfg {
  static constexpr int BM = BM_;                 // tile rows
  static constexpr int WM = WM_, WN = kWaves / WM_;  // wavefront grid
  static constexpr int SA = SA_, SB = SB_;       // LDS stages of the A and B rings
  static constexpr int TM = BM / WM, TN = BN / WN;  // wavefront tile
  static constexpr int MB = TM / 32, NB = TN / 32;  // MFMA blocks per wavefront
  static constexpr int A_LOADS = BM / (8 * kWaves);  // 8-row A blocks per wave per stage
  static constexpr int A_ELEMS = BM * BK, B_ELEMS = BN * BK;  // one stage of each ring
  static constexpr int B_RING = SA * A_ELEMS;    // LDS element offset of the B ring
  static constexpr int LDS_ELEMS = SA * A_ELEMS + SB * B_ELEMS;
  static_assert(MB >= 1 && NB >= 2 && A_LOADS >= 1, "tile shape");
  static_assert(SA >= 2 && (SB == SA || SB == SA + 1), "ring depths");
};
using CfgBig = TileCfg<256, 2, 2, 3>;
using CfgMid = TileCfg<128, 2, 3, 3>;
using CfgSkinny = TileCfg<64, 2, 4, 4>;
constexpr int cmax(int a, int b) { return a > b ? a : b; }
constexpr int kLdsElems = cmax(cmax(CfgBig::LDS_ELEMS, CfgMid::LDS_ELEMS), CfgSkinny::LDS_ELEMS);
static_assert(kLdsElems * 2 <= 160 * 1024, "LDS budget");
constexpr int BM = CfgBig::BM;                   // row-block granularity of the tile list

// 128-byte LDS rows hold eight 16-byte chunks; logical chunk c of row r sits
// at c ^ ((r >> 1) & 7).  A ds_read_b128 phase of 16 lanes reads 16
// consecutive rows at one logical chunk: two rows share each 256-byte bank
// window, and the XOR spreads the 8 rows of each parity over 8 chunks, so the
// 16 reads hit 16 distinct 16-byte groups of the 64 banks.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// s_waitcnt immediates (gfx9 encoding: vmcnt bits 3:0 and 15:14, expcnt
// 6:4, lgkmcnt 11:8).  Issued through the builtin so that the compiler's own
// wait insertion sees them and does not add conservative waits of its own.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
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

// Load slots: in every stage wave w fills A rows (BM/4) w + 8 j + l/8
// (j < BM/32) of the tile, lane l at physical chunk l % 8, i.e. logical chunk
// (l % 8) ^ ((r >> 1) & 7), which is c0 for even j and c0 ^ 4 for odd j
// (every block base is a multiple of 16 rows).  An A load's byte offset is a
// per-lane part (row l/8 of the block and the chunk, by parity of j) plus a
// wave-uniform part (the block's first row and the stage's K offset) passed
// as soffset.  A rows past the buffer's end read zeros; rows past the group's
// end are loaded but their results are discarded.  B comes packed: wave w's
// load j of stage s copies the 1 KB at byte 4096 w + 1024 j of the stage's
// 32 KB block (LDS rows 32 w + 8 j .. + 7), lane l its 16 bytes at 16 l.
struct KLoop {
  bf16_t* smem;
  __amdgpu_buffer_rsrc_t ra, rb;   // buffer descriptors of the A tile and the expert's packed B
  int a_lane[2];                   // per-lane A byte offsets for even / odd j
  int b_lane;                      // per-lane B byte offset (16 l)
  int a_row0;                      // first A row (within the tile) of the wave's load blocks
  int b_tile;                      // byte offset of the wave's first B KB at the item's first stage
  int b_stage;                     // bytes from one K stage's blocks to the next one's
  int row_bytes;                   // K * 2
  int lds_a_load, lds_b_load;      // LDS element offsets of the wave's first A / B load rows
  int lds_a, lds_b;                // LDS element offsets of this lane's fragment rows (chunk-free)
  int sw;                          // this lane's fragment swizzle ((row >> 1) & 7)
  int nk, khalf;
};

template <class C>
struct Frags {
  bf16x8 a[C::MB], b[C::NB];
};

// Load j of the wave's A resp. B loads of stage s (K columns 64 s ..
// 64 s + 63) into A resp. B slot `slot`; issue_a issues all A loads of a stage,
// issue_b_part a quarter of the B loads.
__device__ __forceinline__ void load16_lds(__amdgpu_buffer_rsrc_t r, bf16_t* lds, int voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds, 16, voff, soff, 0, 0);
}
template <class C>
__device__ __forceinline__ void load_a(const KLoop& L, int s, int slot, int j) {
  load16_lds(L.ra, L.smem + slot * C::A_ELEMS + L.lds_a_load + j * 8 * BK, L.a_lane[j & 1],
             (L.a_row0 + 8 * j) * L.row_bytes + s * BK * 2);
}
template <class C>
__device__ __forceinline__ void load_b(const KLoop& L, int s, int slot, int j) {
  load16_lds(L.rb, L.smem + C::B_RING + slot * C::B_ELEMS + L.lds_b_load + j * 8 * BK, L.b_lane,
             L.b_tile + s * L.b_stage + j * 1024);
}
template <class C>
__device__ __forceinline__ void issue_a(const KLoop& L, int s, int slot) {
#pragma unroll
  for (int j = 0; j < C::A_LOADS; ++j) load_a<C>(L, s, slot, j);
}
// Part q (q < BK/16) of the B loads of stage s: loads j = q*kBPart .. +kBPart-1.
template <class C>
__device__ __forceinline__ void issue_b_part(const KLoop& L, int s, int slot, int q) {
#pragma unroll
  for (int i = 0; i < kBPart; ++i) load_b<C>(L, s, slot, q * kBPart + i);
}
template <class C>
__device__ __forceinline__ void issue_b(const KLoop& L, int s, int slot) {
#pragma unroll
  for (int q = 0; q < BK / 16; ++q) issue_b_part<C>(L, s, slot, q);
}

// Load order.  Stage t's A loads and the first quarter of its B loads are
// issued right after the barrier of step t-SA resp. t-SB, A first; the other
// three quarters of B(t) go out before the first three k-steps of the step
// after that, one quarter each, so no wave issues a burst of loads at once.
// The prologue issues stages 0 .. SB-1 in the same order as if the steps
// -SB .. -1 had run (the last three quarters of B(SB-1) go out in step 0).
// Every load is issued, also for stages past the item's last one: those load
// the last stage again into a slot that is never read, so the number of loads
// in flight at every wait is a constant.  Loads complete in issue order, so
// "A(t) and B(t) have landed" is "at most n loads are in flight", n = the
// loads issued after the later of the two.
template <class C>
struct LoadOrder {
  // loads after the last load of stage 0, when the prologue waits
  static constexpr int after_stage0() {
    int n = 0;
    bool after = false;
    for (int j = -C::SB; j < 0; ++j) {
      if (j + C::SA >= 0) {
        if (after) n += C::A_LOADS;
        if (j + C::SA == 0 && C::SB == C::SA + 1) after = true;  // A(0) comes after all of B(0)
      }
      if (j + C::SB >= 0) {
        if (after) n += kBPart;
        if (j + 1 < 0) {
          if (after) n += kBLoads - kBPart;
          if (j + C::SB == 0 && C::SB == C::SA) after = true;    // B(0) ends after A(0)
        }
      }
    }
    return n;
  }
  // loads after the last load of stage kt+1, when step kt waits
  static constexpr int after_next() {
    return C::SB == C::SA ? (C::SA - 2) * (C::A_LOADS + kBLoads)
                          : kBLoads + (C::SA - 2) * (C::A_LOADS + kBLoads);
  }
  static_assert(after_next() < 64 && after_stage0() < 64, "vmcnt range");
};

// Fragment rows of one lane: A rows wm*TM + mb*32 + lrow, B rows
// wn*TN + nb*32 + lrow; (row >> 1) & 7 = (lrow >> 1) & 7 for all of them, so
// one chunk term per k-step serves every block and the block offsets are
// immediates.
template <class C>
__device__ __forceinline__ const bf16_t* frag_base_a(const KLoop& L, int slot, int ks) {
  return L.smem + slot * C::A_ELEMS + ((ks * 2 + L.khalf) ^ L.sw) * 8 + L.lds_a;
}
template <class C>
__device__ __forceinline__ const bf16_t* frag_base_b(const KLoop& L, int slot, int ks) {
  return L.smem + C::B_RING + slot * C::B_ELEMS + ((ks * 2 + L.khalf) ^ L.sw) * 8 + L.lds_b;
}
template <class C, int NACT>
__device__ __forceinline__ void read_frags(const KLoop& L, int slot_a, int slot_b, int ks, Frags<C>& f) {
  const bf16_t* ba = frag_base_a<C>(L, slot_a, ks);
  const bf16_t* bb = frag_base_b<C>(L, slot_b, ks);
#pragma unroll
  for (int nb = 0; nb < C::NB; ++nb) f.b[nb] = *reinterpret_cast<const bf16x8*>(bb + nb * 32 * BK);
#pragma unroll
  for (int mb = 0; mb < NACT; ++mb) f.a[mb] = *reinterpret_cast<const bf16x8*>(ba + mb * 32 * BK);
}

// Buffer loads placed in one k-step: the first NA are A loads 0..NA-1 of
// stage a_s into A slot a_slot, the rest B loads b_j0, b_j0+1, ... of stage
// b_s into B slot b_slot.
struct StepLoads {
  int a_s, a_slot, b_s, b_slot, b_j0;
};
template <class C, int NA>
__device__ __forceinline__ void step_load(const KLoop& L, const StepLoads& ld, int j) {
  if (j < NA) load_a<C>(L, ld.a_s, ld.a_slot, j);
  else load_b<C>(L, ld.b_s, ld.b_slot, ld.b_j0 + j - NA);
}

// One k-step in a fixed issue order.  Its MFMAs run block row by block row
// (mb-major); the other work goes between them: first the fragment reads of
// the next k-step, B blocks then A blocks (the order in which that k-step's
// MFMAs consume them), then the V buffer loads of `ld`.  Op j of
// those R + V goes right after MFMA (j M) / (R + V), so every fragment is
// read at least M - R MFMAs before its first use and no wave issues a burst
// of loads.  Scheduling barriers fence each instruction group: the machine
// scheduler would otherwise move reads next to their consumers, which
// exposes the LDS latency.
// TR: the MFMA takes the weight fragment as its first operand, so the 32 x 32
// accumulator block is (weight row, token row): lane l holds token row
// l % 32 and weight rows 8 (v / 4) + 4 (l / 32) + v % 4, four consecutive
// output columns per group of four registers.  Otherwise the block is
// (token row, weight row): lane l holds output column l % 32 of token rows
// 8 (v / 4) + 4 (l / 32) + v % 4.  Either way every output is the same chain
// of MFMAs over K.
template <class C, int NACT, int NA, int V, bool TR>
__device__ __forceinline__ void kstep(const KLoop& L, const Frags<C>& cur, Frags<C>& nxt, int slot_a, int slot_b,
                                      int ks_next, floatx16 (&acc)[C::MB][C::NB], const StepLoads& ld) {
  constexpr int M = NACT * C::NB;
  constexpr int R = NACT > 0 ? C::NB + NACT : 0;
  constexpr int OPS = R + V;
  if constexpr (M == 0) {
#pragma unroll
    for (int j = 0; j < V; ++j) step_load<C, NA>(L, ld, j);
  } else {
    const bf16_t* ba = frag_base_a<C>(L, slot_a, ks_next);
    const bf16_t* bb = frag_base_b<C>(L, slot_b, ks_next);
#pragma unroll
    for (int i = 0; i < M; ++i) {
      const int mb = i / C::NB, nb = i % C::NB;
      if constexpr (TR)
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur.b[nb], cur.a[mb], acc[mb][nb], 0, 0, 0);
      else
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur.a[mb], cur.b[nb], acc[mb][nb], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < OPS; ++j) {
        if ((j * M) / OPS == i) {
          if (j < C::NB)
            nxt.b[j] = *reinterpret_cast<const bf16x8*>(bb + j * 32 * BK);
          else if (j < R)
            nxt.a[j - C::NB] = *reinterpret_cast<const bf16x8*>(ba + (j - C::NB) * 32 * BK);
          else
            step_load<C, NA>(L, ld, j - R);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  }
}

// One item's K loop.  Stage s (K columns 64 s .. 64 s + 63) lives in A slot
// s % SA and B slot s % SB.  In step kt the four k-steps of stage kt run with
// the next k-step's fragments read ahead; before the MFMAs of the last k-step
// the wave waits for its reads of stage kt and its loads of stage kt+1, the
// barrier publishes stage kt+1 and frees the slots of stage kt, A(kt+SA) and
// B(kt+SB) are issued into them (see the load order above) and the first
// fragments of stage kt+1 are read.  NACT = active 32-row blocks of the wave's
// rows (inactive blocks of a ragged tile get neither LDS reads nor MFMAs).
template <class C, int NACT, bool TR>
__device__ __forceinline__ void k_loop(const KLoop& L, floatx16 (&acc)[C::MB][C::NB]) {
  const int nk = L.nk, last = nk - 1;
#pragma unroll
  for (int j = -C::SB; j < 0; ++j) {
    if (j + C::SA >= 0) issue_a<C>(L, min(j + C::SA, last), j + C::SA);
    if (j + C::SB >= 0) {
      issue_b_part<C>(L, min(j + C::SB, last), j + C::SB, 0);
      if (j + 1 < 0)
#pragma unroll
        for (int q = 1; q < BK / 16; ++q) issue_b_part<C>(L, min(j + C::SB, last), j + C::SB, q);
    }
  }
  int pb_s = min(C::SB - 1, last), pb_slot = C::SB - 1;  // B stage with quarters still to issue
  wait_vm<LoadOrder<C>::after_stage0()>();
  bar();
  Frags<C> f[2];
  if (NACT > 0) read_frags<C, NACT>(L, 0, 0, 0, f[0]);
  int ca = 0, cb = 0;  // slots of stage kt
  for (int kt = 0; kt < nk; ++kt) {
#pragma unroll
    for (int ks = 0; ks < kKsteps - 1; ++ks) {
      const StepLoads ld{0, 0, pb_s, pb_slot, (ks + 1) * kBPart};
      kstep<C, NACT, 0, kBPart, TR>(L, f[ks & 1], f[(ks + 1) & 1], ca, cb, ks + 1, acc, ld);
    }
    // every fragment of stage kt is in registers, stage kt+1 has landed
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    wait_vm<LoadOrder<C>::after_next()>();
    bar();
    pb_s = min(kt + C::SB, last);
    pb_slot = cb;
    const StepLoads ld{min(kt + C::SA, last), ca, pb_s, pb_slot, 0};
    const int na = ca + 1 == C::SA ? 0 : ca + 1;
    const int nb = cb + 1 == C::SB ? 0 : cb + 1;
    kstep<C, NACT, C::A_LOADS, C::A_LOADS + kBPart, TR>(L, f[(kKsteps - 1) & 1], f[0], na, nb, 0, acc, ld);
    ca = na;
    cb = nb;
  }
  // the loads of the stages past the last one must land before the next
  // item's prologue writes the same LDS slots
  wait_vm<0>();
}

// K loop of the wave's nact active 32-row blocks (a compile-time count).
template <class C, bool TR>
__device__ __forceinline__ void k_loop_nact(const KLoop& kl, floatx16 (&acc)[C::MB][C::NB], int nact) {
  if constexpr (C::MB == 4) {
    switch (nact) {
      case 4: k_loop<C, 4, TR>(kl, acc); break;
      case 3: k_loop<C, 3, TR>(kl, acc); break;
      case 2: k_loop<C, 2, TR>(kl, acc); break;
      case 1: k_loop<C, 1, TR>(kl, acc); break;
      default: k_loop<C, 0, TR>(kl, acc); break;
    }
  } else if constexpr (C::MB == 2) {
    switch (nact) {
      case 2: k_loop<C, 2, TR>(kl, acc); break;
      case 1: k_loop<C, 1, TR>(kl, acc); break;
      default: k_loop<C, 0, TR>(kl, acc); break;
    }
  } else {
    static_assert(C::MB == 1, "tile shape");
    if (nact == 1) k_loop<C, 1, TR>(kl, acc); else k_loop<C, 0, TR>(kl, acc);
  }
}

// Float pair to packed bf16, round to nearest even (one hardware conversion).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){a, b}, bf16x2));
}

// bf16 epilogue of transposed accumulators: acc[mb][nb][4 g + q] is token
// row r0w + mb*32 + lrow (r0w = the wavefront row's first row in the tile)
// and weight row wn*TN + nb*32 + 8 g + 4 khalf + q, i.e. four consecutive
// output columns per g.  Gate/up: blocks nb < NB/2 are gate rows and
// nb + NB/2 the up rows of the same f; h = bf16(SwiGLU(gate, up)).  Down:
// o = bf16(acc).  Blocks past nact were not computed (and may be another
// wavefront row's rows).
template <class C, int MODE>
__device__ __forceinline__ void epilogue_tr(const GroupedProblem& p, const floatx16 (&acc)[C::MB][C::NB],
                                            bf16_t* C_out, int row0, int row_end, int ni, int r0w, int wn,
                                            int nact, int lrow, int khalf) {
#pragma unroll
  for (int mb = 0; mb < C::MB; ++mb) {
    const int row = row0 + r0w + mb * 32 + lrow;
    if (mb >= nact || row >= row_end) continue;
    if constexpr (MODE == MODE_GATEUP) {
#pragma unroll
      for (int nb = 0; nb < C::NB / 2; ++nb) {
        const floatx16& gt = acc[mb][nb];
        const floatx16& up = acc[mb][nb + C::NB / 2];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int f = ni * (BN / 2) + wn * (C::TN / 2) + nb * 32 + 8 * g + 4 * khalf;
          uint2 v;
          v.x = pack_bf16x2(swiglu(gt[4 * g], up[4 * g]), swiglu(gt[4 * g + 1], up[4 * g + 1]));
          v.y = pack_bf16x2(swiglu(gt[4 * g + 2], up[4 * g + 2]), swiglu(gt[4 * g + 3], up[4 * g + 3]));
          *reinterpret_cast<uint2*>(C_out + (size_t)row * p.F + f) = v;
        }
      }
    } else {
#pragma unroll
      for (int nb = 0; nb < C::NB; ++nb) {
        const floatx16& c = acc[mb][nb];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = ni * BN + wn * C::TN + nb * 32 + 8 * g + 4 * khalf;
          uint2 v;
          v.x = pack_bf16x2(c[4 * g], c[4 * g + 1]);
          v.y = pack_bf16x2(c[4 * g + 2], c[4 * g + 3]);
          *reinterpret_cast<uint2*>(C_out + (size_t)row * p.H + n) = v;
        }
      }
    }
  }
}

// One work item (m-tile row0.. of group rows ending at row_end, n-tile ni,
// K stages ks0 .. ks0+nks-1) in tile shape C.  part == nullptr: the item
// covers all of K and writes the output; else it writes its fp32 partial
// sums to part (row-major, N = H columns).
template <class C, int MODE>
__device__ __forceinline__ void run_item(const GroupedProblem& p, bf16_t* smem, const bf16_t* A,
                                         bf16_t* C_out, const bf16_t* Bbase, int row0, int row_end,
                                         int ni, int K, int ks0, int nks, float* part, int wave,
                                         int lane) {
  const int wm = wave / C::WN, wn = wave % C::WN;
  const int lrow = lane & 31, khalf = lane >> 5;
  // rows per wavefront row: the tile's rows split evenly over the WM
  // wavefront rows in whole 32-row blocks (a 150-row tile gives each of two
  // wavefront rows 96 rows, 3 blocks, instead of 128 + 22); the slowest
  // wavefront row sets the item's time
  const int tm = min(C::TM, 32 * ((row_end - row0 + 32 * C::WM - 1) / (32 * C::WM)));
  const int lr = lane >> 3, lp = lane & 7;
  const int k_off = ks0 * BK;  // first K column of the item
  const bf16_t* Atile = A + (size_t)row0 * K + k_off;
  const int a_rows = min(C::BM, p.P - row0);  // rows past it read zeros; their results are discarded

  KLoop kl;
  kl.smem = smem;
  kl.ra = buffer_rsrc(Atile, (uint32_t)(a_rows * K * 2 - k_off * 2));
  const int n_rows = MODE == MODE_GATEUP ? 2 * p.F : p.H;  // the expert matrix is n_rows x K
  kl.rb = buffer_rsrc(Bbase, (uint32_t)n_rows * (uint32_t)K * 2u);
  kl.row_bytes = K * 2;
  {
    // swizzle of the wave's first A load row; odd j flips bit 2
    const int ca = lp ^ ((((C::BM / kWaves) * wave + lr) >> 1) & 7);
    kl.a_lane[0] = lr * K * 2 + ca * 16;
    kl.a_lane[1] = lr * K * 2 + (ca ^ 4) * 16;
    kl.a_row0 = (C::BM / kWaves) * wave;
    kl.b_lane = lane * 16;
    kl.b_stage = (n_rows / BN) * (BN * BK * 2);
    kl.b_tile = ks0 * kl.b_stage + ni * (BN * BK * 2) + wave * (BN / kWaves) * BK * 2;
  }
  kl.lds_a_load = (C::BM / kWaves) * wave * BK;
  kl.lds_b_load = (BN / kWaves) * wave * BK;
  kl.lds_a = (wm * tm + lrow) * BK;
  kl.lds_b = (wn * C::TN + lrow) * BK;
  kl.sw = (lrow >> 1) & 7;
  kl.nk = nks;
  kl.khalf = khalf;

  floatx16 acc[C::MB][C::NB];
#pragma unroll
  for (int i = 0; i < C::MB; ++i)
#pragma unroll
    for (int j = 0; j < C::NB; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // 32-row blocks of this wave's TM rows that hold rows of the group
  const int nact = min(tm / 32, max(0, (row_end - (row0 + wm * tm) + 31) / 32));
  // bf16 outputs use the transposed accumulators (one 8-byte store per four
  // consecutive columns); fp32 partial sums the row layout (32 lanes store a
  // whole 128-byte line)
  if (MODE == MODE_GATEUP || part == nullptr) {
    k_loop_nact<C, true>(kl, acc, nact);
    __syncthreads();  // every wave is done with the ring before the next item refills it
    epilogue_tr<C, MODE>(p, acc, C_out, row0, row_end, ni, wm * tm, wn, nact, lrow, khalf);
  } else if constexpr (MODE == MODE_DOWN) {
    k_loop_nact<C, false>(kl, acc, nact);
    __syncthreads();
    // acc[mb][nb][v]: output column wn*TN + nb*32 + lrow of token row
    // wm*tm + mb*32 + 8 (v / 4) + 4 khalf + v % 4
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb) {
      if (mb >= nact) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = row0 + wm * tm + mb * 32 + 8 * (v >> 2) + 4 * khalf + (v & 3);
        if (row >= row_end) continue;
#pragma unroll
        for (int nb = 0; nb < C::NB; ++nb)
          part[(size_t)row * p.H + ni * BN + wn * C::TN + nb * 32 + lrow] = acc[mb][nb][v];
      }
    }
  }
}

// Persistent grouped GEMM.  Work item = (group, n-tile, m-tile); a group of
// R rows has ceil(R / 256) m-tiles sharing its rows evenly, enumerated group
// by group, then by blocks of kMBlock m-tiles, n-tile-major inside a block,
// m-tile fastest, so consecutive items share the weight tile and, running at
// the same pace, read each weight stage from L2 once (unequal m-tiles drift
// apart and fetch the weights again: 2.2-3.5x the weight bytes for two to
// three m-tiles).  The blocks bound how often a large group's activation rows
// are streamed: once per window of n-tiles rather than once per n-tile (with
// tens of m-tiles, 28 times over for a 7168-wide down projection).  Workgroup b runs on XCD b % 8 (round-robin
// dispatch) and takes items from its XCD's contiguous eighth of the list
// through that XCD's atomic counter, so items running together on one L2
// share weight and activation tiles and no workgroup idles while its XCD has
// work; once its XCD's range is drained it takes items from the other XCDs'
// ranges.  Every item is taken exactly once whichever workgroup takes it.
// The counter increment for the next item is issued at the start of the
// current one and its result used at its end.  Each item runs in the tile
// shape of the rows it holds; all shapes accumulate K in the same order, so a
// row's result does not depend on the shape or on which workgroup ran it.
// m-tiles per block of the item order (see grouped_gemm_bf16): a window of
// the 32 items one XCD runs at a time then spans 4 m-tiles x 8 n-tiles, so
// it streams 4 activation and 8 weight tiles instead of 32 and 1.
constexpr int kMBlock = 4;

template <int MODE>
__global__ __launch_bounds__(kThreads, 1) void grouped_gemm_bf16(GroupedProblem p, WeightTable wt,
                                                                 const bf16_t* __restrict__ A,
                                                                 bf16_t* __restrict__ C,
                                                                 int n_ntiles) {
  __shared__ __attribute__((aligned(1024))) bf16_t smem[kLdsElems];
  // the next item index is broadcast through the first word of the ring,
  // which no load writes between an item's last K stage and the next prologue
  int* s_next = reinterpret_cast<int*>(smem);
  // the LDS ring is written by global->LDS loads the compiler does not see
  asm volatile("" ::"v"(smem) : "memory");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int xcd = blockIdx.x % kXcds;
  const int ksplit = MODE == MODE_DOWN ? p.ksplit : 1;
  const int nsub = n_ntiles * ksplit;  // items per m-tile
  const long long total = (long long)(*p.n_tiles) * nsub;
  auto range_lo = [&](int x) { return (int)((x * total) / kXcds); };
  const int K = MODE == MODE_GATEUP ? p.H : p.F;
  const int ES = p.E + p.S;

  // thread 0: the XCD whose range it draws from, and the first item
  int victim = xcd;
  auto settle = [&](int got) {  // item index from a counter value of victim's range, or -1
    int it = range_lo(victim) + got;
    while (it >= range_lo(victim + 1)) {
      victim = victim + 1 == kXcds ? 0 : victim + 1;
      if (victim == xcd) return -1;
      it = range_lo(victim) + atomicAdd(&p.work_ctr[victim], 1);
    }
    return it;
  };
  if (tid == 0) *s_next = settle(atomicAdd(&p.work_ctr[victim], 1));
  __syncthreads();
  int it = *s_next;
  __syncthreads();

  while (it >= 0) {
    int got = 0;
    if (tid == 0) got = atomicAdd(&p.work_ctr[victim], 1);
    // group of this item: a group's items it * nsub .. (it + mt) * nsub - 1
    // cover its m-tiles it .. it + mt - 1, so item / nsub is one of them
    const int4 gd = p.tiles[it / nsub];  // key, first row, rows, first m-tile
    const int mt = (gd.z + BM - 1) / BM;
    // within the group: K part slowest, then blocks of kMBlock m-tiles, then
    // n-tile, m-tile fastest (the last block holds the mt % kMBlock rest)
    const int local = it - gd.w * nsub;
    const int kh = local / (mt * n_ntiles);
    const int rem = local - kh * mt * n_ntiles;
    const int mb = rem / (kMBlock * n_ntiles);
    const int gm = min(kMBlock, mt - mb * kMBlock);
    const int rb = rem - mb * kMBlock * n_ntiles;
    const int ni = rb / gm, mi = mb * kMBlock + (rb - ni * gm);
    const int nks = K / BK / ksplit, ks0 = kh * nks;
    float* part = ksplit > 1 ? p.partial + (size_t)kh * p.P * p.H : nullptr;
    // the group's mt m-tiles share its rows evenly (whole 32-row blocks), so
    // they run at the same pace and meet the same weight stages in L2
    const int rpt = 32 * ((gd.z + 32 * mt - 1) / (32 * mt));
    const int row0 = gd.y + mi * rpt, row_end = min(gd.y + gd.z, row0 + rpt);
    const int layer = gd.x / ES, e = gd.x - layer * ES;
    const bf16_t* Bbase = MODE == MODE_GATEUP
        ? static_cast<const bf16_t*>(wt.gu[layer]) + (size_t)e * 2 * p.F * p.H
        : static_cast<const bf16_t*>(wt.dn[layer]) + (size_t)e * p.H * p.F;
    const int rows = row_end - row0;
    if (rows > CfgMid::BM)
      run_item<CfgBig, MODE>(p, smem, A, C, Bbase, row0, row_end, ni, K, ks0, nks, part, wave, lane);
    else if (rows > CfgSkinny::BM)
      run_item<CfgMid, MODE>(p, smem, A, C, Bbase, row0, row_end, ni, K, ks0, nks, part, wave, lane);
    else
      run_item<CfgSkinny, MODE>(p, smem, A, C, Bbase, row0, row_end, ni, K, ks0, nks, part, wave, lane);
    if (tid == 0) *s_next = settle(got);
    __syncthreads();
    it = *s_next;
    __syncthreads();  // every thread has read it before the next prologue refills the ring
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
  const int4 td = p.tiles[tile];  // the tile's group
  const int key = td.x, row0 = td.y + (tile - td.w) * FBM;
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

// o = dtype(p0 + p1) for the K halves of a split down GEMM, 4 elements per
// thread over the live rows *P_live (H is a multiple of 256); the second
// half starts `stride` floats after the first.
__global__ __launch_bounds__(256) void split_sum_kernel(const float* __restrict__ part, long long stride,
                                                        const int32_t* __restrict__ P_live, int H,
                                                        bf16_t* __restrict__ o) {
  const long long i = ((long long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= (long long)(*P_live) * H) return;
  const float4 a = *reinterpret_cast<const float4*>(part + i);
  const float4 b = *reinterpret_cast<const float4*>(part + stride + i);
  uint2 u;
  u.x = (uint32_t)f32_to_bf16(a.x + b.x) | ((uint32_t)f32_to_bf16(a.y + b.y) << 16);
  u.y = (uint32_t)f32_to_bf16(a.z + b.z) | ((uint32_t)f32_to_bf16(a.w + b.w) << 16);
  *reinterpret_cast<uint2*>(o + i) = u;
}

// Packed bf16 expert weights.  An expert matrix W [N][K] (gate/up: N = 2F
// rows, gate rows f then up rows F + f, K = H; down: N = H, K = F) becomes
// (K / 64) x (N / 256) blocks of 256 x 64 elements (32 KB), block (s, t) at
// index s * (N / 256) + t holding K columns 64 s .. 64 s + 63 of column tile
// t.  Block row r is weight row
//   down:     256 t + r
//   gate/up:  128 t + 32 (r / 64) + (r % 64 < 32 ? r % 64 : r % 64 - 32 + F)
// (the 64 rows of wavefront column r / 64 are 32 gate rows and the matching
// 32 up rows), and its 16-byte chunk at position c holds the 8 K columns
// 64 s + 8 (c ^ ((r >> 1) & 7)) .. + 7 (the LDS swizzle of the ring).
// One thread per 16-byte chunk of dst; n matrices back to back.
__global__ __launch_bounds__(256) void pack_bf16_kernel(const uint4* __restrict__ src,
                                                        uint4* __restrict__ dst, long long chunks,
                                                        int N, int K, int F, int gateup) {
  const long long per_mat = (long long)N * K / 8;
  const int ntiles = N / BN;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < chunks;
       i += (long long)gridDim.x * blockDim.x) {
    const long long mat = i / per_mat;
    const int rem = (int)(i - mat * per_mat);
    const int blk = rem / (BN * BK / 8), in = rem - blk * (BN * BK / 8);
    const int r = in >> 3, c = in & 7;
    const int st = blk / ntiles, t = blk - st * ntiles;
    int row;
    if (gateup) {
      const int q = r & 63;
      row = t * (BN / 2) + (r >> 6) * 32 + (q < 32 ? q : q - 32 + F);
    } else {
      row = t * BN + r;
    }
    const int col = st * BK + 8 * swz(r, c);
    dst[i] = src[mat * per_mat + ((long long)row * K + col) / 8];
  }
}

}  // namespace

int gemm_bm(int dtype) { return dtype == EB_DTYPE_BF16 ? BM : FBM; }

hipError_t launch_pack_weights(int dtype, int gateup, int n, int N, int K, int F, const void* src,
                               void* dst, hipStream_t s) {
  const size_t elem = dtype == EB_DTYPE_BF16 ? 2 : 4;
  const size_t bytes = (size_t)n * N * K * elem;
  if (bytes == 0) return hipSuccess;
  if (dtype != EB_DTYPE_BF16) return hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, s);
  const long long chunks = (long long)(bytes / 16);
  const long long want = (chunks + 255) / 256;
  const unsigned grid = (unsigned)(want < 65536 ? want : 65536);
  hipLaunchKernelGGL(pack_bf16_kernel, dim3(grid), dim3(256), 0, s, static_cast<const uint4*>(src),
                     static_cast<uint4*>(dst), chunks, N, K, F, gateup);
  return hipGetLastError();
}

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
                       void* o, hipStream_t s, bool sum_halves) {
  prof_start(EB_K_DOWN, s);
  if (dtype == EB_DTYPE_BF16) {
    hipLaunchKernelGGL(grouped_gemm_bf16<MODE_DOWN>, dim3(persistent_grid()), dim3(kThreads), 0, s,
                       p, wt, static_cast<const bf16_t*>(h), static_cast<bf16_t*>(o), p.H / BN);
    if (p.ksplit > 1 && sum_halves) {
      const long long n = (long long)p.P * p.H;
      hipLaunchKernelGGL(split_sum_kernel, dim3((unsigned)((n / 4 + 255) / 256)), dim3(256), 0, s,
                         p.partial, n, p.P_live, p.H, static_cast<bf16_t*>(o));
    }
  } else {
    hipLaunchKernelGGL(grouped_gemm_f32<MODE_DOWN>, dim3(p.max_tiles, p.H / FBN), dim3(256), 0, s,
                       p, wt, static_cast<const float*>(h), static_cast<float*>(o));
  }
  prof_stop(EB_K_DOWN, s);
  return hipGetLastError();
}

}  // namespace eb
