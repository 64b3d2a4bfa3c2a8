// Routing of one micro-batch at one layer (Section 2.1: W, I = topk(G(h'))):
//   route_token_kernel   E <= 8 (bf16) / E <= 64 (fp32), H <= 8192: one workgroup
//                        per token computes a = dtype(x * r * gain),
//                        z = a Wg^T + bias and the top-k with its softmax
//                        weights
//   RMSNorm +            other bf16 stacks: RMSNorm, then the router GEMM on
//   route_mfma_kernel /  the matrix cores and the top-k of the workgroup's 32
//   route_lds_kernel     tokens from an LDS logit tile (E <= 64: 32 tokens,
//                        split-K over the 4 wavefronts, operands straight into
//                        registers; E > 64: 128 tokens, 8 wavefronts splitting
//                        tokens and experts, operands staged through LDS as
//                        whole cache lines)
//   RMSNorm +            other fp32 stacks: RMSNorm, an LDS-tiled fp32
//   logits_kernel +      VALU GEMM for z, then the top-k
//   topk_kernel
//   RMSNorm              rmsnorm_row_kernel (H <= 8192: one workgroup per
//                        token, the row read once into registers) or
//                        rmsnorm_kernel (one wavefront per token)
//   counts_kernel        expert counts of each micro-batch from its picks
// Every kernel takes a batch of micro-batches (possibly at different layers)
// and finds its entry from its block index, so routing several micro-batches
// costs one set of launches.
// Every reduction runs in a fixed order, so a token's routing depends on its
// own inputs only (not on the other tokens of the launch).
#include <math.h>

#include "eb_internal.h"
#include "eb_numeric.h"

namespace eb {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Sum of squares of row xr (H floats) by one wavefront: lane l adds the float4
// slices l, l + 64, ... in that order (four slices in flight per iteration);
// the butterfly leaves the bit-identical total in every lane.
__device__ __forceinline__ float row_sumsq(const float4* __restrict__ xr, int n4, int lane) {
  float ss = 0.f;
  int i = lane;
  for (; i + 192 < n4; i += 256) {
    const float4 v0 = xr[i], v1 = xr[i + 64], v2 = xr[i + 128], v3 = xr[i + 192];
    ss = fmaf(v0.x, v0.x, ss); ss = fmaf(v0.y, v0.y, ss); ss = fmaf(v0.z, v0.z, ss); ss = fmaf(v0.w, v0.w, ss);
    ss = fmaf(v1.x, v1.x, ss); ss = fmaf(v1.y, v1.y, ss); ss = fmaf(v1.z, v1.z, ss); ss = fmaf(v1.w, v1.w, ss);
    ss = fmaf(v2.x, v2.x, ss); ss = fmaf(v2.y, v2.y, ss); ss = fmaf(v2.z, v2.z, ss); ss = fmaf(v2.w, v2.w, ss);
    ss = fmaf(v3.x, v3.x, ss); ss = fmaf(v3.y, v3.y, ss); ss = fmaf(v3.z, v3.z, ss); ss = fmaf(v3.w, v3.w, ss);
  }
  for (; i < n4; i += 64) {
    const float4 v = xr[i];
    ss = fmaf(v.x, v.x, ss); ss = fmaf(v.y, v.y, ss); ss = fmaf(v.z, v.z, ss); ss = fmaf(v.w, v.w, ss);
  }
  return wave_sum(ss);
}

// Four consecutive normalised values, stored in the stack's dtype.
__device__ __forceinline__ void store4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
__device__ __forceinline__ void store4(bf16_t* p, float4 v) {
  uint2 u;
  u.x = (uint32_t)f32_to_bf16(v.x) | ((uint32_t)f32_to_bf16(v.y) << 16);
  u.y = (uint32_t)f32_to_bf16(v.z) | ((uint32_t)f32_to_bf16(v.w) << 16);
  *reinterpret_cast<uint2*>(p) = u;
}
__device__ __forceinline__ float4 normed(float4 v, float r, float4 g) {
  return make_float4(v.x * r * g.x, v.y * r * g.y, v.z * r * g.z, v.w * r * g.w);
}

// ---------------------------------------------------------------------------
// RMSNorm + cast, one wavefront per token.
template <typename TA, class RBA>
__global__ __launch_bounds__(256) void rmsnorm_kernel(RBA rba, int H, float eps) {
  const RouteBatch& rb = rba.get();
  const int lane = threadIdx.x & 63;
  const int g = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (g >= rb.tok0[rb.n]) return;
  const int ei = find_entry(rb.tok0, rb.n, g);
  const int t = g - rb.tok0[ei];
  const float* __restrict__ x = in_global(rb.e[ei].x);
  const float* __restrict__ gain = in_global(rb.e[ei].gain);
  TA* __restrict__ a = in_global(static_cast<TA*>(rb.e[ei].a));
  const float4* xr = reinterpret_cast<const float4*>(x + (size_t)t * H);
  const float4* g4 = reinterpret_cast<const float4*>(gain);
  const int n4 = H >> 2;
  const float r = 1.0f / sqrtf(row_sumsq(xr, n4, lane) / (float)H + eps);
  TA* ar = a + (size_t)t * H;
  int i = lane;
  for (; i + 192 < n4; i += 256) {
    const float4 v0 = xr[i], v1 = xr[i + 64], v2 = xr[i + 128], v3 = xr[i + 192];
    const float4 g0 = g4[i], g1 = g4[i + 64], g2 = g4[i + 128], g3 = g4[i + 192];
    store4(ar + 4 * i, normed(v0, r, g0));
    store4(ar + 4 * (i + 64), normed(v1, r, g1));
    store4(ar + 4 * (i + 128), normed(v2, r, g2));
    store4(ar + 4 * (i + 192), normed(v3, r, g3));
  }
  for (; i < n4; i += 64) store4(ar + 4 * i, normed(xr[i], r, g4[i]));
}

// ---------------------------------------------------------------------------
// Top-k and softmax weights of one token by one thread.  zrow(e) gives the
// token's logits e < E.  The picks are kept as a list ordered by the total
// order "larger z first, then lower expert id", built by one ascending pass
// over e with compare-and-swap insertion; NaN never enters the list, so a
// slot left empty means every expert not yet picked has a NaN logit, and it
// takes the lowest such id (NaN ranks after every number, ties by id: the
// k picks are always distinct experts).  The softmax maximum and denominator
// are accumulated over e in ascending order.
__device__ __forceinline__ bool better(float v1, int e1, float v2, int e2) {
  return v1 > v2 || (v1 == v2 && e1 < e2);
}

template <int KMAX, class ZRow>
__device__ __forceinline__ void topk_thread(int E, int k, int norm_topk, ZRow zrow,
                                            int32_t* __restrict__ idx_t, float* __restrict__ w_t) {
  float lv[KMAX];
  int le[KMAX];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    lv[j] = -INFINITY;
    le[j] = E;  // sentinel: loses to every expert
  }
  float mx = -INFINITY;
  for (int e = 0; e < E; ++e) {
    float v = zrow(e);
    mx = fmaxf(mx, v);
    int ve = e;
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      if (j < k && better(v, ve, lv[j], le[j])) {
        const float tv = lv[j];
        const int te = le[j];
        lv[j] = v;
        le[j] = ve;
        v = tv;
        ve = te;
      }
    }
  }
  float se = 0.f;
  for (int e = 0; e < E; ++e) se += expf(zrow(e) - mx);
  float ev[KMAX], esum = 0.f;
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    ev[j] = j < k ? expf(lv[j] - mx) : 0.f;
    esum += ev[j];
  }
  const float denom = norm_topk ? esum : se;
  int fill = 0;  // candidate for the next empty slot (ids ascending)
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    if (j < k) {
      int e = le[j];
      if (e >= E) {
        for (;; ++fill) {
          bool used = false;
#pragma unroll
          for (int i = 0; i < KMAX; ++i) used |= i < j && le[i] == fill;
          if (!used || fill >= E - 1) break;
        }
        e = fill++;
        le[j] = e;
        ev[j] = __builtin_nanf("");
      }
      idx_t[j] = e;
      w_t[j] = ev[j] / denom;
    }
  }
}

// Dispatch on k: KMAX = 8 for k <= 8, else 16.
template <class ZRow>
__device__ __forceinline__ void topk_token(int E, int k, int norm_topk, ZRow zrow,
                                           int32_t* __restrict__ idx_t, float* __restrict__ w_t) {
  if (k <= 8) topk_thread<8>(E, k, norm_topk, zrow, idx_t, w_t);
  else topk_thread<16>(E, k, norm_topk, zrow, idx_t, w_t);
}

// Order key of the logit v of expert e for the top-k: larger z first, then
// lower id; NaN after every number (ties by id); -0 ranks as +0.  The float
// maps to an unsigned integer of the same order (sign flipped for positive
// values, all bits for negative ones), NaN to 1, and the id goes below it as
// ~e, so a pick is one unsigned maximum.  Key 0 (below every expert) marks
// padding.
__device__ __forceinline__ uint64_t pick_key(float v, int e) {
  uint32_t o = 1u;  // NaN
  if (v == v) {
    const uint32_t u = __float_as_uint(v == 0.f ? 0.f : v);
    o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);  // -inf -> 0x007fffff > 1
  }
  return ((uint64_t)o << 32) | (uint32_t)~(uint32_t)e;
}
__device__ __forceinline__ float key_value(uint64_t key) {
  const uint32_t o = (uint32_t)(key >> 32);
  if (o == 1u) return __builtin_nanf("");
  return __uint_as_float((o & 0x80000000u) ? (o ^ 0x80000000u) : ~o);
}

// Top-k and softmax weights of one token by 8 consecutive lanes (sub = lane
// % 8): lane sub holds the keys of the logits e = sub + 8 i (i < PER) and each
// pick is the maximum key over the 8 lanes (the total order above: when only
// NaN logits are left, the lowest unpicked id, so the k picks are distinct
// experts); the softmax maximum and denominator are reduced over the 8 lanes
// in a fixed pattern.  The picks stay in registers (k <= KMAX) and lane sub 0
// writes idx_t and w_t once.
template <int PER, int KMAX>
__device__ __forceinline__ void topk_group8(int sub, int E, int k, int norm_topk, const float* zrow,
                                            int32_t* __restrict__ idx_t, float* __restrict__ w_t) {
  static_assert(PER <= 32, "taken mask");
  uint64_t key[PER];
  uint32_t taken = 0;  // entries already picked
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int e = sub + 8 * i;
    const float v = zrow[min(e, E - 1)];  // entries past E are padding
    mx = fmaxf(mx, e < E ? v : -INFINITY);
    key[i] = e < E ? pick_key(v, e) : 0ull;
  }
#pragma unroll
  for (int off = 1; off < 8; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 8));
  float se = 0.f;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const float ev = expf(key_value(key[i]) - mx);
    se += sub + 8 * i < E ? ev : 0.f;  // +0 leaves the (non-negative) sum's bits alone
  }
#pragma unroll
  for (int off = 1; off < 8; off <<= 1) se += __shfl_xor(se, off, 8);
  float esum = 0.f;
  float pw[KMAX];
  int pe[KMAX];
#pragma unroll
  for (int r = 0; r < KMAX; ++r) {
    pw[r] = 0.f;
    pe[r] = 0;
    if (r < k) {
      uint64_t best = 0;
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const uint64_t ki = (taken >> i) & 1u ? 0ull : key[i];
        best = ki > best ? ki : best;
      }
#pragma unroll
      for (int off = 1; off < 8; off <<= 1) {
        const uint64_t o = __shfl_xor(best, off, 8);
        best = o > best ? o : best;
      }
      int be = (int)~(uint32_t)best;
      be = (be < 0 || be >= E) ? E - 1 : be;  // not reached: r < k <= E leaves an unpicked expert
      if ((be & 7) == sub) taken |= 1u << (be >> 3);
      const float ev = expf(key_value(best) - mx);
      esum += ev;
      pw[r] = ev;
      pe[r] = be;
    }
  }
  if (sub == 0) {
    const float denom = norm_topk ? esum : se;
#pragma unroll
    for (int r = 0; r < KMAX; ++r)
      if (r < k) {
        idx_t[r] = pe[r];
        w_t[r] = pw[r] / denom;
      }
  }
}

// Expert counts of a micro-batch from its picks, one workgroup per batch entry
// (an LDS histogram, then one plain store per expert: nothing to clear
// beforehand; an entry without tokens gets zeros).
template <class RBA>
__global__ __launch_bounds__(1024) void counts_kernel(RBA rba, int k, int E) {
  const RouteBatch& rb = rba.get();
  const int ei = blockIdx.x;
  if (ei >= rb.n) return;  // past the live entries (grid sized for a full batch)
  const int n = (rb.tok0[ei + 1] - rb.tok0[ei]) * k;
  const int32_t* __restrict__ idx = in_global(rb.e[ei].idx);
  int32_t* __restrict__ counts = in_global(rb.e[ei].counts);
  __shared__ int hist[1024];
  for (int e = threadIdx.x; e < E; e += blockDim.x) hist[e] = 0;
  __syncthreads();
  for (int i = threadIdx.x; i < n; i += blockDim.x) atomicAdd(&hist[idx[i]], 1);
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x) counts[e] = hist[e];
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

// RMSNorm + cast, one workgroup of 256 threads per token for long rows:
// thread t holds the float4 slices t + 256 v (v < NV) of the row in
// registers, so x is read once.  Sums of squares: each thread over its
// slices in order, a butterfly per wavefront, then the 4 wavefronts in order.
template <typename TA, int NV, class RBA>
__global__ __launch_bounds__(256) void rmsnorm_row_kernel(RBA rba, int H, float eps) {
  __shared__ float red[4];
  const RouteBatch& rb = rba.get();
  const int g = blockIdx.x;
  if (g >= rb.tok0[rb.n]) return;  // past the live tokens
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ei = find_entry(rb.tok0, rb.n, g);
  const int t = g - rb.tok0[ei];
  const float4* xr = reinterpret_cast<const float4*>(in_global(rb.e[ei].x) + (size_t)t * H);
  const float4* g4 = reinterpret_cast<const float4*>(in_global(rb.e[ei].gain));
  TA* ar = in_global(static_cast<TA*>(rb.e[ei].a)) + (size_t)t * H;
  const int n4 = H >> 2;
  float4 v[NV], gv[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = tid + 256 * j;
    if (i < n4) {
      v[j] = xr[i];
      gv[j] = g4[i];
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NV; ++j)
    if (tid + 256 * j < n4) {
      ss = fmaf(v[j].x, v[j].x, ss); ss = fmaf(v[j].y, v[j].y, ss);
      ss = fmaf(v[j].z, v[j].z, ss); ss = fmaf(v[j].w, v[j].w, ss);
    }
  ss = wave_sum(ss);
  if (lane == 0) red[wave] = ss;
  __syncthreads();
  const float r = 1.0f / sqrtf((((red[0] + red[1]) + red[2]) + red[3]) / (float)H + eps);
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = tid + 256 * j;
    if (i < n4) store4(ar + 4 * i, normed(v[j], r, gv[j]));
  }
}

// ---------------------------------------------------------------------------
// Whole routing of one token for E <= EMAX by one workgroup of 256 threads.
// Thread tid owns the 8-element chunks starting at h = 8 (tid + 256 i), held
// in registers; per chunk it forms and stores the a values and adds their
// (stored, rounded) values times every router row into one accumulator per
// expert.  Sums of squares are reduced by a butterfly per wavefront and then
// over the 4 wavefronts in order, and so are the logits; with E <= 8 the
// per-wavefront logit sums take a reduce-scatter instead (10 lane exchanges
// for the 8 sums rather than 48), the router rows of a chunk are loaded
// together, and 8 lanes of wavefront 0 pick the top-k; otherwise thread 0
// picks it.
template <typename TA> struct Vec8;
template <> struct Vec8<bf16_t> {
  using Raw = uint4;
  __device__ static __forceinline__ Raw load_raw(const bf16_t* p) { return *reinterpret_cast<const uint4*>(p); }
  __device__ static __forceinline__ void unpack(const Raw& u, float (&f)[8]) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      f[2 * q] = __uint_as_float(w[q] << 16);
      f[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);
    }
  }
  // 8 bf16 of a router row / of a
  __device__ static __forceinline__ void load(const bf16_t* p, float (&f)[8]) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      f[2 * q] = __uint_as_float(w[q] << 16);
      f[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);
    }
  }
  // stores dtype(v) and replaces v by it
  __device__ static __forceinline__ void store_round(bf16_t* p, float (&v)[8]) {
    uint32_t w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const bf16_t lo = f32_to_bf16(v[2 * q]), hi = f32_to_bf16(v[2 * q + 1]);
      w[q] = (uint32_t)lo | ((uint32_t)hi << 16);
      v[2 * q] = bf16_to_f32(lo);
      v[2 * q + 1] = bf16_to_f32(hi);
    }
    *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
  }
};
template <> struct Vec8<float> {
  struct Raw { float4 u, v; };
  __device__ static __forceinline__ Raw load_raw(const float* p) {
    return Raw{reinterpret_cast<const float4*>(p)[0], reinterpret_cast<const float4*>(p)[1]};
  }
  __device__ static __forceinline__ void unpack(const Raw& r, float (&f)[8]) {
    f[0] = r.u.x; f[1] = r.u.y; f[2] = r.u.z; f[3] = r.u.w; f[4] = r.v.x; f[5] = r.v.y; f[6] = r.v.z; f[7] = r.v.w;
  }
  __device__ static __forceinline__ void load(const float* p, float (&f)[8]) {
    const float4 u = reinterpret_cast<const float4*>(p)[0], v = reinterpret_cast<const float4*>(p)[1];
    f[0] = u.x; f[1] = u.y; f[2] = u.z; f[3] = u.w; f[4] = v.x; f[5] = v.y; f[6] = v.z; f[7] = v.w;
  }
  __device__ static __forceinline__ void store_round(float* p, float (&v)[8]) {
    reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
    reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
};

constexpr int kTokChunks = 4;  // 8-element chunks per thread: H <= 256 * 8 * 4
constexpr int kTokMaxH = 256 * 8 * kTokChunks;

// KC: 8-element chunks per thread (H <= 256 * 8 * KC).  The 2-chunk form for
// H <= 4096 fits 64 registers, so a CU holds 8 of these workgroups (a
// 2048-token launch in one round).
template <typename TA, int EMAX, int KC, class RBA>
__global__ __launch_bounds__(256, KC == 2 ? 8 : 1) void route_token_kernel(RBA rba, int H, int E, int k,
                                                                           int norm_topk, float eps) {
  __shared__ float red[4];
  __shared__ float red_z[4][EMAX + 1];
  const RouteBatch& rb = rba.get();
  if ((int)blockIdx.x >= rb.tok0[rb.n]) return;  // past the live tokens
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ei = find_entry(rb.tok0, rb.n, blockIdx.x);
  const int t = blockIdx.x - rb.tok0[ei];
  const float* __restrict__ x = in_global(rb.e[ei].x);
  const float* __restrict__ gain = in_global(rb.e[ei].gain);
  const TA* __restrict__ Wg = in_global(static_cast<const TA*>(rb.e[ei].Wg));
  const float* __restrict__ bias = in_global(rb.e[ei].bias);
  TA* __restrict__ a = in_global(static_cast<TA*>(rb.e[ei].a));
  float* __restrict__ z = in_global(rb.e[ei].z);
  int32_t* __restrict__ idx = in_global(rb.e[ei].idx);
  float* __restrict__ w = in_global(rb.e[ei].w);
  const float* xr = x + (size_t)t * H;
  const int nchunk = H >> 3;
  // thread tid owns chunks c = tid + 256 i (8 elements each), kept in registers
  float xs[KC][8];
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < KC; ++i) {
    const int c = tid + 256 * i;
    if (c < nchunk) {
      const float4 u = reinterpret_cast<const float4*>(xr + 8 * c)[0];
      const float4 v = reinterpret_cast<const float4*>(xr + 8 * c)[1];
      xs[i][0] = u.x; xs[i][1] = u.y; xs[i][2] = u.z; xs[i][3] = u.w;
      xs[i][4] = v.x; xs[i][5] = v.y; xs[i][6] = v.z; xs[i][7] = v.w;
    }
  }
#pragma unroll
  for (int i = 0; i < KC; ++i)
    if (tid + 256 * i < nchunk)
#pragma unroll
      for (int q = 0; q < 8; ++q) ss = fmaf(xs[i][q], xs[i][q], ss);
  ss = wave_sum(ss);
  if (lane == 0) red[wave] = ss;
  __syncthreads();
  const float r = 1.0f / sqrtf((((red[0] + red[1]) + red[2]) + red[3]) / (float)H + eps);
  float acc[EMAX];
#pragma unroll
  for (int e = 0; e < EMAX; ++e) acc[e] = 0.f;
  TA* ar = a + (size_t)t * H;
#pragma unroll
  for (int i = 0; i < KC; ++i) {
    const int c = tid + 256 * i;
    if (c < nchunk) {
      const int h = 8 * c;
      const float4 gu = reinterpret_cast<const float4*>(gain + h)[0];
      const float4 gv = reinterpret_cast<const float4*>(gain + h)[1];
      const float g[8] = {gu.x, gu.y, gu.z, gu.w, gv.x, gv.y, gv.z, gv.w};
      float av[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) av[q] = xs[i][q] * r * g[q];
      Vec8<TA>::store_round(ar + h, av);  // the stored (rounded) values feed the router
      if constexpr (EMAX == 8) {
        // the router rows in batches of RB whose loads are in flight together
        // (rows past E repeat row E-1; their sums are never used)
        constexpr int RB = sizeof(TA) == 2 ? 8 : 2;
#pragma unroll
        for (int e0 = 0; e0 < 8; e0 += RB) {
          typename Vec8<TA>::Raw wr[RB];
#pragma unroll
          for (int j = 0; j < RB; ++j) wr[j] = Vec8<TA>::load_raw(Wg + (size_t)min(e0 + j, E - 1) * H + h);
#pragma unroll
          for (int j = 0; j < RB; ++j) {
            float wv[8];
            Vec8<TA>::unpack(wr[j], wv);
#pragma unroll
            for (int q = 0; q < 8; ++q) acc[e0 + j] = fmaf(av[q], wv[q], acc[e0 + j]);
          }
        }
      } else {
#pragma unroll
        for (int e = 0; e < EMAX; ++e) {
          if (e < E) {
            float wv[8];
            Vec8<TA>::load(Wg + (size_t)e * H + h, wv);
#pragma unroll
            for (int q = 0; q < 8; ++q) acc[e] = fmaf(av[q], wv[q], acc[e]);
          }
        }
      }
    }
  }
  if constexpr (EMAX == 8) {
    // the wavefront's 8 sums by a reduce-scatter over the lane bits 5, 4, 3
    // (each step halves the sums a lane carries), then a butterfly over bits
    // 2..0: lanes 8e .. 8e+7 end with the total of expert e
    const bool b5 = lane & 32, b4 = lane & 16, b3 = lane & 8;
    float r1[4], r2[2];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float give = b5 ? acc[j] : acc[j + 4];
      r1[j] = (b5 ? acc[j + 4] : acc[j]) + __shfl_xor(give, 32, 64);  // expert j + 4 b5
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const float give = b4 ? r1[j] : r1[j + 2];
      r2[j] = (b4 ? r1[j + 2] : r1[j]) + __shfl_xor(give, 16, 64);  // expert j + 2 b4 + 4 b5
    }
    float r3 = (b3 ? r2[1] : r2[0]) + __shfl_xor(b3 ? r2[0] : r2[1], 8, 64);
#pragma unroll
    for (int off = 4; off > 0; off >>= 1) r3 += __shfl_xor(r3, off, 64);
    const int e = lane >> 3;
    if ((lane & 7) == 0 && e < E) red_z[wave][e] = r3;
    __syncthreads();
    // lanes 0..7 of wavefront 0: logit of expert `lane` (the 4 wavefronts'
    // sums in order, then the bias), then the top-k over the 8 lanes
    if (tid < 8) {
      if (tid < E) {
        const float ze = (((red_z[0][tid] + red_z[1][tid]) + red_z[2][tid]) + red_z[3][tid]) + bias[tid];
        red_z[0][tid] = ze;  // read back by this lane only
        if (z != nullptr) z[(size_t)t * E + tid] = ze;
      }
      topk_group8<1, 8>(tid, E, k, norm_topk, red_z[0], idx + (size_t)t * k, w + (size_t)t * k);
    }
  } else {
#pragma unroll
    for (int e = 0; e < EMAX; ++e) {
      if (e < E) {
        const float v = wave_sum(acc[e]);
        if (lane == 0) red_z[wave][e] = v;
      }
    }
    __syncthreads();
    if (tid < E) {
      const float ze = (((red_z[0][tid] + red_z[1][tid]) + red_z[2][tid]) + red_z[3][tid]) + bias[tid];
      red_z[0][tid] = ze;  // each thread rewrites only its own entry
      if (z != nullptr) z[(size_t)t * E + tid] = ze;
    }
    __syncthreads();
    if (tid == 0)
      topk_token(E, k, norm_topk, [&](int e) { return red_z[0][e]; }, idx + (size_t)t * k,
                 w + (size_t)t * k);
  }
}

// ---------------------------------------------------------------------------
// Router logits on the matrix cores and top-k (bf16 stacks, E <= 64).
// A workgroup takes 32 tokens and all experts (padded to NB blocks of 32);
// its 4 wavefronts split K into quarters, each accumulating a 32 x 32 NB
// partial with v_mfma_f32_32x32x16_bf16.  Each wavefront streams its quarter
// through a private LDS ring of kRouteKStages stages of 64 K columns, filled
// by buffer loads straight into LDS (8 rows x 128 bytes, whole cache lines,
// per load; 16-byte chunks XOR-swizzled as in the 128-token form below), so
// the K loop needs no barrier.  Waves 1..3 leave their partials in LDS and
// wave 0 adds them in that order, then the bias (a fixed summation order),
// and writes the logits to z and to an LDS tile from which 8 lanes per token
// pick its top-k; partials and tile reuse the rings.
constexpr int kRouteKStages = 3;

template <int NB, class RBA>
__global__ __launch_bounds__(256) void route_mfma_kernel(RBA rba, int H, int E, int k,
                                                         int norm_topk) {
  constexpr int ZS = NB * 32 + 1;                 // padded LDS row of the logit tile
  constexpr int SLOT = (32 + NB * 32) * 64;       // one stage: 32 token rows, NB*32 router rows
  constexpr int WRING = kRouteKStages * SLOT;     // one wavefront's ring
  constexpr int kALd = 4, kBLd = 4 * NB;          // 1 KB loads of one stage
  constexpr int kAhead = (kALd + kBLd) * (kRouteKStages - 1);
  static_assert(kAhead < 64, "vmcnt range");
  static_assert((3 * NB * 16 * 64 + 32 * ZS) * 4 <= 4 * WRING * 2, "partials and logit tile fit in the rings");
  __shared__ __attribute__((aligned(1024))) bf16_t ring[4 * WRING];
  // the rings are written by global->LDS loads the compiler does not see
  asm volatile("" ::"v"(ring) : "memory");
  const RouteBatch& rb = rba.get();
  if ((int)blockIdx.x >= rb.blk0[rb.n]) return;  // past the live 32-token blocks
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lrow = lane & 31, khalf = lane >> 5;
  const int ei = find_entry(rb.blk0, rb.n, blockIdx.x);
  const int T = rb.tok0[ei + 1] - rb.tok0[ei];
  const int t0 = (blockIdx.x - rb.blk0[ei]) * 32;
  const bf16_t* __restrict__ a = in_global(static_cast<const bf16_t*>(rb.e[ei].a));
  const bf16_t* __restrict__ Wg = in_global(static_cast<const bf16_t*>(rb.e[ei].Wg));
  const float* __restrict__ bias = in_global(rb.e[ei].bias);
  float* __restrict__ z = in_global(rb.e[ei].z);
  int32_t* __restrict__ idx = in_global(rb.e[ei].idx);
  float* __restrict__ w = in_global(rb.e[ei].w);
  // buffer descriptors: token rows past T and router rows past E read zeros
  // (their logits are never used)
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16_t*>(a + (size_t)t0 * H), (short)0, min(T - t0, 32) * H * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16_t*>(Wg), (short)0, (int)(E * H * 2), 0x00020000);
  // load lane l: row l / 8 of an 8-row block, physical chunk l % 8 holding
  // logical chunk (l % 8) ^ ((row >> 1) & 7) (row counted within the token or
  // router rows; odd blocks flip bit 2)
  const int lr = lane >> 3, lp = lane & 7;
  const int c_even = lp ^ ((lr >> 1) & 7), c_odd = c_even ^ 4;
  const int row_b = 2 * H;  // bytes of one row
  const int voff_even = lr * row_b + c_even * 16, voff_odd = lr * row_b + c_odd * 16;
  const int kq = H / 4, kbeg = wave * kq, nst = kq / 64;
  bf16_t* wring = ring + wave * WRING;
  auto issue = [&](int st, int slot) {
    st = min(st, nst - 1);  // past the last stage: reload it into a slot nobody reads
    bf16_t* sa = wring + slot * SLOT;
    const int koff = (kbeg + 64 * st) * 2;
#pragma unroll
    for (int j = 0; j < kALd; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, sa + 8 * j * 64, 16, (j & 1) ? voff_odd : voff_even,
                                               8 * j * row_b + koff, 0, 0);
#pragma unroll
    for (int j = 0; j < kBLd; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, sa + (32 + 8 * j) * 64, 16, (j & 1) ? voff_odd : voff_even,
                                               8 * j * row_b + koff, 0, 0);
  };
  floatx16_t acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[nb][v] = 0.f;
  const int sw = (lrow >> 1) & 7;
#pragma unroll
  for (int st = 0; st < kRouteKStages - 1; ++st) issue(st, st);
  for (int st = 0; st < nst; ++st) {
    // this wavefront's fragment reads of stage st-1 are done before its slot
    // is refilled with stage st+2; stage st has landed once only the two later
    // stages' loads are in flight (loads complete in issue order)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4));  // lgkmcnt(0)
    issue(st + kRouteKStages - 1, (st + kRouteKStages - 1) % kRouteKStages);
    __builtin_amdgcn_s_waitcnt((kAhead & 15) | ((kAhead >> 4) << 14) | (7 << 4));
    asm volatile("" ::: "memory");
    const bf16_t* sa = wring + (st % kRouteKStages) * SLOT;
    const bf16_t* sb = sa + 32 * 64;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int ch = ((2 * ks + khalf) ^ sw) * 8;
      const bf16x8_t af = *reinterpret_cast<const bf16x8_t*>(sa + lrow * 64 + ch);
      bf16x8_t bfr[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) bfr[nb] = *reinterpret_cast<const bf16x8_t*>(sb + (nb * 32 + lrow) * 64 + ch);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, bfr[nb], acc[nb], 0, 0, 0);
    }
  }
  // every load (the reloads past the last stage included) has landed and
  // every wave is done with its ring before the partials overwrite them
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(7 << 4);
  __syncthreads();
  float(*part)[NB][16][64] = reinterpret_cast<float(*)[NB][16][64]>(ring);
  float(*zs)[ZS] = reinterpret_cast<float(*)[ZS]>(reinterpret_cast<float*>(ring) + 3 * NB * 16 * 64);
  if (wave > 0) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int v = 0; v < 16; ++v) part[wave - 1][nb][v][lane] = acc[nb][v];
  }
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float sum = acc[nb][v];
#pragma unroll
        for (int q = 0; q < 3; ++q) sum += part[q][nb][v][lane];
        // C[row][col]: col = lane % 32 of block nb (expert), row = 8 (v/4) + 4 (lane/32) + v%4 (token)
        const int tl = 8 * (v >> 2) + 4 * khalf + (v & 3);
        const int e = nb * 32 + lrow;
        if (e < E) {
          const float ze = sum + bias[e];
          zs[tl][e] = ze;
          if (z != nullptr && t0 + tl < T) z[(size_t)(t0 + tl) * E + e] = ze;
        }
      }
    }
  }
  __syncthreads();
  // 8 lanes per token
  const int tl = threadIdx.x >> 3, t = t0 + tl;
  if (t < T) {
    if (k <= 8)
      topk_group8<NB * 4, 8>(threadIdx.x & 7, E, k, norm_topk, zs[tl], idx + (size_t)t * k,
                             w + (size_t)t * k);
    else
      topk_group8<NB * 4, 16>(threadIdx.x & 7, E, k, norm_topk, zs[tl], idx + (size_t)t * k,
                              w + (size_t)t * k);
  }
}

// ---------------------------------------------------------------------------
// Router logits for E > 64 experts (bf16): 128 tokens per workgroup of 8
// wavefronts, wavefront w taking tokens 64 (w / 4) .. + 63 and the NBW
// 32-expert blocks from NBW (w % 4) on, every wavefront over the whole of K.
// Workgroups take the batch's 128-token tiles in order (entry by entry, from
// the batch's 32-token block table), so consecutive tiles run on different
// XCDs.  K advances 64 columns at a time through an
// LDS ring of kRouteStages stages filled by buffer loads straight into LDS:
// 1 KB per load is 8 rows x 128 bytes, whole cache lines, and each row's
// 16-byte chunk c sits at c ^ ((row >> 1) & 7) so the fragment reads are
// conflict-free.  Every logit is one chain of MFMAs over K in ascending order
// plus the bias, so it does not depend on the token's block or batch.  The
// logit tile for the top-k reuses the ring once the K loop is done.
constexpr int kRouteStages = 3;
constexpr int kRouteTokens = 128;

template <int NBW, class RBA>
__global__ __launch_bounds__(512) void route_lds_kernel(RBA rba, int H, int E, int k, int norm_topk) {
  constexpr int NB = 4 * NBW;                       // 32-expert blocks of the workgroup
  constexpr int A_ELEMS = kRouteTokens * 64;        // one stage of the token rows (16 KB)
  constexpr int B_ELEMS = NB * 32 * 64;             // one stage of the router rows
  constexpr int RING = kRouteStages * (A_ELEMS + B_ELEMS);
  constexpr int ZS = NB * 32 + 1;                   // padded row of the logit tile (floats)
  static_assert(kRouteTokens * ZS * 4 <= RING * 2, "logit tile fits in the ring");
  __shared__ __attribute__((aligned(1024))) bf16_t ring[RING];
  // the ring is written by global->LDS loads the compiler does not see
  asm volatile("" ::"v"(ring) : "memory");
  const RouteBatch& rb = rba.get();
  // workgroup q: the q-th 128-token tile of the batch, entries in order
  // (an entry of b 32-token blocks has ceil(b / 4) tiles)
  int ei = -1, t0 = 0;
  for (int i = 0, base = 0; i < rb.n; ++i) {
    const int nt = (rb.blk0[i + 1] - rb.blk0[i] + 3) / 4;
    if ((int)blockIdx.x < base + nt) {
      ei = i;
      t0 = ((int)blockIdx.x - base) * kRouteTokens;
      break;
    }
    base += nt;
  }
  if (ei < 0) return;  // past the live tiles
  const int T = rb.tok0[ei + 1] - rb.tok0[ei];
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 2, wn = wave & 3;
  const int lrow = lane & 31, khalf = lane >> 5;
  const bf16_t* __restrict__ a = in_global(static_cast<const bf16_t*>(rb.e[ei].a));
  const bf16_t* __restrict__ Wg = in_global(static_cast<const bf16_t*>(rb.e[ei].Wg));
  const float* __restrict__ bias = in_global(rb.e[ei].bias);
  float* __restrict__ z = in_global(rb.e[ei].z);
  int32_t* __restrict__ idx = in_global(rb.e[ei].idx);
  float* __restrict__ w = in_global(rb.e[ei].w);
  // buffer descriptors: rows past the tokens' or the experts' end read zeros
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16_t*>(a + (size_t)t0 * H), (short)0, min(T - t0, kRouteTokens) * H * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16_t*>(Wg), (short)0, (int)(E * H * 2), 0x00020000);
  // load lane l: row l / 8 of an 8-row block, physical chunk l % 8 holding
  // logical chunk (l % 8) ^ ((row >> 1) & 7); a block starting at a multiple
  // of 16 rows gives ((l / 8) >> 1) & 7, one starting 8 rows later flips bit 2
  const int lr = lane >> 3, lp = lane & 7;
  const int c_even = lp ^ ((lr >> 1) & 7), c_odd = c_even ^ 4;
  const int row_b = 2 * H;                // bytes of one row
  const int voff_even = lr * row_b + c_even * 16, voff_odd = lr * row_b + c_odd * 16;
  // wave w loads token rows 16 w + 8 j (j < 2) and router rows 4 NB w + 8 j
  // (j < NB / 2); block parity j & 1 in both
  constexpr int kALoads = kRouteTokens / 8 / 8, kBLoads = NB * 32 / 8 / 8;
  const int nst = H / 64;
  auto issue = [&](int st, int slot) {
    st = min(st, nst - 1);  // past the last stage: reload it into a slot nobody reads
    bf16_t* sa = ring + slot * (A_ELEMS + B_ELEMS);
    bf16_t* sb = sa + A_ELEMS;
#pragma unroll
    for (int j = 0; j < kALoads; ++j) {
      const int r0 = kALoads * 8 * wave + 8 * j;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, sa + r0 * 64, 16, (j & 1) ? voff_odd : voff_even,
                                               r0 * row_b + st * 128, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < kBLoads; ++j) {
      const int r0 = kBLoads * 8 * wave + 8 * j;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, sb + r0 * 64, 16, (j & 1) ? voff_odd : voff_even,
                                               r0 * row_b + st * 128, 0, 0);
    }
  };
  constexpr int kLoadsPerStage = kALoads + kBLoads;  // this wavefront's loads of one stage
  constexpr int kWaitAhead = kLoadsPerStage * (kRouteStages - 2);
  static_assert(kWaitAhead < 64, "vmcnt range");
  floatx16_t acc[2][NBW];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[mb][nb][v] = 0.f;
  const int sw = (lrow >> 1) & 7;
#pragma unroll
  for (int s = 0; s < kRouteStages - 1; ++s) issue(s, s);
  for (int s = 0; s < nst; ++s) {
    // stage s has landed once only the later stages' loads are in flight, and
    // this wave's fragment reads of stage s-1 are done (lgkmcnt 0) before the
    // barrier lets another wave refill that slot
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt((kWaitAhead & 15) | ((kWaitAhead >> 4) << 14) | (7 << 4));
    __builtin_amdgcn_s_barrier();  // every wave's part of stage s is in LDS; stage s-1 is read
    asm volatile("" ::: "memory");
    const int slot = s % kRouteStages;
    issue(s + kRouteStages - 1, (s + kRouteStages - 1) % kRouteStages);
    const bf16_t* sa = ring + slot * (A_ELEMS + B_ELEMS) + (64 * wm) * 64;
    const bf16_t* sb = ring + slot * (A_ELEMS + B_ELEMS) + A_ELEMS + (32 * NBW * wn) * 64;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int ch = ((2 * ks + khalf) ^ sw) * 8;
      bf16x8_t af[2], bfr[NBW];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) af[mb] = *reinterpret_cast<const bf16x8_t*>(sa + (mb * 32 + lrow) * 64 + ch);
#pragma unroll
      for (int nb = 0; nb < NBW; ++nb) bfr[nb] = *reinterpret_cast<const bf16x8_t*>(sb + (nb * 32 + lrow) * 64 + ch);
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mb], bfr[nb], acc[mb][nb], 0, 0, 0);
    }
  }
  // every load (including those past the last stage) has landed and every
  // wave is done reading the ring before the logit tile overwrites it
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(7 << 4);
  __syncthreads();
  float* zs = reinterpret_cast<float*>(ring);
  // acc[mb][nb][v]: expert 32 (NBW wn + nb) + lane % 32, token
  // 64 wm + 32 mb + 8 (v / 4) + 4 (lane / 32) + v % 4
#pragma unroll
  for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
      const int e = 32 * (NBW * wn + nb) + lrow;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int tl = 64 * wm + 32 * mb + 8 * (v >> 2) + 4 * khalf + (v & 3);
        if (e < E) {
          const float ze = acc[mb][nb][v] + bias[e];
          zs[tl * ZS + e] = ze;
          if (z != nullptr && t0 + tl < T) z[(size_t)(t0 + tl) * E + e] = ze;
        }
      }
    }
  }
  __syncthreads();
  // 8 lanes per token, two tokens per group of 8 lanes
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    const int tl = (threadIdx.x >> 3) + 64 * half, t = t0 + tl;
    if (t < T) {
      if (k <= 8)
        topk_group8<NB * 4, 8>(threadIdx.x & 7, E, k, norm_topk, zs + tl * ZS, idx + (size_t)t * k,
                               w + (size_t)t * k);
      else
        topk_group8<NB * 4, 16>(threadIdx.x & 7, E, k, norm_topk, zs + tl * ZS, idx + (size_t)t * k,
                                w + (size_t)t * k);
    }
  }
}

// ---------------------------------------------------------------------------
// Top-k from logits in global memory (fp32 stacks without the fused path),
// one thread per token.
__global__ __launch_bounds__(256) void topk_kernel(int T, int E, int k, int norm_topk,
                                                   const float* __restrict__ z,
                                                   int32_t* __restrict__ idx,
                                                   float* __restrict__ w) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
  const float* zr = z + (size_t)t * E;
  topk_token(E, k, norm_topk, [&](int e) { return zr[e]; }, idx + (size_t)t * k, w + (size_t)t * k);
}

// Whether the routing of a batch runs in a fixed set of launches (no launch
// per entry): every bf16 stack, and fp32 stacks on the fused per-token path.
template <typename TA>
bool fused_token_path(const eb_model_desc& d) {
  return (sizeof(TA) == 2 ? d.E <= 8 : d.E <= 64) && d.H <= kTokMaxH;
}

// grid_entries / grid_tokens / grid_blocks: entries, tokens and 32-token
// blocks the grids cover (the live batch's, or a full batch's when the table
// is in device memory); host_rb: the table itself when the host built it
// (the fp32 per-entry path needs it).
template <typename TA, class RBA>
hipError_t route_batch_typed(const eb_model_desc& d, RBA rba, const RouteBatch* host_rb, int grid_entries,
                             int grid_tokens, int grid_blocks, hipStream_t s) {
  if (grid_tokens > 0) {
    if (fused_token_path<TA>(d)) {
      prof_start(EB_K_ROUTE_LOGITS, s);
      if (d.E <= 8 && d.H <= 256 * 8 * 2)
        hipLaunchKernelGGL((route_token_kernel<TA, 8, 2, RBA>), dim3(grid_tokens), dim3(256), 0, s, rba, d.H,
                           d.E, d.k, d.norm_topk, d.rms_eps);
      else if (d.E <= 8)
        hipLaunchKernelGGL((route_token_kernel<TA, 8, kTokChunks, RBA>), dim3(grid_tokens), dim3(256), 0, s,
                           rba, d.H, d.E, d.k, d.norm_topk, d.rms_eps);
      else
        hipLaunchKernelGGL((route_token_kernel<TA, 64, kTokChunks, RBA>), dim3(grid_tokens), dim3(256), 0, s,
                           rba, d.H, d.E, d.k, d.norm_topk, d.rms_eps);
      prof_stop(EB_K_ROUTE_LOGITS, s);
    } else {
      prof_start(EB_K_ROUTE_NORM, s);
      if (d.H > 4096 && d.H <= 256 * 4 * 8)
        hipLaunchKernelGGL((rmsnorm_row_kernel<TA, 8, RBA>), dim3(grid_tokens), dim3(256), 0, s, rba, d.H,
                           d.rms_eps);
      else if (d.H > 2048 && d.H <= 256 * 4 * 4)
        hipLaunchKernelGGL((rmsnorm_row_kernel<TA, 4, RBA>), dim3(grid_tokens), dim3(256), 0, s, rba, d.H,
                           d.rms_eps);
      else if (d.H <= 256 * 4 * 2)
        hipLaunchKernelGGL((rmsnorm_row_kernel<TA, 2, RBA>), dim3(grid_tokens), dim3(256), 0, s, rba, d.H,
                           d.rms_eps);
      else
        hipLaunchKernelGGL((rmsnorm_kernel<TA, RBA>), dim3((grid_tokens + 3) / 4), dim3(256), 0, s, rba, d.H,
                           d.rms_eps);
      prof_stop(EB_K_ROUTE_NORM, s);
      prof_start(EB_K_ROUTE_LOGITS, s);
      if (sizeof(TA) == 2) {
        const dim3 grid(grid_blocks);
        // 128-token tiles: at most a quarter of the blocks plus one per entry
        const dim3 grid_tiles((grid_blocks + 3) / 4 + grid_entries);
        const int nb = (d.E + 31) / 32;
        if (nb <= 2)
          hipLaunchKernelGGL((route_mfma_kernel<2, RBA>), grid, dim3(256), 0, s, rba, d.H, d.E, d.k, d.norm_topk);
        else if (nb <= 4)
          hipLaunchKernelGGL((route_lds_kernel<1, RBA>), grid_tiles, dim3(512), 0, s, rba, d.H, d.E, d.k,
                             d.norm_topk);
        else
          hipLaunchKernelGGL((route_lds_kernel<2, RBA>), grid_tiles, dim3(512), 0, s, rba, d.H, d.E, d.k,
                             d.norm_topk);
        prof_stop(EB_K_ROUTE_LOGITS, s);
      } else {
        if (host_rb == nullptr) return hipErrorInvalidValue;
        const RouteBatch& rb = *host_rb;
        for (int i = 0; i < rb.n; ++i) {
          const int T = rb.tok0[i + 1] - rb.tok0[i];
          if (T == 0) continue;
          const RouteEntry& e = rb.e[i];
          hipLaunchKernelGGL(logits_kernel<TA>, dim3((T + LG_BT - 1) / LG_BT, (d.E + LG_BE - 1) / LG_BE),
                             dim3(256), 0, s, T, d.H, d.E, static_cast<const TA*>(e.a),
                             static_cast<const TA*>(e.Wg), e.bias, e.z);
        }
        prof_stop(EB_K_ROUTE_LOGITS, s);
        prof_start(EB_K_ROUTE_TOPK, s);
        for (int i = 0; i < rb.n; ++i) {
          const int T = rb.tok0[i + 1] - rb.tok0[i];
          if (T == 0) continue;
          const RouteEntry& e = rb.e[i];
          hipLaunchKernelGGL(topk_kernel, dim3((T + 255) / 256), dim3(256), 0, s, T, d.E, d.k,
                             d.norm_topk, e.z, e.idx, e.w);
        }
        prof_stop(EB_K_ROUTE_TOPK, s);
      }
    }
  }
  prof_start(EB_K_ROUTE_TOPK, s);
  if (grid_entries > 0)
    hipLaunchKernelGGL((counts_kernel<RBA>), dim3(grid_entries), dim3(1024), 0, s, rba, d.k, d.E);
  prof_stop(EB_K_ROUTE_TOPK, s);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_route_batch(const eb_model_desc& d, const RouteBatch& rb, hipStream_t s) {
  const ByValue<RouteBatch> a{rb};
  if (d.dtype == EB_DTYPE_BF16)
    return route_batch_typed<bf16_t>(d, a, &rb, rb.n, rb.tok0[rb.n], rb.blk0[rb.n], s);
  return route_batch_typed<float>(d, a, &rb, rb.n, rb.tok0[rb.n], rb.blk0[rb.n], s);
}

bool route_logits_required(const eb_model_desc& d) {
  return d.dtype != EB_DTYPE_BF16 && !fused_token_path<float>(d);
}

bool route_batch_device_ok(const eb_model_desc& d) {
  return d.dtype == EB_DTYPE_BF16 || fused_token_path<float>(d);
}

hipError_t launch_route_batch_dev(const eb_model_desc& d, const RouteBatch* rb, int max_entries, int T,
                                  hipStream_t s) {
  if (!route_batch_device_ok(d) || max_entries > kRouteBatch) return hipErrorInvalidValue;
  const InMemory<RouteBatch> a{rb};
  const int tokens = max_entries * T, blocks = max_entries * ((T + 31) / 32);
  if (d.dtype == EB_DTYPE_BF16) return route_batch_typed<bf16_t>(d, a, nullptr, max_entries, tokens, blocks, s);
  return route_batch_typed<float>(d, a, nullptr, max_entries, tokens, blocks, s);
}

hipError_t launch_route(const eb_model_desc& d, int T, const float* x, const float* gain,
                        const void* Wg, const float* bias, void* a_out, float* logits,
                        int32_t* idx, float* w, int32_t* counts, hipStream_t s) {
  RouteBatch rb;
  rb.n = 1;
  rb.tok0[0] = 0;
  rb.tok0[1] = T;
  rb.blk0[0] = 0;
  rb.blk0[1] = (T + 31) / 32;
  rb.e[0] = RouteEntry{x, gain, Wg, bias, a_out, logits, idx, w, counts};
  return launch_route_batch(d, rb, s);
}

}  // namespace eb
