// Device-side Schedule of Algorithm 1: one workgroup, launched at the start
// of every step of a device-scheduled pass, so that the host never waits for
// the pool's expert counts.
//
//   pool    = micro-batches j with l_j < L
//   RunSet  = MaxUtil / CumUtil / DiffPeak over the pool's per-device loads
//             (Sections 4.2 and 5.2), or the whole pool (lock-step)
//   writes  the step's run table (the micro-batches of RunSet at their layers),
//           the routing table of the micro-batches that advance to a layer
//           < L, the step's records, l_j += 1 for j in RunSet, and a status
//           word in host memory: (pass tag, steps so far, max_j (L - l_j))
//
// The choice is the host scheduler's, bit for bit: the same exact integer
// comparisons of U = sum_d W_d / (D max_d W_d) (128-bit cross products) and
// the same total order on ties (higher U, then more members, then the
// lexicographically smallest set), so the result does not depend on which
// thread evaluates which subset.
#include <algorithm>

#include "eb_internal.h"

namespace eb {
namespace {

constexpr int kSchedThreads = 512;

// a.num / a.den vs b.num / b.den for non-negative operands: the 128-bit
// products a.num * b.den and b.num * a.den, compared high word first.
__device__ __forceinline__ int ratio_cmp(unsigned long long an, unsigned long long ad, unsigned long long bn,
                                         unsigned long long bd) {
  if (((an | ad | bn | bd) >> 32) == 0) {  // the products fit in 64 bits
    const unsigned long long l = an * bd, r = bn * ad;
    return l > r ? 1 : (l < r ? -1 : 0);
  }
  const unsigned long long lh = __umul64hi(an, bd), ll = an * bd;
  const unsigned long long rh = __umul64hi(bn, ad), rl = bn * ad;
  if (lh != rh) return lh > rh ? 1 : -1;
  if (ll != rl) return ll > rl ? 1 : -1;
  return 0;
}

// U of a workload with total `sum` and maximum `mx` as a ratio num / den
// (U = num / (D den)); an all-zero workload has U = 1.
struct Util {
  unsigned long long num, den;
};
__device__ __forceinline__ Util util_of(long long sum, long long mx, int D) {
  return mx == 0 ? Util{(unsigned long long)D, 1ull} : Util{(unsigned long long)sum, (unsigned long long)mx};
}

// Candidate subset of pool indices (bit i = i-th smallest pool id).
struct Cand {
  Util u;
  int size;  // -1: none yet
  unsigned set;
};

// a before b in the MaxUtil order: higher U, then more members, then the
// set holding the lowest pool index where the two differ.
__device__ __forceinline__ bool cand_better(const Cand& a, const Cand& b) {
  if (a.size < 0) return false;
  if (b.size < 0) return true;
  const int c = ratio_cmp(a.u.num, a.u.den, b.u.num, b.u.den);
  if (c != 0) return c > 0;
  if (a.size != b.size) return a.size > b.size;
  const unsigned x = a.set ^ b.set;
  return x != 0 && (a.set & (x & (~x + 1u))) != 0;
}

// The combination of rank r among the j-subsets of {0 .. n-1} in the
// combinatorial number system (r = sum_t C(c_t, t), c_j > ... > c_1 >= 0),
// as a bit mask.  C is Pascal's triangle, C[a * kMaxC + b] = C(a, b).
constexpr int kMaxC = EB_MAXUTIL_MAX_POOL + 1;
struct BinomTable {
  unsigned v[kMaxC * kMaxC];
};
constexpr BinomTable make_binom() {
  BinomTable t{};
  for (int a = 0; a < kMaxC; ++a)
    for (int b = 0; b < kMaxC; ++b)
      t.v[a * kMaxC + b] = b == 0 ? 1u : (b > a ? 0u : t.v[(a - 1) * kMaxC + b - 1] + t.v[(a - 1) * kMaxC + b]);
  return t;
}
__constant__ BinomTable kBinom = make_binom();
constexpr int kDevMaxNzWords = EB_MAX_POOL * 1024 / 32;  // (member, expert) bits, E + S <= 1024
__device__ __forceinline__ unsigned unrank(unsigned r, int j, int n, const unsigned* C) {
  unsigned set = 0;
  int c = n - 1;
  for (int t = j; t >= 1; --t) {
    while (C[c * kMaxC + t] > r) --c;  // the largest c with C(c, t) <= r (c >= t - 1)
    r -= C[c * kMaxC + t];
    set |= 1u << c;
    --c;
  }
  return set;
}

}  // namespace

// Wave-wide maximum of a candidate in the MaxUtil order.
__device__ __forceinline__ Cand wave_best(Cand c) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    Cand o;
    o.u.num = __shfl_xor(c.u.num, off, kWave);
    o.u.den = __shfl_xor(c.u.den, off, kWave);
    o.size = __shfl_xor(c.size, off, kWave);
    o.set = __shfl_xor(c.set, off, kWave);
    if (cand_better(o, c)) c = o;
  }
  return c;
}

// Best subset among ranks [r0, r1) of the excluded sets X (sizes 0 .. max_excl,
// each size in increasing numeric order): one unranking, then Gosper's step
// to the next set of the same size.  W = the pool's total minus X's loads,
// kept in registers (DMAX >= D).
template <int DMAX>
__device__ Cand maxutil_range(unsigned r0, unsigned r1, int n, int D, const unsigned* C, const long long* load,
                              const long long* tot) {
  Cand best{{0ull, 1ull}, -1, 0u};
  if (r0 >= r1) return best;
  int j = 0;
  unsigned rank = r0;
  while (rank >= C[n * kMaxC + j]) rank -= C[n * kMaxC + j++];
  unsigned x = unrank(rank, j, n, C);
  const unsigned full = (1u << n) - 1u;
  for (unsigned r = r0; r < r1; ++r) {
    long long W[DMAX];
#pragma unroll
    for (int d = 0; d < DMAX; ++d) W[d] = d < D ? tot[d] : 0;
    for (unsigned y = x; y != 0; y &= y - 1u) {
      const long long* row = load + (__ffs(y) - 1) * kDevMaxD;
#pragma unroll
      for (int d = 0; d < DMAX; ++d)
        if (d < D) W[d] -= row[d];
    }
    long long sum = 0, mx = 0;
#pragma unroll
    for (int d = 0; d < DMAX; ++d) {
      sum += W[d];
      mx = W[d] > mx ? W[d] : mx;
    }
    const Cand c{util_of(sum, mx, D), n - j, full ^ x};
    if (cand_better(c, best)) best = c;
    // next X: the next set of size j, or the first of size j + 1
    if (++rank < C[n * kMaxC + j]) {
      const unsigned lo = x & (~x + 1u), hi = x + lo;
      x = (((hi ^ x) >> 2) >> (__ffs(lo) - 1)) | hi;
    } else {
      ++j;
      rank = 0;
      x = (1u << j) - 1u;
    }
  }
  return best;
}

template <int DMAX>
__global__ __launch_bounds__(kSchedThreads) void sched_step_kernel(DevPassArgs A) {
  __shared__ int s_layer[EB_MAX_POOL];
  __shared__ int s_pool[EB_MAX_POOL];
  __shared__ int s_pidx[EB_MAX_POOL];  // pool index of micro-batch j, or -1
  __shared__ int s_peak[EB_MAX_POOL];
  __shared__ long long s_W[kDevMaxD];
  __shared__ int s_n;
  __shared__ long long s_load[EB_MAX_POOL * kDevMaxD];
  __shared__ Cand s_cand[kSchedThreads / kWave];
  __shared__ unsigned long long s_chosen;  // over pool indices
  __shared__ unsigned s_bits[kDevMaxKeyWords];
  __shared__ unsigned s_C[kMaxC * kMaxC];
  __shared__ unsigned s_nz[kDevMaxNzWords];  // bit pi * E + e: member pi has pairs on expert e
  __shared__ long long s_tot[kDevMaxD];
  __shared__ unsigned s_lbits[EB_MAX_LAYERS / 32];
  __shared__ int s_groups;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int N = A.N, D = A.D, E = A.E, L = A.L, per = E / D;
  DevPassState* st = A.state;
  // every global read the choice needs is issued up front, in parallel
  const int my_layer = tid < N ? st->layer[tid] : L;  // wave 0: lane j holds l_j
  const int step = st->steps;
  for (int i = tid; i < kMaxC * kMaxC; i += kSchedThreads) s_C[i] = kBinom.v[i];
  for (int w = tid; w < kDevMaxKeyWords; w += kSchedThreads) s_bits[w] = 0u;
  for (int w = tid; w < kDevMaxNzWords; w += kSchedThreads) s_nz[w] = 0u;
  for (int i = tid; i < EB_MAX_POOL * kDevMaxD; i += kSchedThreads) s_load[i] = 0;
  if (tid < kDevMaxD) s_tot[tid] = 0;
  if (tid < EB_MAX_LAYERS / 32) s_lbits[tid] = 0u;
  // the pool, in ascending id: one ballot over wave 0's lanes (N <= 64)
  const unsigned long long pool_mask = __ballot(tid < N && my_layer < L);
  if (wave == 0) {
    const bool in = tid < N && my_layer < L;
    if (tid < N) {
      s_layer[tid] = my_layer;
      s_pidx[tid] = in ? __popcll(pool_mask & ((1ull << lane) - 1ull)) : -1;
    }
    if (in) s_pool[__popcll(pool_mask & ((1ull << lane) - 1ull))] = tid;
    if (tid == 0) {
      s_n = __popcll(pool_mask);
      s_groups = 0;
    }
  }
  __syncthreads();
  const int n = s_n;
  RunTable* rt = A.rt;
  if (tid == 0) {
    rt->E = E;
    rt->k = A.k;
    rt->S = A.S;
    rt->L = L;
    rt->H = A.H;
    rt->chunk_base[0] = 0;
    rt->tok_base[0] = 0;
    for (int b = 0; b < kDevRouteSlots; ++b) {
      A.rb[b].n = 0;
      A.rb[b].tok0[0] = 0;
      A.rb[b].blk0[0] = 0;
    }
  }
  if (n == 0) {  // nothing left: an empty step (every kernel of it exits at once)
    if (tid == 0) rt->n = 0;
    return;
  }

  // per-device loads of the pool members at their current layers, and which
  // (member, expert) pairs hold tokens; the counts are read once, four
  // independent loads per thread at a time
  for (int i0 = tid; i0 < n * E; i0 += 4 * kSchedThreads) {
    int32_t c[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * kSchedThreads;
      c[u] = 0;
      if (i < n * E) {
        const int pi = i / E;
        c[u] = A.counts[(size_t)s_pool[pi] * E + (i - pi * E)];
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * kSchedThreads;
      if (i < n * E && c[u] != 0) {
        const int pi = i / E, e = i - pi * E;
        if (A.place == nullptr) {
          atomicAdd(reinterpret_cast<unsigned long long*>(&s_load[pi * kDevMaxD + e / per]),
                    (unsigned long long)c[u]);
          atomicAdd(reinterpret_cast<unsigned long long*>(&s_tot[e / per]), (unsigned long long)c[u]);
        } else {
          // the expert's pairs split evenly over its copies (validated on the
          // host: 1..R distinct devices < D, ascending, then -1), the lower
          // copies taking the remainder
          const int32_t* cp = A.place + ((size_t)s_layer[s_pool[pi]] * E + e) * A.R;
          int r = 1;
          while (r < A.R && cp[r] >= 0) ++r;
          const int q = c[u] / r, rem = c[u] - q * r;
          for (int ci = 0; ci < r; ++ci) {
            const int dv = cp[ci];
            const unsigned long long share = (unsigned long long)(q + (ci < rem ? 1 : 0));
            atomicAdd(reinterpret_cast<unsigned long long*>(&s_load[pi * kDevMaxD + dv]), share);
            atomicAdd(reinterpret_cast<unsigned long long*>(&s_tot[dv]), share);
          }
        }
        atomicOr(&s_nz[i >> 5], 1u << (i & 31));
      }
    }
  }
  __syncthreads();
  for (int i = tid; i < n * D; i += kSchedThreads) {
    const int pi = i / D, d = i - pi * D;
    const int j = s_pool[pi];
    A.rec_layer_loads[((size_t)j * L + s_layer[j]) * D + d] = (int32_t)s_load[pi * kDevMaxD + d];
  }

  const int need = A.m < n ? A.m : n;
  if (A.policy == EB_POLICY_LOCKSTEP) {
    if (tid == 0) s_chosen = n == 64 ? ~0ull : (1ull << n) - 1ull;
  } else if (A.policy == EB_POLICY_MAXUTIL) {
    // every subset with >= need members (n <= EB_MAXUTIL_MAX_POOL) as the
    // complement of an excluded set X, |X| <= n - need: sum_j C(n, j) of
    // them, numbered consecutively (by |X|, then X's rank) and cut into one
    // contiguous range per thread (one set per lane of wave 0 when there
    // are at most 64); the pool's total workload (summed with the loads)
    // minus X's members gives each one's.  The best of each thread, of each
    // wavefront, then of the block.
    unsigned count = 0;
    for (int j = 0; j <= n - need; ++j) count += s_C[n * kMaxC + j];
    if (count <= (unsigned)kWave) {  // one candidate per lane of wave 0 at most
      if (wave == 0) {
        const unsigned r0 = lane, r1 = min(count, (unsigned)lane + 1u);
        const Cand best = wave_best(maxutil_range<DMAX>(r0, r1, n, D, s_C, s_load, s_tot));
        if (lane == 0) s_chosen = best.set;
      }
    } else {
      const unsigned chunk = (count + kSchedThreads - 1) / kSchedThreads;
      const unsigned r0 = min(count, (unsigned)tid * chunk), r1 = min(count, r0 + chunk);
      Cand best = wave_best(maxutil_range<DMAX>(r0, r1, n, D, s_C, s_load, s_tot));
      if (lane == 0) s_cand[wave] = best;
      __syncthreads();
      if (wave == 0) {
        Cand c = lane < kSchedThreads / kWave ? s_cand[lane] : Cand{{0ull, 1ull}, -1, 0u};
        c = wave_best(c);
        if (lane == 0) s_chosen = c.set;
      }
    }
  } else {
    if (A.policy == EB_POLICY_DIFFPEAK && tid < n) {  // peak device of each member: first maximum
      int p = 0;
      for (int d = 1; d < D; ++d)
        if (s_load[tid * kDevMaxD + d] > s_load[tid * kDevMaxD + p]) p = d;
      s_peak[tid] = p;
    }
    __syncthreads();
    if (tid == 0) {
      unsigned long long set = 1ull;  // the first micro-batch is always scheduled
      if (A.policy == EB_POLICY_CUMUTIL) {
        // add member i when it raises U of the running workload (exact)
        long long* W = s_W;
        long long sum = 0, mx = 0;
        for (int d = 0; d < D; ++d) {
          W[d] = s_load[d];
          sum += W[d];
          mx = W[d] > mx ? W[d] : mx;
        }
        for (int i = 1; i < n; ++i) {
          long long sum2 = 0, mx2 = 0;
          for (int d = 0; d < D; ++d) {
            const long long v = W[d] + s_load[i * kDevMaxD + d];
            sum2 += v;
            mx2 = v > mx2 ? v : mx2;
          }
          const Util u2 = util_of(sum2, mx2, D), u1 = util_of(sum, mx, D);
          if (ratio_cmp(u2.num, u2.den, u1.num, u1.den) > 0) {
            set |= 1ull << i;
            for (int d = 0; d < D; ++d) W[d] += s_load[i * kDevMaxD + d];
            sum = sum2;
            mx = mx2;
          }
        }
      } else {  // DiffPeak: add member i when its peak device is not taken yet
        unsigned long long taken = 1ull << s_peak[0];
        for (int i = 1; i < n; ++i)
          if (!((taken >> s_peak[i]) & 1ull)) {
            taken |= 1ull << s_peak[i];
            set |= 1ull << i;
          }
      }
      // at least min(m, |pool|) members: the lowest unscheduled ones
      int have = __popcll(set);
      for (int i = 0; i < n && have < need; ++i)
        if (!((set >> i) & 1ull)) {
          set |= 1ull << i;
          ++have;
        }
      s_chosen = set;
    }
  }
  __syncthreads();
  const unsigned long long chosen = s_chosen;

  // the step's workload and records
  if (step < A.max_records) {
    for (int d = tid; d < D; d += kSchedThreads) {
      long long v = 0;
      for (int i = 0; i < n; ++i)
        if ((chosen >> i) & 1ull) v += s_load[i * kDevMaxD + d];
      A.rec_load[(size_t)step * D + d] = v;
    }
    if (tid < N) {
      const int i = s_pidx[tid];
      A.rec_layers[(size_t)step * N + tid] = (i >= 0 && ((chosen >> i) & 1ull)) ? s_layer[tid] : -1;
    }
  }
  // run table: chosen members in ascending id order (all hold T tokens)
  const int chunks = (A.T + kPermChunk - 1) / kPermChunk;
  if (tid < n && ((chosen >> tid) & 1ull)) {
    const int r = __popcll(chosen & ((1ull << tid) - 1ull));
    const int j = s_pool[tid];
    rt->chunk_base[r + 1] = (r + 1) * chunks;
    rt->tok_base[r + 1] = (r + 1) * A.T;
    rt->layer[r] = s_layer[j];
    rt->idx[r] = A.idx + (size_t)j * A.T * A.k;
    rt->a[r] = static_cast<const uint8_t*>(A.a) + (size_t)j * A.a_stride;
    rt->w[r] = A.w + (size_t)j * A.T * A.k;
    rt->x[r] = A.x + (size_t)j * A.T * A.H;
    atomicOr(&s_lbits[s_layer[j] >> 5], 1u << (s_layer[j] & 31));
  }
  // distinct (layer, routed expert) groups with a pair in this step
  const int n_run = __popcll(chosen);
  for (int i = tid; i < n * E; i += kSchedThreads) {
    const int pi = i / E, e = i - pi * E;
    if (!((chosen >> pi) & 1ull) || !((s_nz[i >> 5] >> (i & 31)) & 1u)) continue;
    const int key = s_layer[s_pool[pi]] * E + e;
    atomicOr(&s_bits[key >> 5], 1u << (key & 31));
  }
  __syncthreads();
  {
    int g = 0;
    for (int w = tid; w < (L * E + 31) / 32; w += kSchedThreads) g += __popc(s_bits[w]);
    if (tid < EB_MAX_LAYERS / 32) g += A.S * __popc(s_lbits[tid]);
    if (g) atomicAdd(&s_groups, g);
  }
  // wave 0, lane j: micro-batch j advances, is routed at its next layer if
  // that is < L, and reports how many layers it is still short
  if (wave == 0) {
    const int i = tid < N ? s_pidx[tid] : -1;
    const bool run = i >= 0 && ((chosen >> i) & 1ull);
    const int l_new = tid < N ? my_layer + (run ? 1 : 0) : L;
    const bool adv = run && l_new < L;
    const unsigned long long adv_mask = __ballot(adv);
    if (adv) {
      const int r = __popcll(adv_mask & ((1ull << lane) - 1ull));
      const int j = tid;
      RouteBatch& rb = A.rb[r / kRouteBatch];
      const int q = r % kRouteBatch;
      rb.tok0[q + 1] = (q + 1) * A.T;
      rb.blk0[q + 1] = (q + 1) * ((A.T + 31) / 32);
      rb.e[q] = RouteEntry{A.x + (size_t)j * A.T * A.H,
                           A.gain + (size_t)l_new * A.H,
                           A.Wg[l_new],
                           A.bias + (size_t)l_new * E,
                           static_cast<uint8_t*>(A.a) + (size_t)j * A.a_stride,
                           A.z + (size_t)j * A.T * E,
                           A.idx + (size_t)j * A.T * A.k,
                           A.w + (size_t)j * A.T * A.k,
                           A.counts + (size_t)j * E};
    }
    if (run) st->layer[tid] = l_new;
    int lag = L - l_new;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) lag = max(lag, __shfl_xor(lag, off, kWave));
    if (tid == 0) {
      const int n_adv = __popcll(adv_mask);
      for (int b = 0; b < kDevRouteSlots; ++b) {
        const int nb = n_adv - b * kRouteBatch;
        A.rb[b].n = nb < 0 ? 0 : (nb > kRouteBatch ? kRouteBatch : nb);
      }
      rt->n = n_run;
      st->steps = step + 1;
      if (step < A.max_records) {
        unsigned long long ids = 0;
        for (int q = 0; q < n; ++q)
          if ((chosen >> q) & 1ull) ids |= 1ull << s_pool[q];
        A.rec_mask[step] = ids;
      }
    }
    // s_groups is final only after the barrier below; the status word goes
    // last, after it
    if (tid == 0) s_W[0] = lag;
  }
  __syncthreads();
  if (tid == 0) {
    if (step < A.max_records) A.rec_groups[step] = s_groups;
    // the host reads this word while the rest of the step runs: a
    // system-scope store into host memory, no cache maintenance
    const unsigned long long word = ((unsigned long long)A.tag << 48) |
                                    ((unsigned long long)(step + 1) << 16) | (unsigned long long)s_W[0];
    __hip_atomic_store(A.status, word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  }
}

// Start of a device-scheduled pass: every micro-batch at layer 0, no steps,
// per-layer loads unknown (-1).
__global__ __launch_bounds__(256) void pass_init_kernel(DevPassArgs A) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < (size_t)A.N) A.state->layer[i] = 0;
  if (i == 0) A.state->steps = 0;
  const size_t n_ll = (size_t)A.N * A.L * A.D;
  for (size_t q = i; q < n_ll; q += (size_t)gridDim.x * blockDim.x) A.rec_layer_loads[q] = -1;
}

hipError_t launch_pass_init(const DevPassArgs& A, hipStream_t s) {
  const size_t n_ll = (size_t)A.N * A.L * A.D;
  const unsigned grid = (unsigned)std::min<size_t>(1024, (n_ll + 255) / 256 + 1);
  hipLaunchKernelGGL(pass_init_kernel, dim3(grid), dim3(256), 0, s, A);
  return hipGetLastError();
}

hipError_t launch_sched_step(const DevPassArgs& A, hipStream_t s) {
  if (A.D <= 8)
    hipLaunchKernelGGL(sched_step_kernel<8>, dim3(1), dim3(kSchedThreads), 0, s, A);
  else if (A.D <= 16)
    hipLaunchKernelGGL(sched_step_kernel<16>, dim3(1), dim3(kSchedThreads), 0, s, A);
  else if (A.D <= 32)
    hipLaunchKernelGGL(sched_step_kernel<32>, dim3(1), dim3(kSchedThreads), 0, s, A);
  else
    hipLaunchKernelGGL(sched_step_kernel<kDevMaxD>, dim3(1), dim3(kSchedThreads), 0, s, A);
  return hipGetLastError();
}

}  // namespace eb
