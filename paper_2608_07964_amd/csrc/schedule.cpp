// Host scheduler: RunSet_i = Schedule(S_{i-1}, m) of Algorithm 1 (EasyBalance).
//
// MaxUtil (Section 4.2) picks, among subsets of the pool with at least
// min(m, |pool|) members, the one whose combined per-device workload has the
// highest utilization U = sum_d W_d / (D * max_d W_d) (Eq. 3 for one step).
// CumUtil and DiffPeak are the linear-time heuristics of Section 5.2.
// Everything is exact integer arithmetic so that every rank of a real EP
// group, given the same counts, picks the same RunSet.
#include <stdint.h>
#include <string.h>

#include <vector>

#include "eb_internal.h"

namespace eb {
namespace {

// U as a comparable ratio: U = num / (D * den).  U of an all-zero workload is
// 1, i.e. num/den = D.
struct Ratio {
  int64_t num, den;
};

inline Ratio util_ratio(const int64_t* W, int D) {
  int64_t sum = 0, mx = 0;
  for (int d = 0; d < D; ++d) {
    sum += W[d];
    if (W[d] > mx) mx = W[d];
  }
  if (mx == 0) return Ratio{D, 1};
  return Ratio{sum, mx};
}

// +1 if a > b, -1 if a < b, 0 if equal.
inline int ratio_cmp(const Ratio& a, const Ratio& b) {
  const __int128 l = (__int128)a.num * b.den;
  const __int128 r = (__int128)b.num * a.den;
  return l > r ? 1 : (l < r ? -1 : 0);
}

// Among equal-size subsets (bit i = i-th smallest id), `a` is lexicographically
// smaller iff it holds the lowest bit where the two differ.
inline bool lex_smaller(uint32_t a, uint32_t b) {
  const uint32_t x = a ^ b;
  return x != 0 && (a & (x & (~x + 1u))) != 0;
}

// Depth-first walk over the subsets with at least `need` members, as the
// complements of excluded sets X with |X| <= n - need (members of X in
// ascending order): sum_{j <= n-need} C(n, j) subsets instead of all 2^n,
// e.g. 2517 instead of 65536 for n = 16, need = 12.  The per-device workload
// of each subset is the parent's minus one micro-batch's load, its maximum
// taken in the same pass.  The choice (highest U, then more members, then the
// lexicographically smallest set) is a total order on subsets, so the result
// does not depend on the walk order.
struct MaxUtilSearch {
  int n, D, max_excl;
  uint32_t full;
  const int64_t* load;   // [n][D]
  const int64_t* lsum;   // [n] sum over devices of load
  int64_t* level;        // [max_excl + 1][D] workload per depth
  uint32_t best = 0;
  Ratio best_u{0, 1};
  int best_size = -1;

  void consider(uint32_t set, int size, int64_t sum, int64_t mx) {
    const Ratio u = mx == 0 ? Ratio{D, 1} : Ratio{sum, mx};
    int c;
    if (best_size < 0) {
      c = 1;
    } else {
      // num/den <= D; the doubles decide unless the two ratios agree to
      // within their rounding, then the exact 128-bit products do
      const double l = (double)u.num * (double)best_u.den, r = (double)best_u.num * (double)u.den;
      if (l > r * (1.0 + 1e-12)) c = 1;
      else if (r > l * (1.0 + 1e-12)) c = -1;
      else c = ratio_cmp(u, best_u);
    }
    if (c > 0 || (c == 0 && (size > best_size || (size == best_size && lex_smaller(set, best))))) {
      best = set;
      best_u = u;
      best_size = size;
    }
  }

  // X = excl (depth members, all below `first`); its complement's workload is
  // level[depth] and has been considered
  void walk(int depth, int first, uint32_t excl, int64_t sum) {
    const int64_t* W = level + (size_t)depth * D;
    int64_t* W2 = level + (size_t)(depth + 1) * D;
    for (int i = first; i < n; ++i) {
      const int64_t* li = load + (size_t)i * D;
      int64_t mx = 0;
      for (int d = 0; d < D; ++d) {
        const int64_t v = W[d] - li[d];
        W2[d] = v;
        mx = v > mx ? v : mx;
      }
      const uint32_t x2 = excl | (1u << i);
      const int64_t sum2 = sum - lsum[i];
      consider(full ^ x2, n - depth - 1, sum2, mx);
      if (depth + 1 < max_excl) walk(depth + 1, i + 1, x2, sum2);
    }
  }
};

uint32_t maxutil(int n, const std::vector<int64_t>& load, int D, int need) {
  MaxUtilSearch s;
  s.n = n;
  s.D = D;
  s.max_excl = n - need;  // need >= 1, so the empty set is never visited
  s.full = n == 32 ? 0xffffffffu : (1u << n) - 1u;
  s.load = load.data();
  std::vector<int64_t> lsum(n, 0), level((size_t)(s.max_excl + 1) * D, 0);
  int64_t sum = 0, mx = 0;
  for (int i = 0; i < n; ++i)
    for (int d = 0; d < D; ++d) {
      lsum[i] += load[(size_t)i * D + d];
      level[d] += load[(size_t)i * D + d];
    }
  for (int d = 0; d < D; ++d) {
    sum += level[d];
    mx = level[d] > mx ? level[d] : mx;
  }
  s.lsum = lsum.data();
  s.level = level.data();
  s.consider(s.full, n, sum, mx);
  if (s.max_excl > 0) s.walk(0, 0, 0u, sum);
  return s.best;
}

uint64_t pad(uint64_t set, int n, int need) {
  int have = __builtin_popcountll(set);
  for (int i = 0; i < n && have < need; ++i)
    if (!(set & (1ull << i))) {
      set |= 1ull << i;
      ++have;
    }
  return set;
}

uint64_t cumutil(int n, const std::vector<int64_t>& load, int D, int need) {
  std::vector<int64_t> W(D), W2(D);
  uint64_t set = 1;  // the first micro-batch is always scheduled
  for (int d = 0; d < D; ++d) W[d] = load[d];
  for (int i = 1; i < n; ++i) {
    for (int d = 0; d < D; ++d) W2[d] = W[d] + load[(size_t)i * D + d];
    if (ratio_cmp(util_ratio(W2.data(), D), util_ratio(W.data(), D)) > 0) {
      set |= 1ull << i;
      W.swap(W2);
    }
  }
  return pad(set, n, need);
}

int peak_device(const int64_t* w, int D) {
  int p = 0;
  for (int d = 1; d < D; ++d)
    if (w[d] > w[p]) p = d;
  return p;
}

uint64_t diffpeak(int n, const std::vector<int64_t>& load, int D, int need) {
  std::vector<char> peak_taken(D, 0);
  uint64_t set = 1;
  peak_taken[peak_device(&load[0], D)] = 1;
  for (int i = 1; i < n; ++i) {
    const int p = peak_device(&load[(size_t)i * D], D);
    if (!peak_taken[p]) {
      peak_taken[p] = 1;
      set |= 1ull << i;
    }
  }
  return pad(set, n, need);
}

}  // namespace

int check_placement(const eb_placement* p, int L, int E, int D) {
  if (p->L != L || p->E != E || p->D != D)
    return set_error(EB_ERR_INVALID_ARG, "placement is for L=%d E=%d D=%d, not L=%d E=%d D=%d", p->L, p->E,
                     p->D, L, E, D);
  if (p->R < 1 || p->R > D || p->R > kDevMaxD)
    return set_error(EB_ERR_INVALID_ARG, "placement R=%d outside [1, min(D=%d, %d)]", p->R, D, kDevMaxD);
  if (p->copies == nullptr) return set_error(EB_ERR_INVALID_ARG, "placement copies is NULL");
  for (int l = 0; l < L; ++l)
    for (int e = 0; e < E; ++e) {
      const int32_t* c = p->copies + ((size_t)l * E + e) * p->R;
      if (c[0] < 0 || c[0] >= D)
        return set_error(EB_ERR_INVALID_ARG, "placement: expert %d of layer %d has no copy on a device", e, l);
      bool ended = false;
      for (int i = 1; i < p->R; ++i) {
        if (c[i] < 0) {
          if (c[i] != -1) return set_error(EB_ERR_INVALID_ARG, "placement: entry %d of (%d, %d) is %d", i, l, e, c[i]);
          ended = true;
        } else if (ended || c[i] >= D || c[i] <= c[i - 1]) {
          return set_error(EB_ERR_INVALID_ARG,
                           "placement: copies of expert %d at layer %d must be distinct devices < %d, ascending, "
                           "then -1", e, l, D);
        }
      }
    }
  return EB_OK;
}

void add_device_loads(const int32_t* counts, int E, int D, const eb_placement* p, int layer, int64_t* out) {
  if (p == nullptr) {
    const int per = E / D;
    for (int e = 0; e < E; ++e) out[e / per] += counts[e];
    return;
  }
  const int32_t* row = p->copies + (size_t)layer * E * p->R;
  for (int e = 0; e < E; ++e) {
    const int32_t* c = row + (size_t)e * p->R;
    int r = 1;
    while (r < p->R && c[r] >= 0) ++r;
    const int64_t q = counts[e] / r, rem = counts[e] % r;
    for (int i = 0; i < r; ++i) out[c[i]] += q + (i < rem ? 1 : 0);
  }
}

int schedule_impl(int32_t n_pool, const int32_t* pool_ids, const int32_t* counts, int32_t E,
                  int32_t D, int32_t m, int32_t policy, uint64_t* runset_mask,
                  int64_t* step_load, const int32_t* pool_layers, const eb_placement* placement) {
  if (runset_mask == nullptr) return set_error(EB_ERR_INVALID_ARG, "runset_mask is NULL");
  if (n_pool < 0 || n_pool > EB_MAX_POOL)
    return set_error(EB_ERR_INVALID_ARG, "n_pool=%d outside [0, %d]", n_pool, EB_MAX_POOL);
  if (E < 1 || D < 1 || E % D != 0)
    return set_error(EB_ERR_INVALID_ARG, "E=%d must be a positive multiple of D=%d", E, D);
  if (m < 1) return set_error(EB_ERR_INVALID_ARG, "m=%d must be >= 1", m);
  if (policy != EB_POLICY_MAXUTIL && policy != EB_POLICY_CUMUTIL && policy != EB_POLICY_DIFFPEAK)
    return set_error(EB_ERR_INVALID_ARG, "unknown policy %d", policy);
  if (n_pool > 0 && (pool_ids == nullptr || counts == nullptr))
    return set_error(EB_ERR_INVALID_ARG, "pool_ids/counts is NULL");
  for (int i = 0; i < n_pool; ++i) {
    if (pool_ids[i] < 0 || pool_ids[i] >= EB_MAX_POOL)
      return set_error(EB_ERR_INVALID_ARG, "pool_ids[%d]=%d outside [0, 64)", i, pool_ids[i]);
    if (i > 0 && pool_ids[i] <= pool_ids[i - 1])
      return set_error(EB_ERR_INVALID_ARG, "pool_ids must be strictly ascending");
  }
  if (placement != nullptr) {
    const int rc = check_placement(placement, placement->L, E, D);
    if (rc) return rc;
    if (n_pool > 0 && pool_layers == nullptr)
      return set_error(EB_ERR_INVALID_ARG, "pool_layers is NULL (required with a placement)");
    for (int i = 0; i < n_pool; ++i)
      if (pool_layers[i] < 0 || pool_layers[i] >= placement->L)
        return set_error(EB_ERR_INVALID_ARG, "pool_layers[%d]=%d outside [0, %d)", i, pool_layers[i],
                         placement->L);
  }
  if (policy == EB_POLICY_MAXUTIL && n_pool > EB_MAXUTIL_MAX_POOL)
    return set_error(EB_ERR_UNSUPPORTED, "MaxUtil enumerates up to 2^n subsets; n_pool=%d > %d",
                     n_pool, EB_MAXUTIL_MAX_POOL);
  *runset_mask = 0;
  if (n_pool == 0) {
    if (step_load) memset(step_load, 0, sizeof(int64_t) * (size_t)D);
    return EB_OK;
  }
  std::vector<int64_t> load((size_t)n_pool * D, 0);
  for (int i = 0; i < n_pool; ++i) {
    for (int e = 0; e < E; ++e)
      if (counts[(size_t)i * E + e] < 0) return set_error(EB_ERR_INVALID_ARG, "negative count at [%d][%d]", i, e);
    add_device_loads(counts + (size_t)i * E, E, D, placement, placement ? pool_layers[i] : 0,
                     load.data() + (size_t)i * D);
  }
  const int need = m < n_pool ? m : n_pool;
  uint64_t set;
  if (policy == EB_POLICY_MAXUTIL)
    set = maxutil(n_pool, load, D, need);
  else if (policy == EB_POLICY_CUMUTIL)
    set = cumutil(n_pool, load, D, need);
  else
    set = diffpeak(n_pool, load, D, need);
  uint64_t mask = 0;
  for (int i = 0; i < n_pool; ++i)
    if (set & (1ull << i)) mask |= 1ull << pool_ids[i];
  *runset_mask = mask;
  if (step_load) {
    std::vector<int64_t> W(D);
    for (int d = 0; d < D; ++d) W[d] = 0;
    for (int i = 0; i < n_pool; ++i)
      if (set & (1ull << i))
        for (int d = 0; d < D; ++d) W[d] += load[(size_t)i * D + d];
    memcpy(step_load, W.data(), sizeof(int64_t) * (size_t)D);
  }
  return EB_OK;
}

}  // namespace eb
