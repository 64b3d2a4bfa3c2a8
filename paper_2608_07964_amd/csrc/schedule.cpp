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

uint32_t maxutil(int n, const std::vector<int64_t>& load, int D, int need) {
  std::vector<int64_t> W(D, 0);
  uint32_t best = 0;
  Ratio best_u{0, 1};
  int best_size = -1;
  uint32_t gray = 0;
  int size = 0;
  const uint32_t total = 1u << n;
  for (uint32_t i = 1; i < total; ++i) {
    const int bit = __builtin_ctz(i);
    const uint32_t g = gray ^ (1u << bit);
    const int64_t* lb = &load[(size_t)bit * D];
    if (g & (1u << bit)) {
      for (int d = 0; d < D; ++d) W[d] += lb[d];
      ++size;
    } else {
      for (int d = 0; d < D; ++d) W[d] -= lb[d];
      --size;
    }
    gray = g;
    if (size < need) continue;
    const Ratio u = util_ratio(W.data(), D);
    bool take;
    if (best_size < 0) {
      take = true;
    } else {
      const int c = ratio_cmp(u, best_u);
      take = c > 0 || (c == 0 && (size > best_size || (size == best_size && lex_smaller(g, best))));
    }
    if (take) {
      best = g;
      best_u = u;
      best_size = size;
    }
  }
  return best;
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

int schedule_impl(int32_t n_pool, const int32_t* pool_ids, const int32_t* counts, int32_t E,
                  int32_t D, int32_t m, int32_t policy, uint64_t* runset_mask,
                  int64_t* step_load) {
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
  if (policy == EB_POLICY_MAXUTIL && n_pool > EB_MAXUTIL_MAX_POOL)
    return set_error(EB_ERR_UNSUPPORTED, "MaxUtil enumerates 2^n subsets; n_pool=%d > %d",
                     n_pool, EB_MAXUTIL_MAX_POOL);
  *runset_mask = 0;
  if (n_pool == 0) {
    if (step_load) memset(step_load, 0, sizeof(int64_t) * (size_t)D);
    return EB_OK;
  }
  const int per = E / D;
  std::vector<int64_t> load((size_t)n_pool * D, 0);
  for (int i = 0; i < n_pool; ++i)
    for (int e = 0; e < E; ++e) {
      const int32_t c = counts[(size_t)i * E + e];
      if (c < 0) return set_error(EB_ERR_INVALID_ARG, "negative count at [%d][%d]", i, e);
      load[(size_t)i * D + e / per] += c;
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
