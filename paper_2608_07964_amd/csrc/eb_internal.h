// Internal declarations shared by the translation units of libeasybalance.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "easybalance.h"

namespace eb {

constexpr int kWave = 64;
constexpr int kPermChunk = 256;     // tokens per permutation block (one per thread)
constexpr int kMaxSlots = 16;       // k + S per token handled by the permutation

// Per-step table of RunSet entries, passed by value as a kernel argument.
struct RunTable {
  int32_t n;                               // entries
  int32_t E, k, S, L, H;
  int32_t chunk_base[EB_MAX_RUN + 1];      // prefix sums of ceil(T / kPermChunk)
  int32_t tok_base[EB_MAX_RUN + 1];        // prefix sums of T
  int32_t layer[EB_MAX_RUN];
  const int32_t* idx[EB_MAX_RUN];
  const void* a[EB_MAX_RUN];
  const float* w[EB_MAX_RUN];
  float* x[EB_MAX_RUN];
};

// Per-layer expert weight tables, passed by value.
struct WeightTable {
  const void* gu[EB_MAX_LAYERS];           // [E+S][2F][H]
  const void* dn[EB_MAX_LAYERS];           // [E+S][H][F]
};

// Grouped-GEMM problem of one step.
struct GroupedProblem {
  int32_t H, F, E, S;                      // E+S expert slots per layer
  int32_t P;                               // grouped rows
  const int32_t* offsets;                  // [L*(E+S)+1]
  const int4* tiles;                       // [n_tiles] the row block's group: (key, first row,
                                           // rows, index of the group's first row block)
  const int32_t* n_tiles;                  // device scalar: row blocks over all groups
  const int4* groups;                      // [n_groups] (key, first row, rows, first row block)
  const int32_t* n_groups;                 // device scalar: non-empty keys
  int32_t max_tiles;                       // grid bound
  int32_t* work_ctr;                       // [8] per-XCD work counters of this launch, zeroed
  int32_t ksplit;                          // 1, or 2: K halves computed by separate items
  float* partial;                          // ksplit 2: [2][P][N] fp32 partial sums
};

// K split of the down GEMM: two halves for long K (a rule on the shape only,
// so every schedule computes a row the same way).
inline int down_ksplit(int dtype, int F) { return dtype == EB_DTYPE_BF16 && F >= 8192 ? 2 : 1; }

constexpr int kWorkCounters = 16;          // 8 per grouped GEMM launch (gate/up, down)

// Device-side entry lookup: largest rho with base[rho] <= v (bases ascending).
__device__ __forceinline__ int find_entry(const int32_t* base, int n, int v) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (base[mid] <= v) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Routing of up to kRouteBatch micro-batches in one set of launches: entry i
// holds tokens tok0[i] .. tok0[i+1]-1 of the batch and 32-token blocks
// blk0[i] .. blk0[i+1]-1; gain/Wg/bias are those of the entry's layer.
constexpr int kRouteBatch = 32;
struct RouteEntry {
  const float* x;
  const float* gain;
  const void* Wg;
  const float* bias;
  void* a;
  float* z;
  int32_t* idx;
  float* w;
  int32_t* counts;
};
struct RouteBatch {
  int32_t n;
  int32_t tok0[kRouteBatch + 1];
  int32_t blk0[kRouteBatch + 1];
  RouteEntry e[kRouteBatch];
};

// ---- launchers (return hipError_t of the launch) ---------------------------
hipError_t launch_route_batch(const eb_model_desc& d, const RouteBatch& rb, hipStream_t s);
hipError_t launch_route(const eb_model_desc& d, int T, const float* x, const float* gain,
                        const void* Wg, const float* bias, void* a_out, float* logits,
                        int32_t* idx, float* w, int32_t* counts, hipStream_t s);

hipError_t launch_perm_count(const RunTable& rt, int n_chunks, int32_t* hist, hipStream_t s);
hipError_t launch_perm_scan(const RunTable& rt, int n_chunks, const int32_t* hist,
                            int32_t* chunk_base, int32_t* offsets, int4* tiles,
                            int32_t* n_tiles, int4* groups, int32_t* n_groups, int bm,
                            int max_tiles, int32_t* work_ctr, hipStream_t s);
hipError_t launch_perm_scatter(const RunTable& rt, int n_chunks, int P, int elem_bytes,
                               const int32_t* chunk_base, int32_t* perm, int32_t* inv,
                               void* a_perm, hipStream_t s);

// Row-block height of the grouped GEMM tiles for a dtype.
int gemm_bm(int dtype);

// Expert weights in the layout the grouped GEMMs read (bf16: packed blocks,
// see gemm.hip; fp32: row-major, a copy).  n matrices of N x K.
hipError_t launch_pack_weights(int dtype, int gateup, int n, int N, int K, int F, const void* src,
                               void* dst, hipStream_t s);

hipError_t launch_gateup(int dtype, const GroupedProblem& p, const WeightTable& wt,
                         const void* a_perm, void* h, hipStream_t s);
hipError_t launch_down(int dtype, const GroupedProblem& p, const WeightTable& wt,
                       const void* h, void* o, hipStream_t s);

hipError_t launch_combine(const RunTable& rt, int total_tokens, int dtype, const void* o,
                          const int32_t* inv, hipStream_t s);

// Profiling hooks (api.cpp): bracket one launch of kernel class `kind`.
void prof_start(int kind, hipStream_t s);
void prof_stop(int kind, hipStream_t s);

// Host scheduler (schedule.cpp); returns EB_OK or an EB_ERR_* code and sets
// the message through set_error.
int schedule_impl(int32_t n_pool, const int32_t* pool_ids, const int32_t* counts, int32_t E,
                  int32_t D, int32_t m, int32_t policy, uint64_t* runset_mask,
                  int64_t* step_load);
int set_error(int code, const char* fmt, ...);

}  // namespace eb
