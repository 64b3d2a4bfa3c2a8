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

// A kernel's view of a per-step table: in the kernel arguments (the host
// built it) or in device memory (the device-side scheduler wrote it).  The
// kernels take the live counts (entries, chunks, tokens) from the table
// itself, so a grid sized for the largest step is cut to the live one.
template <class Tab>
struct ByValue {
  Tab v;
  __device__ __forceinline__ const Tab& get() const { return v; }
};
template <class Tab>
struct InMemory {
  const Tab* p;
  __device__ __forceinline__ const Tab& get() const { return *p; }
};

// Per-layer expert weight tables, passed by value.
struct WeightTable {
  const void* gu[EB_MAX_LAYERS];           // [E+S][2F][H]
  const void* dn[EB_MAX_LAYERS];           // [E+S][H][F]
};

// Grouped-GEMM problem of one step.
struct GroupedProblem {
  int32_t H, F, E, S;                      // E+S expert slots per layer
  int32_t P;                               // grouped rows the buffers hold (the live
                                           // rows or, device-scheduled, the largest step's)
  const int32_t* offsets;                  // [L*(E+S)+1]
  const int32_t* P_live;                   // device scalar: the live grouped rows
                                           // (offsets[L*(E+S)])
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

// A pointer read from a table in device memory is a generic address to the
// compiler, so its loads and stores become flat instructions, which also
// count on the LDS counter (every wait for them waits for LDS traffic too,
// and the other way round).  Every table pointer here points into device
// global memory; rebuilt from its integer value in the global address space,
// it (and every pointer derived from it) gets global loads and stores; a
// null pointer stays null.
template <class T>
__device__ __forceinline__ T* in_global(T* p) {
  return (T*)(__attribute__((address_space(1))) T*)(uintptr_t)p;
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

// ---- device-scheduled pass --------------------------------------------------
constexpr int kDevMaxD = 64;                       // virtual devices the device scheduler handles
constexpr int kDevRouteSlots = (EB_MAX_POOL + kRouteBatch - 1) / kRouteBatch;
constexpr int kDevMaxKeyWords = 15360 / 32;        // bitmap words over L * E <= 15360 keys

// State of a device-scheduled pass, in device memory.
struct DevPassState {
  int32_t layer[EB_MAX_POOL];  // l_j; L once micro-batch j has finished
  int32_t steps;               // steps scheduled so far
};

// Everything the scheduler kernel needs, by value.  Micro-batch j's buffers
// sit at j * (its size) from each base: a (a_stride bytes), z [T][E],
// idx / w [T][k], x [T][H] fp32, counts [E].
struct DevPassArgs {
  int32_t N, T, L, H, E, k, S, D, m, policy;
  int32_t max_records;           // steps the record arrays hold (N * L)
  int32_t tag;                   // pass tag echoed in the status word (16 bits)
  void* a;
  size_t a_stride;
  float* z;
  int32_t* idx;
  float* w;
  float* x;
  int32_t* counts;
  const float* gain;             // [L][H]
  const float* bias;             // [L][E]
  const void* Wg[EB_MAX_LAYERS]; // router weights of each layer
  DevPassState* state;
  RunTable* rt;                  // the step's run table
  RouteBatch* rb;                // [kDevRouteSlots] routing after the step
  uint64_t* rec_mask;            // [max_records] RunSet (bit j = micro-batch j)
  int32_t* rec_layers;           // [max_records][N] layer of each member, -1 if not run
  int64_t* rec_load;             // [max_records][D] the step's per-device workload
  int32_t* rec_groups;           // [max_records] distinct (layer, expert) groups
  int32_t* rec_layer_loads;      // [N][L][D] per-device load of (j, l), -1 until seen
  unsigned long long* status;    // host-mapped: tag << 48 | steps << 16 | max_j (L - l_j)
  const int32_t* place;          // [L][E][R] expert copies (eb_placement), or NULL: E/D
                                 // contiguous experts per device
  int32_t R;                     // copy entries per expert of place
};

hipError_t launch_pass_init(const DevPassArgs& A, hipStream_t s);
hipError_t launch_sched_step(const DevPassArgs& A, hipStream_t s);
// Permute, GEMMs and combine of one device-scheduled step (api.cpp);
// returns EB_OK or an EB_ERR_* code.
int enqueue_step_dev(const eb_model_desc& d, int N, int T, const RunTable* rt, const WeightTable& wt,
                     void* ws, void* o, int32_t* inv, hipStream_t s);

// ---- launchers (return hipError_t of the launch) ---------------------------
hipError_t launch_route_batch(const eb_model_desc& d, const RouteBatch& rb, hipStream_t s);
// A batch table in device memory (written by the device-side scheduler);
// grids cover max_entries entries of T tokens.  Only for stacks whose
// routing needs no launch per entry (route_batch_device_ok).
bool route_batch_device_ok(const eb_model_desc& d);
// Whether the top-k of this stack reads the logits back from global memory
// (fp32 stacks off the one-workgroup-per-token path), so z must be stored.
bool route_logits_required(const eb_model_desc& d);
hipError_t launch_route_batch_dev(const eb_model_desc& d, const RouteBatch* rb, int max_entries, int T,
                                  hipStream_t s);
hipError_t launch_route(const eb_model_desc& d, int T, const float* x, const float* gain,
                        const void* Wg, const float* bias, void* a_out, float* logits,
                        int32_t* idx, float* w, int32_t* counts, hipStream_t s);

hipError_t launch_perm_count(const RunTable& rt, int n_chunks, int32_t* hist, hipStream_t s);
hipError_t launch_perm_scan(const RunTable& rt, const int32_t* hist, int32_t* chunk_base,
                            int32_t* offsets, int4* tiles, int32_t* n_tiles, int4* groups,
                            int32_t* n_groups, int bm, int max_tiles, int32_t* work_ctr,
                            hipStream_t s);
hipError_t launch_perm_scatter(const RunTable& rt, int n_chunks, int elem_bytes,
                               const int32_t* chunk_base, int32_t* perm, int32_t* inv,
                               void* a_perm, hipStream_t s);

// Workspace buffers of one step (see the workspace layout in api.cpp).
struct StepBuffers {
  int32_t* hist;
  int32_t* chunk_base;
  int32_t* offsets;
  int4* tiles;
  int32_t* n_tiles;
  int4* groups;
  int32_t* n_groups;
  int32_t* work_ctr;
  int32_t max_tiles;
  int32_t* perm;
  int32_t* inv;
  void* a_perm;
};

// Count, scan, scatter and gather of a step whose run table a device-side
// scheduler wrote to `rt` (device memory); grids cover max_chunks chunks and
// max_tokens tokens, the largest step's.
hipError_t launch_permute_dev(const eb_model_desc& d, const RunTable* rt, int max_chunks,
                              int max_tokens, const StepBuffers& b, hipStream_t s);

// Row-block height of the grouped GEMM tiles for a dtype.
int gemm_bm(int dtype);

// Expert weights in the layout the grouped GEMMs read (bf16: packed blocks,
// see gemm.hip; fp32: row-major, a copy).  n matrices of N x K.
hipError_t launch_pack_weights(int dtype, int gateup, int n, int N, int K, int F, const void* src,
                               void* dst, hipStream_t s);

hipError_t launch_gateup(int dtype, const GroupedProblem& p, const WeightTable& wt,
                         const void* a_perm, void* h, hipStream_t s);
// sum_halves false (split K only): the fp32 halves stay in p.partial and o
// is not written (launch_combine_split_dev reads them).
hipError_t launch_down(int dtype, const GroupedProblem& p, const WeightTable& wt,
                       const void* h, void* o, hipStream_t s, bool sum_halves = true);

hipError_t launch_combine(const RunTable& rt, int dtype, const void* o, const int32_t* inv,
                          hipStream_t s);
hipError_t launch_combine_dev(const RunTable* rt, int slots, int max_tokens, int dtype, const void* o,
                              const int32_t* inv, hipStream_t s);
// bf16 combine straight from a split-K down GEMM's fp32 halves (part and
// part + stride), rounded as the split-K sum would round them.  slots: k + S
// (the device-resident table's, known to the caller).
hipError_t launch_combine_split_dev(const RunTable* rt, int slots, int max_tokens, const float* part, long long stride,
                                    const int32_t* inv, hipStream_t s);

// Profiling hooks (api.cpp): bracket one launch of kernel class `kind`.
void prof_start(int kind, hipStream_t s);
void prof_stop(int kind, hipStream_t s);

// Body of easybalance_moe_step on workspace ws (api.cpp).  static_scratch:
// ws is the library's static scratch array (a shortfall is then
// EB_ERR_UNSUPPORTED instead of EB_ERR_WORKSPACE_TOO_SMALL).
int moe_step_common(const eb_model_desc* desc, int32_t n_run, const eb_work* run, const void* const* W_gu,
                    const void* const* W_dn, void* ws, size_t ws_bytes, void* o_out, int32_t* inv_out,
                    const eb_step_views* views, void* stream, bool static_scratch);

// Host scheduler (schedule.cpp); returns EB_OK or an EB_ERR_* code and sets
// the message through set_error.
int schedule_impl(int32_t n_pool, const int32_t* pool_ids, const int32_t* counts, int32_t E,
                  int32_t D, int32_t m, int32_t policy, uint64_t* runset_mask,
                  int64_t* step_load, const int32_t* pool_layers, const eb_placement* placement);
// Checks a placement against the model's L, E, D (EB_OK or EB_ERR_INVALID_ARG).
int check_placement(const eb_placement* p, int L, int E, int D);
// out[d] += pairs of counts[E] that device d carries at `layer` (placement
// NULL: E/D contiguous experts per device; else the even split over each
// expert's copies, the lower copies taking the remainder).
void add_device_loads(const int32_t* counts, int E, int D, const eb_placement* p, int layer, int64_t* out);
int set_error(int code, const char* fmt, ...);

}  // namespace eb
