// One pass of Algorithm 1 (Section 4.2) driven natively: the host loop of
// EasyBalance over the library's own entry points.
//
//   route every micro-batch at layer 0                    (Attn_Route_Dispatch)
//   while the pool is not empty:
//     RunSet <- Schedule(pool, m)                          (the pool's expert counts)
//     expert FFNs of RunSet jointly, then the combine      (MoECompute_Combine)
//     l_j += 1 for j in RunSet; route those not finished
//
// Host-scheduled, the only host<->device synchronisation per step is the
// copy of the pool's expert counts into pinned host memory that the
// scheduler needs; everything else is queued on the caller's stream without
// waiting.  Device-scheduled (EB_PASS_DEVICE_SCHEDULE), a one-workgroup
// kernel at the start of each step makes the same choice on the GPU and
// writes the step's tables, and the host queues steps ahead of the GPU: it
// never waits for the counts.  It queues only steps that must run: after s
// steps with the furthest-behind micro-batch L - l layers short, at least
// s + (L - l) steps are needed in all, and the scheduler kernel publishes
// (s, L - l) in host memory as soon as it has chosen.
#include <hip/hip_runtime.h>
#include <string.h>

#include <algorithm>
#include <chrono>
#include <vector>

#include "eb_internal.h"

namespace eb {
namespace {

constexpr size_t kAlignP = 256;
size_t align_p(size_t v) { return (v + kAlignP - 1) / kAlignP * kAlignP; }

struct PassLayout {
  size_t a, logits, idx, w, counts, o, inv, ws, ws_bytes;
  // device-scheduled pass: scheduler state, step tables, records (N * L steps)
  size_t dstate, drt, drb, rec_mask, rec_layers, rec_load, rec_groups, rec_ll, place;
  size_t total;
};

PassLayout pass_layout(const eb_model_desc& d, int N, int T) {
  const size_t eb = d.dtype == EB_DTYPE_BF16 ? 2 : 4;
  const size_t NT = (size_t)N * T, slots = (size_t)(d.k + d.S);
  PassLayout p{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_p(bytes);
    return o;
  };
  p.a = take(eb * NT * d.H);
  p.logits = take(sizeof(float) * NT * d.E);
  p.idx = take(sizeof(int32_t) * NT * d.k);
  p.w = take(sizeof(float) * NT * d.k);
  p.counts = take(sizeof(int32_t) * (size_t)N * d.E);
  p.o = take(eb * NT * slots * d.H);
  p.inv = take(sizeof(int32_t) * NT * slots);
  std::vector<int32_t> Ts(N, T);
  size_t wsb = 0;
  easybalance_moe_step_workspace_size(&d, N, Ts.data(), &wsb);
  p.ws_bytes = wsb;
  p.ws = take(wsb);
  const size_t steps = (size_t)N * d.L;  // every step advances a micro-batch by a layer
  p.dstate = take(sizeof(DevPassState));
  p.drt = take(sizeof(RunTable));
  p.drb = take(sizeof(RouteBatch) * kDevRouteSlots);
  p.rec_mask = take(sizeof(uint64_t) * steps);
  p.rec_layers = take(sizeof(int32_t) * steps * N);
  p.rec_load = take(sizeof(int64_t) * steps * d.D);
  p.rec_groups = take(sizeof(int32_t) * steps);
  p.rec_ll = take(sizeof(int32_t) * (size_t)N * d.L * d.D);
  // a placement's copy table, R <= min(D, 64) entries per (layer, expert)
  p.place = take(sizeof(int32_t) * (size_t)d.L * d.E * std::min(d.D, kDevMaxD));
  p.total = off;
  return p;
}

// Pinned host buffer for the counts, one per host thread, grown on demand.
struct PinnedCounts {
  int32_t* p = nullptr;
  size_t n = 0;
  ~PinnedCounts() {
    if (p) (void)hipHostFree(p);
  }
  int32_t* get(size_t count) {
    if (count > n) {
      if (p) (void)hipHostFree(p);
      p = nullptr;
      n = 0;
      if (hipHostMalloc(reinterpret_cast<void**>(&p), count * sizeof(int32_t), hipHostMallocDefault) != hipSuccess)
        return nullptr;
      n = count;
    }
    return p;
  }
};
thread_local PinnedCounts t_pinned;

// Host-mapped status word of device-scheduled passes, one per host thread;
// the tag tells this pass's words from an earlier pass's.
struct PinnedStatus {
  unsigned long long* h = nullptr;
  unsigned long long* d = nullptr;
  uint32_t tag = 0;
  ~PinnedStatus() {
    if (h) (void)hipHostFree(h);
  }
  bool ready() {
    if (h) return true;
    void* p = nullptr;
    if (hipHostMalloc(&p, 256, hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess) return false;
    void* dp = nullptr;
    if (hipHostGetDevicePointer(&dp, p, 0) != hipSuccess) {
      (void)hipHostFree(p);
      return false;
    }
    h = static_cast<unsigned long long*>(p);
    d = static_cast<unsigned long long*>(dp);
    __atomic_store_n(h, 0ull, __ATOMIC_RELEASE);
    return true;
  }
};
thread_local PinnedStatus t_status;

struct PassStatus {
  int steps, maxlag;
};

// Waits until the scheduler kernel of this pass (tag) has reported at least
// `steps` steps.  The stream is polled now and then: if it has drained or
// failed without the word, or a minute passes, the wait ends with an error.
int wait_status(hipStream_t s, uint32_t tag, int steps, PassStatus* out) {
  const auto t0 = std::chrono::steady_clock::now();
  for (long iter = 0;; ++iter) {
    const unsigned long long v = __atomic_load_n(t_status.h, __ATOMIC_ACQUIRE);
    if ((uint32_t)(v >> 48) == (tag & 0xffffu) && (int)((v >> 16) & 0xffffffffull) >= steps) {
      out->steps = (int)((v >> 16) & 0xffffffffull);
      out->maxlag = (int)(v & 0xffffull);
      return EB_OK;
    }
    if ((iter & 1023) == 1023) {
      const hipError_t q = hipStreamQuery(s);
      if (q == hipSuccess) {
        const unsigned long long w = __atomic_load_n(t_status.h, __ATOMIC_ACQUIRE);
        if ((uint32_t)(w >> 48) == (tag & 0xffffu) && (int)((w >> 16) & 0xffffffffull) >= steps) continue;
        return set_error(EB_ERR_HIP, "device-scheduled pass: the stream drained before step %d reported", steps);
      }
      if (q != hipErrorNotReady)
        return set_error(EB_ERR_HIP, "device-scheduled pass: %s", hipGetErrorString(q));
      if (std::chrono::steady_clock::now() - t0 > std::chrono::seconds(60))
        return set_error(EB_ERR_HIP, "device-scheduled pass: no report of step %d within 60 s", steps);
    }
    __builtin_ia32_pause();
  }
}

// Algorithm 1 with the Schedule step on the GPU (see the file comment).
// Inputs as validated by easybalance_run_pass; the layer-0 routing is queued.
int run_pass_device(const eb_model_desc& d, int N, int T, const PassLayout& P, uint8_t* base, float* x,
                    const float* gain, const void* const* Wg, const float* bias,
                    const void* const* W_gu, const void* const* W_dn, int policy, int m,
                    int max_steps, int32_t* n_steps_out, uint64_t* runsets_out, int32_t* layers_out,
                    int64_t* step_load_out, int32_t* groups_out, int32_t* layer_loads_out,
                    const eb_placement* placement, hipStream_t s) {
  const size_t eb = d.dtype == EB_DTYPE_BF16 ? 2 : 4;
  DevPassArgs A;
  memset(&A, 0, sizeof(A));
  A.N = N;
  A.T = T;
  A.L = d.L;
  A.H = d.H;
  A.E = d.E;
  A.k = d.k;
  A.S = d.S;
  A.D = d.D;
  A.m = m;
  A.policy = policy;
  A.max_records = N * d.L;
  if ((++t_status.tag & 0xffffu) == 0) ++t_status.tag;  // tag 0 is the word's initial value
  A.tag = (int32_t)(t_status.tag & 0xffffu);
  A.a = base + P.a;
  A.a_stride = eb * (size_t)T * d.H;
  A.z = reinterpret_cast<float*>(base + P.logits);
  A.idx = reinterpret_cast<int32_t*>(base + P.idx);
  A.w = reinterpret_cast<float*>(base + P.w);
  A.x = x;
  A.counts = reinterpret_cast<int32_t*>(base + P.counts);
  A.gain = gain;
  A.bias = bias;
  for (int l = 0; l < d.L; ++l) A.Wg[l] = Wg[l];
  A.state = reinterpret_cast<DevPassState*>(base + P.dstate);
  A.rt = reinterpret_cast<RunTable*>(base + P.drt);
  A.rb = reinterpret_cast<RouteBatch*>(base + P.drb);
  A.rec_mask = reinterpret_cast<uint64_t*>(base + P.rec_mask);
  A.rec_layers = reinterpret_cast<int32_t*>(base + P.rec_layers);
  A.rec_load = reinterpret_cast<int64_t*>(base + P.rec_load);
  A.rec_groups = reinterpret_cast<int32_t*>(base + P.rec_groups);
  A.rec_layer_loads = reinterpret_cast<int32_t*>(base + P.rec_ll);
  A.status = t_status.d;
  if (placement) {
    // the copy table goes to device memory for the scheduler kernel; the
    // wait makes the caller's table free for reuse when the call returns
    int32_t* dplace = reinterpret_cast<int32_t*>(base + P.place);
    const size_t bytes = sizeof(int32_t) * (size_t)d.L * d.E * placement->R;
    if (hipMemcpyAsync(dplace, placement->copies, bytes, hipMemcpyHostToDevice, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
      return set_error(EB_ERR_HIP, "placement copy: %s", hipGetErrorString(hipGetLastError()));
    A.place = dplace;
    A.R = placement->R;
  }
  WeightTable wt;
  memset(&wt, 0, sizeof(wt));
  for (int l = 0; l < d.L; ++l) {
    wt.gu[l] = W_gu[l];
    wt.dn[l] = W_dn[l];
  }
  void* o = base + P.o;
  int32_t* inv = reinterpret_cast<int32_t*>(base + P.inv);
  void* ws = base + P.ws;
  if (launch_pass_init(A, s) != hipSuccess) return set_error(EB_ERR_HIP, "pass init launch");

  int rc;
  auto enqueue_step = [&]() -> int {
    if (launch_sched_step(A, s) != hipSuccess) return set_error(EB_ERR_HIP, "scheduler launch");
    if ((rc = enqueue_step_dev(d, N, T, A.rt, wt, ws, o, inv, s))) return rc;
    for (int b = 0; b * kRouteBatch < N; ++b)
      if (launch_route_batch_dev(d, A.rb + b, std::min(kRouteBatch, N - b * kRouteBatch), T, s) != hipSuccess)
        return set_error(EB_ERR_HIP, "route launch");
    return EB_OK;
  };
  // every micro-batch needs L steps; queue what is known to run, then wait
  // for a report one step behind the last queued one
  int queued = 0, bound = d.L;
  PassStatus st{0, 0};
  for (;;) {
    for (; queued < bound; ++queued)
      if ((rc = enqueue_step())) return rc;
    if ((rc = wait_status(s, A.tag, queued >= 2 ? queued - 1 : queued, &st))) return rc;
    if (st.maxlag == 0) break;  // st.steps == queued: the pass is complete
    if (st.steps + st.maxlag == queued) {
      if ((rc = wait_status(s, A.tag, queued, &st))) return rc;
      if (st.maxlag == 0) break;
    }
    if (st.steps + st.maxlag <= queued)
      return set_error(EB_ERR_HIP, "device-scheduled pass: report (%d steps, %d to go) below %d queued", st.steps,
                       st.maxlag, queued);
    bound = st.steps + st.maxlag;
  }
  const int n_steps = queued;
  if (n_steps_out) *n_steps_out = n_steps;
  const int rec = std::min(n_steps, max_steps);
  auto fetch = [&](void* dst, const void* src, size_t bytes) -> int {
    if (bytes == 0) return EB_OK;
    if (hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, s) != hipSuccess)
      return set_error(EB_ERR_HIP, "record copy");
    return EB_OK;
  };
  if (runsets_out && (rc = fetch(runsets_out, A.rec_mask, sizeof(uint64_t) * rec))) return rc;
  if (layers_out && (rc = fetch(layers_out, A.rec_layers, sizeof(int32_t) * (size_t)rec * N))) return rc;
  if (step_load_out && (rc = fetch(step_load_out, A.rec_load, sizeof(int64_t) * (size_t)rec * d.D))) return rc;
  if (groups_out && (rc = fetch(groups_out, A.rec_groups, sizeof(int32_t) * rec))) return rc;
  if (layer_loads_out &&
      (rc = fetch(layer_loads_out, A.rec_layer_loads, sizeof(int32_t) * (size_t)N * d.L * d.D)))
    return rc;
  if ((runsets_out || layers_out || step_load_out || groups_out || layer_loads_out) &&
      hipStreamSynchronize(s) != hipSuccess)
    return set_error(EB_ERR_HIP, "record copy: %s", hipGetErrorString(hipGetLastError()));
  return EB_OK;
}

}  // namespace
}  // namespace eb

using namespace eb;

extern "C" {

int easybalance_pass_state_size(const eb_model_desc* desc, int32_t N, int32_t T, size_t* bytes) {
  if (desc == nullptr || bytes == nullptr) return set_error(EB_ERR_INVALID_ARG, "desc/bytes is NULL");
  if (N < 1 || N > EB_MAX_POOL || T < 1) return set_error(EB_ERR_INVALID_ARG, "N=%d T=%d out of range", N, T);
  size_t wsb = 0;
  std::vector<int32_t> Ts(N, T);
  const int rc = easybalance_moe_step_workspace_size(desc, N, Ts.data(), &wsb);
  if (rc) return rc;
  *bytes = pass_layout(*desc, N, T).total;
  return EB_OK;
}

int easybalance_run_pass(const eb_model_desc* desc, int32_t N, int32_t T, float* x,
                         const float* gain, const void* const* Wg, const float* bias,
                         const void* const* W_gu, const void* const* W_dn, int32_t policy,
                         int32_t m, void* state, size_t state_bytes, int32_t max_steps,
                         int32_t* n_steps_out, uint64_t* runsets_out, int32_t* layers_out,
                         int64_t* step_load_out, int32_t* groups_out, int32_t* layer_loads_out,
                         const eb_placement* placement, void* stream) {
  size_t need = 0;
  int rc = easybalance_pass_state_size(desc, N, T, &need);
  if (rc) return rc;
  const eb_model_desc& d = *desc;
  if (x == nullptr || gain == nullptr || Wg == nullptr || bias == nullptr || W_gu == nullptr ||
      W_dn == nullptr)
    return set_error(EB_ERR_INVALID_ARG, "a required pass pointer is NULL");
  const bool device = (policy & EB_PASS_DEVICE_SCHEDULE) != 0;
  policy &= ~EB_PASS_DEVICE_SCHEDULE;
  if (policy < EB_POLICY_MAXUTIL || policy > EB_POLICY_LOCKSTEP)
    return set_error(EB_ERR_INVALID_ARG, "policy %d unknown", policy);
  if (policy == EB_POLICY_MAXUTIL && N > EB_MAXUTIL_MAX_POOL)
    return set_error(EB_ERR_UNSUPPORTED, "MaxUtil enumerates subsets of at most %d micro-batches",
                     EB_MAXUTIL_MAX_POOL);
  if (m < 1) return set_error(EB_ERR_INVALID_ARG, "m=%d < 1", m);
  if (device && d.D > kDevMaxD)
    return set_error(EB_ERR_UNSUPPORTED, "device-scheduled pass: D=%d > %d", d.D, kDevMaxD);
  if (device && !route_batch_device_ok(d))
    return set_error(EB_ERR_UNSUPPORTED, "device-scheduled pass: fp32 routing with E=%d needs a launch per entry",
                     d.E);
  if (state == nullptr || (reinterpret_cast<uintptr_t>(state) % kAlignP) != 0)
    return set_error(EB_ERR_INVALID_ARG, "state must be non-NULL and 256-byte aligned");
  if (state_bytes < need)
    return set_error(EB_ERR_WORKSPACE_TOO_SMALL, "state %zu < %zu bytes", state_bytes, need);
  if (max_steps < 0 || ((runsets_out || layers_out || step_load_out || groups_out) && max_steps == 0))
    return set_error(EB_ERR_INVALID_ARG, "max_steps=%d", max_steps);
  if (placement && (rc = check_placement(placement, d.L, d.E, d.D))) return rc;

  const PassLayout P = pass_layout(d, N, T);
  uint8_t* base = static_cast<uint8_t*>(state);
  const size_t eb = d.dtype == EB_DTYPE_BF16 ? 2 : 4;
  auto a_of = [&](int j) { return base + P.a + eb * (size_t)j * T * d.H; };
  auto logits_of = [&](int j) { return reinterpret_cast<float*>(base + P.logits) + (size_t)j * T * d.E; };
  auto idx_of = [&](int j) { return reinterpret_cast<int32_t*>(base + P.idx) + (size_t)j * T * d.k; };
  auto w_of = [&](int j) { return reinterpret_cast<float*>(base + P.w) + (size_t)j * T * d.k; };
  int32_t* counts_dev = reinterpret_cast<int32_t*>(base + P.counts);
  auto x_of = [&](int j) { return x + (size_t)j * T * d.H; };
  void* o = base + P.o;
  int32_t* inv = reinterpret_cast<int32_t*>(base + P.inv);
  void* ws = base + P.ws;
  hipStream_t s = static_cast<hipStream_t>(stream);

  if (layer_loads_out) {
    for (size_t i = 0; i < (size_t)N * d.L * d.D; ++i) layer_loads_out[i] = -1;
  }

  for (int l = 0; l < d.L; ++l)
    if (Wg[l] == nullptr || W_gu[l] == nullptr || W_dn[l] == nullptr)
      return set_error(EB_ERR_INVALID_ARG, "weights of layer %d are NULL", l);
  std::vector<int32_t> layer(N, 0), pool(N);
  // routes micro-batches js (each at its layer) in batches of kRouteBatch
  auto route = [&](const std::vector<int32_t>& js) -> int {
    for (size_t b = 0; b < js.size(); b += kRouteBatch) {
      RouteBatch rb;
      rb.n = (int)std::min<size_t>(kRouteBatch, js.size() - b);
      rb.tok0[0] = 0;
      rb.blk0[0] = 0;
      for (int i = 0; i < rb.n; ++i) {
        const int j = js[b + i], l = layer[j];
        rb.tok0[i + 1] = rb.tok0[i] + T;
        rb.blk0[i + 1] = rb.blk0[i] + (T + 31) / 32;
        rb.e[i] = RouteEntry{x_of(j), gain + (size_t)l * d.H, Wg[l], bias + (size_t)l * d.E, a_of(j),
                             logits_of(j), idx_of(j), w_of(j), counts_dev + (size_t)j * d.E};
      }
      const hipError_t e = launch_route_batch(d, rb, s);
      if (e != hipSuccess) return set_error(EB_ERR_HIP, "route launch: %s", hipGetErrorString(e));
    }
    return EB_OK;
  };
  if (device && !t_status.ready()) return set_error(EB_ERR_HIP, "pinned status allocation failed");
  for (int j = 0; j < N; ++j) pool[j] = j;
  if ((rc = route(pool))) return rc;
  if (device)
    return run_pass_device(d, N, T, P, base, x, gain, Wg, bias, W_gu, W_dn, policy, m, max_steps, n_steps_out,
                           runsets_out, layers_out, step_load_out, groups_out, layer_loads_out, placement, s);
  // host-scheduled: the pool's counts come back through this thread's pinned buffer
  int32_t* counts = t_pinned.get((size_t)N * d.E);
  if (counts == nullptr) return set_error(EB_ERR_HIP, "pinned host allocation failed");
  std::vector<int32_t> pool_counts, pool_layers;
  std::vector<int64_t> load(d.D), lj(d.D);
  std::vector<eb_work> run;
  std::vector<float*> xs;
  int n_steps = 0;
  while (!pool.empty()) {
    if (hipMemcpyAsync(counts, counts_dev, sizeof(int32_t) * (size_t)N * d.E, hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
      return set_error(EB_ERR_HIP, "counts copy: %s", hipGetErrorString(hipGetLastError()));
    const int n_pool = (int)pool.size();
    if (layer_loads_out) {
      for (int j : pool) {
        std::fill(lj.begin(), lj.end(), 0);
        add_device_loads(counts + (size_t)j * d.E, d.E, d.D, placement, layer[j], lj.data());
        for (int dv = 0; dv < d.D; ++dv)
          layer_loads_out[((size_t)j * d.L + layer[j]) * d.D + dv] = (int32_t)lj[dv];
      }
    }
    uint64_t mask = 0;
    if (policy == EB_POLICY_LOCKSTEP) {
      for (int dv = 0; dv < d.D; ++dv) load[dv] = 0;
      for (int j : pool) {
        mask |= 1ull << j;
        add_device_loads(counts + (size_t)j * d.E, d.E, d.D, placement, layer[j], load.data());
      }
    } else {
      pool_counts.resize((size_t)n_pool * d.E);
      pool_layers.resize(n_pool);
      for (int i = 0; i < n_pool; ++i) {
        memcpy(&pool_counts[(size_t)i * d.E], counts + (size_t)pool[i] * d.E, sizeof(int32_t) * d.E);
        pool_layers[i] = layer[pool[i]];
      }
      if ((rc = schedule_impl(n_pool, pool.data(), pool_counts.data(), d.E, d.D, m, policy, &mask,
                              load.data(), pool_layers.data(), placement)))
        return rc;
    }
    run.clear();
    xs.clear();
    for (int j : pool)
      if ((mask >> j) & 1) {
        run.push_back(eb_work{j, layer[j], T, 0, a_of(j), idx_of(j), w_of(j)});
        xs.push_back(x_of(j));
      }
    if (n_steps < max_steps) {
      if (runsets_out) runsets_out[n_steps] = mask;
      if (layers_out)
        for (int j = 0; j < N; ++j) layers_out[(size_t)n_steps * N + j] = ((mask >> j) & 1) ? layer[j] : -1;
      if (step_load_out)
        for (int dv = 0; dv < d.D; ++dv) step_load_out[(size_t)n_steps * d.D + dv] = load[dv];
      if (groups_out) {
        // distinct (layer, expert) keys with a token among the RunSet's entries
        std::vector<uint8_t> seen((size_t)d.L * d.E, 0);
        std::vector<uint8_t> layer_seen(d.L, 0);
        int g = 0;
        for (const eb_work& r : run) {
          if (!layer_seen[r.layer]) {
            layer_seen[r.layer] = 1;
            g += d.S;
          }
          for (int e = 0; e < d.E; ++e)
            if (counts[(size_t)r.mb_id * d.E + e] > 0 && !seen[(size_t)r.layer * d.E + e]) {
              seen[(size_t)r.layer * d.E + e] = 1;
              ++g;
            }
        }
        groups_out[n_steps] = g;
      }
    }
    ++n_steps;
    const int n_run = (int)run.size();
    if ((rc = easybalance_moe_step(desc, n_run, run.data(), W_gu, W_dn, ws, P.ws_bytes, o, inv,
                                   nullptr, stream)))
      return rc;
    if ((rc = easybalance_combine(desc, n_run, run.data(), xs.data(), o, inv, stream))) return rc;
    std::vector<int32_t> next, advanced;
    for (int j : pool) {
      if ((mask >> j) & 1) {
        if (++layer[j] < d.L) {
          advanced.push_back(j);
          next.push_back(j);
        }
      } else {
        next.push_back(j);
      }
    }
    if ((rc = route(advanced))) return rc;
    pool.swap(next);
  }
  if (n_steps_out) *n_steps_out = n_steps;
  return EB_OK;
}

}  // extern "C"
