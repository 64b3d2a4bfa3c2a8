// C ABI of libeasybalance.so: argument checks, workspace layout, per-step
// tables, kernel-timing hooks.  The compute lives in the kernels of
// route.hip, permute.hip, gemm.hip and combine.hip; the scheduler in
// schedule.cpp.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <vector>

#include "eb_internal.h"

namespace eb {

namespace {
thread_local char g_err[512] = "";

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

int check_desc(const eb_model_desc* d) {
  if (d == nullptr) return set_error(EB_ERR_INVALID_ARG, "desc is NULL");
  if (d->L < 1 || d->H < 1 || d->F < 1 || d->E < 1 || d->k < 1 || d->S < 0 || d->D < 1)
    return set_error(EB_ERR_INVALID_ARG, "desc has a non-positive size (L=%d H=%d F=%d E=%d k=%d S=%d D=%d)",
                     d->L, d->H, d->F, d->E, d->k, d->S, d->D);
  if (d->dtype != EB_DTYPE_F32 && d->dtype != EB_DTYPE_BF16)
    return set_error(EB_ERR_INVALID_ARG, "dtype %d is not EB_DTYPE_F32/BF16", d->dtype);
  if (d->k > d->E) return set_error(EB_ERR_INVALID_ARG, "k=%d > E=%d", d->k, d->E);
  if (d->E % d->D != 0) return set_error(EB_ERR_INVALID_ARG, "E=%d not a multiple of D=%d", d->E, d->D);
  if (!(d->rms_eps >= 0.f)) return set_error(EB_ERR_INVALID_ARG, "rms_eps must be >= 0");
  if (d->norm_topk != 0 && d->norm_topk != 1) return set_error(EB_ERR_INVALID_ARG, "norm_topk must be 0/1");
  if (d->H % 256 != 0) return set_error(EB_ERR_UNSUPPORTED, "H=%d is not a multiple of 256", d->H);
  if (d->F % 128 != 0) return set_error(EB_ERR_UNSUPPORTED, "F=%d is not a multiple of 128", d->F);
  if (d->E + d->S > 1024) return set_error(EB_ERR_UNSUPPORTED, "E+S=%d > 1024", d->E + d->S);
  if (d->dtype == EB_DTYPE_BF16 && d->E > 256)
    return set_error(EB_ERR_UNSUPPORTED, "bf16 router supports E <= 256 (E=%d)", d->E);
  if (d->k + d->S > kMaxSlots) return set_error(EB_ERR_UNSUPPORTED, "k+S=%d > %d", d->k + d->S, kMaxSlots);
  if (d->L > EB_MAX_LAYERS) return set_error(EB_ERR_UNSUPPORTED, "L=%d > %d", d->L, EB_MAX_LAYERS);
  if (d->dtype == EB_DTYPE_BF16 && 2LL * d->F * d->H * 2 >= (1LL << 31))
    return set_error(EB_ERR_UNSUPPORTED, "an expert's gate/up matrix (2F x H bf16) must be < 2 GiB");
  if ((long)d->L * (d->E + d->S) > 15360)
    return set_error(EB_ERR_UNSUPPORTED, "L*(E+S)=%ld > 15360", (long)d->L * (d->E + d->S));
  return EB_OK;
}

// Sizes that fix the workspace layout of one step.
struct StepShape {
  int n_chunks;
  long long P;         // grouped rows
  long long tokens;
  int max_tiles;
};

StepShape step_shape(const eb_model_desc& d, int n_run, const int32_t* T) {
  StepShape s{0, 0, 0, 0};
  for (int i = 0; i < n_run; ++i) {
    s.n_chunks += (T[i] + kPermChunk - 1) / kPermChunk;
    s.tokens += T[i];
  }
  s.P = s.tokens * (d.k + d.S);
  const long long bm = gemm_bm(d.dtype);
  const long long groups = (long long)n_run * (d.E + d.S);
  s.max_tiles = (int)((s.P + bm - 1) / bm + (groups < s.P ? groups : s.P));
  return s;
}

struct WsLayout {
  size_t hist, chunk_base, offsets, tiles, n_tiles, groups, n_groups, work_ctr, partial, perm, a_perm,
      h, total;
};

WsLayout ws_layout(const eb_model_desc& d, const StepShape& s, const eb_step_views* v) {
  const size_t eb = d.dtype == EB_DTYPE_BF16 ? 2 : 4;
  WsLayout w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes);
    return o;
  };
  w.hist = take(sizeof(int32_t) * (size_t)s.n_chunks * d.E);
  w.chunk_base = take(sizeof(int32_t) * (size_t)s.n_chunks * (d.E + d.S));
  w.offsets = (v && v->offsets) ? 0 : take(sizeof(int32_t) * ((size_t)d.L * (d.E + d.S) + 1));
  w.tiles = take(sizeof(int4) * (size_t)(s.max_tiles > 0 ? s.max_tiles : 1));
  w.n_tiles = take(sizeof(int32_t));
  w.groups = take(sizeof(int4) * (size_t)d.L * (d.E + d.S));
  w.n_groups = take(sizeof(int32_t));
  w.work_ctr = take(sizeof(int32_t) * kWorkCounters);
  w.partial = down_ksplit(d.dtype, d.F) > 1 ? take(sizeof(float) * 2 * (size_t)s.P * d.H) : 0;
  w.perm = (v && v->perm) ? 0 : take(sizeof(int32_t) * (size_t)s.P);
  w.a_perm = (v && v->a_perm) ? 0 : take(eb * (size_t)s.P * d.H);
  w.h = (v && v->h) ? 0 : take(eb * (size_t)s.P * d.F);
  w.total = off;
  return w;
}

int check_run(const eb_model_desc& d, int32_t n_run, const eb_work* run, bool need_idx) {
  if (n_run < 1 || n_run > EB_MAX_RUN)
    return set_error(EB_ERR_INVALID_ARG, "n_run=%d outside [1, %d]", n_run, EB_MAX_RUN);
  if (run == nullptr) return set_error(EB_ERR_INVALID_ARG, "run is NULL");
  long long tokens = 0;
  for (int i = 0; i < n_run; ++i) {
    const eb_work& r = run[i];
    if (r.layer < 0 || r.layer >= d.L)
      return set_error(EB_ERR_INVALID_ARG, "run[%d].layer=%d outside [0, %d)", i, r.layer, d.L);
    if (r.T < 0) return set_error(EB_ERR_INVALID_ARG, "run[%d].T=%d < 0", i, r.T);
    if (r.reserved != 0) return set_error(EB_ERR_INVALID_ARG, "run[%d].reserved must be 0", i);
    if (r.T > 0 && (r.w == nullptr || (need_idx && (r.a == nullptr || r.idx == nullptr))))
      return set_error(EB_ERR_INVALID_ARG, "run[%d] has a NULL a/idx/w pointer", i);
    tokens += r.T;
  }
  if (tokens * (d.k + d.S) > 0x7fffffffLL)
    return set_error(EB_ERR_UNSUPPORTED, "step has %lld pairs (> 2^31-1)", tokens * (d.k + d.S));
  return EB_OK;
}

RunTable make_run_table(const eb_model_desc& d, int32_t n_run, const eb_work* run,
                        float* const* x) {
  RunTable rt;
  memset(&rt, 0, sizeof(rt));
  rt.n = n_run;
  rt.E = d.E;
  rt.k = d.k;
  rt.S = d.S;
  rt.L = d.L;
  rt.H = d.H;
  rt.chunk_base[0] = 0;
  rt.tok_base[0] = 0;
  for (int i = 0; i < n_run; ++i) {
    rt.chunk_base[i + 1] = rt.chunk_base[i] + (run[i].T + kPermChunk - 1) / kPermChunk;
    rt.tok_base[i + 1] = rt.tok_base[i] + run[i].T;
    rt.layer[i] = run[i].layer;
    rt.idx[i] = run[i].idx;
    rt.a[i] = run[i].a;
    rt.w[i] = run[i].w;
    rt.x[i] = x ? x[i] : nullptr;
  }
  return rt;
}

int hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return EB_OK;
  return set_error(EB_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// A step's buffers carved from its workspace (laid out for shape sh); views
// that the caller provides replace their workspace slots.
struct StepWs {
  StepBuffers b;
  float* partial;
  void* h;
};

StepWs carve_step(const eb_model_desc& d, const StepShape& sh, const eb_step_views* views, void* ws,
                  int32_t* inv) {
  const WsLayout L = ws_layout(d, sh, views);
  uint8_t* base = static_cast<uint8_t*>(ws);
  StepWs w;
  StepBuffers& b = w.b;
  b.hist = reinterpret_cast<int32_t*>(base + L.hist);
  b.chunk_base = reinterpret_cast<int32_t*>(base + L.chunk_base);
  b.offsets = (views && views->offsets) ? views->offsets : reinterpret_cast<int32_t*>(base + L.offsets);
  b.tiles = reinterpret_cast<int4*>(base + L.tiles);
  b.n_tiles = reinterpret_cast<int32_t*>(base + L.n_tiles);
  b.groups = reinterpret_cast<int4*>(base + L.groups);
  b.n_groups = reinterpret_cast<int32_t*>(base + L.n_groups);
  b.work_ctr = reinterpret_cast<int32_t*>(base + L.work_ctr);
  b.max_tiles = sh.max_tiles;
  b.perm = (views && views->perm) ? views->perm : reinterpret_cast<int32_t*>(base + L.perm);
  b.inv = inv;
  b.a_perm = (views && views->a_perm) ? views->a_perm : base + L.a_perm;
  w.partial = L.partial ? reinterpret_cast<float*>(base + L.partial) : nullptr;
  w.h = (views && views->h) ? views->h : base + L.h;
  return w;
}

// The two grouped GEMMs of a step whose permutation is queued before them.
// sh.P rows are held by the buffers; the live rows come from the offsets.
int run_gemms(const eb_model_desc& d, const StepShape& sh, const StepWs& w, const WeightTable& wt,
              void* o, hipStream_t s, bool sum_halves = true) {
  GroupedProblem gp;
  gp.H = d.H;
  gp.F = d.F;
  gp.E = d.E;
  gp.S = d.S;
  gp.P = (int32_t)sh.P;
  gp.offsets = w.b.offsets;
  gp.P_live = w.b.offsets + (size_t)d.L * (d.E + d.S);
  gp.tiles = w.b.tiles;
  gp.n_tiles = w.b.n_tiles;
  gp.groups = w.b.groups;
  gp.n_groups = w.b.n_groups;
  gp.max_tiles = sh.max_tiles;
  gp.work_ctr = w.b.work_ctr;
  gp.ksplit = 1;
  gp.partial = nullptr;
  int rc;
  if ((rc = hip_status(launch_gateup(d.dtype, gp, wt, w.b.a_perm, w.h, s), "gate/up GEMM"))) return rc;
  gp.work_ctr = w.b.work_ctr + kWorkCounters / 2;
  gp.ksplit = down_ksplit(d.dtype, d.F);
  gp.partial = w.partial;
  return hip_status(launch_down(d.dtype, gp, wt, w.h, o, s, sum_halves), "down GEMM");
}

// ---- kernel timing ---------------------------------------------------------
struct EventPair {
  hipEvent_t start, stop;
  int kind;
};
std::mutex g_prof_mu;
std::atomic<bool> g_prof_on{false};
std::atomic<uint32_t> g_prof_mask{0};
std::vector<EventPair> g_prof_done;
std::vector<hipEvent_t> g_prof_free;
thread_local hipEvent_t t_pending = nullptr;

hipEvent_t prof_event() {
  if (!g_prof_free.empty()) {
    hipEvent_t e = g_prof_free.back();
    g_prof_free.pop_back();
    return e;
  }
  // timing only: no system-scope fence (cache writeback and invalidate) when
  // the event is recorded, which would stall the kernels around it
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

}  // namespace

// One step of a device-scheduled pass: its run table is at rt (device
// memory, written by the scheduler kernel queued before), its workspace laid
// out for all N micro-batches of T tokens, every grid sized for that step.
int enqueue_step_dev(const eb_model_desc& d, int N, int T, const RunTable* rt, const WeightTable& wt,
                     void* ws, void* o, int32_t* inv, hipStream_t s) {
  std::vector<int32_t> Ts(N, T);
  const StepShape sh = step_shape(d, N, Ts.data());
  const StepWs w = carve_step(d, sh, nullptr, ws, inv);
  int rc;
  if ((rc = hip_status(launch_permute_dev(d, rt, sh.n_chunks, (int)sh.tokens, w.b, s), "permute")))
    return rc;
  // a split-K down GEMM leaves its two fp32 halves for the combine, which
  // rounds their sum as the split-K sum kernel would (o is not stored)
  const bool fuse = w.partial != nullptr;
  if ((rc = run_gemms(d, sh, w, wt, o, s, !fuse))) return rc;
  if (fuse)
    return hip_status(
        launch_combine_split_dev(rt, d.k + d.S, (int)sh.tokens, w.partial, (long long)sh.P * d.H, inv, s),
        "combine");
  return hip_status(launch_combine_dev(rt, d.k + d.S, (int)sh.tokens, d.dtype, o, inv, s), "combine");
}

int set_error(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

void prof_start(int kind, hipStream_t s) {
  if (!g_prof_on.load(std::memory_order_relaxed) ||
      !((g_prof_mask.load(std::memory_order_relaxed) >> kind) & 1u))
    return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  t_pending = prof_event();
  if (t_pending && hipEventRecord(t_pending, s) != hipSuccess) {
    g_prof_free.push_back(t_pending);
    t_pending = nullptr;
  }
}

void prof_stop(int kind, hipStream_t s) {
  if (!g_prof_on.load(std::memory_order_relaxed) || t_pending == nullptr) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  hipEvent_t stop = prof_event();
  if (stop != nullptr && hipEventRecord(stop, s) == hipSuccess) {
    g_prof_done.push_back(EventPair{t_pending, stop, kind});
  } else {
    g_prof_free.push_back(t_pending);
    if (stop) g_prof_free.push_back(stop);
  }
  t_pending = nullptr;
}

}  // namespace eb

using namespace eb;

extern "C" {

const char* easybalance_version(void) { return "easybalance-mi355x 0.1.0"; }

const char* easybalance_last_error(void) { return g_err; }

int easybalance_route(const eb_model_desc* desc, int32_t layer, int32_t T, const float* x,
                      const float* gain, const void* Wg, const float* bias, void* a_out,
                      float* logits_out, int32_t* idx_out, float* w_out, int32_t* counts_out,
                      void* stream) {
  int rc = check_desc(desc);
  if (rc) return rc;
  if (layer < 0 || layer >= desc->L)
    return set_error(EB_ERR_INVALID_ARG, "layer=%d outside [0, %d)", layer, desc->L);
  if (T < 0) return set_error(EB_ERR_INVALID_ARG, "T=%d < 0", T);
  if (counts_out == nullptr) return set_error(EB_ERR_INVALID_ARG, "counts_out is NULL");
  if (T > 0 && (x == nullptr || gain == nullptr || Wg == nullptr || bias == nullptr ||
                a_out == nullptr || idx_out == nullptr || w_out == nullptr))
    return set_error(EB_ERR_INVALID_ARG, "a required route pointer is NULL");
  if (T > 0 && logits_out == nullptr && route_logits_required(*desc))
    return set_error(EB_ERR_INVALID_ARG,
                     "logits_out is NULL, but this stack's top-k reads the logits back (fp32, E=%d, H=%d)",
                     desc->E, desc->H);
  return hip_status(launch_route(*desc, T, x, gain, Wg, bias, a_out, logits_out, idx_out, w_out,
                                 counts_out, static_cast<hipStream_t>(stream)),
                    "route launch");
}

int easybalance_schedule(int32_t n_pool, const int32_t* pool_ids, const int32_t* counts,
                         int32_t E, int32_t D, int32_t m, int32_t policy, uint64_t* runset_mask,
                         int64_t* step_load, const int32_t* pool_layers, const eb_placement* placement) {
  return schedule_impl(n_pool, pool_ids, counts, E, D, m, policy, runset_mask, step_load, pool_layers,
                       placement);
}

int easybalance_moe_step_workspace_size(const eb_model_desc* desc, int32_t n_run,
                                        const int32_t* T, size_t* bytes) {
  int rc = check_desc(desc);
  if (rc) return rc;
  if (n_run < 1 || n_run > EB_MAX_RUN || T == nullptr || bytes == nullptr)
    return set_error(EB_ERR_INVALID_ARG, "bad n_run/T/bytes");
  for (int i = 0; i < n_run; ++i)
    if (T[i] < 0) return set_error(EB_ERR_INVALID_ARG, "T[%d] < 0", i);
  *bytes = ws_layout(*desc, step_shape(*desc, n_run, T), nullptr).total;
  return EB_OK;
}

int easybalance_moe_step(const eb_model_desc* desc, int32_t n_run, const eb_work* run,
                         const void* const* W_gu, const void* const* W_dn, void* ws,
                         size_t ws_bytes, void* o_out, int32_t* inv_out,
                         const eb_step_views* views, void* stream) {
  return moe_step_common(desc, n_run, run, W_gu, W_dn, ws, ws_bytes, o_out, inv_out, views, stream, false);
}

}  // extern "C"

namespace eb {

int moe_step_common(const eb_model_desc* desc, int32_t n_run, const eb_work* run, const void* const* W_gu,
                    const void* const* W_dn, void* ws, size_t ws_bytes, void* o_out, int32_t* inv_out,
                    const eb_step_views* views, void* stream, bool static_scratch) {
  int rc = check_desc(desc);
  if (rc) return rc;
  rc = check_run(*desc, n_run, run, true);
  if (rc) return rc;
  const eb_model_desc& d = *desc;
  int32_t Ts[EB_MAX_RUN];  // no heap allocation on this path (n_run <= EB_MAX_RUN, checked)
  for (int i = 0; i < n_run; ++i) Ts[i] = run[i].T;
  const StepShape sh = step_shape(d, n_run, Ts);
  if (sh.P == 0) return EB_OK;
  if (W_gu == nullptr || W_dn == nullptr) return set_error(EB_ERR_INVALID_ARG, "W_gu/W_dn is NULL");
  WeightTable wt;
  memset(&wt, 0, sizeof(wt));
  for (int i = 0; i < n_run; ++i) {
    const int l = run[i].layer;
    if (run[i].T > 0 && (W_gu[l] == nullptr || W_dn[l] == nullptr))
      return set_error(EB_ERR_INVALID_ARG, "weights of layer %d are NULL", l);
  }
  for (int l = 0; l < d.L; ++l) {
    wt.gu[l] = W_gu[l];
    wt.dn[l] = W_dn[l];
  }
  if (o_out == nullptr || inv_out == nullptr) return set_error(EB_ERR_INVALID_ARG, "o_out/inv_out is NULL");
  if (ws == nullptr || (reinterpret_cast<uintptr_t>(ws) % kAlign) != 0)
    return set_error(EB_ERR_INVALID_ARG, "workspace must be non-NULL and 256-byte aligned");
  const WsLayout L = ws_layout(d, sh, views);
  if (ws_bytes < L.total) {
    if (static_scratch)
      return set_error(EB_ERR_UNSUPPORTED, "the step needs %zu bytes of scratch, more than the static %zu",
                       L.total, ws_bytes);
    return set_error(EB_ERR_WORKSPACE_TOO_SMALL, "workspace %zu < %zu bytes", ws_bytes, L.total);
  }
  const StepWs w = carve_step(d, sh, views, ws, inv_out);
  hipStream_t s = static_cast<hipStream_t>(stream);

  const RunTable rt = make_run_table(d, n_run, run, nullptr);
  const int eb = d.dtype == EB_DTYPE_BF16 ? 2 : 4;
  const StepBuffers& b = w.b;
  if ((rc = hip_status(launch_perm_count(rt, sh.n_chunks, b.hist, s), "perm_count"))) return rc;
  if ((rc = hip_status(launch_perm_scan(rt, b.hist, b.chunk_base, b.offsets, b.tiles, b.n_tiles, b.groups,
                                        b.n_groups, gemm_bm(d.dtype), b.max_tiles, b.work_ctr, s),
                       "perm_scan")))
    return rc;
  if ((rc = hip_status(launch_perm_scatter(rt, sh.n_chunks, eb, b.chunk_base, b.perm, inv_out, b.a_perm, s),
                       "perm_scatter")))
    return rc;
  return run_gemms(d, sh, w, wt, o_out, s);
}

}  // namespace eb

extern "C" {

int easybalance_combine(const eb_model_desc* desc, int32_t n_run, const eb_work* run,
                        float* const* x_inout, const void* o, const int32_t* inv, void* stream) {
  int rc = check_desc(desc);
  if (rc) return rc;
  rc = check_run(*desc, n_run, run, false);
  if (rc) return rc;
  if (x_inout == nullptr) return set_error(EB_ERR_INVALID_ARG, "x_inout is NULL");
  long long tokens = 0;
  for (int i = 0; i < n_run; ++i) {
    if (run[i].T > 0 && x_inout[i] == nullptr)
      return set_error(EB_ERR_INVALID_ARG, "x_inout[%d] is NULL", i);
    tokens += run[i].T;
  }
  if (tokens == 0) return EB_OK;
  if (o == nullptr || inv == nullptr) return set_error(EB_ERR_INVALID_ARG, "o/inv is NULL");
  const RunTable rt = make_run_table(*desc, n_run, run, x_inout);
  return hip_status(launch_combine(rt, desc->dtype, o, inv,
                                   static_cast<hipStream_t>(stream)),
                    "combine");
}

int easybalance_pack_weights(const eb_model_desc* desc, int32_t kind, int32_t n, const void* src,
                            void* dst, void* stream) {
  int rc = check_desc(desc);
  if (rc) return rc;
  if (kind != EB_WEIGHTS_GATE_UP && kind != EB_WEIGHTS_DOWN)
    return set_error(EB_ERR_INVALID_ARG, "kind %d is not EB_WEIGHTS_GATE_UP/DOWN", kind);
  if (n < 0) return set_error(EB_ERR_INVALID_ARG, "n=%d < 0", n);
  if (n == 0) return EB_OK;
  if (src == nullptr || dst == nullptr) return set_error(EB_ERR_INVALID_ARG, "src/dst is NULL");
  const int N = kind == EB_WEIGHTS_GATE_UP ? 2 * desc->F : desc->H;
  const int K = kind == EB_WEIGHTS_GATE_UP ? desc->H : desc->F;
  const size_t bytes = (size_t)n * N * K * (desc->dtype == EB_DTYPE_BF16 ? 2 : 4);
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
  if (s0 < d0 + bytes && d0 < s0 + bytes) return set_error(EB_ERR_INVALID_ARG, "src and dst overlap");
  if ((s0 | d0) % 16 != 0) return set_error(EB_ERR_INVALID_ARG, "src/dst not 16-byte aligned");
  return hip_status(launch_pack_weights(desc->dtype, kind == EB_WEIGHTS_GATE_UP, n, N, K, desc->F, src,
                                        dst, static_cast<hipStream_t>(stream)),
                    "pack_weights");
}

int easybalance_profile_begin(uint32_t kernel_mask) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_mask.store(kernel_mask & EB_PROFILE_ALL);
  for (auto& p : g_prof_done) {
    g_prof_free.push_back(p.start);
    g_prof_free.push_back(p.stop);
  }
  g_prof_done.clear();
  g_prof_on.store(true);
  return EB_OK;
}

int easybalance_profile_end(double* ms_out, int64_t* launches_out) {
  g_prof_on.store(false);
  std::lock_guard<std::mutex> lk(g_prof_mu);
  double ms[EB_NUM_KERNELS] = {0};
  int64_t n[EB_NUM_KERNELS] = {0};
  int rc = EB_OK;
  for (auto& p : g_prof_done) {
    float t = 0.f;
    hipError_t e = hipEventSynchronize(p.stop);
    if (e == hipSuccess) e = hipEventElapsedTime(&t, p.start, p.stop);
    if (e != hipSuccess && rc == EB_OK) rc = hip_status(e, "profile events");
    ms[p.kind] += t;
    n[p.kind] += 1;
    g_prof_free.push_back(p.start);
    g_prof_free.push_back(p.stop);
  }
  g_prof_done.clear();
  if (ms_out) memcpy(ms_out, ms, sizeof(ms));
  if (launches_out) memcpy(launches_out, n, sizeof(n));
  return rc;
}

}  // extern "C"
