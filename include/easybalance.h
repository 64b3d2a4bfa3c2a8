/*
 * easybalance.h -- C ABI of libeasybalance.so, the one-GPU hot path of
 * EasyBalance (cross-layer load balancing for expert-parallel MoE inference,
 * arXiv 2608.07964) on AMD Instinct MI355X (gfx950).
 *
 * Algorithm 1 of the paper runs, per step, three operations:
 *   Attn_Route_Dispatch(RunSet_{i-1})  -> easybalance_route (routing part)
 *   RunSet_i = Schedule(S_{i-1}, m)    -> easybalance_schedule
 *   MoECompute_Combine(RunSet_i)       -> easybalance_moe_step + easybalance_combine
 * The expert-parallel group of D devices is virtual: all experts of all layers
 * live on this one GPU, E/D contiguous experts per virtual device, and the work
 * every virtual device would do in a step runs in one grouped launch.
 *
 * Conventions shared by every call
 *  - Return value: EB_OK (0) or a negative EB_ERR_* code.  On error the
 *    outputs are unspecified and easybalance_last_error() (thread-local)
 *    describes the first failed check.  No C++ exception crosses the ABI.
 *  - Memory: every buffer passed in is owned by the caller.  "device"
 *    pointers are HIP device allocations on the current device; "host"
 *    pointers are ordinary host memory.  The library allocates no device
 *    memory; scratch space of easybalance_moe_step is a caller workspace
 *    sized by easybalance_moe_step_workspace_size.  What the library does
 *    hold, until the process (or the calling thread) ends:
 *      easybalance_run_pass: per host thread, a pinned host buffer of the
 *        pool's expert counts (host-scheduled passes, N * E int32, grown on
 *        demand) and a 256-byte host-mapped status word (device-scheduled
 *        passes); freed when the thread exits;
 *      easybalance_profile_*: a process-wide pool of timing events;
 *      easybalance_moe_step_noalloc: its static device array
 *        (EB_NOALLOC_SCRATCH_BYTES per device, allocated by the HIP loader).
 *  - Streams: `stream` is a hipStream_t passed as void* (NULL = null stream).
 *    Device calls only enqueue work on it and never synchronize; the caller
 *    orders calls on one stream or with events.
 *  - Layouts are row-major and densely packed, except the expert weights
 *    that easybalance_moe_step reads (see easybalance_pack_weights).
 *    "dtype" is the model's storage type (EB_DTYPE_F32 or EB_DTYPE_BF16,
 *    bf16 as raw 16-bit patterns); accumulation is always fp32.
 *  - Shape limits (EB_ERR_UNSUPPORTED otherwise): H % 256 == 0,
 *    F % 128 == 0, 1 <= k <= E, E + S <= 1024, k + S <= 16, E % D == 0,
 *    L <= EB_MAX_LAYERS, L * (E + S) <= 15360; bf16 stacks: E <= 256 and
 *    2F * H * 2 bytes < 2 GiB (one gate/up matrix).
 */
#ifndef EASYBALANCE_H
#define EASYBALANCE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define EB_OK 0
#define EB_ERR_INVALID_ARG (-1)
#define EB_ERR_UNSUPPORTED (-2)
#define EB_ERR_HIP (-3)
#define EB_ERR_WORKSPACE_TOO_SMALL (-4)

#define EB_DTYPE_F32 0
#define EB_DTYPE_BF16 1

#define EB_POLICY_MAXUTIL 0
#define EB_POLICY_CUMUTIL 1
#define EB_POLICY_DIFFPEAK 2
#define EB_WEIGHTS_GATE_UP 0     /* easybalance_pack_weights kinds */
#define EB_WEIGHTS_DOWN 1

#define EB_POLICY_LOCKSTEP 3    /* easybalance_run_pass only: every pooled
                                   micro-batch every step (per-layer baseline) */
#define EB_PASS_DEVICE_SCHEDULE 0x100  /* easybalance_run_pass only, OR-ed into
                                   policy: Schedule runs on the GPU */

#define EB_MAX_POOL 64          /* micro-batch ids are 0..63 (one bit each)   */
#define EB_MAXUTIL_MAX_POOL 20  /* MaxUtil enumerates up to 2^n subsets       */
#define EB_MAX_RUN 64
#define EB_MAX_LAYERS 128

/* Kernel classes reported by the profiling calls. */
#define EB_K_ROUTE_NORM 0
#define EB_K_ROUTE_LOGITS 1
#define EB_K_ROUTE_TOPK 2
#define EB_K_PERM_COUNT 3
#define EB_K_PERM_SCAN 4
#define EB_K_PERM_SCATTER 5
#define EB_K_GATEUP 6
#define EB_K_DOWN 7
#define EB_K_COMBINE 8
#define EB_K_PERM_GATHER 9
#define EB_NUM_KERNELS 10

/* Model shape.  L MoE layers, hidden H, expert FFN size F, E routed experts
 * with top-k routing, S always-on shared experts, D virtual EP devices.
 * rms_eps: RMSNorm epsilon.  norm_topk: 0 = routing weights are the softmax
 * over all E experts taken at the k picks (Eq. 1 as written), 1 = renormalised
 * over the k picks. */
typedef struct eb_model_desc {
  int32_t L, H, F, E, k, S, D;
  int32_t dtype;
  float rms_eps;
  int32_t norm_topk;
} eb_model_desc;

/* One micro-batch of a step's RunSet, at its own layer (Algorithm 1 keeps
 * l_j per micro-batch; Section 4.1 lets micro-batches at different layers run
 * jointly).  All pointers are device pointers produced by easybalance_route
 * for this micro-batch at `layer`. */
typedef struct eb_work {
  int32_t mb_id;        /* micro-batch id j (informational)              */
  int32_t layer;        /* l_j, 0 <= layer < L                           */
  int32_t T;            /* tokens, >= 0                                  */
  int32_t reserved;     /* must be 0                                     */
  const void* a;        /* [T][H] dtype: normalised activations          */
  const int32_t* idx;   /* [T][k] routed expert ids                      */
  const float* w;       /* [T][k] routing weights                        */
} eb_work;

/* Optional extra outputs of easybalance_moe_step (any member may be NULL;
 * a NULL member lives in the workspace instead).  P = sum_rho T_rho * (k+S). */
typedef struct eb_step_views {
  void* a_perm;         /* [P][H] dtype: rows grouped by (layer, expert)  */
  void* h;              /* [P][F] dtype: SwiGLU activations               */
  int32_t* perm;        /* [P]: pair index at each grouped position       */
  int32_t* offsets;     /* [L*(E+S)+1]: first grouped row of each key     */
} eb_step_views;

/* Library version string, e.g. "easybalance-mi355x 0.1.0". */
const char* easybalance_version(void);

/* Message of the last failed call on this thread ("" if none). */
const char* easybalance_last_error(void);

/*
 * easybalance_route -- RMSNorm, router and top-k of one micro-batch at one
 * layer: the routing half of Attn_Route_Dispatch (Algorithm 1), i.e.
 * W_l, I_l = topk(G(h'_l)) of Section 2.1, plus the expert pair counts from
 * which the per-device workload vector of Section 2.3 is formed.
 *
 *   a   = dtype( x * r * gain ),  r = 1 / sqrt(mean(x^2) + rms_eps)   per token
 *   z   = a Wg^T + bias                                  (fp32 accumulate)
 *   idx = the k largest z per token, largest first; equal z -> lower expert id
 *   w   = softmax(z over all E)[idx]   (norm_topk=1: renormalised over the k)
 *   counts[e] = #{(t, r) : idx[t][r] == e}
 *
 * layer      0 <= layer < L (checked; weights are passed for this layer)
 * T          tokens (>= 0)
 * x          device [T][H] fp32 residual stream (read only)
 * gain       device [H] fp32 RMSNorm gain
 * Wg         device [E][H] dtype router weights
 * bias       device [E] fp32 router logit bias
 * a_out      device [T][H] dtype
 * logits_out device [T][E] fp32: the router's output z, or NULL when it is
 *            not wanted -- except on fp32 stacks with E > 64 or H > 8192,
 *            whose top-k reads z back (EB_ERR_INVALID_ARG there)
 * idx_out    device [T][k] int32
 * w_out      device [T][k] fp32
 * counts_out device [E] int32 (overwritten, not accumulated)
 * NaN logits rank after every number: a token whose remaining logits are all
 * NaN takes the lowest expert ids not yet picked, in ascending order (weight
 * NaN), so every token's k picks are distinct experts.
 */
int easybalance_route(const eb_model_desc* desc, int32_t layer, int32_t T, const float* x,
                      const float* gain, const void* Wg, const float* bias, void* a_out,
                      float* logits_out, int32_t* idx_out, float* w_out, int32_t* counts_out,
                      void* stream);

/*
 * Static placement of every layer's experts on the D (virtual) devices, with
 * replicas: the redundant-expert placement that Section 5 combines with
 * EasyBalance to show the two are orthogonal (EPLB; the paper's appendix on
 * redundant experts).  NULL wherever a placement is optional means the
 * paper's even mapping: E/D contiguous experts per device, device(e) =
 * e div (E/D).
 *
 * copies[(l*E + e)*R + i], i < R, is the device of copy i of expert e at
 * layer l; an expert has 1..R copies, on distinct devices listed in
 * ascending order, and the unused entries after them are -1.  An expert's c
 * routed pairs are split as evenly as possible over its r copies: copy i
 * carries c div r pairs, plus one if i < c mod r.  Shared experts stay out
 * of the workload vectors, as without a placement.
 */
typedef struct eb_placement {
  int32_t L, E, D;        /* must equal the model's (checked)                    */
  int32_t R;              /* copy entries per expert, 1 <= R <= min(D, 64)       */
  const int32_t* copies;  /* host [L][E][R]                                      */
} eb_placement;

/*
 * easybalance_schedule -- RunSet_i = Schedule(S_{i-1}, m) of Algorithm 1.
 * Host only, pure, re-entrant; no GPU access.
 *
 * Workload of micro-batch pool_ids[i] (Section 2.3): for device d,
 *   load_i[d] = sum over experts e in [d*E/D, (d+1)*E/D) of counts[i*E + e]
 * (placement NULL), or the pairs its experts' copies on d carry under the
 * placement at the micro-batch's layer pool_layers[i] (see eb_placement).
 * Utilization of a set R (Eq. 3 for one step): U(R) = sum_d W_d / (D max_d W_d)
 * with W = sum_{i in R} load_i; U = 1 if W is all zero.
 *   EB_POLICY_MAXUTIL (Section 4.2): the R with |R| >= min(m, n_pool) of
 *     highest U; ties -> larger |R| -> lexicographically smallest id list.
 *     n_pool <= EB_MAXUTIL_MAX_POOL.  Cost: one visit per candidate set,
 *     sum_{j <= n_pool - min(m, n_pool)} C(n_pool, j) of them, O(D) each.
 *   EB_POLICY_CUMUTIL (Section 5.2): scan ids ascending, take the first, add
 *     each next one iff it strictly raises U.
 *   EB_POLICY_DIFFPEAK (Section 5.2): scan ids ascending, take the first, add
 *     each next one iff its peak device (lowest index among maxima) is not yet
 *     a peak of the chosen set.
 *   CumUtil/DiffPeak then pad with the lowest unchosen ids up to min(m, n_pool).
 * All comparisons are exact integer arithmetic.
 *
 * n_pool      0 <= n_pool <= EB_MAX_POOL (0 gives an empty RunSet)
 * pool_ids    host [n_pool], strictly ascending, each in [0, 64)
 * counts      host [n_pool][E] int32 >= 0, row i belongs to pool_ids[i]
 * m           >= 1
 * runset_mask host out: bit j set iff micro-batch j runs in this step
 * step_load   host out [D] int64 (nullable): combined workload W of the RunSet
 * pool_layers host [n_pool] (required with a placement, else ignored): l_j of
 *             each pool member, 0 <= l_j < placement->L
 * placement   host (nullable): see eb_placement (E and D must match)
 */
int easybalance_schedule(int32_t n_pool, const int32_t* pool_ids, const int32_t* counts,
                         int32_t E, int32_t D, int32_t m, int32_t policy,
                         uint64_t* runset_mask, int64_t* step_load, const int32_t* pool_layers,
                         const eb_placement* placement);

/* Workspace bytes easybalance_moe_step needs for these per-entry token
 * counts (host [n_run]), assuming every eb_step_views member is NULL. */
int easybalance_moe_step_workspace_size(const eb_model_desc* desc, int32_t n_run,
                                        const int32_t* T, size_t* bytes);

/*
 * easybalance_moe_step -- the expert half of MoECompute_Combine(RunSet_i)
 * (Algorithm 1): every (token, expert) pair of every micro-batch in the step,
 * whatever its layer, through its expert in one grouped launch per GEMM
 * (Section 4.1, cross-layer workload combination).  On a real EP group this
 * is dispatch all-to-all -> expert FFNs -> gather all-to-all (Section 2.2);
 * here the dispatch is a stable grouping of the pairs by key
 * (layer, expert slot), slot E+s being shared expert s:
 *   pairs enumerated entry by entry in `run` order, then token, then slot
 *   (k routed slots, then S shared), q = global pair index;
 *   key(q) = layer * (E+S) + slot expert;  grouped position inv[q] = stable
 *   rank of q by key;  a_perm[inv[q]] = a of q's token.
 * For each group g = (l, e):   (W_gu rows 0..F-1 gate, F..2F-1 up)
 *   h = dtype( SiLU(a_perm W_gate^T) * (a_perm W_up^T) ),  o = dtype( h W_down^T ).
 * Every row is computed with the same K order whatever group or tile it sits
 * in, so results do not depend on the schedule (batch invariance).
 *
 * run      host [n_run] (1 <= n_run <= EB_MAX_RUN); `run` order defines q
 * W_gu     host [L] of device pointers, each the E+S matrices [2F][H] dtype
 *          as easybalance_pack_weights(EB_WEIGHTS_GATE_UP) wrote them
 * W_dn     host [L] of device pointers, each the E+S matrices [H][F] dtype
 *          as easybalance_pack_weights(EB_WEIGHTS_DOWN) wrote them
 * ws       device workspace of ws_bytes >= easybalance_moe_step_workspace_size
 *          (else EB_ERR_WORKSPACE_TOO_SMALL); 256-byte aligned
 * o_out    device [P][H] dtype: expert outputs at grouped positions
 * inv_out  device [P] int32: grouped position of pair q
 * views    host pointer to optional outputs (nullable)
 * Expert ids outside [0, E) in idx are clamped into range (no fault).
 * A step whose entries all have T = 0 (P = 0) enqueues nothing and writes
 * no output, views->offsets included; the weight and output pointers are
 * then not checked.
 */
int easybalance_moe_step(const eb_model_desc* desc, int32_t n_run, const eb_work* run,
                         const void* const* W_gu, const void* const* W_dn, void* ws,
                         size_t ws_bytes, void* o_out, int32_t* inv_out,
                         const eb_step_views* views, void* stream);

/*
 * easybalance_moe_step_noalloc -- easybalance_moe_step for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same kernels, same results bit for bit;
 * the call allocates nothing (no hipMalloc/hipFree, no host heap).  The step's
 * scratch -- permutation histograms and bases, tile and group lists, work
 * counters, perm and offsets unless views supplies them, and for long K
 * (bf16, F >= 8192) the two fp32 partial-sum planes 2 * P * H * 4 bytes --
 * sits in a static device array of EB_NOALLOC_SCRATCH_BYTES that the library
 * holds on every device it runs on until the process ends.
 *
 * Arguments as for easybalance_moe_step, without ws/ws_bytes; views is
 * required, with a_perm [P][H] and h [P][F] (dtype, the caller's buffers).
 * Errors: EB_ERR_INVALID_ARG (as easybalance_moe_step, or views / a_perm / h
 * NULL), EB_ERR_UNSUPPORTED when the step needs more scratch than the array
 * holds (the message states the need; e.g. at H = 4096, F = 14336 steps of up
 * to ~5000 pairs fit), EB_ERR_HIP.
 * Every call on a device shares that device's array and leaves its contents
 * behind (nothing in it needs to start at zero: each table is written before
 * it is read).  Calls that overlap on one device race: order them on one
 * stream or with events.
 */
#define EB_NOALLOC_SCRATCH_BYTES (160u * 1024u * 1024u)
int easybalance_moe_step_noalloc(const eb_model_desc* desc, int32_t n_run, const eb_work* run,
                                 const void* const* W_gu, const void* const* W_dn, void* o_out,
                                 int32_t* inv_out, const eb_step_views* views, void* stream);

/*
 * easybalance_pack_weights -- expert weights into the layout the grouped
 * GEMMs of easybalance_moe_step stream (once, when the weights are loaded;
 * the expert computation of Section 2.1 / Eq. 1 is unchanged, only where its
 * weights sit in memory).
 *
 * kind  EB_WEIGHTS_GATE_UP: n matrices [2F][H] (rows 0..F-1 the gate
 *       projection, F..2F-1 the up projection), row-major, back to back;
 *       EB_WEIGHTS_DOWN: n matrices [H][F], row-major, back to back.
 * src   device, the row-major matrices (dtype of desc); unchanged
 * dst   device, same size, written; must not overlap src; 16-byte aligned
 * bf16: each N x K matrix (N its rows) becomes (K/64) x (N/256) blocks of
 *   256 x 64 elements, block (s, t) at index s*(N/256) + t with K columns
 *   64s .. 64s+63 of column tile t; block row r is weight row 256t + r
 *   (down) or 128t + 32(r/64) + (r%64 < 32 ? r%64 : r%64 - 32 + F) (gate/up);
 *   its 16-byte chunk at position c holds K columns 64s + 8(c ^ ((r>>1)&7))
 *   .. +7.  fp32: dst is a copy of src (row-major).
 * Enqueued on `stream`; errors: EB_ERR_INVALID_ARG (bad kind, n < 0, NULL,
 * overlap, misalignment), EB_ERR_UNSUPPORTED (descriptor outside the shape
 * limits above), EB_ERR_HIP.
 */
int easybalance_pack_weights(const eb_model_desc* desc, int32_t kind, int32_t n, const void* src,
                             void* dst, void* stream);

/*
 * easybalance_combine -- the weighted sum of Eq. (1) plus the residual of
 * Section 2.1, for every micro-batch of the step (the gather half of
 * MoECompute_Combine):
 *   x[t] <- x[t] + ( sum_{r<k} w[t][r] * o[inv[q(t,r)]] + sum_{s<S} o[inv[q(t,k+s)]] )
 * summed in fp32 in exactly that order (routed slots ascending, then shared).
 *
 * run, n_run  the same array passed to easybalance_moe_step
 * x_inout     host [n_run] of device pointers, entry rho -> [T_rho][H] fp32
 * o, inv      device outputs of that easybalance_moe_step call
 */
int easybalance_combine(const eb_model_desc* desc, int32_t n_run, const eb_work* run,
                        float* const* x_inout, const void* o, const int32_t* inv,
                        void* stream);

/*
 * easybalance_run_pass -- one pass of Algorithm 1 (Section 4.2) for N
 * micro-batches of T tokens through all L layers, driven by the library:
 *   route every micro-batch at layer 0 (easybalance_route);
 *   while the pool S is not empty:
 *     RunSet = Schedule(S, m) (easybalance_schedule's policies on the pool's
 *       expert counts, or EB_POLICY_LOCKSTEP: RunSet = S);
 *     easybalance_moe_step + easybalance_combine on the RunSet, entries in
 *       ascending micro-batch id, each at its own layer;
 *     l_j += 1 for j in RunSet; route those with l_j < L; drop the finished.
 * The results are the ones the same sequence of calls through the other entry
 * points gives.  The only host<->device synchronisation per step is the copy
 * of the pool's expert counts to pinned host memory for the scheduler (a
 * buffer the calling thread keeps for later passes, freed at thread exit).
 *
 * policy | EB_PASS_DEVICE_SCHEDULE: the same pass with Schedule on the GPU (a
 * one-workgroup kernel at the start of each step, exact integer arithmetic,
 * the same RunSets bit for bit), every step's kernels reading their tables
 * from device memory, and the host queueing steps ahead instead of waiting
 * for the counts: it queues only steps that must run (s steps done and a
 * micro-batch L - l layers short need s + L - l in all) and reads a status
 * word the scheduler kernel writes to host-mapped memory (256 bytes the
 * calling thread keeps for later passes, freed at thread exit).  The call returns
 * once the last step is queued (after the records are copied, if any are
 * asked for).  EB_ERR_UNSUPPORTED if D > 64 or, for fp32, E > 64.
 *
 * x            device [N][T][H] fp32, updated in place (the residual stream)
 * gain         device [L][H] fp32;  bias  device [L][E] fp32
 * Wg           host [L] of device pointers, each [E][H] dtype
 * W_gu, W_dn   host [L] of device pointers as for easybalance_moe_step
 * policy, m    EB_POLICY_* and the minimum RunSet size of Algorithm 1
 *              (MaxUtil: N <= EB_MAXUTIL_MAX_POOL)
 * state        device scratch of state_bytes >= easybalance_pass_state_size
 *              (routing outputs, grouped rows, step workspace), 256-byte
 *              aligned, caller-owned; contents undefined afterwards
 * max_steps    capacity of the per-step host outputs below
 * n_steps_out  host out (nullable): steps the pass took (at most N * L)
 * runsets_out  host out [max_steps] (nullable): RunSet bit masks
 * layers_out   host out [max_steps][N] (nullable): layer each RunSet member
 *              ran at, -1 for micro-batches not in the RunSet
 * step_load_out host out [max_steps][D] (nullable): combined workload W
 * groups_out   host out [max_steps] (nullable): (layer, expert slot) groups
 *              with rows in the step (routed experts with a token, plus the
 *              S shared experts of every layer in the RunSet)
 * layer_loads_out host out [N][L][D] (nullable): per-device load of each
 *              micro-batch at each layer, as its routing produced it
 * placement    host (nullable): static expert placement with replicas (see
 *              eb_placement) from which every per-device load above and
 *              every Schedule decision is formed; NULL = E/D contiguous
 *              experts per device.  The expert computation does not depend on
 *              it (on one GPU every copy of an expert is the same weights), so
 *              the hidden states are those of any other schedule.
 * Steps past max_steps are run but not recorded.
 */
int easybalance_pass_state_size(const eb_model_desc* desc, int32_t N, int32_t T, size_t* bytes);
int easybalance_run_pass(const eb_model_desc* desc, int32_t N, int32_t T, float* x,
                         const float* gain, const void* const* Wg, const float* bias,
                         const void* const* W_gu, const void* const* W_dn, int32_t policy,
                         int32_t m, void* state, size_t state_bytes, int32_t max_steps,
                         int32_t* n_steps_out, uint64_t* runsets_out, int32_t* layers_out,
                         int64_t* step_load_out, int32_t* groups_out, int32_t* layer_loads_out,
                         const eb_placement* placement, void* stream);

/*
 * Kernel timing for measurement.  Between easybalance_profile_begin(mask) and
 * easybalance_profile_end(), every kernel the library launches whose class
 * EB_K_* has its bit (1u << EB_K_*) set in kernel_mask is bracketed by HIP
 * events recorded on the stream it is launched on (EB_PROFILE_ALL selects
 * every class).  The events only time: they are recorded without a
 * system-scope fence, so they do not order memory for the host; each pair
 * still adds a little time to the stream, so a caller timing a whole pass
 * selects only the kernels it needs.  profile_end waits
 * for those events and returns, per kernel class, the summed duration in ms
 * (ms_out[EB_NUM_KERNELS]) and the launch count (launches_out[EB_NUM_KERNELS]);
 * both host arrays are nullable.  Process-wide state, guarded by a mutex.
 */
#define EB_PROFILE_ALL ((1u << EB_NUM_KERNELS) - 1u)
int easybalance_profile_begin(uint32_t kernel_mask);
int easybalance_profile_end(double* ms_out, int64_t* launches_out);

#ifdef __cplusplus
}
#endif

#endif /* EASYBALANCE_H */
