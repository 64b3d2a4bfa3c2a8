// Stable grouping of a step's (token, expert) pairs by key (layer, expert slot).
//
// On an EP group this is the dispatch all-to-all (Section 2.2); with several
// micro-batches at different layers in one step (Section 4.1) the key carries
// the layer, so one grouped GEMM launch covers every (layer, expert) group.
//
//   perm_count_kernel    per 256-token chunk: routed pairs per expert (LDS atomics)
//   perm_scan_kernel     one workgroup: per-key totals, offsets, per-chunk bases,
//                        the GEMM tile list (each BM-row block's group record) and
//                        the list of non-empty groups (key, first row, rows,
//                        index of its first row block); it also clears the
//                        work counters of the step's grouped GEMM launches
//   perm_scatter_kernel  per chunk: stable rank of each pair inside its key from
//                        per-wavefront 64-bit expert masks (popcount of the lanes
//                        below), then inv and perm
//   gather_tokens_kernel one wavefront per (token, 1 KB piece of its row):
//                        the piece, read once, to a_perm[inv[q]] for each of
//                        the token's k+S pairs q
//
// Pair q = (tok_base[rho] + t) * (k+S) + r; key = layer*(E+S) + slot expert.
// All results are integers fixed by the inputs (no order-dependent atomics).
#include "eb_internal.h"
#include "eb_numeric.h"

namespace eb {
namespace {

constexpr int kScanThreads = 1024;

__device__ __forceinline__ int clamp_expert(int e, int E) { return e < 0 ? 0 : (e >= E ? E - 1 : e); }

template <class RTA>
__global__ __launch_bounds__(kPermChunk) void perm_count_kernel(RTA rta, int32_t* __restrict__ hist) {
  const RunTable& rt = rta.get();
  __shared__ int cnt[1024];
  const int b = blockIdx.x;
  if (b >= rt.chunk_base[rt.n]) return;  // past the live chunks (grid sized for the largest step)
  for (int e = threadIdx.x; e < rt.E; e += blockDim.x) cnt[e] = 0;
  __syncthreads();
  const int rho = find_entry(rt.chunk_base, rt.n, b);
  const int T = rt.tok_base[rho + 1] - rt.tok_base[rho];
  const int t = (b - rt.chunk_base[rho]) * kPermChunk + threadIdx.x;
  if (t < T) {
    const int32_t* ix = in_global(rt.idx[rho]) + (size_t)t * rt.k;
    for (int r = 0; r < rt.k; ++r) atomicAdd(&cnt[clamp_expert(ix[r], rt.E)], 1);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < rt.E; e += blockDim.x) hist[(size_t)b * rt.E + e] = cnt[e];
}

constexpr int kScanWaves = kScanThreads / kWave;
constexpr int kMaxKeys = 15360;      // L * (E + S) limit of the descriptor check
constexpr int kHistWindow = 16384;   // histogram cells held in LDS at once

// Block-wide exclusive scan of one value per thread (1024 threads): a
// shuffle scan inside each wavefront, then over the 16 wavefront totals;
// returns the exclusive prefix and writes the total to *total.
__device__ int block_exclusive_scan(int v, int* wtot, int* total) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  int x = v;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int y = __shfl_up(x, off, kWave);
    if (lane >= off) x += y;
  }
  if (lane == kWave - 1) wtot[wave] = x;
  __syncthreads();
  if (wave == 0) {
    int t = lane < kScanWaves ? wtot[lane] : 0;
#pragma unroll
    for (int off = 1; off < kScanWaves; off <<= 1) {
      const int y = __shfl_up(t, off, kWave);
      if (lane >= off) t += y;
    }
    if (lane < kScanWaves) wtot[lane] = t;
  }
  __syncthreads();
  const int before = wave > 0 ? wtot[wave - 1] : 0;
  *total = wtot[kScanWaves - 1];
  __syncthreads();  // wtot is reused by the next scan
  return before + x - v;
}

// offsets: [L*(E+S)+1]; chunk_base: [n_chunks][E+S]; tiles: [max_tiles].
// The histogram cells (chunk b, column c) go through LDS in windows of
// kHistWindow / (E+S) chunks (one window unless the step is very large);
// every global load of a phase is independent of the others.
template <class RTA>
__global__ __launch_bounds__(kScanThreads) void perm_scan_kernel(
    RTA rta, const int32_t* __restrict__ hist, int32_t* __restrict__ chunk_base,
    int32_t* __restrict__ offsets, int4* __restrict__ tiles, int32_t* __restrict__ n_tiles,
    int4* __restrict__ groups, int32_t* __restrict__ n_groups, int bm, int max_tiles,
    int32_t* __restrict__ work_ctr) {
  __shared__ int running[kMaxKeys];              // per-key totals, then offsets / cursors
  __shared__ int hl[kHistWindow];                // one window of histogram cells
  __shared__ int wtot[kScanWaves];
  __shared__ int s_cb[EB_MAX_RUN + 1], s_tb[EB_MAX_RUN + 1], s_ly[EB_MAX_RUN];
  const RunTable& rt = rta.get();
  const int tid = threadIdx.x;
  if (tid < kWorkCounters) work_ctr[tid] = 0;
  const int E = rt.E, ES = rt.E + rt.S, n = rt.n;
  const int n_chunks = rt.chunk_base[n];
  const int n_keys = rt.L * ES;
  for (int i = tid; i < n_keys; i += kScanThreads) running[i] = 0;
  if (tid <= n) {
    s_cb[tid] = rt.chunk_base[tid];
    s_tb[tid] = rt.tok_base[tid];
  }
  if (tid < n) s_ly[tid] = rt.layer[tid];
  __syncthreads();

  // cell (b, c): routed pairs of chunk b on expert c, or (shared slot c >= E)
  // the chunk's tokens; *key = (layer of b's entry, c)
  auto cell = [&](int b, int c, int* key) {
    const int rho = find_entry(s_cb, n, b);
    *key = s_ly[rho] * ES + c;
    if (c < E) return (int)hist[(size_t)b * E + c];
    return min(kPermChunk, s_tb[rho + 1] - s_tb[rho] - (b - s_cb[rho]) * kPermChunk);
  };
  const int win = kHistWindow / ES;  // >= 16 chunks (ES <= 1024)
  const int n_win = (n_chunks + win - 1) / win;

  // 1) per-key totals (integer LDS atomics: order-free); the last window
  //    stays in hl
  for (int w0 = 0; w0 < n_chunks; w0 += win) {
    const int cells = min(win, n_chunks - w0) * ES;
    for (int i = tid; i < cells; i += kScanThreads) {
      int key;
      const int v = cell(w0 + i / ES, i % ES, &key);
      hl[i] = v;
      atomicAdd(&running[key], v);
    }
  }
  __syncthreads();

  // 2) exclusive scan over keys -> offsets; thread tid owns a contiguous span
  const int span = (n_keys + kScanThreads - 1) / kScanThreads;
  const int k0 = min(tid * span, n_keys), k1 = min(k0 + span, n_keys);
  int local = 0;
  for (int i = k0; i < k1; ++i) local += running[i];
  int total = 0;
  int base = block_exclusive_scan(local, wtot, &total);
  for (int i = k0; i < k1; ++i) {
    const int v = running[i];
    offsets[i] = base;
    running[i] = base;  // becomes the running cursor of key i
    base += v;
  }
  if (tid == 0) offsets[n_keys] = total;
  __syncthreads();

  // 3) tile and group lists: ceil(M/bm) row blocks per non-empty key, keys ascending
  auto rows_of = [&](int i) { return (i + 1 < n_keys ? running[i + 1] : total) - running[i]; };
  int local_tiles = 0, local_groups = 0;
  for (int i = k0; i < k1; ++i) {
    const int M = rows_of(i);
    local_tiles += (M + bm - 1) / bm;
    local_groups += M > 0;
  }
  int tiles_total = 0, groups_total = 0;
  int tb = block_exclusive_scan(local_tiles, wtot, &tiles_total);
  int gb = block_exclusive_scan(local_groups, wtot, &groups_total);
  for (int i = k0; i < k1; ++i) {
    const int r0 = running[i], M = rows_of(i);
    if (M == 0) continue;
    const int4 g = make_int4(i, r0, M, tb);
    groups[gb++] = g;
    for (int m = 0; m < M; m += bm) {
      if (tb < max_tiles) tiles[tb] = g;
      ++tb;
    }
  }
  if (tid == 0) {
    *n_tiles = min(tiles_total, max_tiles);
    *n_groups = groups_total;
  }
  __syncthreads();  // running[] becomes the cursors below

  // 4) per-chunk bases: for every column, the entries' chunks in order; a
  //    key's cursor lives in LDS across entries, in a register within one
  for (int w = 0; w < n_win; ++w) {
    const int w0 = w * win, nw = min(win, n_chunks - w0);
    if (n_win > 1) {
      for (int i = tid; i < nw * ES; i += kScanThreads) {
        int key;
        hl[i] = cell(w0 + i / ES, i % ES, &key);
      }
      __syncthreads();
    }
    for (int c = tid; c < ES; c += kScanThreads) {
      for (int rho = 0; rho < n; ++rho) {
        const int b_lo = max(s_cb[rho], w0), b_hi = min(s_cb[rho + 1], w0 + nw);
        if (b_lo >= b_hi) continue;
        const int key = s_ly[rho] * ES + c;
        int cur = running[key];
        for (int b = b_lo; b < b_hi; ++b) {
          chunk_base[(size_t)b * ES + c] = cur;
          cur += hl[(b - w0) * ES + c];
        }
        running[key] = cur;
      }
    }
    __syncthreads();  // hl is refilled by the next window
  }
}

// One block per chunk, one token per thread.  `elem_bytes` is 2 (bf16) or 4.
template <class RTA>
__global__ __launch_bounds__(kPermChunk) void perm_scatter_kernel(
    RTA rta, const int32_t* __restrict__ chunk_base, int32_t* __restrict__ perm,
    int32_t* __restrict__ inv) {
  __shared__ unsigned long long mask[kPermChunk / kWave][1024];
  const RunTable& rt = rta.get();
  const int E = rt.E, S = rt.S, k = rt.k, ES = E + S, slots = k + S;
  const int b = blockIdx.x;
  if (b >= rt.chunk_base[rt.n]) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int i = threadIdx.x; i < (kPermChunk / kWave) * E; i += blockDim.x)
    mask[i / E][i % E] = 0ull;
  __syncthreads();
  const int rho = find_entry(rt.chunk_base, rt.n, b);
  const int T = rt.tok_base[rho + 1] - rt.tok_base[rho];
  const int t0 = (b - rt.chunk_base[rho]) * kPermChunk;
  const int t = t0 + threadIdx.x;
  const bool valid = t < T;
  const int32_t* ix = in_global(rt.idx[rho]) + (size_t)t * k;
  if (valid)
    for (int r = 0; r < k; ++r) atomicOr(&mask[wave][clamp_expert(ix[r], E)], 1ull << lane);
  __syncthreads();
  if (valid) {
    const unsigned long long below = (1ull << lane) - 1ull;
    const int32_t* cb = chunk_base + (size_t)b * ES;
    const size_t q0 = (size_t)(rt.tok_base[rho] + t) * slots;
    for (int r = 0; r < slots; ++r) {
      int pos;
      if (r < k) {
        const int e = clamp_expert(ix[r], E);
        int rank = __popcll(mask[wave][e] & below);
        for (int w2 = 0; w2 < wave; ++w2) rank += __popcll(mask[w2][e]);
        pos = cb[e] + rank;
      } else {
        pos = cb[E + (r - k)] + threadIdx.x;  // every token of the chunk has it
      }
      inv[q0 + r] = pos;
      perm[pos] = (int32_t)(q0 + r);
    }
  }
}

// One wavefront per (token, 1 KB piece of its row): the piece is read once
// (one 16-byte load per lane) and written to the grouped positions inv[q]
// of all the token's k+S pairs.  Reading each row once per pair instead (one
// wavefront per grouped row) moves up to k+S times the read bytes; pieces of
// 2 KB keep fewer wavefronts in flight.
constexpr int kGatherU = 1;                  // 16-byte loads per lane per piece
constexpr int kGatherPiece = 64 * kGatherU;  // 16-byte chunks per piece

template <class RTA>
__global__ __launch_bounds__(256) void gather_tokens_kernel(RTA rta, int pieces, int elem_bytes,
                                                          const int32_t* __restrict__ inv,
                                                          uint8_t* __restrict__ a_perm) {
  const RunTable& rt = rta.get();
  const int total = rt.tok_base[rt.n];
  const int lane = threadIdx.x & 63;
  const long long wv = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wv >= (long long)total * pieces) return;
  const int g = (int)(wv / pieces);  // global token of the step
  const int c0 = (int)(wv - (long long)g * pieces) * kGatherPiece;
  const int slots = rt.k + rt.S;
  const int P = total * slots;
  const int rho = find_entry(rt.tok_base, rt.n, g);
  const int t = g - rt.tok_base[rho];
  const size_t row_bytes = (size_t)rt.H * elem_bytes;
  const uint4* src = reinterpret_cast<const uint4*>(in_global(static_cast<const uint8_t*>(rt.a[rho])) + (size_t)t * row_bytes);
  // lane r < slots holds the grouped position of slot r (clamped into range)
  const int pos = lane < slots ? min(max(inv[(size_t)g * slots + lane], 0), P - 1) : 0;
  const int n16 = (int)(row_bytes / 16);
  uint4 v[kGatherU];
#pragma unroll
  for (int j = 0; j < kGatherU; ++j) {
    const int c = c0 + 64 * j + lane;
    if (c < n16) v[j] = src[c];
  }
  for (int r = 0; r < slots; ++r) {
    uint4* dst = reinterpret_cast<uint4*>(a_perm + (size_t)__shfl(pos, r, 64) * row_bytes);
#pragma unroll
    for (int j = 0; j < kGatherU; ++j) {
      const int c = c0 + 64 * j + lane;
      if (c < n16) dst[c] = v[j];
    }
  }
}

}  // namespace

// Launch helpers shared by the host-built (ByValue) and device-written
// (InMemory) tables; grids are the live sizes or the largest step's.
namespace {

template <class RTA>
void perm_count_impl(RTA a, int grid, int32_t* hist, hipStream_t s) {
  prof_start(EB_K_PERM_COUNT, s);
  if (grid > 0) hipLaunchKernelGGL(perm_count_kernel<RTA>, dim3(grid), dim3(kPermChunk), 0, s, a, hist);
  prof_stop(EB_K_PERM_COUNT, s);
}

template <class RTA>
void perm_scan_impl(RTA a, const int32_t* hist, int32_t* chunk_base, int32_t* offsets, int4* tiles,
                    int32_t* n_tiles, int4* groups, int32_t* n_groups, int bm, int max_tiles,
                    int32_t* work_ctr, hipStream_t s) {
  prof_start(EB_K_PERM_SCAN, s);
  hipLaunchKernelGGL(perm_scan_kernel<RTA>, dim3(1), dim3(kScanThreads), 0, s, a, hist, chunk_base,
                     offsets, tiles, n_tiles, groups, n_groups, bm, max_tiles, work_ctr);
  prof_stop(EB_K_PERM_SCAN, s);
}

// grid_chunks / grid_tokens: chunks and tokens the grids cover
template <class RTA>
void perm_scatter_impl(RTA a, int H, int grid_chunks, int grid_tokens, int elem_bytes,
                       const int32_t* chunk_base, int32_t* perm, int32_t* inv, void* a_perm,
                       hipStream_t s) {
  prof_start(EB_K_PERM_SCATTER, s);
  if (grid_chunks > 0)
    hipLaunchKernelGGL(perm_scatter_kernel<RTA>, dim3(grid_chunks), dim3(kPermChunk), 0, s, a,
                       chunk_base, perm, inv);
  prof_stop(EB_K_PERM_SCATTER, s);
  const size_t row_bytes = (size_t)H * elem_bytes;
  prof_start(EB_K_PERM_GATHER, s);
  if (grid_tokens > 0) {
    const int n16 = (int)(row_bytes / 16);
    const int pieces = (n16 + kGatherPiece - 1) / kGatherPiece;
    const long long waves = (long long)grid_tokens * pieces;
    hipLaunchKernelGGL(gather_tokens_kernel<RTA>, dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s, a,
                       pieces, elem_bytes, inv, static_cast<uint8_t*>(a_perm));
  }
  prof_stop(EB_K_PERM_GATHER, s);
}

bool scan_fits(int L, int E, int S, int n) {
  return (long)L * (E + S) <= kMaxKeys && E + S <= kScanThreads && n <= EB_MAX_RUN;
}

}  // namespace

hipError_t launch_perm_count(const RunTable& rt, int n_chunks, int32_t* hist, hipStream_t s) {
  perm_count_impl(ByValue<RunTable>{rt}, n_chunks, hist, s);
  return hipGetLastError();
}

hipError_t launch_perm_scan(const RunTable& rt, const int32_t* hist, int32_t* chunk_base,
                            int32_t* offsets, int4* tiles, int32_t* n_tiles, int4* groups,
                            int32_t* n_groups, int bm, int max_tiles, int32_t* work_ctr,
                            hipStream_t s) {
  if (!scan_fits(rt.L, rt.E, rt.S, rt.n)) return hipErrorInvalidValue;
  perm_scan_impl(ByValue<RunTable>{rt}, hist, chunk_base, offsets, tiles, n_tiles, groups, n_groups,
                 bm, max_tiles, work_ctr, s);
  return hipGetLastError();
}

hipError_t launch_perm_scatter(const RunTable& rt, int n_chunks, int elem_bytes,
                               const int32_t* chunk_base, int32_t* perm, int32_t* inv,
                               void* a_perm, hipStream_t s) {
  perm_scatter_impl(ByValue<RunTable>{rt}, rt.H, n_chunks, rt.tok_base[rt.n], elem_bytes,
                    chunk_base, perm, inv, a_perm, s);
  return hipGetLastError();
}

hipError_t launch_permute_dev(const eb_model_desc& d, const RunTable* rt, int max_chunks,
                              int max_tokens, const StepBuffers& b, hipStream_t s) {
  if (!scan_fits(d.L, d.E, d.S, 0)) return hipErrorInvalidValue;
  const InMemory<RunTable> a{rt};
  const int eb = d.dtype == EB_DTYPE_BF16 ? 2 : 4;
  perm_count_impl(a, max_chunks, b.hist, s);
  perm_scan_impl(a, b.hist, b.chunk_base, b.offsets, b.tiles, b.n_tiles, b.groups, b.n_groups,
                 gemm_bm(d.dtype), b.max_tiles, b.work_ctr, s);
  perm_scatter_impl(a, d.H, max_chunks, max_tokens, eb, b.chunk_base, b.perm, b.inv,
                    b.a_perm, s);
  return hipGetLastError();
}

}  // namespace eb
