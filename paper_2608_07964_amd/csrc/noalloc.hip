// easybalance_moe_step_noalloc: easybalance_moe_step for callers that cannot
// allocate device memory.  The step's scratch (permutation histograms and
// bases, key offsets, tile and group lists, work counters, perm, the split-K
// partial sums) lives in a file-scope device array instead of a caller
// workspace; the kernels are the same, so the results are the same bits.
//
// In host code `scratch` names a host-side stand-in, not device memory: the
// array's device address is taken once per device with hipGetSymbolAddress
// (with that device current) and only that address is handed to kernels.
#include <mutex>

#include "eb_internal.h"

namespace eb {
namespace {

static_assert(EB_NOALLOC_SCRATCH_BYTES % 256 == 0, "scratch size");

// One copy per device, held from the code object's load until the process ends.
static __device__ __align__(256) unsigned char scratch[EB_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array (taken on the first
// call on that device).
int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return set_error(EB_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return set_error(EB_ERR_UNSUPPORTED, "device %d: the static scratch serves devices 0..%d", dev,
                     kMaxDevices - 1);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return set_error(EB_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return EB_OK;
}

}  // namespace
}  // namespace eb

using namespace eb;

extern "C" int easybalance_moe_step_noalloc(const eb_model_desc* desc, int32_t n_run, const eb_work* run,
                                            const void* const* W_gu, const void* const* W_dn, void* o_out,
                                            int32_t* inv_out, const eb_step_views* views, void* stream) {
  if (views == nullptr || views->a_perm == nullptr || views->h == nullptr)
    return set_error(EB_ERR_INVALID_ARG, "views with a_perm and h are required (the caller's buffers)");
  void* ws = nullptr;
  const int rc = scratch_address(&ws);
  if (rc) return rc;
  return moe_step_common(desc, n_run, run, W_gu, W_dn, ws, EB_NOALLOC_SCRATCH_BYTES, o_out, inv_out, views,
                         stream, true);
}
