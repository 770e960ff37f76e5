// Forward-only token log-probabilities without a caller workspace: the same
// kernels as agrl_token_logprob, with their workspace in a fixed array of
// device memory that the library holds on every GPU it runs on.  For callers
// that cannot allocate device memory around the call.
#include <stdio.h>

#include <mutex>

#include "../../include/agrl.h"
#include "common.hpp"

namespace {

// AGRL_NOALLOC_SCRATCH_BYTES of device memory per GPU, held until the process
// ends.  In host code `scratch` is only a stand-in for the symbol: its device
// address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) uint8_t scratch[AGRL_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::once_flag g_once[kMaxDevices];
void* g_scratch[kMaxDevices];
hipError_t g_status[kMaxDevices];

void init_scratch(int dev) {
  void* p = nullptr;
  g_status[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  g_scratch[dev] = g_status[dev] == hipSuccess ? p : nullptr;
}

}  // namespace

extern "C" int agrl_token_logprob_noalloc(int64_t T, int64_t max_act, int32_t d, int32_t V,
                                          int32_t dtype, const void* H, const void* W,
                                          const int32_t* token_id, const uint8_t* action_mask,
                                          const agrl_options* opt, float* logp, float* lse,
                                          void* stream) {
  int dev = 0;
  int rc = agrl::hip_status(hipGetDevice(&dev));
  if (rc) return rc;
  if (dev < 0 || dev >= kMaxDevices) {
    agrl::set_last_error("agrl_token_logprob_noalloc: device index out of range");
    return AGRL_E_HIP;
  }
  std::call_once(g_once[dev], init_scratch, dev);
  if (!g_scratch[dev]) return agrl::hip_status(g_status[dev]);
  if (T > 0) {
    const size_t need = agrl_token_logprob_workspace_size(T, max_act, d, V, dtype, opt);
    if (need > (size_t)AGRL_NOALLOC_SCRATCH_BYTES) {
      char buf[256];
      snprintf(buf, sizeof buf,
               "agrl_token_logprob_noalloc: these sizes need %zu bytes of scratch, more than "
               "the %lld the library holds per device; call agrl_token_logprob with a workspace",
               need, (long long)AGRL_NOALLOC_SCRATCH_BYTES);
      agrl::set_last_error(buf);
      return AGRL_E_WORKSPACE;
    }
  }
  return agrl_token_logprob(T, max_act, d, V, dtype, H, W, token_id, action_mask, opt,
                            g_scratch[dev], (size_t)AGRL_NOALLOC_SCRATCH_BYTES, logp, lse, stream);
}
