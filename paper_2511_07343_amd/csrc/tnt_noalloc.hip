// tnt_mem_fwd_noalloc: the forward pass for callers that cannot allocate
// device memory.  Its workspace is `scratch`, a file-scope device array the
// library owns; the kernels are those of tnt_mem_fwd, given the array's device
// address in place of the caller's workspace.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/tnt.h"
#include "tnt_entry.h"

namespace {

static __device__ __align__(256) unsigned char scratch[TNT_NOALLOC_WORKSPACE_BYTES];

// Device address of `scratch` per device, taken once per device (with that
// device current) on its first call.  The array's host-side name is only a
// stand-in for the symbol: every use below goes through this address.
constexpr int MAX_DEV = 64;
void* g_scratch[MAX_DEV] = {};
std::mutex g_scratch_mu;

hipError_t scratch_of_current_device(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= MAX_DEV) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

}  // namespace

extern "C" tnt_status tnt_mem_fwd_noalloc(const tnt_config* cfg, const void* q, const void* k,
                                          const void* v, const float* lr, const float* mom,
                                          const float* decay, const float* W1_init,
                                          const float* W2_init, void* o, float* final_state,
                                          void* stream) {
  if (!cfg) return TNT_ERR_NULL;
  if (tnt_mem_workspace_size(cfg, TNT_WS_FWD_MIN) > (size_t)TNT_NOALLOC_WORKSPACE_BYTES) {
    // an invalid configuration sizes to 0 and gets its own error below
    return TNT_ERR_WORKSPACE;
  }
  void* ws = nullptr;
  if (scratch_of_current_device(&ws) != hipSuccess) return TNT_ERR_HIP;
  return tnt::forward_entry(cfg, q, k, v, lr, mom, decay, W1_init, W2_init, o, final_state,
                            nullptr, 0, ws, (size_t)TNT_NOALLOC_WORKSPACE_BYTES, false,
                            (hipStream_t)stream);
}
