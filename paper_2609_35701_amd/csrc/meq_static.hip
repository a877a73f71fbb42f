// meq_step for callers that cannot allocate device memory: the workspace is the library's own
// file-scope device array `scratch` of MEQ_STATIC_SCRATCH_BYTES, one copy per GPU the library
// runs on, held until the process ends.  Host code never passes `scratch` itself (its host-side
// name is only a stand-in for the device symbol): the device address of each GPU's copy comes
// from hipGetSymbolAddress, called once per device with that device current, and is cached.
#include <mutex>

#include "meq.h"
#include "meq_internal.h"

#define MEQ_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

static __device__ __align__(256) uint8_t scratch[MEQ_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of the current device's copy of `scratch` (nullptr on a HIP error).
void* scratch_address() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

MEQ_EXPORT meq_status meq_step_static(meq_plan* plan, void* const* params, const void* const* grads,
                                      float* const* momenta, float lr, hipStream_t stream) {
  if (!plan) return MEQ_ERR_INVALID_ARG;
  const size_t need = meq_workspace_bytes(plan);
  if (need > MEQ_STATIC_SCRATCH_BYTES) return MEQ_ERR_WORKSPACE;
  if (need == 0) return meq_step(plan, params, grads, momenta, lr, nullptr, 0, stream);  // nothing to update
  void* ws = scratch_address();
  if (!ws) return MEQ_ERR_HIP;
  return meq_step(plan, params, grads, momenta, lr, ws, MEQ_STATIC_SCRATCH_BYTES, stream);
}
