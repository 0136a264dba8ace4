// Stage 2 without a workspace argument, for callers that cannot allocate
// device memory.  The workspace lives in one file-scope device array; every
// GPU the library runs on holds its own copy of it until the process ends.
//
// In host code `scratch` names a host-side stand-in, not device memory: its
// device address on the current GPU comes from hipGetSymbolAddress, looked up
// once per device on the first call there and kept.  Only that address is
// ever passed on to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/trevs.h"

namespace {

static __device__ __align__(256) uint8_t scratch[TREVS_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_lookup;
void* g_scratch[kMaxDevices];  // device address of `scratch` per device, null until looked up

// Device address of this device's scratch array (the calling thread's
// current device).
trevs_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return TREVS_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return TREVS_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_lookup);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return TREVS_ERR_HIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return TREVS_OK;
}

}  // namespace

extern "C" trevs_status trevs_inllm_prune_noalloc(const trevs_inllm_args* a, void* stream) {
  // the workspace this call needs; 0 means invalid arguments, which the
  // regular entry point reports with the precise status before any launch
  const size_t need = trevs_inllm_workspace_size(a);
  if (need == 0) return trevs_inllm_prune(a, nullptr, 0, stream);
  if (need > TREVS_NOALLOC_SCRATCH_BYTES) return TREVS_ERR_WORKSPACE;
  void* ws = nullptr;
  const trevs_status st = scratch_address(&ws);
  if (st != TREVS_OK) return st;
  // the stage-2 kernels write every workspace element they read, so the
  // previous call's contents need no clearing
  return trevs_inllm_prune(a, ws, TREVS_NOALLOC_SCRATCH_BYTES, stream);
}
