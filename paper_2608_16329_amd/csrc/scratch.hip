// Fixed device scratch of the entry point that allocates nothing
// (mlip_compute_noalloc): the fused kernel's per-work-group workspace, the
// block totals and the active-pair counter live in one file-scope device
// array instead of context buffers.  Each device holds its own copy of the
// array from the call that first resolves it there until the process ends.
#include <mutex>

#include "mlip_internal.h"

// In host code `scratch` names a host-side stand-in, not device memory: only
// the address that hipGetSymbolAddress returns on the current device may be
// given to kernels and copies.
static __device__ __align__(256) unsigned char scratch[mlip::kStaticScratchBytes];

namespace mlip {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_lock;
void* g_address[kMaxDevices] = {};  // per device, resolved once

}  // namespace

hipError_t static_scratch_address(int device, void** out) {
  *out = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> guard(g_lock);
  if (!g_address[device]) {
    // the symbol resolves on the current device, which must be this one
    int current = -1;
    hipError_t e = hipGetDevice(&current);
    if (e != hipSuccess) return e;
    if (current != device) return hipErrorInvalidDevice;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_address[device] = p;
  }
  *out = g_address[device];
  return hipSuccess;
}

}  // namespace mlip
