// static_scratch.hip -- the fixed device scratch behind kb_follow_noalloc.
//
// Callers that cannot allocate device memory (code under graph capture,
// serving loops, harnesses that forbid hipMalloc) get the forward pass with
// its split-row partials in this file-scope array instead of a caller
// workspace.  The array lives in this file's own code object, so a device
// holds it from the first kb_follow_noalloc call on that device until the
// process ends.
//
// In host code `scratch` names a host-side stand-in, not device memory: the
// device address of each device's copy comes from hipGetSymbolAddress, called
// once per device with that device current, and only that address is ever
// handed to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.h"

namespace {

static __device__ __align__(256) unsigned char scratch[kbf::kStaticScratchBytes];

}  // namespace

namespace kbf {

hipError_t static_scratch(int device, void **ptr) {
  *ptr = nullptr;
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void *addr[kMaxDevices] = {};
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[device]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device) return hipErrorInvalidDevice;  // resolved with its own device current
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[device] = p;
  }
  *ptr = addr[device];
  return hipSuccess;
}

}  // namespace kbf
