// The static scratch behind ojbkq_quantize_layer_noalloc: a file-scope device
// array that stands in for the caller's workspace, so that the entry point
// needs no device allocation.  Each GPU holds its own copy (the module's
// .bss), created when the library's code object is loaded on that device and
// kept until the process ends.
#include <hip/hip_runtime.h>

#include <mutex>

#include "ojbkq.h"

namespace {

static __device__ __align__(256) unsigned char scratch[OJBKQ_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_lock;
void* g_ptr[kMaxDevices] = {};   // device address of `scratch` per device

}  // namespace

namespace ojbkq {

// Device address of the current device's copy of the scratch array (looked up
// once per device, with that device current).  The array's name is not a
// device address in host code, so every host-side use goes through this.
hipError_t noalloc_scratch(void** out) {
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> guard(g_lock);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return hipSuccess;
}

}  // namespace ojbkq
