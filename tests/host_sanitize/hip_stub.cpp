// A stand-in for the HIP runtime for the host-only sanitizer build of the
// library: "device" memory is host memory, copies and fills are memcpy and
// memset, and kernel launches return success without running anything.  It
// lets AddressSanitizer and UndefinedBehaviorSanitizer check every host-side
// line of the library -- argument checks, workspace layouts, task lists,
// geometry, error paths -- without a GPU.  Test infrastructure only.
#include <hip/hip_runtime_api.h>

#include <chrono>
#include <cstdlib>
#include <cstring>

namespace {

struct Config {
  dim3 grid, block;
  size_t shmem = 0;
  hipStream_t stream = nullptr;
};
thread_local Config g_cfg;

struct Event {
  std::chrono::steady_clock::time_point t;
};

}  // namespace

extern "C" {

hipError_t hipMemsetAsync(void* dst, int value, size_t sizeBytes, hipStream_t) {
  if (sizeBytes && !dst) return hipErrorInvalidValue;
  if (sizeBytes) std::memset(dst, value, sizeBytes);
  return hipSuccess;
}

hipError_t hipMemcpyAsync(void* dst, const void* src, size_t sizeBytes, hipMemcpyKind,
                          hipStream_t) {
  if (sizeBytes && (!dst || !src)) return hipErrorInvalidValue;
  if (sizeBytes) std::memmove(dst, src, sizeBytes);
  return hipSuccess;
}

hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }

hipError_t hipGetDevice(int* dev) {
  *dev = 0;
  return hipSuccess;
}

hipError_t hipDeviceGetAttribute(int* pi, hipDeviceAttribute_t attr, int) {
  *pi = attr == hipDeviceAttributeMultiprocessorCount ? 256 : 0;
  return hipSuccess;
}

const char* hipGetErrorString(hipError_t e) { return e == hipSuccess ? "no error" : "stub error"; }

hipError_t hipGetLastError(void) { return hipSuccess; }

hipError_t hipEventCreate(hipEvent_t* ev) {
  *ev = reinterpret_cast<hipEvent_t>(new Event());
  return hipSuccess;
}

hipError_t hipEventDestroy(hipEvent_t ev) {
  delete reinterpret_cast<Event*>(ev);
  return hipSuccess;
}

hipError_t hipEventRecord(hipEvent_t ev, hipStream_t) {
  reinterpret_cast<Event*>(ev)->t = std::chrono::steady_clock::now();
  return hipSuccess;
}

hipError_t hipEventElapsedTime(float* ms, hipEvent_t a, hipEvent_t b) {
  *ms = std::chrono::duration<float, std::milli>(reinterpret_cast<Event*>(b)->t -
                                                 reinterpret_cast<Event*>(a)->t)
            .count();
  return hipSuccess;
}

hipError_t hipFuncSetAttribute(const void*, hipFuncAttribute, int) { return hipSuccess; }

// The no-allocation entry point's static array: a host buffer of the same size.
hipError_t hipGetSymbolAddress(void** devPtr, const void*) {
  static void* buf = std::calloc(256u * 1024u * 1024u, 1);
  *devPtr = buf;
  return buf ? hipSuccess : hipErrorOutOfMemory;
}

hipError_t hipLaunchKernel(const void*, dim3, dim3, void**, size_t, hipStream_t) {
  return hipSuccess;
}

hipError_t __hipPushCallConfiguration(dim3 gridDim, dim3 blockDim, size_t sharedMem,
                                      hipStream_t stream) {
  g_cfg.grid = gridDim;
  g_cfg.block = blockDim;
  g_cfg.shmem = sharedMem;
  g_cfg.stream = stream;
  return hipSuccess;
}

hipError_t __hipPopCallConfiguration(dim3* gridDim, dim3* blockDim, size_t* sharedMem,
                                     hipStream_t* stream) {
  *gridDim = g_cfg.grid;
  *blockDim = g_cfg.block;
  *sharedMem = g_cfg.shmem;
  *stream = g_cfg.stream;
  return hipSuccess;
}

// Code-object registration (present only when device code is compiled in).
void** __hipRegisterFatBinary(const void*) {
  static void* handle = nullptr;
  return &handle;
}
void __hipRegisterFunction(void**, const void*, char*, const char*, unsigned int, void*, void*,
                           void*, void*, int*) {}
void __hipRegisterVar(void**, void*, char*, char*, int, size_t, int, int) {}
void __hipUnregisterFatBinary(void**) {}

}  // extern "C"
