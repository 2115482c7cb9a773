// Library-held scratch memory for losa_sparse_attn_fwd_noalloc, the forward
// entry point for callers that cannot allocate device memory (code under HIP
// graph capture, serving loops, harnesses that forbid allocation).
//
// The scratch is a file-scope device array of kNoAllocScratchBytes.  Every GPU
// the library runs on holds its own copy, at its own address, from the moment
// this code object is loaded on that device until the process ends.  In host
// code the array's name is only a handle for the symbol lookup below; kernels
// receive the device address the lookup returns, never the name.
//
// Calls on one GPU share that GPU's copy and leave the last call's contents in
// it.  The forward rewrites everything it reads from the scratch (V^T and the
// dispatch order) before reading it, so nothing needs to start at zero, but
// two calls that overlap in time on one GPU (different streams, or different
// host threads without ordering) race on it.
#include <hip/hip_runtime.h>

#include <mutex>

#include "launch.hpp"

namespace losa {

namespace {

static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
void* g_scratch[kMaxDevices] = {};  // device address of `scratch` per device, once looked up

}  // namespace

hipError_t noalloc_scratch(hipStream_t stream, void** ptr, int* device) {
  *ptr = nullptr;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  *device = dev;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  if (stream != nullptr) {
    // the lookup below is made with the current device; a stream of another
    // device would run the kernels against that device's copy
    int sdev = -1;
    e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) return e;
    if (sdev != dev) return hipErrorInvalidResourceHandle;
  }
  std::lock_guard<std::mutex> lock(g_mutex);
  if (g_scratch[dev] == nullptr) {
    // once per device, with that device current: its copy's address
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch[dev] = p;
  }
  *ptr = g_scratch[dev];
  return hipSuccess;
}

}  // namespace losa
