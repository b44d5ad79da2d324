// The fixed per-device scratch array of the allocation-free qlinear entry point
// (subspec_qlinear_noalloc): split-K completion counters, per-group sums of x and
// partial sums live here instead of in the growable workspace, so that entry point
// never allocates.  Each device holds its own copy of the array, at its own address,
// from module load until the process ends.
#include <hip/hip_runtime.h>

#include <mutex>
#include <vector>

#include "kernels.h"

namespace {

static __device__ __align__(256) unsigned char scratch[subspec::kNoAllocScratchBytes];

std::mutex g_mutex;
std::vector<void*> g_scratch;  // per device: the array's device address once set up

}  // namespace

namespace subspec {

hipError_t noalloc_scratch(hipStream_t st, void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (static_cast<int>(g_scratch.size()) <= dev) g_scratch.resize(dev + 1, nullptr);
  if (!g_scratch[dev]) {
    // Set-up, once per device with that device current.  In host code `scratch`
    // names a host-side stand-in; the device address comes from the runtime.
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    e = hipStreamIsCapturing(st, &cs);
    if (e != hipSuccess) return e;
    if (cs != hipStreamCaptureStatusNone) return hipErrorStreamCaptureUnsupported;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    // The completion counters must start at zero (every launch leaves them so).
    e = hipMemsetAsync(p, 0, kSplitCounterBytes, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return e;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

}  // namespace subspec
