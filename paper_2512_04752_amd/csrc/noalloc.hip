// Static device scratch for spec_verify_noalloc: the verify step's workspace
// (residual stream, activations, attention and split-K partials, descriptors)
// in a file-scope device array instead of caller memory, for callers that
// cannot allocate.  Each device the library runs on holds its own copy of
// the array from the first lookup until the process ends.  The array lives in
// a translation unit of its own, so that its code object, which holds no
// kernel, is only loaded by processes that look it up.
#include <mutex>

#include "common.h"
#include "specverify.h"

namespace {

static __device__ __align__(256) unsigned char scratch[SPEC_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

}  // namespace

namespace spec {

// Device address of the current device's copy of `scratch`.  In host code
// the array's name only stands in for it: the address comes from
// hipGetSymbolAddress, called once per device with that device current.
hipError_t noalloc_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return hipSuccess;
}

}  // namespace spec
