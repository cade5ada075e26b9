// Fixed device scratch of adaptcore_matmul_noalloc: the workspace of split-K
// partials, stream-K pieces and row-major copies of column-major operands for
// callers that cannot allocate device memory (code under graph capture,
// serving loops, harnesses that forbid allocation). Every GPU the library
// runs on holds one copy of the array, at its own address, until the process
// ends.
#include <hip/hip_runtime.h>

#include <mutex>

#include "noalloc.h"

static __device__ __align__(256) char scratch[ac::NOALLOC_SCRATCH_BYTES];

namespace ac {
namespace {
std::mutex g_mu;
void* g_ptr[NOALLOC_MAX_DEVICES] = {};
}  // namespace

// In host code `scratch` names a host-side stand-in, not device memory: the
// device address is resolved once per device, with that device current, and
// only that address is ever handed to kernels.
hipError_t noalloc_scratch(int dev, void** out) {
  if (dev < 0 || dev >= NOALLOC_MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ptr[dev]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != dev) return hipErrorInvalidDevice;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return hipSuccess;
}

}  // namespace ac
