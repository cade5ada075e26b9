// Fixed device scratch for adaptcore_matmul_noalloc (see noalloc.hip).
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace ac {

// Size of the per-device scratch array: the largest workspace a plan run by
// adaptcore_matmul_noalloc may need.
constexpr int64_t NOALLOC_SCRATCH_BYTES = 64LL << 20;
constexpr int NOALLOC_MAX_DEVICES = 64;

// Device address of the scratch array on device `dev`, which must be the
// calling thread's current device the first time (resolved then, cached).
hipError_t noalloc_scratch(int dev, void** out);

}  // namespace ac
