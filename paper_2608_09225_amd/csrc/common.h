// Shared host/device helpers of libkvgov (error latching, launch checks).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/kvgov.h"

namespace kvgov {

// Store `code` into *status unless an earlier error is already there.
__device__ __forceinline__ void latch(int32_t *status, int32_t code) {
  atomicCAS(status, 0, code);
}

inline hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

inline int launch_status() {
  return hipGetLastError() == hipSuccess ? KVGOV_OK : KVGOV_E_HIP;
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

constexpr int kWave = 64;

// Number of compute units of the current device (cached per device).
int device_cu_count();

}  // namespace kvgov
