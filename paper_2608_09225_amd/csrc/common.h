// Shared host/device helpers of libkvgov (error latching, launch checks).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <mutex>

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

// Scratch device memory the library keeps per (device, stream), grown on
// demand and held until the process ends.  A stream runs its work in order,
// so the buffer of stream s serves one call of s at a time without any
// stream-ordered allocation (no memory handed between streams).  The caller
// keeps `lk` (it is returned locked) while it enqueues the kernels that use
// the buffer, so that calls from several host threads on one stream do not
// interleave their kernels.  Growth waits for s, then frees the old buffer.
// Returns KVGOV_OK, KVGOV_E_NOMEM or KVGOV_E_HIP.
int stream_scratch(hipStream_t s, size_t bytes, void **ptr, std::unique_lock<std::mutex> &lk);

}  // namespace kvgov
