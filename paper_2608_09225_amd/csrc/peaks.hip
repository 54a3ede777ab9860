// Measured-peak microbenchmarks for gfx950 (libkvgov_peaks.so).
//
// Not part of the hashing / cache path: these two kernels give the ceilings
// against which the path's kernels are also reported, beside the published
// figures.  k_peak_valu issues only independent 32-bit integer vector ops
// (rotate, 3-input add, 3-input xor: the op mix of a SHA-256 round);
// k_peak_gather reads 32-byte records at pseudo-random slots of a table, the
// access pattern of a hash-table probe.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/kvgov_peaks.h"

namespace {

constexpr int kThreads = 256;
constexpr int kChains = 8;   // independent dependency chains per lane
constexpr int kUnroll = 4;   // iterations unrolled per loop trip
constexpr int kOpsPerStep = 3;
constexpr int kLoadsPerTrip = 4;

__global__ __launch_bounds__(kThreads) void k_peak_valu(uint32_t *out, int32_t trips,
                                                        uint32_t seed) {
  const uint32_t gid = blockIdx.x * kThreads + threadIdx.x;
  uint32_t a[kChains], b[kChains];
#pragma unroll
  for (int k = 0; k < kChains; ++k) {
    a[k] = gid * 0x9E3779B9u + seed + k;
    b[k] = gid ^ (seed * (k + 1));
  }
  // Each step is exactly three VALU instructions per chain (written as asm so
  // that the compiler cannot split or merge them); the eight chains are
  // independent, so consecutive instructions never wait on each other.
  for (int t = 0; t < trips; ++t) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
      for (int k = 0; k < kChains; ++k)
        asm("v_alignbit_b32 %0, %1, %1, %2" : "=v"(a[k]) : "v"(a[k]), "i"(7 + k));
#pragma unroll
      for (int k = 0; k < kChains; ++k)
        asm("v_add3_u32 %0, %1, %2, %3" : "=v"(b[k]) : "v"(a[k]), "v"(b[k]), "s"(seed));
#pragma unroll
      for (int k = 0; k < kChains; ++k)
        asm("v_bitop3_b32 %0, %1, %2, %3 bitop3:0x96"
            : "=v"(a[k]) : "v"(a[k]), "v"(b[k]), "s"(seed));
    }
  }
  uint32_t r = 0;
#pragma unroll
  for (int k = 0; k < kChains; ++k) r ^= a[k] + b[k];
  out[gid] = r;
}

__device__ __forceinline__ uint32_t mix32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7FEB352Du;
  x ^= x >> 15;
  x *= 0x846CA68Bu;
  x ^= x >> 16;
  return x;
}

__global__ __launch_bounds__(kThreads) void k_peak_gather(const uint4 *__restrict__ table,
                                                          uint32_t mask, uint32_t *out,
                                                          int32_t trips, uint32_t seed) {
  const uint32_t gid = blockIdx.x * kThreads + threadIdx.x;
  uint32_t x = mix32(gid ^ seed);
  uint32_t acc = 0;
  for (int t = 0; t < trips; ++t) {
    uint4 v[kLoadsPerTrip][2];
#pragma unroll
    for (int u = 0; u < kLoadsPerTrip; ++u) {
      x = mix32(x + 0x9E3779B9u);
      const uint64_t slot = x & mask;
      v[u][0] = table[2 * slot];
      v[u][1] = table[2 * slot + 1];
    }
#pragma unroll
    for (int u = 0; u < kLoadsPerTrip; ++u)
      acc ^= v[u][0].x ^ v[u][0].y ^ v[u][0].z ^ v[u][0].w ^ v[u][1].x ^ v[u][1].y ^
             v[u][1].z ^ v[u][1].w;
  }
  out[gid] = acc;
}

}  // namespace

extern "C" int kvgov_peak_valu(uint32_t *out, int32_t grid, int32_t trips, int64_t *ops,
                               void *stream) {
  if (!out || grid <= 0 || trips <= 0 || !ops) return KVGOV_PEAK_E_INVAL;
  hipLaunchKernelGGL(k_peak_valu, dim3(grid), dim3(kThreads), 0,
                     reinterpret_cast<hipStream_t>(stream), out, trips, 0x2026u);
  if (hipGetLastError() != hipSuccess) return KVGOV_PEAK_E_HIP;
  *ops = int64_t(grid) * kThreads * trips * kUnroll * kChains * kOpsPerStep;
  return 0;
}

extern "C" int kvgov_peak_gather(const uint8_t *table, int64_t slots, uint32_t *out,
                                 int32_t grid, int32_t trips, int64_t *bytes, void *stream) {
  if (!table || !out || grid <= 0 || trips <= 0 || !bytes) return KVGOV_PEAK_E_INVAL;
  if (slots <= 0 || (slots & (slots - 1)) || slots > (int64_t(1) << 32))
    return KVGOV_PEAK_E_INVAL;
  if (reinterpret_cast<uintptr_t>(table) % 16) return KVGOV_PEAK_E_INVAL;
  hipLaunchKernelGGL(k_peak_gather, dim3(grid), dim3(kThreads), 0,
                     reinterpret_cast<hipStream_t>(stream), reinterpret_cast<const uint4 *>(table),
                     uint32_t(slots - 1), out, trips, 0x2026u);
  if (hipGetLastError() != hipSuccess) return KVGOV_PEAK_E_HIP;
  *bytes = int64_t(grid) * kThreads * trips * kLoadsPerTrip * 32;
  return 0;
}
