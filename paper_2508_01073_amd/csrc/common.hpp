// Device and host helpers shared by the library's HIP sources (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "rdf2v.h"

#define RDF2V_API extern "C" __attribute__((visibility("default")))

namespace rdf2v {

constexpr int kWave = 64;

// Return RDF2V_ERR_HIP from the enclosing function if a HIP call or the last
// launch failed.
#define RDF2V_HIP_TRY(expr)                              \
  do {                                                   \
    if ((expr) != hipSuccess) return RDF2V_ERR_HIP;      \
  } while (0)
#define RDF2V_LAUNCH_CHECK() RDF2V_HIP_TRY(hipGetLastError())

__host__ __device__ inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Lane index inside the wavefront and the mask of lower lanes.
__device__ __forceinline__ int lane_id() { return __lane_id(); }
__device__ __forceinline__ uint64_t lanes_below(int lane) { return (uint64_t(1) << lane) - 1; }

// Exclusive scan of one value per thread over a block of NT threads (NT a
// multiple of 64, at most 1024). `scratch` holds NT/64 values of LDS. Returns
// the thread's exclusive prefix; `total` receives the block-wide sum. Contains
// two block barriers, so every thread of the block must call it.
template <int NT, typename T = int>
__device__ __forceinline__ T block_exclusive_scan(T x, T *scratch, T &total) {
  constexpr int kWaves = NT / kWave;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  T v = x;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const T y = __shfl_up(v, off, kWave);
    if (lane >= off) v += y;
  }
  if (lane == kWave - 1) scratch[wave] = v;
  __syncthreads();
  T before = 0, sum = 0;
#pragma unroll
  for (int i = 0; i < kWaves; ++i) {
    const T s = scratch[i];
    before += (i < wave) ? s : T(0);
    sum += s;
  }
  __syncthreads();
  total = sum;
  return before + v - x;
}

// Sum of one value per thread over the block (same contract as above).
template <int NT, typename T = int>
__device__ __forceinline__ T block_sum(T x, T *scratch) {
  T total;
  (void)block_exclusive_scan<NT, T>(x, scratch, total);
  return total;
}

}  // namespace rdf2v
