// Workgroup order across the XCDs of gfx950.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace rdf2v {

// Work item (tile) handled by workgroup b of a grid of `items` workgroups.
// Workgroups are dealt to the 8 XCDs in turn (b mod 8), and each XCD has its
// own L2; this mapping gives XCD x one contiguous range of items, which its
// workgroups take in order. Where consecutive items write adjacent output
// ranges, the cache line at the boundary of two ranges is written partly by
// each; with both items on one XCD the two halves meet in the same L2 instead
// of going to memory as two partial writes. A bijection of [0, items), so it
// changes speed only. It pays where an item writes many short runs (a radix
// scatter tile writes one run per digit); kernels whose workgroups each write
// one long contiguous range were measured slower with it (the 8 XCDs then
// stream to 8 distant regions at once) and keep the workgroup order.
constexpr int kXcds = 8;
__device__ __forceinline__ int64_t xcd_tile(int64_t b, int64_t items) {
  const int64_t x = b % kXcds, slot = b / kXcds;
  const int64_t per = items / kXcds, rem = items % kXcds;
  return x * per + min(x, rem) + slot;
}

}  // namespace rdf2v
