// Walk records on gfx950: walk_edges[k] = (pred, obj, row_ptr[obj], row_ptr[obj + 1])
// for every out-edge record k of the CSR, so that a walk reads one 16-byte record
// per hop instead of the edge record and then the next entity's row bounds.
//
// The edge records stream through once (non-temporal loads and stores); the row
// bounds are a random gather into row_ptr, L2-resident up to a few MB (the
// compiler fetches the two adjacent bounds with one 8-byte load).

#include "common.hpp"
#include "walk.hpp"

namespace rdf2v {
namespace {

typedef int32_t v4i32 __attribute__((ext_vector_type(4)));
typedef int32_t v2i32 __attribute__((ext_vector_type(2)));

// Each thread handles kWalkEdgeItems records strided by the block size, issuing
// all loads, then all row-bound gathers, then all stores, so that several
// independent memory operations per lane are in flight.
constexpr int kWalkEdgeThreads = 256;
constexpr int kWalkEdgeItems = 2;
constexpr int kWalkEdgeTile = kWalkEdgeThreads * kWalkEdgeItems;

__global__ __launch_bounds__(kWalkEdgeThreads) void walk_edges_kernel(
    const int32_t *__restrict__ row_ptr, const int2 *__restrict__ edges, int64_t n,
    int32_t num_entities, v4i32 *__restrict__ out, int32_t *status) {
  const int64_t base = int64_t(blockIdx.x) * kWalkEdgeTile + threadIdx.x;
  int2 rec[kWalkEdgeItems];
  int2 bounds[kWalkEdgeItems];
  int bad = 0;
#pragma unroll
  for (int j = 0; j < kWalkEdgeItems; ++j) {
    const int64_t i = base + j * kWalkEdgeThreads;
    rec[j] = make_int2(0, 0);
    if (i < n) {
      // streamed once: non-temporal, so the row_ptr lines gathered below stay in L2
      const v2i32 v = __builtin_nontemporal_load(reinterpret_cast<const v2i32 *>(edges) + i);
      rec[j] = make_int2(v.x, v.y);
    }
  }
  // The gathers of all items are issued together. An object id out of range is
  // flagged, not read, and gets the bounds (0, 0) of an empty row; otherwise
  // o + 1 <= num_entities, the last index of row_ptr.
#pragma unroll
  for (int j = 0; j < kWalkEdgeItems; ++j) {
    const int64_t i = base + j * kWalkEdgeThreads;
    const bool ok = uint32_t(rec[j].y) < uint32_t(num_entities);
    bad |= (i < n && !ok) ? 1 : 0;
    bounds[j] = make_int2(0, 0);
    if (i < n && ok) bounds[j] = make_int2(row_ptr[rec[j].y], row_ptr[rec[j].y + 1]);
  }
#pragma unroll
  for (int j = 0; j < kWalkEdgeItems; ++j) {
    const int64_t i = base + j * kWalkEdgeThreads;
    if (i < n) __builtin_nontemporal_store(v4i32{rec[j].x, rec[j].y, bounds[j].x, bounds[j].y}, out + i);
  }
  if (bad && status != nullptr) atomicOr(status, RDF2V_STATUS_ID_OUT_OF_RANGE);
}

}  // namespace

rdf2v_status launch_walk_edges(const int32_t *row_ptr, const int32_t *edges, int64_t num_edges,
                               int32_t num_entities, int32_t *walk_edges_out, int32_t *status_dev,
                               hipStream_t stream) {
  if (num_edges == 0) return RDF2V_OK;
  const int64_t blocks = (num_edges + kWalkEdgeTile - 1) / kWalkEdgeTile;
  walk_edges_kernel<<<dim3(unsigned(blocks)), dim3(kWalkEdgeThreads), 0, stream>>>(
      row_ptr, reinterpret_cast<const int2 *>(edges), num_edges, num_entities,
      reinterpret_cast<v4i32 *>(walk_edges_out), status_dev);
  RDF2V_LAUNCH_CHECK();
  return RDF2V_OK;
}

}  // namespace rdf2v
