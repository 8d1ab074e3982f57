// Launchers of the walk kernels (random walks and walk records). Kept apart
// from the other launchers so that the walk kernel's sources are exactly
// random_walk.hip, common.hpp and this header.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "rdf2v.h"

namespace rdf2v {

struct WalkArgs {
  const int32_t *row_ptr;
  const int32_t *edges;       // (predicate, object) pairs, 8-byte aligned
  const int32_t *walk_edges;  // optional (predicate, object, row lo, row hi), 16-byte aligned
  const int32_t *start;
  int32_t *tokens;
  int32_t *lens;
  int32_t *status;
  int64_t walk_begin;
  int64_t walk_count;
  int64_t num_edges;
  int32_t num_entities;
  int32_t num_predicates;
  int32_t walks_per_node;
  int32_t depth;
  int32_t token_kind;  // rdf2v_walk_tokens
  uint32_t key_lo;
  uint32_t key_hi;
};
rdf2v_status launch_random_walks(const WalkArgs &args, hipStream_t stream);

rdf2v_status launch_walk_edges(const int32_t *row_ptr, const int32_t *edges, int64_t num_edges,
                               int32_t num_entities, int32_t *walk_edges_out, int32_t *status_dev,
                               hipStream_t stream);

}  // namespace rdf2v
