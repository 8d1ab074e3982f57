// Host-side launchers of the library's kernels. The extern "C" entry points in
// api.hip validate arguments and call these; each launcher only enqueues.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "rdf2v.h"
#include "walk.hpp"

namespace rdf2v {

// Layout of the rdf2v_build_csr workspace for (num_triples, num_entities).
struct SortPlan {
  int passes = 0;      // LSD radix passes over the subject id
  int digit_bits = 0;  // bits of the widest pass (<= 9); sizes the count table
  int pass_bits[4] = {0, 0, 0, 0};  // bits of each pass, lowest digit first
  int64_t tiles = 0;   // 4096-triple tiles
  int64_t count_len = 0;     // digit-major count table length = bins * tiles
  int64_t count_blocks = 0;  // scan blocks over the count table
  size_t off_keys_a = 0, off_keys_b = 0, off_payload = 0, off_counts = 0, off_partials = 0;
  size_t bytes = 0;
};
SortPlan plan_csr_build(int64_t num_triples, int32_t num_entities);

rdf2v_status launch_csr_build(const int32_t *subj, const int32_t *pred, const int32_t *obj,
                              int64_t num_triples, int32_t num_entities, int32_t num_predicates,
                              int32_t *row_ptr_out, int32_t *edges_out, void *workspace,
                              const SortPlan &plan, int32_t *status_dev, hipStream_t stream);

size_t nonsink_workspace_bytes(int32_t num_entities);
rdf2v_status launch_nonsink_starts(const int32_t *row_ptr, int32_t num_entities, int32_t *starts_out,
                                   int64_t *count_out, void *workspace, hipStream_t stream);

size_t skipgram_workspace_bytes(int64_t num_walks);
rdf2v_status launch_cbow_examples(const int32_t *tokens, const int32_t *len, int64_t num_walks, int32_t width,
                                  int32_t window, int32_t *centers_out, int32_t *contexts_out, int64_t capacity,
                                  int64_t *count_out, void *workspace, int32_t *status_dev, hipStream_t stream);
rdf2v_status launch_skipgram_pairs(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                                   int32_t width, int32_t window, int32_t *pairs_out, int64_t capacity,
                                   int64_t *count_out, void *workspace, int32_t *status_dev,
                                   hipStream_t stream);

size_t unique_walks_workspace_bytes(int64_t num_walks);
rdf2v_status launch_unique_walks(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                                 int32_t group, int32_t width, int32_t *tokens_out, int32_t *len_out,
                                 int64_t *count_out, void *workspace, int32_t *status_dev,
                                 hipStream_t stream);

size_t bfs_walks_workspace_bytes(int32_t num_entities, int64_t num_roots);
rdf2v_status launch_bfs_walks(const int32_t *row_ptr, const int32_t *edges, int64_t num_edges,
                              int32_t num_entities, int32_t num_predicates, const int32_t *roots,
                              int64_t num_roots, int32_t depth, int32_t max_walks, int32_t *tokens_out,
                              int32_t *len_out, int32_t *counts_out, void *workspace, int32_t *status_dev,
                              hipStream_t stream);

// The three string columns of rdf2v_build_vocabulary, in the order subject,
// predicate, object.
struct VocabColumns {
  const uint8_t *chars[3];
  const int64_t *offsets[3];
  int64_t bytes[3];
};
size_t vocabulary_workspace_bytes(int64_t num_triples, int64_t max_entities, int64_t max_predicates);
rdf2v_status launch_build_vocabulary(const VocabColumns &cols, int64_t num_triples, int64_t max_entities,
                                     int64_t max_predicates, int32_t *subj_ids, int32_t *pred_ids,
                                     int32_t *obj_ids, int64_t *counts_out, void *workspace,
                                     int32_t *status_dev, hipStream_t stream);

}  // namespace rdf2v
