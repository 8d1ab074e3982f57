// extern "C" entry points: host-side argument checks, then the launchers.
// The declarations, argument meanings and error behaviour are in rdf2v.h.

#include <climits>

#include "common.hpp"
#include "launch.hpp"

namespace {

constexpr int64_t kInt32Limit = int64_t(1) << 31;
// Most walk rows one skip-gram call takes: far beyond any device memory, and
// small enough that workspace sizes and pair offsets (fewer than 2^15 pairs
// per row) stay exact in 64 bits.
constexpr int64_t kMaxRows = int64_t(1) << 46;
constexpr int64_t kMaxUniqueRows = (int64_t(1) << 31) * 255;  // block counts fit the compaction's index type

bool id_space_too_large(int32_t num_entities, int32_t num_predicates) {
  return int64_t(num_entities) + int64_t(num_predicates) >= kInt32Limit;
}

}  // namespace

RDF2V_API size_t rdf2v_build_csr_workspace_size(int64_t num_triples, int32_t num_entities) {
  if (num_triples <= 0 || num_triples >= kInt32Limit || num_entities < 0) return 0;
  return rdf2v::plan_csr_build(num_triples, num_entities).bytes;
}

RDF2V_API rdf2v_status rdf2v_build_csr(const int32_t *subj, const int32_t *pred, const int32_t *obj,
                                       int64_t num_triples, int32_t num_entities,
                                       int32_t num_predicates, int32_t *row_ptr_out,
                                       int32_t *edges_out, void *workspace, size_t workspace_bytes,
                                       int32_t *status_dev, void *stream) {
  if (num_triples < 0 || num_entities < 0 || num_predicates < 0) return RDF2V_ERR_INVALID_ARGUMENT;
  if (row_ptr_out == nullptr) return RDF2V_ERR_INVALID_ARGUMENT;
  if (num_triples >= kInt32Limit || id_space_too_large(num_entities, num_predicates))
    return RDF2V_ERR_TOO_LARGE;
  if (num_triples > 0) {
    if (subj == nullptr || pred == nullptr || obj == nullptr || edges_out == nullptr)
      return RDF2V_ERR_INVALID_ARGUMENT;
    if ((reinterpret_cast<uintptr_t>(edges_out) & 7) != 0) return RDF2V_ERR_INVALID_ARGUMENT;
    // Every subject must be < num_entities; with no entities that is impossible.
    if (num_entities == 0 || num_predicates == 0) return RDF2V_ERR_ID_OUT_OF_RANGE;
  }
  const rdf2v::SortPlan plan = rdf2v::plan_csr_build(num_triples, num_entities);
  if (plan.bytes > 0) {
    if (workspace == nullptr || workspace_bytes < plan.bytes) return RDF2V_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return RDF2V_ERR_WORKSPACE;
  }
  return rdf2v::launch_csr_build(subj, pred, obj, num_triples, num_entities, num_predicates,
                                 row_ptr_out, edges_out, workspace, plan, status_dev,
                                 static_cast<hipStream_t>(stream));
}

RDF2V_API rdf2v_status rdf2v_build_walk_edges(const rdf2v_csr *csr, int32_t *walk_edges_out,
                                              int32_t *status_dev, void *stream) {
  if (csr == nullptr || csr->row_ptr == nullptr) return RDF2V_ERR_INVALID_ARGUMENT;
  if (csr->num_entities < 0 || csr->num_predicates < 0 || csr->num_edges < 0)
    return RDF2V_ERR_INVALID_ARGUMENT;
  if (csr->num_edges >= kInt32Limit || id_space_too_large(csr->num_entities, csr->num_predicates))
    return RDF2V_ERR_TOO_LARGE;
  if (csr->num_edges == 0) return RDF2V_OK;
  if (csr->edges == nullptr || walk_edges_out == nullptr) return RDF2V_ERR_INVALID_ARGUMENT;
  // Every object must be < num_entities; with no entities that is impossible.
  if (csr->num_entities == 0) return RDF2V_ERR_ID_OUT_OF_RANGE;
  if ((reinterpret_cast<uintptr_t>(csr->edges) & 7) != 0) return RDF2V_ERR_INVALID_ARGUMENT;
  if ((reinterpret_cast<uintptr_t>(walk_edges_out) & 15) != 0) return RDF2V_ERR_INVALID_ARGUMENT;
  return rdf2v::launch_walk_edges(csr->row_ptr, csr->edges, csr->num_edges, csr->num_entities,
                                  walk_edges_out, status_dev, static_cast<hipStream_t>(stream));
}

RDF2V_API int32_t rdf2v_walk_edges_recommended(int32_t num_entities, int64_t num_edges) {
  constexpr int64_t kRowPtrL2Bytes = int64_t(3) << 19;  // 1.5 MiB of row_ptr
  if (num_entities < 0 || num_edges <= 0) return 0;
  return (int64_t(num_entities) + 1) * 4 > kRowPtrL2Bytes ? 1 : 0;
}

RDF2V_API size_t rdf2v_nonsink_starts_workspace_size(int32_t num_entities) {
  return rdf2v::nonsink_workspace_bytes(num_entities);
}

RDF2V_API rdf2v_status rdf2v_nonsink_starts(const rdf2v_csr *csr, int32_t *starts_out,
                                            int64_t *count_out, void *workspace,
                                            size_t workspace_bytes, void *stream) {
  if (csr == nullptr || count_out == nullptr || csr->row_ptr == nullptr) return RDF2V_ERR_INVALID_ARGUMENT;
  if (csr->num_entities < 0) return RDF2V_ERR_INVALID_ARGUMENT;
  if (csr->num_entities > 0 && starts_out == nullptr) return RDF2V_ERR_INVALID_ARGUMENT;
  const size_t need = rdf2v::nonsink_workspace_bytes(csr->num_entities);
  if (workspace == nullptr || workspace_bytes < need) return RDF2V_ERR_WORKSPACE;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return RDF2V_ERR_WORKSPACE;
  return rdf2v::launch_nonsink_starts(csr->row_ptr, csr->num_entities, starts_out, count_out,
                                      workspace, static_cast<hipStream_t>(stream));
}

RDF2V_API rdf2v_status rdf2v_random_walks(const rdf2v_csr *csr, const int32_t *start_nodes,
                                          int64_t num_start, int32_t walks_per_node, int32_t depth,
                                          uint64_t seed, int64_t walk_begin, int64_t walk_count,
                                          int32_t *tokens_out, int32_t *len_out,
                                          int32_t *status_dev, void *stream) {
  return rdf2v_random_walks_tokens(csr, start_nodes, num_start, walks_per_node, depth, seed, walk_begin,
                                   walk_count, RDF2V_TOKENS_TRIPLES, tokens_out, len_out, status_dev,
                                   stream);
}

RDF2V_API rdf2v_status rdf2v_random_walks_tokens(const rdf2v_csr *csr, const int32_t *start_nodes,
                                                 int64_t num_start, int32_t walks_per_node, int32_t depth,
                                                 uint64_t seed, int64_t walk_begin, int64_t walk_count,
                                                 int32_t token_kind, int32_t *tokens_out, int32_t *len_out,
                                                 int32_t *status_dev, void *stream) {
  if (token_kind != RDF2V_TOKENS_TRIPLES && token_kind != RDF2V_TOKENS_ENTITIES &&
      token_kind != RDF2V_TOKENS_PROPERTIES)
    return RDF2V_ERR_INVALID_ARGUMENT;
  if (csr == nullptr) return RDF2V_ERR_INVALID_ARGUMENT;
  if (csr->num_entities < 0 || csr->num_predicates < 0 || csr->num_edges < 0)
    return RDF2V_ERR_INVALID_ARGUMENT;
  if (num_start < 0 || walks_per_node < 0 || depth < 0 || depth > RDF2V_MAX_DEPTH)
    return RDF2V_ERR_INVALID_ARGUMENT;
  if (walk_begin < 0 || walk_count < 0) return RDF2V_ERR_INVALID_ARGUMENT;
  if (csr->num_edges >= kInt32Limit || id_space_too_large(csr->num_entities, csr->num_predicates))
    return RDF2V_ERR_TOO_LARGE;
  if (walks_per_node > 0 && num_start > INT64_MAX / walks_per_node) return RDF2V_ERR_TOO_LARGE;
  const int64_t num_walks = num_start * int64_t(walks_per_node);
  if (walk_begin > num_walks || walk_count > num_walks - walk_begin) return RDF2V_ERR_INVALID_ARGUMENT;
  if (walk_count == 0) return RDF2V_OK;
  if (start_nodes == nullptr || tokens_out == nullptr || len_out == nullptr || csr->row_ptr == nullptr)
    return RDF2V_ERR_INVALID_ARGUMENT;
  if (csr->walk_edges != nullptr) {
    if ((reinterpret_cast<uintptr_t>(csr->walk_edges) & 15) != 0) return RDF2V_ERR_INVALID_ARGUMENT;
  } else {
    if (csr->num_edges > 0 && csr->edges == nullptr) return RDF2V_ERR_INVALID_ARGUMENT;
    if ((reinterpret_cast<uintptr_t>(csr->edges) & 7) != 0) return RDF2V_ERR_INVALID_ARGUMENT;
  }
  if (walk_count > INT64_MAX / (2 * int64_t(depth) + 1)) return RDF2V_ERR_TOO_LARGE;

  rdf2v::WalkArgs a;
  a.row_ptr = csr->row_ptr;
  a.edges = csr->edges;
  a.walk_edges = csr->walk_edges;
  a.start = start_nodes;
  a.tokens = tokens_out;
  a.lens = len_out;
  a.status = status_dev;
  a.walk_begin = walk_begin;
  a.walk_count = walk_count;
  a.num_edges = csr->num_edges;
  a.num_entities = csr->num_entities;
  a.num_predicates = csr->num_predicates;
  a.walks_per_node = walks_per_node;
  a.depth = depth;
  a.token_kind = token_kind;
  a.key_lo = uint32_t(seed);
  a.key_hi = uint32_t(seed >> 32);
  return rdf2v::launch_random_walks(a, static_cast<hipStream_t>(stream));
}

RDF2V_API size_t rdf2v_skipgram_pairs_workspace_size(int64_t num_walks) {
  if (num_walks < 0 || num_walks > kMaxRows) return 0;
  return rdf2v::skipgram_workspace_bytes(num_walks);
}

RDF2V_API rdf2v_status rdf2v_skipgram_pairs(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                                            int32_t row_width, int32_t window, int32_t *pairs_out,
                                            int64_t pair_capacity, int64_t *pair_count_out,
                                            void *workspace, size_t workspace_bytes,
                                            int32_t *status_dev, void *stream) {
  if (num_walks < 0 || window < 0 || pair_capacity < 0) return RDF2V_ERR_INVALID_ARGUMENT;
  if (row_width < 1 || row_width > 2 * RDF2V_MAX_DEPTH + 1) return RDF2V_ERR_INVALID_ARGUMENT;
  if (pair_count_out == nullptr) return RDF2V_ERR_INVALID_ARGUMENT;
  if (num_walks > 0 && (tokens == nullptr || len == nullptr)) return RDF2V_ERR_INVALID_ARGUMENT;
  if (pair_capacity > 0 && pairs_out == nullptr) return RDF2V_ERR_INVALID_ARGUMENT;
  if ((reinterpret_cast<uintptr_t>(pairs_out) & 7) != 0) return RDF2V_ERR_INVALID_ARGUMENT;
  if (num_walks > kMaxRows) return RDF2V_ERR_TOO_LARGE;
  const size_t need = rdf2v::skipgram_workspace_bytes(num_walks);
  if (workspace == nullptr || workspace_bytes < need) return RDF2V_ERR_WORKSPACE;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return RDF2V_ERR_WORKSPACE;
  return rdf2v::launch_skipgram_pairs(tokens, len, num_walks, row_width, window, pairs_out,
                                      pair_capacity, pair_count_out, workspace, status_dev,
                                      static_cast<hipStream_t>(stream));
}

RDF2V_API size_t rdf2v_cbow_examples_workspace_size(int64_t num_walks) {
  if (num_walks < 0 || num_walks > kMaxRows) return 0;
  return rdf2v::skipgram_workspace_bytes(num_walks);  // the same per-walk offsets and block sums
}

RDF2V_API rdf2v_status rdf2v_cbow_examples(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                                           int32_t row_width, int32_t window, int32_t *centers_out,
                                           int32_t *contexts_out, int64_t capacity, int64_t *count_out,
                                           void *workspace, size_t workspace_bytes, int32_t *status_dev,
                                           void *stream) {
  if (num_walks < 0 || capacity < 0) return RDF2V_ERR_INVALID_ARGUMENT;
  if (window < 1 || window > 2 * RDF2V_MAX_DEPTH) return RDF2V_ERR_INVALID_ARGUMENT;
  if (row_width < 1 || row_width > 2 * RDF2V_MAX_DEPTH + 1) return RDF2V_ERR_INVALID_ARGUMENT;
  if (count_out == nullptr) return RDF2V_ERR_INVALID_ARGUMENT;
  if (num_walks > 0 && (tokens == nullptr || len == nullptr)) return RDF2V_ERR_INVALID_ARGUMENT;
  if (capacity > 0 && (centers_out == nullptr || contexts_out == nullptr)) return RDF2V_ERR_INVALID_ARGUMENT;
  if (((reinterpret_cast<uintptr_t>(centers_out) | reinterpret_cast<uintptr_t>(contexts_out)) & 3) != 0)
    return RDF2V_ERR_INVALID_ARGUMENT;
  if (num_walks > kMaxRows || capacity > kMaxRows * (2 * RDF2V_MAX_DEPTH + 1)) return RDF2V_ERR_TOO_LARGE;
  const size_t need = rdf2v::skipgram_workspace_bytes(num_walks);
  if (workspace == nullptr || workspace_bytes < need) return RDF2V_ERR_WORKSPACE;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return RDF2V_ERR_WORKSPACE;
  return rdf2v::launch_cbow_examples(tokens, len, num_walks, row_width, window, centers_out, contexts_out,
                                     capacity, count_out, workspace, status_dev, static_cast<hipStream_t>(stream));
}

RDF2V_API size_t rdf2v_unique_walks_workspace_size(int64_t num_walks) {
  if (num_walks < 0 || num_walks > kMaxUniqueRows) return 0;
  return rdf2v::unique_walks_workspace_bytes(num_walks);
}

RDF2V_API rdf2v_status rdf2v_unique_walks(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                                          int32_t group_size, int32_t row_width, int32_t *tokens_out,
                                          int32_t *len_out, int64_t *count_out, void *workspace,
                                          size_t workspace_bytes, int32_t *status_dev, void *stream) {
  if (num_walks < 0 || group_size < 1 || row_width < 1) return RDF2V_ERR_INVALID_ARGUMENT;
  if (count_out == nullptr) return RDF2V_ERR_INVALID_ARGUMENT;
  if (num_walks > 0 && (tokens == nullptr || len == nullptr || tokens_out == nullptr || len_out == nullptr))
    return RDF2V_ERR_INVALID_ARGUMENT;
  if (num_walks > kMaxUniqueRows || num_walks > INT64_MAX / row_width) return RDF2V_ERR_TOO_LARGE;
  const size_t need = rdf2v::unique_walks_workspace_bytes(num_walks);
  if (workspace == nullptr || workspace_bytes < need) return RDF2V_ERR_WORKSPACE;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return RDF2V_ERR_WORKSPACE;
  return rdf2v::launch_unique_walks(tokens, len, num_walks, group_size, row_width, tokens_out, len_out,
                                    count_out, workspace, status_dev, static_cast<hipStream_t>(stream));
}

RDF2V_API size_t rdf2v_bfs_walks_workspace_size(int32_t num_entities, int64_t num_roots) {
  // rdf2v_bfs_walks takes fewer than 2^31 roots (its per-level stamps are int32)
  if (num_entities < 0 || num_roots < 0 || num_roots >= kInt32Limit) return 0;
  return rdf2v::bfs_walks_workspace_bytes(num_entities, num_roots);
}

RDF2V_API rdf2v_status rdf2v_bfs_walks(const rdf2v_csr *csr, const int32_t *roots, int64_t num_roots,
                                       int32_t depth, int32_t max_walks, int32_t *tokens_out,
                                       int32_t *len_out, int32_t *counts_out, void *workspace,
                                       size_t workspace_bytes, int32_t *status_dev, void *stream) {
  if (csr == nullptr || csr->row_ptr == nullptr) return RDF2V_ERR_INVALID_ARGUMENT;
  if (csr->num_entities < 0 || csr->num_predicates < 0 || csr->num_edges < 0)
    return RDF2V_ERR_INVALID_ARGUMENT;
  if (num_roots < 0 || depth < 0 || depth > RDF2V_MAX_DEPTH || max_walks < 1) return RDF2V_ERR_INVALID_ARGUMENT;
  if (csr->num_edges >= kInt32Limit || id_space_too_large(csr->num_entities, csr->num_predicates))
    return RDF2V_ERR_TOO_LARGE;
  // the per-level stamps of one workgroup (int32) must not run out
  if (num_roots >= kInt32Limit || (num_roots > 0 && (num_roots + 1) * int64_t(depth + 1) >= kInt32Limit))
    return RDF2V_ERR_TOO_LARGE;
  if (num_roots > INT64_MAX / max_walks / (2 * int64_t(depth) + 1)) return RDF2V_ERR_TOO_LARGE;
  if (num_roots == 0) return RDF2V_OK;
  if (roots == nullptr || tokens_out == nullptr || len_out == nullptr || counts_out == nullptr)
    return RDF2V_ERR_INVALID_ARGUMENT;
  if (csr->num_edges > 0 && csr->edges == nullptr) return RDF2V_ERR_INVALID_ARGUMENT;
  if ((reinterpret_cast<uintptr_t>(csr->edges) & 7) != 0) return RDF2V_ERR_INVALID_ARGUMENT;
  const size_t need = rdf2v::bfs_walks_workspace_bytes(csr->num_entities, num_roots);
  if (workspace == nullptr || workspace_bytes < need) return RDF2V_ERR_WORKSPACE;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return RDF2V_ERR_WORKSPACE;
  return rdf2v::launch_bfs_walks(csr->row_ptr, csr->edges, csr->num_edges, csr->num_entities,
                                 csr->num_predicates, roots, num_roots, depth, max_walks, tokens_out, len_out,
                                 counts_out, workspace, status_dev, static_cast<hipStream_t>(stream));
}

namespace {

bool vocab_sizes_ok(int64_t num_triples, int64_t max_entities, int64_t max_predicates) {
  return num_triples >= 0 && num_triples <= RDF2V_VOCAB_MAX_TRIPLES && max_entities >= 1 &&
         max_entities <= RDF2V_VOCAB_MAX_DISTINCT && max_predicates >= 1 &&
         max_predicates <= RDF2V_VOCAB_MAX_DISTINCT;
}

bool column_ok(const uint8_t *chars, const int64_t *offsets, int64_t bytes, int64_t num_triples) {
  if (bytes < 0) return false;
  if (num_triples > 0 && offsets == nullptr) return false;
  if (bytes > 0 && chars == nullptr) return false;
  return (reinterpret_cast<uintptr_t>(chars) & 3) == 0;
}

}  // namespace

RDF2V_API size_t rdf2v_build_vocabulary_workspace_size(int64_t num_triples, int64_t max_entities,
                                                       int64_t max_predicates) {
  if (!vocab_sizes_ok(num_triples, max_entities, max_predicates)) return 0;
  return rdf2v::vocabulary_workspace_bytes(num_triples, max_entities, max_predicates);
}

RDF2V_API rdf2v_status rdf2v_build_vocabulary(const uint8_t *subj_chars, const int64_t *subj_offsets,
                                              int64_t subj_bytes, const uint8_t *pred_chars,
                                              const int64_t *pred_offsets, int64_t pred_bytes,
                                              const uint8_t *obj_chars, const int64_t *obj_offsets,
                                              int64_t obj_bytes, int64_t num_triples, int64_t max_entities,
                                              int64_t max_predicates, int32_t *subj_ids, int32_t *pred_ids,
                                              int32_t *obj_ids, int64_t *counts_out, void *workspace,
                                              size_t workspace_bytes, int32_t *status_dev, void *stream) {
  if (num_triples > RDF2V_VOCAB_MAX_TRIPLES || max_entities > RDF2V_VOCAB_MAX_DISTINCT ||
      max_predicates > RDF2V_VOCAB_MAX_DISTINCT)
    return RDF2V_ERR_TOO_LARGE;
  if (!vocab_sizes_ok(num_triples, max_entities, max_predicates) || counts_out == nullptr)
    return RDF2V_ERR_INVALID_ARGUMENT;
  if (!column_ok(subj_chars, subj_offsets, subj_bytes, num_triples) ||
      !column_ok(pred_chars, pred_offsets, pred_bytes, num_triples) ||
      !column_ok(obj_chars, obj_offsets, obj_bytes, num_triples))
    return RDF2V_ERR_INVALID_ARGUMENT;
  if (num_triples > 0 && (subj_ids == nullptr || pred_ids == nullptr || obj_ids == nullptr))
    return RDF2V_ERR_INVALID_ARGUMENT;
  const size_t need = rdf2v::vocabulary_workspace_bytes(num_triples, max_entities, max_predicates);
  if (workspace == nullptr || workspace_bytes < need) return RDF2V_ERR_WORKSPACE;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return RDF2V_ERR_WORKSPACE;
  const rdf2v::VocabColumns cols{{subj_chars, pred_chars, obj_chars},
                                 {subj_offsets, pred_offsets, obj_offsets},
                                 {subj_bytes, pred_bytes, obj_bytes}};
  return rdf2v::launch_build_vocabulary(cols, num_triples, max_entities, max_predicates, subj_ids, pred_ids,
                                        obj_ids, counts_out, workspace, status_dev,
                                        static_cast<hipStream_t>(stream));
}

RDF2V_API const char *rdf2v_status_string(int status) {
  switch (status) {
    case RDF2V_OK: return "RDF2V_OK";
    case RDF2V_ERR_INVALID_ARGUMENT: return "RDF2V_ERR_INVALID_ARGUMENT";
    case RDF2V_ERR_ID_OUT_OF_RANGE: return "RDF2V_ERR_ID_OUT_OF_RANGE";
    case RDF2V_ERR_TOO_LARGE: return "RDF2V_ERR_TOO_LARGE";
    case RDF2V_ERR_WORKSPACE: return "RDF2V_ERR_WORKSPACE";
    case RDF2V_ERR_HIP: return "RDF2V_ERR_HIP";
  }
  return "RDF2V_UNKNOWN_STATUS";
}
