/*
 * Host-side paths of every rdf2v.h entry point, for a library built with
 * AddressSanitizer and UndefinedBehaviorSanitizer on its host code: the
 * workspace-size functions at extreme sizes, and each call with arguments
 * that the host rejects before any HIP call (so no device is needed and the
 * fake device pointers are never dereferenced). Any undefined behaviour in the
 * size arithmetic or the checks ends the run with an error.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "rdf2v.h"

#define EXPECT(cond)                                                  \
  do {                                                                \
    if (!(cond)) {                                                    \
      fprintf(stderr, "failed: %s (line %d)\n", #cond, __LINE__);     \
      exit(1);                                                        \
    }                                                                 \
  } while (0)

static void *fake(uintptr_t addr) { return (void *)addr; }

int main(void) {
  const int64_t big64[] = {0, 1, 4095, 4096, 4097, (int64_t)1 << 30, ((int64_t)1 << 31) - 1, (int64_t)1 << 31,
                           (int64_t)1 << 40, INT64_MAX, -1, INT64_MIN};
  const int32_t big32[] = {0, 1, 2, 255, 256, 1 << 17, (1 << 18) + 1, 1 << 26, INT32_MAX, -1, INT32_MIN};
  const size_t n64 = sizeof(big64) / sizeof(big64[0]), n32 = sizeof(big32) / sizeof(big32[0]);
  size_t sink = 0;
  for (size_t i = 0; i < n64; ++i) {
    for (size_t j = 0; j < n32; ++j) {
      sink += rdf2v_build_csr_workspace_size(big64[i], big32[j]);
      sink += rdf2v_bfs_walks_workspace_size(big32[j], big64[i]);
      sink += (size_t)rdf2v_walk_edges_recommended(big32[j], big64[i]);
      for (size_t k = 0; k < n64; ++k) sink += rdf2v_build_vocabulary_workspace_size(big64[i], big64[k], big64[k]);
    }
    sink += rdf2v_skipgram_pairs_workspace_size(big64[i]);
    sink += rdf2v_cbow_examples_workspace_size(big64[i]);
    sink += rdf2v_unique_walks_workspace_size(big64[i]);
  }
  for (size_t j = 0; j < n32; ++j) sink += rdf2v_nonsink_starts_workspace_size(big32[j]);
  EXPECT(rdf2v_build_csr_workspace_size(INT64_MAX, INT32_MAX) == 0);

  void *F = fake((uintptr_t)1 << 40);
  int32_t *FI = (int32_t *)F;
  rdf2v_csr csr = {10, 3, 20, FI, FI, NULL};
  rdf2v_csr bad = {-1, 3, 20, FI, FI, NULL};

  /* CSR build */
  EXPECT(rdf2v_build_csr(FI, FI, FI, -1, 10, 3, FI, FI, F, 1 << 20, NULL, NULL) == RDF2V_ERR_INVALID_ARGUMENT);
  EXPECT(rdf2v_build_csr(FI, FI, FI, (int64_t)1 << 31, 10, 3, FI, FI, F, 1 << 20, NULL, NULL) == RDF2V_ERR_TOO_LARGE);
  EXPECT(rdf2v_build_csr(FI, FI, FI, 100, INT32_MAX, INT32_MAX, FI, FI, F, 1 << 20, NULL, NULL) == RDF2V_ERR_TOO_LARGE);
  EXPECT(rdf2v_build_csr(FI, FI, FI, 100, 10, 3, FI, FI, NULL, 0, NULL, NULL) == RDF2V_ERR_WORKSPACE);
  EXPECT(rdf2v_build_walk_edges(&bad, FI, NULL, NULL) == RDF2V_ERR_INVALID_ARGUMENT);
  EXPECT(rdf2v_nonsink_starts(&bad, FI, (int64_t *)F, F, 1 << 20, NULL) == RDF2V_ERR_INVALID_ARGUMENT);

  /* walks */
  EXPECT(rdf2v_random_walks(&csr, FI, INT64_MAX, INT32_MAX, 4, 42, 0, 1, FI, FI, NULL, NULL) == RDF2V_ERR_TOO_LARGE);
  EXPECT(rdf2v_random_walks(&csr, FI, 5, 2, 65, 42, 0, 1, FI, FI, NULL, NULL) == RDF2V_ERR_INVALID_ARGUMENT);
  EXPECT(rdf2v_random_walks(&csr, FI, 5, 2, 4, 42, INT64_MAX, INT64_MAX, FI, FI, NULL, NULL) ==
         RDF2V_ERR_INVALID_ARGUMENT);
  EXPECT(rdf2v_random_walks(&csr, FI, (int64_t)1 << 61, 4, 64, 42, 0, (int64_t)1 << 62, FI, FI, NULL, NULL) ==
         RDF2V_ERR_TOO_LARGE);
  EXPECT(rdf2v_random_walks_tokens(&csr, FI, 5, 2, 4, 42, 0, 10, 7, FI, FI, NULL, NULL) == RDF2V_ERR_INVALID_ARGUMENT);

  /* skip-gram pairs, duplicate-free walks, BFS walks */
  EXPECT(rdf2v_skipgram_pairs(FI, FI, INT64_MAX, 129, 5, FI, 1, (int64_t *)F, F, 1 << 20, NULL, NULL) ==
         RDF2V_ERR_TOO_LARGE);
  EXPECT(rdf2v_skipgram_pairs(FI, FI, 10, 0, 5, FI, 1, (int64_t *)F, F, 1 << 20, NULL, NULL) ==
         RDF2V_ERR_INVALID_ARGUMENT);
  EXPECT(rdf2v_skipgram_pairs_noalloc(FI, FI, INT64_MAX, 9, 5, FI, 1, (int64_t *)F, NULL, NULL) ==
         RDF2V_ERR_TOO_LARGE);
  EXPECT(rdf2v_skipgram_pairs_noalloc(FI, FI, RDF2V_NOALLOC_MAX_WALKS + 1, 9, 5, FI, 1, (int64_t *)F, NULL, NULL) ==
         RDF2V_ERR_TOO_LARGE);
  EXPECT(rdf2v_skipgram_pairs_noalloc(FI, FI, 10, 0, 5, FI, 1, (int64_t *)F, NULL, NULL) ==
         RDF2V_ERR_INVALID_ARGUMENT);
  EXPECT(rdf2v_cbow_examples(FI, FI, INT64_MAX, 129, 5, FI, FI, 1, (int64_t *)F, F, 1 << 20, NULL, NULL) ==
         RDF2V_ERR_TOO_LARGE);
  EXPECT(rdf2v_cbow_examples(FI, FI, 10, 9, 5, FI, FI, INT64_MAX, (int64_t *)F, F, 1 << 20, NULL, NULL) ==
         RDF2V_ERR_TOO_LARGE);
  EXPECT(rdf2v_cbow_examples(FI, FI, 10, 9, 0, FI, FI, 1, (int64_t *)F, F, 1 << 20, NULL, NULL) ==
         RDF2V_ERR_INVALID_ARGUMENT);
  EXPECT(rdf2v_unique_walks(FI, FI, INT64_MAX, 3, INT32_MAX, FI, FI, (int64_t *)F, F, 1 << 20, NULL, NULL) ==
         RDF2V_ERR_TOO_LARGE);
  EXPECT(rdf2v_unique_walks(FI, FI, 10, 0, 9, FI, FI, (int64_t *)F, F, 1 << 20, NULL, NULL) ==
         RDF2V_ERR_INVALID_ARGUMENT);
  EXPECT(rdf2v_bfs_walks(&csr, FI, INT64_MAX, 64, INT32_MAX, FI, FI, FI, F, 1 << 20, NULL, NULL) ==
         RDF2V_ERR_TOO_LARGE);
  EXPECT(rdf2v_bfs_walks(&csr, FI, 10, 2, 0, FI, FI, FI, F, 1 << 20, NULL, NULL) == RDF2V_ERR_INVALID_ARGUMENT);

  /* vocabulary */
  const uint8_t *C = (const uint8_t *)F;
  const int64_t *O = (const int64_t *)F;
  int64_t *counts = (int64_t *)F;
  EXPECT(rdf2v_build_vocabulary(C, O, 10, C, O, 10, C, O, 10, INT64_MAX, 10, 10, FI, FI, FI, counts, F, 1 << 20,
                                NULL, NULL) == RDF2V_ERR_TOO_LARGE);
  EXPECT(rdf2v_build_vocabulary(C, O, -1, C, O, 10, C, O, 10, 5, 10, 10, FI, FI, FI, counts, F, 1 << 20, NULL,
                                NULL) == RDF2V_ERR_INVALID_ARGUMENT);
  EXPECT(rdf2v_build_vocabulary(C, O, 10, C, O, 10, C, O, 10, 5, 10, 10, FI, FI, FI, counts, NULL, 0, NULL,
                                NULL) == RDF2V_ERR_WORKSPACE);

  for (int s = -1; s < 7; ++s) EXPECT(rdf2v_status_string(s) != NULL);
  printf("abi sanitize: ok (%zu)\n", sink % 7);
  return 0;
}
