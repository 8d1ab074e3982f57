/*
 * A plain C99 client of librdf2v: reads id triples and walk parameters from a
 * binary file, builds the CSR, the start set and the random walks on the GPU
 * through the C ABI of rdf2v.h (device memory from the HIP runtime API), and
 * writes the start set, the token rows and the lengths to a binary file.
 *
 * Input  (little-endian): int64 T, int32 V, int32 P, int32 walks_per_node,
 *        int32 depth, uint64 seed, then int32 subj[T], pred[T], obj[T].
 * Output: int64 num_start, int64 num_walks, int32 starts[num_start],
 *         int32 tokens[num_walks][2*depth+1], int32 len[num_walks].
 * Exit status 0 on success; any library or HIP error is printed and ends the
 * program with status 1.
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "rdf2v.h"

#define HIP_OK(call)                                                            \
  do {                                                                          \
    hipError_t e_ = (call);                                                     \
    if (e_ != hipSuccess) {                                                     \
      fprintf(stderr, "%s:%d: %s\n", __FILE__, __LINE__, hipGetErrorString(e_)); \
      exit(1);                                                                  \
    }                                                                           \
  } while (0)

#define RDF2V_OK_(call)                                                         \
  do {                                                                          \
    rdf2v_status s_ = (call);                                                   \
    if (s_ != RDF2V_OK) {                                                       \
      fprintf(stderr, "%s:%d: %s\n", __FILE__, __LINE__, rdf2v_status_string(s_)); \
      exit(1);                                                                  \
    }                                                                           \
  } while (0)

static void read_all(FILE *f, void *dst, size_t bytes) {
  if (bytes > 0 && fread(dst, 1, bytes, f) != bytes) {
    fprintf(stderr, "short input\n");
    exit(1);
  }
}

static void write_all(FILE *f, const void *src, size_t bytes) {
  if (bytes > 0 && fwrite(src, 1, bytes, f) != bytes) {
    fprintf(stderr, "short output\n");
    exit(1);
  }
}

static void *dev_alloc(size_t bytes) {
  void *p = NULL;
  HIP_OK(hipMalloc(&p, bytes > 0 ? bytes : 1));
  return p;
}

int main(int argc, char **argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: %s input.bin output.bin\n", argv[0]);
    return 2;
  }
  FILE *in = fopen(argv[1], "rb");
  if (in == NULL) return 1;
  int64_t T;
  int32_t V, P, wpn, depth;
  uint64_t seed;
  read_all(in, &T, 8);
  read_all(in, &V, 4);
  read_all(in, &P, 4);
  read_all(in, &wpn, 4);
  read_all(in, &depth, 4);
  read_all(in, &seed, 8);
  if (T < 0 || V < 1 || P < 1 || wpn < 0 || depth < 0 || depth > RDF2V_MAX_DEPTH) return 1;
  const size_t tb = (size_t)T * 4;
  int32_t *host = (int32_t *)malloc(3 * tb + 4);
  if (host == NULL) return 1;
  read_all(in, host, 3 * tb);
  fclose(in);

  int32_t *s = (int32_t *)dev_alloc(tb), *p = (int32_t *)dev_alloc(tb), *o = (int32_t *)dev_alloc(tb);
  HIP_OK(hipMemcpy(s, host, tb, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(p, host + T, tb, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(o, host + 2 * T, tb, hipMemcpyHostToDevice));
  int32_t *status = (int32_t *)dev_alloc(4);
  HIP_OK(hipMemset(status, 0, 4));

  /* triples -> CSR (+ walk records when they pay for this size) */
  int32_t *row_ptr = (int32_t *)dev_alloc((size_t)(V + 1) * 4);
  int32_t *edges = (int32_t *)dev_alloc((size_t)T * 8);
  const size_t ws_bytes = rdf2v_build_csr_workspace_size(T, V);
  void *ws = dev_alloc(ws_bytes);
  RDF2V_OK_(rdf2v_build_csr(s, p, o, T, V, P, row_ptr, edges, ws, ws_bytes, status, NULL));
  rdf2v_csr csr = {V, P, T, row_ptr, edges, NULL};
  int32_t *records = NULL;
  if (rdf2v_walk_edges_recommended(V, T)) {
    records = (int32_t *)dev_alloc((size_t)T * 16);
    RDF2V_OK_(rdf2v_build_walk_edges(&csr, records, status, NULL));
    csr.walk_edges = records;
  }

  /* start set: entities with out-degree >= 1 */
  int32_t *starts = (int32_t *)dev_alloc((size_t)V * 4);
  int64_t *count = (int64_t *)dev_alloc(8);
  const size_t sws_bytes = rdf2v_nonsink_starts_workspace_size(V);
  void *sws = dev_alloc(sws_bytes);
  RDF2V_OK_(rdf2v_nonsink_starts(&csr, starts, count, sws, sws_bytes, NULL));
  int64_t num_start = 0;
  HIP_OK(hipMemcpy(&num_start, count, 8, hipMemcpyDeviceToHost));

  /* every walk of every start entity in one call */
  const int64_t num_walks = num_start * wpn;
  const int64_t width = 2 * (int64_t)depth + 1;
  int32_t *tokens = (int32_t *)dev_alloc((size_t)(num_walks * width) * 4);
  int32_t *lens = (int32_t *)dev_alloc((size_t)num_walks * 4);
  RDF2V_OK_(rdf2v_random_walks(&csr, starts, num_start, wpn, depth, seed, 0, num_walks, tokens, lens, status,
                               NULL));
  HIP_OK(hipDeviceSynchronize());
  int32_t flags = 0;
  HIP_OK(hipMemcpy(&flags, status, 4, hipMemcpyDeviceToHost));
  if (flags != 0) {
    fprintf(stderr, "device status bits 0x%x\n", (unsigned)flags);
    return 1;
  }

  int32_t *h_starts = (int32_t *)malloc((size_t)num_start * 4 + 4);
  int32_t *h_tokens = (int32_t *)malloc((size_t)(num_walks * width) * 4 + 4);
  int32_t *h_lens = (int32_t *)malloc((size_t)num_walks * 4 + 4);
  if (h_starts == NULL || h_tokens == NULL || h_lens == NULL) return 1;
  HIP_OK(hipMemcpy(h_starts, starts, (size_t)num_start * 4, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(h_tokens, tokens, (size_t)(num_walks * width) * 4, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(h_lens, lens, (size_t)num_walks * 4, hipMemcpyDeviceToHost));
  FILE *out = fopen(argv[2], "wb");
  if (out == NULL) return 1;
  write_all(out, &num_start, 8);
  write_all(out, &num_walks, 8);
  write_all(out, h_starts, (size_t)num_start * 4);
  write_all(out, h_tokens, (size_t)(num_walks * width) * 4);
  write_all(out, h_lens, (size_t)num_walks * 4);
  fclose(out);

  void *bufs[] = {s, p, o, status, row_ptr, edges, ws, records, starts, count, sws, tokens, lens};
  for (size_t i = 0; i < sizeof(bufs) / sizeof(bufs[0]); ++i)
    if (bufs[i] != NULL) HIP_OK(hipFree(bufs[i]));
  free(host);
  free(h_starts);
  free(h_tokens);
  free(h_lens);
  return 0;
}
