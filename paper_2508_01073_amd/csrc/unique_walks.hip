// Duplicate-free walks on gfx950 (gpuRDF2vec Tab. 1: "random walk duplicate
// free"): within each group of consecutive rows (the walks of one start
// entity) keep the first occurrence of every distinct walk, in row order.
//
//   1. row_hash_kernel:  a 64-bit hash of (len, valid tokens) per row;
//   2. keep_kernel:      row r is kept unless an earlier row of its group has
//                        the same hash, the same length and the same tokens
//                        (equal hashes are always confirmed token by token, so
//                        collisions cannot drop a walk);
//   3. count / scan / compact: an order-preserving stream compaction of the
//                        kept rows (int64 offsets).
// Integer streaming work; the group scan of step 2 reads hashes that are
// L1/L2-resident because the rows of a group are adjacent.

#include "common.hpp"
#include "launch.hpp"

namespace rdf2v {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = 16;
constexpr int kTile = kThreads * kItems;

// 64-bit FNV-1a over the length and the valid tokens of a row.
__device__ __forceinline__ uint64_t row_hash(const int32_t *row, int32_t L) {
  uint64_t h = 0xcbf29ce484222325ull;
  h = (h ^ uint32_t(L)) * 0x100000001b3ull;
  for (int32_t j = 0; j < L; ++j) h = (h ^ uint32_t(row[j])) * 0x100000001b3ull;
  return h;
}

__device__ __forceinline__ int32_t clamp_len(int32_t L, int32_t width, int &bad) {
  if (L < 0 || L > width) {
    bad = 1;
    return L < 0 ? 0 : width;
  }
  return L;
}

// kStage: the block's kThreads rows (one contiguous span) are first copied to
// LDS with consecutive loads, then each thread hashes its row from LDS.
constexpr int kStageInts = 64 * 256;  // rows of up to 64 tokens

template <bool kStage>
__global__ __launch_bounds__(kThreads) void row_hash_kernel(const int32_t *__restrict__ tokens,
                                                            const int32_t *__restrict__ len, int64_t n,
                                                            int32_t width, uint64_t *__restrict__ hash,
                                                            int32_t *status) {
  __shared__ int32_t tile[kStage ? kStageInts : 1];
  const int64_t r0 = int64_t(blockIdx.x) * kThreads;
  const int64_t r = r0 + threadIdx.x;
  const int rows = int(min(int64_t(kThreads), n - r0));
  if (kStage) {
    const int64_t total = int64_t(rows) * width;
    const int32_t *src = tokens + r0 * width;
    for (int64_t q = threadIdx.x; q < total; q += kThreads) tile[q] = src[q];
    __syncthreads();
  }
  if (r >= n) return;
  int bad = 0;
  const int32_t L = clamp_len(len[r], width, bad);
  hash[r] = row_hash(kStage ? tile + int64_t(threadIdx.x) * width : tokens + r * width, L);
  if (bad && status != nullptr) atomicOr(status, RDF2V_STATUS_BAD_LENGTH);
}

__global__ __launch_bounds__(kThreads) void keep_kernel(const int32_t *__restrict__ tokens,
                                                        const int32_t *__restrict__ len, int64_t n,
                                                        int32_t width, int32_t group,
                                                        const uint64_t *__restrict__ hash,
                                                        int32_t *__restrict__ keep) {
  const int64_t r = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (r >= n) return;
  const int64_t g0 = r / group * group;
  const uint64_t h = hash[r];
  int bad = 0;
  const int32_t L = clamp_len(len[r], width, bad);
  const int32_t *row = tokens + r * width;
  bool dup = false;
  for (int64_t q = g0; q < r && !dup; ++q) {
    if (hash[q] != h) continue;
    int b2 = 0;
    if (clamp_len(len[q], width, b2) != L) continue;
    const int32_t *other = tokens + q * width;
    bool same = true;
    for (int32_t j = 0; j < L && same; ++j) same = other[j] == row[j];
    dup = same;
  }
  keep[r] = dup ? 0 : 1;
}

__global__ __launch_bounds__(kThreads) void keep_count_kernel(const int32_t *__restrict__ keep, int64_t n,
                                                              int64_t *__restrict__ partials) {
  __shared__ int64_t scratch[kThreads / kWave];
  const int64_t base = int64_t(blockIdx.x) * kTile;
  int64_t s = 0;
#pragma unroll 4
  for (int i = 0; i < kItems; ++i) {
    const int64_t r = base + int64_t(i) * kThreads + threadIdx.x;
    if (r < n) s += keep[r];
  }
  const int64_t total = block_sum<kThreads, int64_t>(s, scratch);
  if (threadIdx.x == 0) partials[blockIdx.x] = total;
}

__global__ __launch_bounds__(kThreads) void keep_partials_kernel(int64_t *partials, int64_t nb,
                                                                 int64_t *total_out) {
  __shared__ int64_t scratch[kThreads / kWave];
  int64_t carry = 0;
  for (int64_t base = 0; base < nb; base += kThreads) {
    const int64_t idx = base + threadIdx.x;
    const int64_t x = idx < nb ? partials[idx] : 0;
    int64_t tot;
    const int64_t ex = block_exclusive_scan<kThreads, int64_t>(x, scratch, tot);
    if (idx < nb) partials[idx] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) {
    partials[nb] = carry;
    *total_out = carry;
  }
}

// Each round of kThreads rows: a block scan of the keep flags gives every kept
// row its output slot; the kept rows of the round form one contiguous output
// span, which the block writes with consecutive stores, reading the tokens
// back from the (cache-resident) rows of the round.
__global__ __launch_bounds__(kThreads) void compact_kernel(const int32_t *__restrict__ tokens,
                                                           const int32_t *__restrict__ len, int64_t n,
                                                           int32_t width, const int32_t *__restrict__ keep,
                                                           const int64_t *__restrict__ partials,
                                                           int32_t *__restrict__ tokens_out,
                                                           int32_t *__restrict__ len_out) {
  __shared__ int64_t scratch[kThreads / kWave];
  __shared__ int32_t kept_rows[kThreads];
  const int64_t base = int64_t(blockIdx.x) * kTile;
  int64_t carry = partials[blockIdx.x];
  for (int i = 0; i < kItems; ++i) {
    const int64_t round0 = base + int64_t(i) * kThreads;
    if (round0 >= n) break;  // uniform across the block
    const int64_t r = round0 + threadIdx.x;
    const int64_t k = r < n ? keep[r] : 0;
    int64_t tot;
    const int64_t ex = block_exclusive_scan<kThreads, int64_t>(k, scratch, tot);
    if (k) {
      kept_rows[ex] = threadIdx.x;
      len_out[carry + ex] = len[r];
    }
    __syncthreads();
    const int32_t span = int32_t(tot) * width;  // at most kThreads rows of <= 129 tokens
    int32_t *dst = tokens_out + carry * width;
    const int32_t *src = tokens + round0 * width;
    for (int32_t q = threadIdx.x; q < span; q += kThreads) {
      const int32_t kr = q / width;
      const int32_t col = q - kr * width;
      dst[q] = src[kept_rows[kr] * width + col];
    }
    __syncthreads();  // kept_rows is rewritten by the next round
    carry += tot;
  }
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

size_t unique_walks_workspace_bytes(int64_t num_walks) {
  const int64_t nb = ceil_div(num_walks, kTile);
  return align_up(size_t(num_walks) * 8, 256) + align_up(size_t(num_walks) * 4, 256) +
         align_up(size_t(nb + 1) * 8, 256);
}

rdf2v_status launch_unique_walks(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                                 int32_t group, int32_t width, int32_t *tokens_out, int32_t *len_out,
                                 int64_t *count_out, void *workspace, int32_t *status_dev,
                                 hipStream_t stream) {
  char *ws = static_cast<char *>(workspace);
  uint64_t *hash = reinterpret_cast<uint64_t *>(ws);
  int32_t *keep = reinterpret_cast<int32_t *>(ws + align_up(size_t(num_walks) * 8, 256));
  int64_t *partials = reinterpret_cast<int64_t *>(ws + align_up(size_t(num_walks) * 8, 256) +
                                                  align_up(size_t(num_walks) * 4, 256));
  const int64_t nb = ceil_div(num_walks, kTile);
  if (num_walks > 0) {
    const unsigned rows_blocks = unsigned(ceil_div(num_walks, kThreads));
    if (int64_t(width) * kThreads <= kStageInts)
      row_hash_kernel<true><<<dim3(rows_blocks), dim3(kThreads), 0, stream>>>(tokens, len, num_walks, width,
                                                                             hash, status_dev);
    else
      row_hash_kernel<false><<<dim3(rows_blocks), dim3(kThreads), 0, stream>>>(tokens, len, num_walks, width,
                                                                              hash, status_dev);
    RDF2V_LAUNCH_CHECK();
    keep_kernel<<<dim3(rows_blocks), dim3(kThreads), 0, stream>>>(tokens, len, num_walks, width, group, hash,
                                                                 keep);
    RDF2V_LAUNCH_CHECK();
    keep_count_kernel<<<dim3(unsigned(nb)), dim3(kThreads), 0, stream>>>(keep, num_walks, partials);
    RDF2V_LAUNCH_CHECK();
  }
  keep_partials_kernel<<<dim3(1), dim3(kThreads), 0, stream>>>(partials, nb, count_out);
  RDF2V_LAUNCH_CHECK();
  if (num_walks > 0) {
    compact_kernel<<<dim3(unsigned(nb)), dim3(kThreads), 0, stream>>>(tokens, len, num_walks, width, keep,
                                                                     partials, tokens_out, len_out);
    RDF2V_LAUNCH_CHECK();
  }
  return RDF2V_OK;
}

}  // namespace rdf2v
