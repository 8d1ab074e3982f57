// Duplicate-free walks on gfx950 (gpuRDF2vec Tab. 1: "random walk duplicate
// free"): within each group of consecutive rows (the walks of one start
// entity) keep the first occurrence of every distinct walk, in row order.
//
// Main path (groups of at most 1024 rows whose block of rows fits the LDS
// stage): a block owns whole groups.
//   1. group_keep_kernel: the block copies its rows to LDS (batched coalesced
//      loads), hashes every row there (64-bit FNV-1a over length and valid
//      tokens), and keeps a row unless an earlier row of its group has the same
//      hash, length and tokens (equal hashes are always confirmed token by
//      token, so collisions cannot drop a walk). Keep flags go to global
//      memory, the block's kept count to a partial sum.
//   2. an exclusive scan of the block counts (tiles scanned in parallel, then
//      the tile totals, then each tile's prefix added).
//   3. group_compact_kernel: the block stages its rows again, scans its keep
//      flags and writes its kept rows as one contiguous range.
// Other shapes use the general path: a hash per row, a group scan over the
// hashes in global memory, and the same scan and order-preserving compaction
// over tiles of rows. Integer streaming work.

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

// Exclusive scan of the nb block counts, in place, in three launches:
// tile_scan_kernel scans each tile of kTile counts and writes the tile's total
// to tile_sums; keep_partials_kernel (one block) scans the tile totals; and
// tile_add_kernel adds each tile's prefix to its counts.
__global__ __launch_bounds__(kThreads) void tile_scan_kernel(int64_t *partials, int64_t nb,
                                                             int64_t *tile_sums) {
  __shared__ int64_t scratch[kThreads / kWave];
  const int64_t first = int64_t(blockIdx.x) * kTile + int64_t(threadIdx.x) * kItems;
  int64_t v[kItems];
  int64_t s = 0;
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    v[i] = first + i < nb ? partials[first + i] : 0;
    s += v[i];
  }
  int64_t tot;
  int64_t ex = block_exclusive_scan<kThreads, int64_t>(s, scratch, tot);
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    if (first + i < nb) partials[first + i] = ex;
    ex += v[i];
  }
  if (threadIdx.x == 0) tile_sums[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kThreads) void tile_add_kernel(int64_t *partials, int64_t nb,
                                                            const int64_t *tile_sums) {
  const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (i < nb) partials[i] += tile_sums[i / kTile];
}

// One block: exclusive scan of the nb counts in place, kItems consecutive
// counts per thread per round; the total goes to partials[nb] and *total_out.
__global__ __launch_bounds__(kThreads) void keep_partials_kernel(int64_t *partials, int64_t nb,
                                                                 int64_t *total_out) {
  __shared__ int64_t scratch[kThreads / kWave];
  int64_t carry = 0;
  for (int64_t base = 0; base < nb; base += kTile) {
    const int64_t first = base + int64_t(threadIdx.x) * kItems;
    int64_t v[kItems];
    int64_t s = 0;
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
      v[i] = first + i < nb ? partials[first + i] : 0;
      s += v[i];
    }
    int64_t tot;
    int64_t ex = carry + block_exclusive_scan<kThreads, int64_t>(s, scratch, tot);
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
      if (first + i < nb) partials[first + i] = ex;
      ex += v[i];
    }
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

// Exclusive scan of nb counts in place, total to *total_out; tile_sums holds
// ceil(nb / kTile) + 1 entries, counts nb + 1.
rdf2v_status scan_counts(int64_t *counts, int64_t nb, int64_t *tile_sums, int64_t *total_out,
                         hipStream_t stream) {
  const int64_t tiles = ceil_div(nb, kTile);
  if (tiles > 1) {
    tile_scan_kernel<<<dim3(unsigned(tiles)), dim3(kThreads), 0, stream>>>(counts, nb, tile_sums);
    RDF2V_LAUNCH_CHECK();
    keep_partials_kernel<<<dim3(1), dim3(kThreads), 0, stream>>>(tile_sums, tiles, total_out);
    RDF2V_LAUNCH_CHECK();
    tile_add_kernel<<<dim3(unsigned(ceil_div(nb, kThreads))), dim3(kThreads), 0, stream>>>(counts, nb, tile_sums);
  } else {
    keep_partials_kernel<<<dim3(1), dim3(kThreads), 0, stream>>>(counts, nb, total_out);
  }
  RDF2V_LAUNCH_CHECK();
  return RDF2V_OK;
}

// ---------------------------------------------------------------------------
// Main path: blocks of whole groups.
// ---------------------------------------------------------------------------

constexpr int kGroupStageInts = 12288;  // at most 48 KiB of rows per block (dynamic LDS, sized per launch)
constexpr int kBatch = 8;               // loads in flight per thread while staging

// Copies `count` ints from global memory to LDS, kBatch independent loads per
// thread at a time (NT threads).
template <int NT>
__device__ __forceinline__ void stage_ints(int32_t *__restrict__ dst, const int32_t *__restrict__ src,
                                           int32_t count) {
  for (int32_t base = 0; base < count; base += kBatch * NT) {
    int32_t v[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int32_t q = base + k * NT + int32_t(threadIdx.x);
      v[k] = q < count ? src[q] : 0;
    }
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int32_t q = base + k * NT + int32_t(threadIdx.x);
      if (q < count) dst[q] = v[k];
    }
  }
}

// Rows [b * rows_per_block, ...) of block b, rows_per_block = (NT / group) * group.
template <int NT>
__global__ __launch_bounds__(NT) void group_keep_kernel(const int32_t *__restrict__ tokens,
                                                              const int32_t *__restrict__ len, int64_t n,
                                                              int32_t width, int32_t group, int32_t rows_per_block,
                                                              uint8_t *__restrict__ keep,
                                                              int64_t *__restrict__ partials, int32_t *status) {
  constexpr int kSlots = 2 * NT;      // open-addressing table of (group, hash) keys
  constexpr uint64_t kNoKey = ~uint64_t(0);
  extern __shared__ int32_t tile[];  // rows_per_block * width ints
  __shared__ uint64_t hashes[NT];
  __shared__ int32_t lens[NT];
  __shared__ int64_t scratch[NT / kWave];
  __shared__ uint64_t tab_key[kSlots];
  __shared__ int32_t tab_first[kSlots];  // smallest row of the block with the slot's key
  const int t = threadIdx.x;
  for (int i = t; i < kSlots; i += NT) {
    tab_key[i] = kNoKey;
    tab_first[i] = INT32_MAX;
  }
  const int64_t r0 = int64_t(blockIdx.x) * rows_per_block;
  const int32_t rows = int32_t(min(int64_t(rows_per_block), n - r0));
  // The row's length is read before the barrier, alongside the rows.
  const int32_t raw_len = t < rows ? len[r0 + t] : 0;
  stage_ints<NT>(tile, tokens + r0 * width, rows * width);
  __syncthreads();
  int bad = 0;
  int32_t L = 0, slot = 0;
  if (t < rows) {
    L = clamp_len(raw_len, width, bad);
    const uint64_t h = row_hash(tile + t * width, L);
    hashes[t] = h;
    lens[t] = L;
    // Key: the hash with the row's group mixed in (two groups' keys may still
    // meet: rows are always compared before one is dropped).
    uint64_t key = h ^ (uint64_t(t / group + 1) * 0x9e3779b97f4a7c15ull);
    if (key == kNoKey) key = kNoKey - 1;
    slot = int32_t((key ^ (key >> 29)) & uint64_t(kSlots - 1));
    for (int n_probe = 0; n_probe < kSlots; ++n_probe) {  // the table has more slots than rows
      const uint64_t cur = atomicCAS(reinterpret_cast<unsigned long long *>(tab_key + slot),
                                     static_cast<unsigned long long>(kNoKey), static_cast<unsigned long long>(key));
      if (cur == kNoKey || cur == key) break;
      slot = (slot + 1) & (kSlots - 1);
    }
    atomicMin(tab_first + slot, t);
  }
  __syncthreads();
  int32_t k = 0;
  if (t < rows) {
    const uint64_t h = hashes[t];
    const int32_t *row = tile + t * width;
    auto same_row = [&](int32_t q) {
      if (hashes[q] != h || lens[q] != L) return false;
      const int32_t *other = tile + q * width;
      for (int32_t j = 0; j < L; ++j)
        if (other[j] != row[j]) return false;
      return true;
    };
    // The first row with this key is usually the first occurrence of this
    // walk; when it is not (a key collision), scan the group's earlier rows.
    const int32_t first = tab_first[slot];
    bool dup = false;
    if (first != t) {
      dup = first / group == t / group && same_row(first);
      for (int32_t q = t / group * group; q < t && !dup; ++q) dup = same_row(q);
    }
    k = dup ? 0 : 1;
    keep[r0 + t] = uint8_t(k);
  }
  const int64_t total = block_sum<NT, int64_t>(k, scratch);
  if (t == 0) partials[blockIdx.x] = total;
  if (bad && status != nullptr) atomicOr(status, RDF2V_STATUS_BAD_LENGTH);
}

template <int NT>
__global__ __launch_bounds__(NT) void group_compact_kernel(const int32_t *__restrict__ tokens,
                                                                 const int32_t *__restrict__ len, int64_t n,
                                                                 int32_t width, int32_t rows_per_block,
                                                                 const uint8_t *__restrict__ keep,
                                                                 const int64_t *__restrict__ partials,
                                                                 int32_t *__restrict__ tokens_out,
                                                                 int32_t *__restrict__ len_out) {
  extern __shared__ int32_t tile[];  // rows_per_block * width ints
  __shared__ int32_t kept_rows[NT];
  __shared__ int64_t scratch[NT / kWave];
  const int64_t r0 = int64_t(blockIdx.x) * rows_per_block;
  const int32_t rows = int32_t(min(int64_t(rows_per_block), n - r0));
  const int t = threadIdx.x;
  // Every global read is issued before the scan's barriers: the keep flag, the
  // row's length, the block's output offset, and the rows themselves.
  const int64_t k = t < rows ? keep[r0 + t] : 0;
  const int32_t row_len = t < rows ? len[r0 + t] : 0;
  const int64_t out0 = partials[blockIdx.x];
  stage_ints<NT>(tile, tokens + r0 * width, rows * width);
  int64_t tot;
  const int64_t ex = block_exclusive_scan<NT, int64_t>(k, scratch, tot);  // also orders the stage
  if (k) {
    kept_rows[ex] = t;
    len_out[out0 + ex] = row_len;
  }
  __syncthreads();
  // The block's kept rows form one contiguous output range.
  const int32_t span = int32_t(tot) * width;
  int32_t *dst = tokens_out + out0 * width;
  for (int32_t q = t; q < span; q += NT) {
    const int32_t kr = q / width;
    dst[q] = tile[kept_rows[kr] * width + (q - kr * width)];
  }
}

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
  // Main path: blocks of whole groups (256 threads, or 1024 for groups of up
  // to 1024 rows), when the block's rows fit the LDS stage. Workspace: the
  // block partials where the general path keeps its hashes (8 B per row >=
  // 8 B per block + 1), the keep flags after them.
  int64_t *block_counts = reinterpret_cast<int64_t *>(ws);
  uint8_t *keep_flags = reinterpret_cast<uint8_t *>(ws + align_up(size_t(num_walks) * 8, 256));
  // the scan's tile sums where the general path keeps its partials
  int64_t *tile_sums = reinterpret_cast<int64_t *>(ws + align_up(size_t(num_walks) * 8, 256) +
                                                   align_up(size_t(num_walks) * 4, 256));
  auto main_path = [&](auto keep_kernel, auto compact_kernel, int nt) -> rdf2v_status {
    const int32_t rows_per_block = (nt / group) * group;
    const size_t tile_bytes = size_t(rows_per_block) * width * sizeof(int32_t);
    const int64_t nb = ceil_div(num_walks, rows_per_block);
    if (nb >= (int64_t(1) << 31)) return RDF2V_ERR_TOO_LARGE;
    if (nb > 0) {
      keep_kernel<<<dim3(unsigned(nb)), dim3(nt), tile_bytes, stream>>>(tokens, len, num_walks, width, group,
                                                                        rows_per_block, keep_flags, block_counts,
                                                                        status_dev);
      RDF2V_LAUNCH_CHECK();
    }
    const rdf2v_status st = scan_counts(block_counts, nb, tile_sums, count_out, stream);
    if (st != RDF2V_OK) return st;
    if (nb > 0) {
      compact_kernel<<<dim3(unsigned(nb)), dim3(nt), tile_bytes, stream>>>(tokens, len, num_walks, width,
                                                                           rows_per_block, keep_flags, block_counts,
                                                                           tokens_out, len_out);
      RDF2V_LAUNCH_CHECK();
    }
    return RDF2V_OK;
  };
  auto fits = [&](int nt) { return group <= nt && int64_t(nt / group) * group * width <= kGroupStageInts; };
  if (fits(kThreads)) return main_path(group_keep_kernel<kThreads>, group_compact_kernel<kThreads>, kThreads);
  if (fits(1024)) return main_path(group_keep_kernel<1024>, group_compact_kernel<1024>, 1024);
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
  // the hashes are no longer needed: their space holds the tile sums of the scan
  const rdf2v_status st = scan_counts(partials, nb, reinterpret_cast<int64_t *>(ws), count_out, stream);
  if (st != RDF2V_OK) return st;
  if (num_walks > 0) {
    compact_kernel<<<dim3(unsigned(nb)), dim3(kThreads), 0, stream>>>(tokens, len, num_walks, width, keep,
                                                                     partials, tokens_out, len_out);
    RDF2V_LAUNCH_CHECK();
  }
  return RDF2V_OK;
}

}  // namespace rdf2v
