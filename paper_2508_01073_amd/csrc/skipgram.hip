// Skip-gram training pairs and CBOW training examples from walk rows on gfx950.
//
// gpuRDF2vec turns the walk corpus into center-context pairs for SkipGram
// (Sec. 3.2) after dropping the -1 padding (Sec. 3.1). For walk r with
// L = len[r] valid tokens t_0 .. t_{L-1}, every center i and every context j
// with 1 <= |i - j| <= window, 0 <= j < L, give the pair (t_i, t_j), ordered
// by walk, then i, then j.
//
// The number of pairs of a walk is a closed form of L and the window, so the
// output offsets of all walks are one exclusive scan (int64: a corpus easily
// exceeds 2^31 pairs) and the emit kernel needs no atomics: one thread per
// (walk, center) computes where its pairs start, again in closed form, and
// places them. Pure integer streaming work, bound by HBM writes.
//
// CBOW (Sec. 3.2: the library trains Continuous Bag of Words next to
// Skip-Gram; it predicts a center token from the tokens around it) takes one
// example per valid token: the center t_i and its contexts, the t_j with
// 1 <= |i - j| <= window in ascending j, padded with -1 to 2 * window entries.
// Examples are ordered by walk, then i; a walk of L tokens gives L of them, so
// the offsets are a scan of the lengths and the same kernels serve both.

#include <algorithm>

#include "common.hpp"
#include "launch.hpp"

namespace rdf2v {
namespace {

typedef int32_t v2i32 __attribute__((ext_vector_type(2)));
typedef int32_t v4i32 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kItems = 16;
constexpr int kTile = kThreads * kItems;  // walks per scan block

// Pairs of a walk with L valid tokens: 2 * sum_{d=1}^{m} (L - d), m = min(window, L - 1).
__device__ __forceinline__ int64_t walk_pairs(int64_t L, int64_t window) {
  const int64_t m = min(window, L - 1);
  return m <= 0 ? 0 : 2 * (m * L - m * (m + 1) / 2);
}

// sum_{k=0}^{n-1} min(k, window)
__device__ __forceinline__ int64_t capped_prefix(int64_t n, int64_t window) {
  if (n <= 0) return 0;
  if (n <= window + 1) return n * (n - 1) / 2;
  return window * (window + 1) / 2 + (n - 1 - window) * window;
}

// Training items of one walk of L valid tokens: pairs, or CBOW examples.
template <bool kCbow>
__device__ __forceinline__ int64_t walk_items(int64_t L, int64_t window) {
  return kCbow ? L : walk_pairs(L, window);
}

// Valid length of walk r, clamped to the row; out-of-range lengths raise a flag.
__device__ __forceinline__ int32_t clamped_len(const int32_t *len, int64_t r, int32_t width, int &bad) {
  const int32_t L = len[r];
  if (L < 0 || L > width) {
    bad = 1;
    return L < 0 ? 0 : width;
  }
  return L;
}

template <bool kCbow>
__global__ __launch_bounds__(kThreads) void pair_count_reduce_kernel(const int32_t *__restrict__ len,
                                                                     int64_t n, int32_t width,
                                                                     int32_t window,
                                                                     int64_t *__restrict__ partials,
                                                                     int32_t *status) {
  __shared__ int64_t scratch[kThreads / kWave];
  const int64_t base = int64_t(blockIdx.x) * kTile;
  int64_t s = 0;
  int bad = 0;
#pragma unroll 4
  for (int i = 0; i < kItems; ++i) {
    const int64_t r = base + int64_t(i) * kThreads + threadIdx.x;
    if (r < n) s += walk_items<kCbow>(clamped_len(len, r, width, bad), window);
  }
  const int64_t total = block_sum<kThreads, int64_t>(s, scratch);
  if (threadIdx.x == 0) partials[blockIdx.x] = total;
  if (bad && status != nullptr) atomicOr(status, RDF2V_STATUS_BAD_LENGTH);
}

// One block: exclusive scan of the block sums in place; the total goes to *total_out.
__global__ __launch_bounds__(kThreads) void pair_partials_kernel(int64_t *partials, int64_t nb,
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

template <bool kCbow>
__global__ __launch_bounds__(kThreads) void pair_offsets_kernel(const int32_t *__restrict__ len, int64_t n,
                                                                int32_t width, int32_t window,
                                                                const int64_t *__restrict__ partials,
                                                                int64_t *__restrict__ offsets) {
  __shared__ int64_t scratch[kThreads / kWave];
  const int64_t base = int64_t(blockIdx.x) * kTile;
  int64_t carry = partials[blockIdx.x];
  int bad = 0;
  for (int i = 0; i < kItems; ++i) {
    const int64_t r = base + int64_t(i) * kThreads + threadIdx.x;
    const int64_t x = r < n ? walk_items<kCbow>(clamped_len(len, r, width, bad), window) : 0;
    int64_t tot;
    const int64_t ex = block_exclusive_scan<kThreads, int64_t>(x, scratch, tot);
    if (r < n) offsets[r] = carry + ex;
    carry += tot;
  }
}

// One thread per (walk, center); walks_per_block = kBlock / width walks per
// block, whose rows are contiguous in the input and whose pairs form one
// contiguous output range. With kStage, the block first copies its rows to LDS
// with one coalesced load, the threads place their pairs in an LDS stage sized
// at launch to the block's most pairs (dynamic LDS), and the block streams the
// range out with consecutive, non-temporal 16-byte stores; otherwise each
// thread reads its row from global memory and writes its pairs directly.

template <bool kStage, int kBlock>
__global__ __launch_bounds__(kBlock) void pair_emit_kernel(const int32_t *__restrict__ tokens,
                                                             const int32_t *__restrict__ len, int64_t n,
                                                             int32_t width, int32_t window,
                                                             const int64_t *__restrict__ offsets,
                                                             int2 *__restrict__ pairs, int64_t capacity,
                                                             int32_t *status) {
  extern __shared__ int2 stage[];                // kStage: the block's pairs
  __shared__ int32_t rows[kStage ? kBlock : 1];  // the block's walk rows, walks_per_block * width tokens
  const int walks_per_block = kBlock / width;
  const int t = threadIdx.x;
  const int64_t r0 = int64_t(blockIdx.x) * walks_per_block;
  const int64_t r_end = min(n, r0 + walks_per_block);
  const int64_t r = r0 + t / width;
  const int64_t i = t % width;
  const bool active = t < walks_per_block * width && r < n;
  int bad = 0;
  const int64_t w = window;
  const int64_t block_first = offsets[r0];
  int64_t first = 0, L = 0;
  if (active) {
    L = clamped_len(len, r, width, bad);
    first = offsets[r] + capped_prefix(i, w) + capped_prefix(L, w) - capped_prefix(L - i, w);
  }
  // The block's pairs end where the next block's begin: the offset of walk
  // r_end, or the pair count of the last walk added to its offset.
  __shared__ int64_t block_end;
  if (kStage) {
    const int64_t span = (r_end - r0) * width;  // <= kBlock
    if (t < span) rows[t] = tokens[r0 * width + t];
    if (t == 0) {
      if (r_end < n) {
        block_end = offsets[r_end];
      } else {
        int b2 = 0;
        block_end = offsets[n - 1] + walk_pairs(clamped_len(len, n - 1, width, b2), w);
      }
    }
    __syncthreads();
  }
  bool full = false;
  if (active && i < L) {
    const int32_t *row = kStage ? rows + (t / width) * width : tokens + r * width;
    const int32_t center = row[i];
    const int64_t j0 = max(int64_t(0), i - w), j1 = min(L - 1, i + w);
    int64_t k = first;
    for (int64_t j = j0; j <= j1; ++j) {
      if (j == i) continue;
      const int2 pr = make_int2(center, row[j]);
      if (kStage) {
        stage[k - block_first] = pr;
      } else if (k < capacity) {
        __builtin_nontemporal_store(v2i32{pr.x, pr.y}, reinterpret_cast<v2i32 *>(pairs + k));
      } else {
        full = true;
      }
      ++k;
    }
  }
  if (kStage) {
    __syncthreads();
    const int64_t cnt = block_end - block_first;
    if (block_end > capacity) full = true;
    const int64_t lim = min(cnt, capacity - block_first);  // pairs of this block that fit
    // One leading pair if the range does not start 16-byte aligned, then two
    // pairs per 16-byte store, then a possible trailing pair.
    const int64_t head = (reinterpret_cast<uintptr_t>(pairs + block_first) & 15) ? 1 : 0;
    if (t == 0 && head && lim > 0)
      __builtin_nontemporal_store(v2i32{stage[0].x, stage[0].y}, reinterpret_cast<v2i32 *>(pairs + block_first));
    const int64_t body = lim > head ? (lim - head) >> 1 : 0;
    v4i32 *dst = reinterpret_cast<v4i32 *>(pairs + block_first + head);
    for (int64_t q = t; q < body; q += kBlock) {
      const int2 a = stage[head + 2 * q], b = stage[head + 2 * q + 1];
      __builtin_nontemporal_store(v4i32{a.x, a.y, b.x, b.y}, dst + q);
    }
    const int64_t tail = head + 2 * body;
    if (t == 0 && tail < lim)
      __builtin_nontemporal_store(v2i32{stage[tail].x, stage[tail].y},
                                  reinterpret_cast<v2i32 *>(pairs + block_first + tail));
  }
  if ((full || bad) && status != nullptr)
    atomicOr(status, (full ? RDF2V_STATUS_CAPACITY : 0) | (bad ? RDF2V_STATUS_BAD_LENGTH : 0));
}

// Streams `total` int32 from LDS to dst (4-byte aligned) with the whole block:
// a scalar head up to 16-byte alignment, 16-byte non-temporal stores, a scalar
// tail.
template <int kBlock>
__device__ __forceinline__ void stream_run(const int32_t *src, int32_t *dst, int64_t total) {
  const int t = threadIdx.x;
  const int64_t head = min(total, int64_t((16 - (reinterpret_cast<uintptr_t>(dst) & 15)) & 15) / 4);
  if (t < head) __builtin_nontemporal_store(src[t], dst + t);
  const int64_t body = (total - head) >> 2;
  v4i32 *dst4 = reinterpret_cast<v4i32 *>(dst + head);
  for (int64_t q = t; q < body; q += kBlock) {
    const int32_t *s4 = src + head + 4 * q;
    __builtin_nontemporal_store(v4i32{s4[0], s4[1], s4[2], s4[3]}, dst4 + q);
  }
  for (int64_t q = head + 4 * body + t; q < total; q += kBlock) __builtin_nontemporal_store(src[q], dst + q);
}

// CBOW, staged: one thread per (walk, position); walks_per_block = kBlock / width
// walks per block, whose examples form one contiguous output range. The block
// copies its rows to LDS, places its centers and context rows in LDS stages
// (at most kBlock examples, 2 * window ints per context row) and streams each
// out as one contiguous run of 16-byte non-temporal stores.
template <int kBlock>
__global__ __launch_bounds__(kBlock) void cbow_emit_kernel(const int32_t *__restrict__ tokens,
                                                            const int32_t *__restrict__ len, int64_t n,
                                                            int32_t width, int32_t window,
                                                            const int64_t *__restrict__ offsets,
                                                            int32_t *__restrict__ centers,
                                                            int32_t *__restrict__ contexts, int64_t capacity,
                                                            int32_t *status) {
  extern __shared__ int32_t ctx_stage[];  // the block's context rows
  __shared__ int32_t rows[kBlock];        // the block's walk rows
  __shared__ int32_t ctr_stage[kBlock];   // the block's centers
  const int walks_per_block = kBlock / width;
  const int t = threadIdx.x;
  const int64_t r0 = int64_t(blockIdx.x) * walks_per_block;
  const int64_t r_end = min(n, r0 + walks_per_block);
  const int64_t r = r0 + t / width;
  const int64_t i = t % width;
  const bool active = t < walks_per_block * width && r < n;
  const int64_t cw = 2 * int64_t(window);  // context entries per example
  int bad = 0;
  const int64_t block_first = offsets[r0];
  // Every global read the block needs is issued before the first barrier, so
  // none of them waits behind it: the walk's length and first example, the
  // rows, and (thread 0) where the next block's examples begin.
  int64_t L = 0, walk_first = 0;
  if (active) {
    L = clamped_len(len, r, width, bad);
    walk_first = offsets[r];
  }
  __shared__ int64_t block_end;
  const int64_t span = (r_end - r0) * width;  // <= kBlock
  if (t < span) rows[t] = tokens[r0 * width + t];
  if (t == 0) {
    if (r_end < n) {
      block_end = offsets[r_end];
    } else {
      int b2 = 0;
      block_end = offsets[n - 1] + clamped_len(len, n - 1, width, b2);
    }
  }
  __syncthreads();
  if (active && i < L) {
    const int32_t *row = rows + (t / width) * width;
    const int64_t e = walk_first + i;
    ctr_stage[e - block_first] = row[i];
    int32_t *ctx = ctx_stage + (e - block_first) * cw;
    const int64_t j0 = max(int64_t(0), i - window), j1 = min(L - 1, i + int64_t(window));
    int64_t m = 0;
    for (int64_t j = j0; j <= j1; ++j)
      if (j != i) ctx[m++] = row[j];
    for (; m < cw; ++m) ctx[m] = -1;
  }
  __syncthreads();
  // The block's examples end where the next block's begin.
  const bool full = block_end > capacity;
  const int64_t lim = max(int64_t(0), min(block_end, capacity) - block_first);  // examples that fit
  stream_run<kBlock>(ctr_stage, centers + block_first, lim);
  stream_run<kBlock>(ctx_stage, contexts + block_first * cw, lim * cw);
  // `full` holds for the whole block: one thread reports it
  if (((full && threadIdx.x == 0) || bad) && status != nullptr)
    atomicOr(status, (full ? RDF2V_STATUS_CAPACITY : 0) | (bad ? RDF2V_STATUS_BAD_LENGTH : 0));
}

// CBOW, written in output order. A block of kBlock threads takes
// kBlock / width walks, whose examples form one contiguous output range. It
// stages only its walk rows and, per walk, where its examples start and how
// many there are, plus the walk of each example; then every thread produces
// context entries directly in output order, four per 16-byte non-temporal
// store: entry m of example e is the m-th context of that example's position
// (the tokens j0 .. j1 of its window, skipping the position itself), or -1
// past the last one. No context row is ever staged, so the block's LDS does
// not grow with the window.
template <int kBlock>
__global__ __launch_bounds__(kBlock) void cbow_direct_kernel(const int32_t *__restrict__ tokens,
                                                              const int32_t *__restrict__ len, int64_t n,
                                                              int32_t width, int32_t window,
                                                              const int64_t *__restrict__ offsets,
                                                              int32_t *__restrict__ centers,
                                                              int32_t *__restrict__ contexts, int64_t capacity,
                                                              int32_t *status) {
  __shared__ int32_t rows[kBlock];        // the block's walk rows
  __shared__ int32_t walk_first[kBlock];  // per walk of the block: its first example, block-relative
  __shared__ int32_t walk_len[kBlock];    // per walk of the block: its examples (valid tokens)
  __shared__ int32_t ex_walk[kBlock];     // per example of the block: its walk
  __shared__ int64_t block_end;
  const int walks_per_block = kBlock / width;
  const int t = threadIdx.x;
  const int64_t r0 = int64_t(blockIdx.x) * walks_per_block;
  const int64_t r_end = min(n, r0 + walks_per_block);
  const int k_walk = t / width;  // this thread's walk within the block
  const int64_t r = r0 + k_walk;
  const int i = t % width;
  const bool active = t < walks_per_block * width && r < n;
  int bad = 0;
  // Every global read the block needs is issued before the first barrier.
  const int64_t block_first = offsets[r0];
  int32_t L = 0;
  int64_t walk_first_g = 0;
  if (active) {
    L = clamped_len(len, r, width, bad);
    walk_first_g = offsets[r];
  }
  const int64_t span = (r_end - r0) * width;  // <= kBlock
  if (t < span) rows[t] = tokens[r0 * width + t];
  if (t == 0) {
    if (r_end < n) {
      block_end = offsets[r_end];
    } else {
      int b2 = 0;
      block_end = offsets[n - 1] + clamped_len(len, n - 1, width, b2);
    }
  }
  // Block-relative example indices: a block holds at most one example per thread.
  const int32_t wf = int32_t(walk_first_g - block_first);
  if (active && i == 0) {
    walk_first[k_walk] = wf;
    walk_len[k_walk] = L;
  }
  if (active && i < L) ex_walk[wf + i] = k_walk;
  __syncthreads();

  const int64_t cnt = block_end - block_first;                          // examples of the block
  const int32_t lim = int32_t(max(int64_t(0), min(cnt, capacity - block_first)));  // those that fit
  const bool full = block_end > capacity;
  const int32_t w = window, cw = 2 * window;
  // Centers: example e of the block is position e - walk_first of its walk.
  for (int32_t e = t; e < lim; e += kBlock) {
    const int32_t k = ex_walk[e];
    __builtin_nontemporal_store(rows[k * width + (e - walk_first[k])], centers + block_first + e);
  }
  // Context entry q = e * cw + m of the block; `next` steps to entry q + 1.
  struct Cursor {
    int32_t e, m, base, nleft, nctx;  // example, entry; the example's window start, contexts before / in all
  };
  auto at = [&](int32_t e, int32_t m) {
    Cursor c;
    c.e = e;
    c.m = m;
    const int32_t k = ex_walk[e];
    const int32_t pos = e - walk_first[k];
    const int32_t j0 = max(0, pos - w), j1 = min(walk_len[k] - 1, pos + w);
    c.base = k * width + j0;
    c.nleft = pos - j0;
    c.nctx = j1 - j0;
    return c;
  };
  auto value = [&](const Cursor &c) {
    return c.m < c.nleft ? rows[c.base + c.m] : (c.m < c.nctx ? rows[c.base + c.m + 1] : -1);
  };
  auto next = [&](Cursor &c) {
    if (++c.m == cw && c.e + 1 < lim) c = at(c.e + 1, 0);
  };
  const int32_t total = lim * cw;  // entries that fit (<= kBlock * 2 * RDF2V_MAX_DEPTH * 2)
  int32_t *dst = contexts + block_first * int64_t(cw);
  const int32_t head = min(total, int32_t(((16 - (reinterpret_cast<uintptr_t>(dst) & 15)) & 15) / 4));
  if (t < head) {
    const Cursor c = at(t / cw, t % cw);
    __builtin_nontemporal_store(value(c), dst + t);
  }
  const int32_t body = (total - head) >> 2;
  v4i32 *dst4 = reinterpret_cast<v4i32 *>(dst + head);
  for (int32_t q4 = t; q4 < body; q4 += kBlock) {
    const int32_t q = head + 4 * q4;
    Cursor c = at(q / cw, q % cw);
    v4i32 v;
    v.x = value(c);
    next(c);
    v.y = value(c);
    next(c);
    v.z = value(c);
    next(c);
    v.w = value(c);
    __builtin_nontemporal_store(v, dst4 + q4);
  }
  for (int32_t q = head + 4 * body + t; q < total; q += kBlock) {
    const Cursor c = at(q / cw, q % cw);
    __builtin_nontemporal_store(value(c), dst + q);
  }
  // `full` holds for the whole block: one thread reports it
  if (((full && threadIdx.x == 0) || bad) && status != nullptr)
    atomicOr(status, (full ? RDF2V_STATUS_CAPACITY : 0) | (bad ? RDF2V_STATUS_BAD_LENGTH : 0));
}

constexpr size_t kMaxStageBytes = 32 << 10;

// Most pairs one walk of this width can give.
inline int64_t max_walk_pairs(int64_t width, int64_t window) {
  const int64_t m = std::min(window, width - 1);
  return m <= 0 ? 0 : 2 * (m * width - m * (m + 1) / 2);
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

size_t skipgram_workspace_bytes(int64_t num_walks) {
  const int64_t nb = ceil_div(num_walks, kTile);
  return align_up(size_t(num_walks) * 8, 256) + align_up(size_t(nb + 1) * 8, 256);
}

rdf2v_status launch_skipgram_pairs(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                                   int32_t width, int32_t window, int32_t *pairs_out, int64_t capacity,
                                   int64_t *count_out, void *workspace, int32_t *status_dev,
                                   hipStream_t stream) {
  char *ws = static_cast<char *>(workspace);
  int64_t *offsets = reinterpret_cast<int64_t *>(ws);
  int64_t *partials = reinterpret_cast<int64_t *>(ws + align_up(size_t(num_walks) * 8, 256));
  const int64_t nb = ceil_div(num_walks, kTile);
  if (nb > 0) {
    pair_count_reduce_kernel<false><<<dim3(unsigned(nb)), dim3(kThreads), 0, stream>>>(len, num_walks, width,
                                                                                      window, partials,
                                                                                      status_dev);
    RDF2V_LAUNCH_CHECK();
  }
  pair_partials_kernel<<<dim3(1), dim3(kThreads), 0, stream>>>(partials, nb, count_out);
  RDF2V_LAUNCH_CHECK();
  if (nb == 0) return RDF2V_OK;
  pair_offsets_kernel<false><<<dim3(unsigned(nb)), dim3(kThreads), 0, stream>>>(len, num_walks, width, window,
                                                                               partials, offsets);
  RDF2V_LAUNCH_CHECK();
  if (capacity > 0) {
    int2 *out = reinterpret_cast<int2 *>(pairs_out);
    // Blocks of 256 threads when their pairs fit a stage of at most
    // kMaxStageBytes, else of 128 or 64: several small blocks per CU keep the
    // write stream going while others load rows and place pairs (measured:
    // 256 threads with a ~17 KB stage beat 512 and 1024 with 33-67 KB).
    const int64_t per_walk = max_walk_pairs(width, window);
    auto stage_bytes = [&](int block) { return size_t(per_walk * (block / width)) * sizeof(int2); };
    auto launch = [&](auto kernel, int block, size_t lds) -> rdf2v_status {
      const int64_t blocks = ceil_div(num_walks, block / width);
      if (blocks >= (int64_t(1) << 31)) return RDF2V_ERR_TOO_LARGE;
      kernel<<<dim3(unsigned(blocks)), dim3(block), lds, stream>>>(tokens, len, num_walks, width, window, offsets,
                                                                   out, capacity, status_dev);
      RDF2V_LAUNCH_CHECK();
      return RDF2V_OK;
    };
    if (width <= 256 && stage_bytes(256) <= kMaxStageBytes)
      return launch(pair_emit_kernel<true, 256>, 256, stage_bytes(256));
    if (width <= 128 && stage_bytes(128) <= kMaxStageBytes)
      return launch(pair_emit_kernel<true, 128>, 128, stage_bytes(128));
    if (width <= 64 && stage_bytes(64) <= kMaxStageBytes)
      return launch(pair_emit_kernel<true, 64>, 64, stage_bytes(64));
    return launch(pair_emit_kernel<false, kThreads>, kThreads, 0);
  }
  return RDF2V_OK;
}

rdf2v_status launch_cbow_examples(const int32_t *tokens, const int32_t *len, int64_t num_walks, int32_t width,
                                  int32_t window, int32_t *centers_out, int32_t *contexts_out, int64_t capacity,
                                  int64_t *count_out, void *workspace, int32_t *status_dev, hipStream_t stream) {
  char *ws = static_cast<char *>(workspace);
  int64_t *offsets = reinterpret_cast<int64_t *>(ws);
  int64_t *partials = reinterpret_cast<int64_t *>(ws + align_up(size_t(num_walks) * 8, 256));
  const int64_t nb = ceil_div(num_walks, kTile);
  if (nb > 0) {
    pair_count_reduce_kernel<true><<<dim3(unsigned(nb)), dim3(kThreads), 0, stream>>>(len, num_walks, width, window,
                                                                                     partials, status_dev);
    RDF2V_LAUNCH_CHECK();
  }
  pair_partials_kernel<<<dim3(1), dim3(kThreads), 0, stream>>>(partials, nb, count_out);
  RDF2V_LAUNCH_CHECK();
  if (nb == 0) return RDF2V_OK;
  pair_offsets_kernel<true><<<dim3(unsigned(nb)), dim3(kThreads), 0, stream>>>(len, num_walks, width, window,
                                                                              partials, offsets);
  RDF2V_LAUNCH_CHECK();
  if (capacity == 0) return RDF2V_OK;
  // The staged kernel holds a block's context rows in LDS: B rows of
  // 2 * window ints for B threads, 256-thread blocks up to 32 KB, else 128.
  // The output-order kernel needs no stage. Measured on 8M walks of 17 tokens
  // (ms, staged / output order): windows 1: 0.95 / 0.93, 2: 1.12 / 1.00,
  // 5: 1.55 / 1.55, 10: 2.62 / 2.68, 20 (128 threads): 4.88 / 5.09, 40 (then
  // 64-thread staged blocks): 14.2 / 9.1; so the staged kernel serves windows
  // of 5 and more while a block of at least 128 threads holds its stage.
  // (Earlier, at window 5 on 48.9M walks: 512-thread blocks, or two or four
  // positions per thread, were 2-50 % slower.)
  const size_t row_bytes = size_t(2) * size_t(window) * sizeof(int32_t);
  auto launch = [&](auto kernel, int block, size_t lds) -> rdf2v_status {
    const int64_t blocks = ceil_div(num_walks, block / width);
    if (blocks >= (int64_t(1) << 31)) return RDF2V_ERR_TOO_LARGE;
    kernel<<<dim3(unsigned(blocks)), dim3(block), lds, stream>>>(tokens, len, num_walks, width, window, offsets,
                                                                 centers_out, contexts_out, capacity, status_dev);
    RDF2V_LAUNCH_CHECK();
    return RDF2V_OK;
  };
  if (window >= 5) {
    if (width <= 256 && 256 * row_bytes <= kMaxStageBytes)
      return launch(cbow_emit_kernel<256>, 256, 256 * row_bytes);
    if (width <= 128 && 128 * row_bytes <= kMaxStageBytes)
      return launch(cbow_emit_kernel<128>, 128, 128 * row_bytes);
  }
  return launch(cbow_direct_kernel<256>, 256, 0);
}

}  // namespace rdf2v
