// Triples -> subject-indexed CSR on gfx950.
//
// The CSR's rows must keep the triples' input order (a stable sort by subject),
// so that walk parity is exact and independent of scheduling. Atomics cannot
// give that order; an LSD radix sort on the subject id can, because every pass
// is a stable counting sort on one digit. Each pass runs three kernels:
//   1. radix_count:   per 4096-triple tile, a histogram of the pass's digit
//                     (LDS atomics), written digit-major to a count table;
//   2. scan:          exclusive scan of that table (reduce, scan of block
//                     sums, apply) -> the global start of (digit, tile);
//   3. radix_scatter: per tile, the stable rank of every triple among the
//                     tile's triples with the same digit (wave ballots give the
//                     lanes sharing a digit, per-wave LDS counters carry the
//                     count across rounds), a local reorder through LDS, then
//                     writes of runs of equal digits to their global slots.
// The first pass also checks every id range. After the last pass the sorted
// subjects give row_ptr[v] = (number of subjects < v) by binary search, so no
// kernel needs global atomics (power-law hubs would serialise them).
//
// Workspace: two key buffers (4 B/triple each), one payload buffer (8 B/triple;
// edges_out is the other), the count table and the scan's block sums.

#include "common.hpp"
#include "launch.hpp"
#include "xcd.hpp"

namespace rdf2v {
namespace {

constexpr int kSortThreads = 512;
constexpr int kSortItems = 8;
constexpr int kTile = kSortThreads * kSortItems;     // triples per tile
constexpr int kMaxDigitBits = 9;
constexpr int kMaxBins = 1 << kMaxDigitBits;
constexpr int kTileWaves = kSortThreads / kWave;
constexpr int kWaveItems = kTile / kTileWaves;       // consecutive triples per wave
constexpr int kRounds = kWaveItems / kWave;          // rounds of 64 per wave

constexpr int kScanThreads = 256;
constexpr int kScanItems = 16;
constexpr int kScanTile = kScanThreads * kScanItems;

static_assert(kMaxBins <= kSortThreads, "one thread per digit in the tile prefix step");

// ---------------------------------------------------------------------------
// Radix pass, step 1: per-tile digit histogram (+ subject id validation on
// pass 0; the first scatter, which reads predicates and objects anyway,
// validates those).
// ---------------------------------------------------------------------------
// Each thread reads kCountItems keys as 16-byte vectors (all loads issued
// before any histogram update) and counts them in its wave's own LDS
// histogram, so lanes of different waves never contend for a bin.
constexpr int kCountThreads = 256;
constexpr int kCountWaves = kCountThreads / kWave;
constexpr int kCountItems = kTile / kCountThreads;  // keys per thread

template <bool kValidate>
__global__ __launch_bounds__(kCountThreads) void radix_count_kernel(
    const uint32_t *__restrict__ keys, int64_t n, int shift, int bits, int32_t num_entities,
    int32_t *__restrict__ counts, int64_t tiles, int32_t *status) {
  __shared__ int hist[kCountWaves * kMaxBins];
  constexpr int kVec = 4;
  constexpr int kLoads = kCountItems / kVec;
  const int bins = 1 << bits;
  const uint32_t mask = uint32_t(bins - 1);
  const int wave = threadIdx.x / kWave;
  for (int i = threadIdx.x; i < kCountWaves * bins; i += kCountThreads) hist[i] = 0;
  __syncthreads();
  int *wave_hist = hist + wave * bins;
  const int64_t tile = xcd_tile(blockIdx.x, tiles);
  const int64_t base = tile * kTile;
  const bool full = base + kTile <= n && (reinterpret_cast<uintptr_t>(keys) & 15) == 0;
  uint32_t k[kCountItems];
  int bad = 0;
  if (full) {
    // 16-byte loads: vector v of the tile holds keys 4v .. 4v+3.
    const uint4 *k4 = reinterpret_cast<const uint4 *>(keys + base);
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
      const uint4 v = k4[i * kCountThreads + threadIdx.x];
      k[kVec * i + 0] = v.x; k[kVec * i + 1] = v.y; k[kVec * i + 2] = v.z; k[kVec * i + 3] = v.w;
    }
    if (kValidate) {
#pragma unroll
      for (int i = 0; i < kCountItems; ++i) bad |= k[i] >= uint32_t(num_entities);
    }
    // After the first pass the keys of a tile are grouped by their lower digits, and in
    // power-law graphs many tiles hold one hub's triples only: a wave's 64 increments of one
    // bin would serialise on one LDS address. The lanes that share lane 0's digit add their
    // number with one atomic instead.
    const int lane = lane_id();
#pragma unroll
    for (int i = 0; i < kCountItems; ++i) {
      const uint32_t d = (k[i] >> shift) & mask;
      const uint32_t d0 = __builtin_amdgcn_readfirstlane(d);
      const uint64_t same = __ballot(d == d0);
      if (d != d0)
        atomicAdd(&wave_hist[d], 1);
      else if (lane == 0)
        atomicAdd(&wave_hist[d0], __popcll(same));
    }
  } else {
    // ragged last tile or unaligned input: scalar loads of the same items
#pragma unroll
    for (int i = 0; i < kCountItems; ++i) {
      const int64_t idx = base + int64_t(i / kVec) * (kCountThreads * kVec) + threadIdx.x * kVec + (i % kVec);
      if (idx < n) {
        const uint32_t key = keys[idx];
        atomicAdd(&wave_hist[(key >> shift) & mask], 1);
        if (kValidate) bad |= key >= uint32_t(num_entities);
      }
    }
  }
  if (kValidate) {
    if (__syncthreads_or(bad) && threadIdx.x == 0 && status != nullptr)
      atomicOr(status, RDF2V_STATUS_ID_OUT_OF_RANGE);
  } else {
    __syncthreads();
  }
  for (int d = threadIdx.x; d < bins; d += kCountThreads) {
    int c = 0;
#pragma unroll
    for (int w = 0; w < kCountWaves; ++w) c += hist[w * bins + d];
    counts[int64_t(d) * tiles + tile] = c;
  }
}

// ---------------------------------------------------------------------------
// Radix pass, step 3: stable scatter of one tile.
// ---------------------------------------------------------------------------
template <bool kFirst>
__global__ __launch_bounds__(kSortThreads) void radix_scatter_kernel(
    const uint32_t *__restrict__ keys_in, const int2 *__restrict__ pay_in,
    const int32_t *__restrict__ pred_in, const int32_t *__restrict__ obj_in,
    uint32_t *__restrict__ keys_out, int2 *__restrict__ pay_out, int64_t n, int shift, int bits,
    const int32_t *__restrict__ offsets, int64_t tiles, int32_t num_entities, int32_t num_predicates,
    int32_t *status) {
  __shared__ int wave_count[kTileWaves][kMaxBins];
  __shared__ int global_minus_local[kMaxBins];
  __shared__ uint32_t s_keys[kTile];
  __shared__ int2 s_pay[kTile];
  __shared__ int scan_scratch[kSortThreads / kWave];

  const int bins = 1 << bits;
  const uint32_t mask = uint32_t(bins - 1);
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int64_t tile = xcd_tile(blockIdx.x, tiles);
  const int64_t base = tile * kTile;
  const int tile_n = int(min(int64_t(kTile), n - base));

  for (int i = threadIdx.x; i < kTileWaves * kMaxBins; i += kSortThreads) (&wave_count[0][0])[i] = 0;
  __syncthreads();

  // Thread d's global start of digit d in this tile, issued with the tile's loads
  // below so that it is not waited for on its own after the ranking barrier.
  const int32_t digit_global = threadIdx.x < bins ? offsets[int64_t(threadIdx.x) * tiles + tile] : 0;

  // Wave `wave` owns tile items [wave*kWaveItems, (wave+1)*kWaveItems), visited in order.
  // All of the wave's loads are issued before any ranking, so they are in
  // flight together.
  uint32_t key[kRounds];
  int2 pay[kRounds];
  int rank[kRounds];
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const int local = wave * kWaveItems + r * kWave + lane;
    const int64_t idx = base + local;
    key[r] = 0;
    pay[r] = make_int2(0, 0);
    if (local < tile_n) {
      key[r] = keys_in[idx];
      pay[r] = kFirst ? make_int2(pred_in[idx], obj_in[idx]) : pay_in[idx];
    }
  }
  if (kFirst) {  // predicate and object ids (subjects were checked by the count pass)
    int bad = 0;
#pragma unroll
    for (int r = 0; r < kRounds; ++r)
      bad |= (uint32_t(pay[r].x) >= uint32_t(num_predicates)) | (uint32_t(pay[r].y) >= uint32_t(num_entities));
    if (__ballot(bad) != 0 && lane == 0 && status != nullptr) atomicOr(status, RDF2V_STATUS_ID_OUT_OF_RANGE);
  }
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const int local = wave * kWaveItems + r * kWave + lane;
    const bool valid = local < tile_n;
    const uint32_t k = key[r];
    const uint32_t d = (k >> shift) & mask;
    // Lanes of this round holding the same digit.
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < bits; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t m = __ballot(bit);
      peers &= bit ? m : ~m;
    }
    const int below = __popcll(peers & lanes_below(lane));
    const int before = valid ? wave_count[wave][d] : 0;
    rank[r] = before + below;
    // The lowest lane of each digit group advances the wave's counter; its
    // store depends on the load above, so every lane's load precedes it.
    if (valid && below == 0) wave_count[wave][d] = before + __popcll(peers);
  }
  __syncthreads();

  // Tile-local start of every (wave, digit) run, and the shift from tile-local
  // to global slot per digit.
  {
    const int d = threadIdx.x;
    int c[kTileWaves];
    int total = 0;
#pragma unroll
    for (int w = 0; w < kTileWaves; ++w) {
      c[w] = d < bins ? wave_count[w][d] : 0;
      total += c[w];
    }
    int tile_total;
    const int start = block_exclusive_scan<kSortThreads>(total, scan_scratch, tile_total);
    if (d < bins) {
      int run = start;
#pragma unroll
      for (int w = 0; w < kTileWaves; ++w) {
        wave_count[w][d] = run;
        run += c[w];
      }
      global_minus_local[d] = digit_global - start;
    }
  }
  __syncthreads();

#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const int local = wave * kWaveItems + r * kWave + lane;
    if (local < tile_n) {
      const int pos = wave_count[wave][(key[r] >> shift) & mask] + rank[r];
      if (pos < kTile) {  // always true; keeps a logic slip from leaving the tile
        s_keys[pos] = key[r];
        s_pay[pos] = pay[r];
      }
    }
  }
  __syncthreads();

  for (int j = threadIdx.x; j < tile_n; j += kSortThreads) {
    const uint32_t k = s_keys[j];
    const int64_t g = int64_t(global_minus_local[(k >> shift) & mask]) + j;
    if (g >= 0 && g < n) {  // always true for consistent counts; never write outside the arrays
      keys_out[g] = k;
      pay_out[g] = s_pay[j];
    }
  }
}

// ---------------------------------------------------------------------------
// Exclusive scan of int32 (reduce -> scan of block sums -> apply).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kScanThreads) void scan_reduce_kernel(const int32_t *__restrict__ in,
                                                                   int64_t n,
                                                                   int32_t *__restrict__ partials) {
  __shared__ int scratch[kScanThreads / kWave];
  const int64_t base = int64_t(blockIdx.x) * kScanTile;
  int s = 0;
#pragma unroll 4
  for (int i = 0; i < kScanItems; ++i) {
    const int64_t idx = base + int64_t(i) * kScanThreads + threadIdx.x;
    if (idx < n) s += in[idx];
  }
  const int total = block_sum<kScanThreads>(s, scratch);
  if (threadIdx.x == 0) partials[blockIdx.x] = total;
}

// One block: exclusive scan of the block sums in place; partials[nb] = total.
__global__ __launch_bounds__(kScanThreads) void scan_partials_kernel(int32_t *partials, int64_t nb,
                                                                     int64_t *total_out) {
  __shared__ int scratch[kScanThreads / kWave];
  int carry = 0;
  for (int64_t base = 0; base < nb; base += kScanThreads) {
    const int64_t idx = base + threadIdx.x;
    const int x = idx < nb ? partials[idx] : 0;
    int tot;
    const int ex = block_exclusive_scan<kScanThreads>(x, scratch, tot);
    if (idx < nb) partials[idx] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) {
    partials[nb] = carry;
    if (total_out != nullptr) *total_out = carry;
  }
}

__global__ __launch_bounds__(kScanThreads) void scan_apply_kernel(const int32_t *in, int64_t n,
                                                                  const int32_t *__restrict__ partials,
                                                                  int32_t *out) {
  __shared__ int scratch[kScanThreads / kWave];
  const int64_t base = int64_t(blockIdx.x) * kScanTile;
  int carry = partials[blockIdx.x];
  for (int i = 0; i < kScanItems; ++i) {
    const int64_t idx = base + int64_t(i) * kScanThreads + threadIdx.x;
    const int x = idx < n ? in[idx] : 0;
    int tot;
    const int ex = block_exclusive_scan<kScanThreads>(x, scratch, tot);
    if (idx < n) out[idx] = carry + ex;
    carry += tot;
  }
}

rdf2v_status scan_exclusive(int32_t *data, int64_t n, int32_t *partials, int64_t nb,
                            hipStream_t stream) {
  scan_reduce_kernel<<<dim3(unsigned(nb)), dim3(kScanThreads), 0, stream>>>(data, n, partials);
  RDF2V_LAUNCH_CHECK();
  scan_partials_kernel<<<dim3(1), dim3(kScanThreads), 0, stream>>>(partials, nb, nullptr);
  RDF2V_LAUNCH_CHECK();
  scan_apply_kernel<<<dim3(unsigned(nb)), dim3(kScanThreads), 0, stream>>>(data, n, partials, data);
  RDF2V_LAUNCH_CHECK();
  return RDF2V_OK;
}

// ---------------------------------------------------------------------------
// row_ptr[v] = number of sorted subjects < v, for v in [0, V], from the sorted
// subjects in one pass: where the subject changes from a (at position i-1) to
// b (at i), every v in (a, b] has row_ptr[v] = i; the subjects v above the
// last one get n. A thread writes at most kGapRun of those entries; longer
// runs of entities without out-edges keep the -1 that row_ptr_fill_kernel put
// there, and row_ptr_fixup_kernel finds each of them by binary search.
// ---------------------------------------------------------------------------
constexpr int kGapRun = 64;

__global__ __launch_bounds__(256) void row_ptr_fill_kernel(int32_t *__restrict__ row_ptr, int64_t nv) {
  const int64_t v = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (v < nv) row_ptr[v] = -1;
}

// Each thread takes kBoundItems consecutive positions (two 16-byte loads).
constexpr int kBoundItems = 8;

__global__ __launch_bounds__(256) void row_ptr_bounds_kernel(const uint32_t *__restrict__ sorted_keys,
                                                             int64_t n, int32_t num_entities,
                                                             int32_t *__restrict__ row_ptr) {
  const int64_t i0 = (int64_t(blockIdx.x) * 256 + threadIdx.x) * kBoundItems;
  if (i0 > n) return;
  uint32_t k[kBoundItems];
  if (i0 + kBoundItems <= n && (reinterpret_cast<uintptr_t>(sorted_keys) & 15) == 0) {
    const uint4 *k4 = reinterpret_cast<const uint4 *>(sorted_keys + i0);
    const uint4 v0 = k4[0], v1 = k4[1];
    k[0] = v0.x; k[1] = v0.y; k[2] = v0.z; k[3] = v0.w;
    k[4] = v1.x; k[5] = v1.y; k[6] = v1.z; k[7] = v1.w;
  } else {
#pragma unroll
    for (int j = 0; j < kBoundItems; ++j) k[j] = i0 + j < n ? sorted_keys[i0 + j] : 0u;
  }
  // entities in (a, b] start at position i; a = -1 before the first subject, b = V after the last
  int64_t a = i0 == 0 ? -1 : int64_t(sorted_keys[i0 - 1]);
#pragma unroll
  for (int j = 0; j < kBoundItems; ++j) {
    const int64_t i = i0 + j;
    if (i > n) break;
    const int64_t b = i == n ? int64_t(num_entities) : int64_t(k[j]);
    if (b != a) {
      const int64_t hi = min(b, int64_t(num_entities));  // ids >= V cannot occur after validation
      const int64_t lo = max(a + 1, hi - (kGapRun - 1));
      for (int64_t v = lo; v <= hi; ++v) row_ptr[v] = int32_t(i);
    }
    a = b;
  }
}

__global__ __launch_bounds__(256) void row_ptr_fixup_kernel(const uint32_t *__restrict__ sorted_keys,
                                                            int64_t n, int32_t num_entities,
                                                            int32_t *__restrict__ row_ptr) {
  const int64_t v = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (v > num_entities || row_ptr[v] >= 0) return;
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (sorted_keys[mid] < uint32_t(v)) lo = mid + 1;
    else hi = mid;
  }
  row_ptr[v] = int32_t(lo);
}

__global__ __launch_bounds__(256) void fill_kernel(int32_t *p, int64_t n, int32_t value) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) p[i] = value;
}

// ---------------------------------------------------------------------------
// Entities with out-degree >= 1, ascending (count per block, scan, compact).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kScanThreads) void nonsink_count_kernel(const int32_t *__restrict__ row_ptr,
                                                                     int32_t num_entities,
                                                                     int32_t *__restrict__ partials) {
  __shared__ int scratch[kScanThreads / kWave];
  const int64_t base = int64_t(blockIdx.x) * kScanTile;
  int s = 0;
  for (int i = 0; i < kScanItems; ++i) {
    const int64_t v = base + int64_t(i) * kScanThreads + threadIdx.x;
    if (v < num_entities) s += row_ptr[v + 1] > row_ptr[v];
  }
  const int total = block_sum<kScanThreads>(s, scratch);
  if (threadIdx.x == 0) partials[blockIdx.x] = total;
}

__global__ __launch_bounds__(kScanThreads) void nonsink_compact_kernel(const int32_t *__restrict__ row_ptr,
                                                                       int32_t num_entities,
                                                                       const int32_t *__restrict__ partials,
                                                                       int32_t *__restrict__ out) {
  __shared__ int scratch[kScanThreads / kWave];
  const int64_t base = int64_t(blockIdx.x) * kScanTile;
  int carry = partials[blockIdx.x];
  for (int i = 0; i < kScanItems; ++i) {
    const int64_t v = base + int64_t(i) * kScanThreads + threadIdx.x;
    const int f = (v < num_entities) ? (row_ptr[v + 1] > row_ptr[v]) : 0;
    int tot;
    const int ex = block_exclusive_scan<kScanThreads>(f, scratch, tot);
    if (f) out[carry + ex] = int32_t(v);
    carry += tot;
  }
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

SortPlan plan_csr_build(int64_t num_triples, int32_t num_entities) {
  SortPlan p;
  if (num_triples <= 0) return p;
  int total_bits = 0;
  if (num_entities > 1) total_bits = 32 - __builtin_clz(uint32_t(num_entities - 1));
  // Digits of at most 8 bits, except that ids of 17 or 18 bits take two 9-bit
  // passes instead of three: a 512-bin pass costs about 1.4x a 256-bin one
  // (shorter runs per tile, a count table twice as long), which pays when it
  // saves one pass in three but not one in four.
  p.passes = total_bits == 0 ? 1 : int(ceil_div(total_bits, 8));
  if (p.passes == 3 && total_bits <= 2 * kMaxDigitBits) p.passes = 2;
  // The bits are spread as evenly as the pass count allows, the first passes
  // taking the odd ones: a pass of fewer bits has fewer bins and longer runs.
  for (int k = 0; k < p.passes; ++k)
    p.pass_bits[k] = total_bits == 0 ? 1 : total_bits / p.passes + (k < total_bits % p.passes ? 1 : 0);
  p.digit_bits = p.pass_bits[0];
  p.tiles = ceil_div(num_triples, kTile);
  p.count_len = (int64_t(1) << p.digit_bits) * p.tiles;
  p.count_blocks = ceil_div(p.count_len, kScanTile);
  size_t off = 0;
  p.off_keys_a = off;   off = align_up(off + size_t(num_triples) * 4, 256);
  p.off_keys_b = off;   off = align_up(off + size_t(num_triples) * 4, 256);
  p.off_payload = off;  off = align_up(off + size_t(num_triples) * 8, 256);
  p.off_counts = off;   off = align_up(off + size_t(p.count_len) * 4, 256);
  p.off_partials = off; off = align_up(off + size_t(p.count_blocks + 1) * 4, 256);
  p.bytes = off;
  return p;
}

rdf2v_status launch_csr_build(const int32_t *subj, const int32_t *pred, const int32_t *obj,
                              int64_t num_triples, int32_t num_entities, int32_t num_predicates,
                              int32_t *row_ptr_out, int32_t *edges_out, void *workspace,
                              const SortPlan &plan, int32_t *status_dev, hipStream_t stream) {
  const int64_t T = num_triples;
  if (T == 0) {
    const int64_t n = int64_t(num_entities) + 1;
    fill_kernel<<<dim3(unsigned(ceil_div(n, 256))), dim3(256), 0, stream>>>(row_ptr_out, n, 0);
    RDF2V_LAUNCH_CHECK();
    return RDF2V_OK;
  }
  char *ws = static_cast<char *>(workspace);
  uint32_t *keys_a = reinterpret_cast<uint32_t *>(ws + plan.off_keys_a);
  uint32_t *keys_b = reinterpret_cast<uint32_t *>(ws + plan.off_keys_b);
  int2 *pay_tmp = reinterpret_cast<int2 *>(ws + plan.off_payload);
  int32_t *counts = reinterpret_cast<int32_t *>(ws + plan.off_counts);
  int32_t *partials = reinterpret_cast<int32_t *>(ws + plan.off_partials);
  int2 *edges2 = reinterpret_cast<int2 *>(edges_out);

  const uint32_t *keys_in = reinterpret_cast<const uint32_t *>(subj);
  const int2 *pay_in = nullptr;
  int shift = 0;
  for (int pass = 0; pass < plan.passes; ++pass) {
    const int bits = plan.pass_bits[pass];
    const int64_t count_len = (int64_t(1) << bits) * plan.tiles;
    uint32_t *keys_out = (pass % 2 == 0) ? keys_a : keys_b;
    // The last pass must land in edges_out, so the payload alternates backwards from it.
    int2 *pay_out = ((plan.passes - 1 - pass) % 2 == 0) ? edges2 : pay_tmp;
    const dim3 grid(unsigned(plan.tiles));
    if (pass == 0)
      radix_count_kernel<true><<<grid, dim3(kCountThreads), 0, stream>>>(
          keys_in, T, shift, bits, num_entities, counts, plan.tiles, status_dev);
    else
      radix_count_kernel<false><<<grid, dim3(kCountThreads), 0, stream>>>(
          keys_in, T, shift, bits, num_entities, counts, plan.tiles, nullptr);
    RDF2V_LAUNCH_CHECK();
    const rdf2v_status st = scan_exclusive(counts, count_len, partials, ceil_div(count_len, kScanTile), stream);
    if (st != RDF2V_OK) return st;
    if (pass == 0)
      radix_scatter_kernel<true><<<grid, dim3(kSortThreads), 0, stream>>>(
          keys_in, nullptr, pred, obj, keys_out, pay_out, T, shift, bits, counts,
          plan.tiles, num_entities, num_predicates, status_dev);
    else
      radix_scatter_kernel<false><<<grid, dim3(kSortThreads), 0, stream>>>(
          keys_in, pay_in, nullptr, nullptr, keys_out, pay_out, T, shift, bits, counts,
          plan.tiles, num_entities, num_predicates, nullptr);
    RDF2V_LAUNCH_CHECK();
    keys_in = keys_out;
    pay_in = pay_out;
    shift += bits;
  }
  const int64_t nv = int64_t(num_entities) + 1;
  row_ptr_fill_kernel<<<dim3(unsigned(ceil_div(nv, 256))), dim3(256), 0, stream>>>(row_ptr_out, nv);
  RDF2V_LAUNCH_CHECK();
  row_ptr_bounds_kernel<<<dim3(unsigned(ceil_div(T + 1, 256 * kBoundItems))), dim3(256), 0, stream>>>(
      keys_in, T, num_entities, row_ptr_out);
  RDF2V_LAUNCH_CHECK();
  row_ptr_fixup_kernel<<<dim3(unsigned(ceil_div(nv, 256))), dim3(256), 0, stream>>>(keys_in, T, num_entities,
                                                                                   row_ptr_out);
  RDF2V_LAUNCH_CHECK();
  return RDF2V_OK;
}

size_t nonsink_workspace_bytes(int32_t num_entities) {
  const int64_t nb = ceil_div(int64_t(num_entities > 0 ? num_entities : 0), kScanTile);
  return align_up(size_t(nb + 1) * 4, 256);
}

rdf2v_status launch_nonsink_starts(const int32_t *row_ptr, int32_t num_entities, int32_t *starts_out,
                                   int64_t *count_out, void *workspace, hipStream_t stream) {
  const int64_t nb = ceil_div(int64_t(num_entities), kScanTile);
  int32_t *partials = static_cast<int32_t *>(workspace);
  if (nb > 0) {
    nonsink_count_kernel<<<dim3(unsigned(nb)), dim3(kScanThreads), 0, stream>>>(row_ptr, num_entities,
                                                                               partials);
    RDF2V_LAUNCH_CHECK();
  }
  scan_partials_kernel<<<dim3(1), dim3(kScanThreads), 0, stream>>>(partials, nb, count_out);
  RDF2V_LAUNCH_CHECK();
  if (nb > 0) {
    nonsink_compact_kernel<<<dim3(unsigned(nb)), dim3(kScanThreads), 0, stream>>>(
        row_ptr, num_entities, partials, starts_out);
    RDF2V_LAUNCH_CHECK();
  }
  return RDF2V_OK;
}

}  // namespace rdf2v
