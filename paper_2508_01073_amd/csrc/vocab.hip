// Vocabulary on gfx950 (gpuRDF2vec Sec. 3.1: entities and predicates are
// tokenised to integer ids at the start of the pipeline): string triples ->
// dense ids, numbered by first appearance (entities over s_0, o_0, s_1, o_1,
// ...; predicates over p_0, p_1, ...).
//
// Per sequence (entities, then predicates):
//   1. insert_kernel:  one thread per occurrence q hashes its string and finds
//                      or claims its slot in an open-addressing table (linear
//                      probing, lock-free). A slot's 64-bit key is
//                      (hash tag << 32 | representative occurrence), claimed
//                      by one compare-and-swap; equal tags are always
//                      confirmed byte by byte against the representative, so
//                      hash collisions cannot merge two strings. The slot's
//                      minpos becomes the smallest occurrence of its string
//                      (read first, atomicMin only if smaller). The slot index
//                      is parked in the id output.
//   2. mark_kernel:    every used slot sets bit minpos of a bitset over the
//                      occurrences: the first occurrences of all strings.
//   3. popcount scan:  the rank of a first occurrence among all first
//                      occurrences is its id (int32 prefix per 64-bit word).
//   4. slot_id_kernel: the id of every used slot; assign_kernel replaces the
//                      parked slot indices by ids.
// The table is sized to a power of two >= 2 * the caller's bound on distinct
// strings, so probing stays short; the result does not depend on which thread
// wins a slot, only on minpos, so it is deterministic.

#include <algorithm>

#include "common.hpp"
#include "launch.hpp"

namespace rdf2v {
namespace {

constexpr int kThreads = 256;
constexpr int kWordsPerThread = 16;
constexpr int kWordTile = kThreads * kWordsPerThread;
constexpr uint64_t kEmpty = ~uint64_t(0);

struct alignas(16) Slot {
  uint64_t key;    // kEmpty, or (tag << 32) | representative occurrence
  int32_t minpos;  // smallest occurrence of the slot's string
  int32_t id;      // dense id, once ranked
};

struct StrCol {
  const uint8_t *chars;
  const int64_t *off;
  int64_t bytes;
};

struct Seq {
  StrCol col[2];  // occurrence q: column (q & 1), row q >> 1 when paired; else column 0, row q
  int32_t *out[2];
};

template <bool kPaired>
__device__ __forceinline__ int seq_col(int64_t q) {
  return kPaired ? int(q & 1) : 0;
}
template <bool kPaired>
__device__ __forceinline__ int64_t seq_row(int64_t q) {
  return kPaired ? (q >> 1) : q;
}

// Byte range of string `row`; an inconsistent range is read as empty and flagged.
__device__ __forceinline__ void string_range(const StrCol &c, int64_t row, int64_t &start, int64_t &len,
                                             int &bad) {
  const int64_t a = c.off[row], b = c.off[row + 1];
  if (a < 0 || b < a || b > c.bytes) {
    bad = 1;
    start = 0;
    len = 0;
    return;
  }
  start = a;
  len = b - a;
}

// Little-endian 4-byte word j of a column's chars (bytes past the end read 0).
__device__ __forceinline__ uint32_t load_word(const StrCol &c, int64_t j) {
  const int64_t p = 4 * j;
  if (p + 4 <= c.bytes) return reinterpret_cast<const uint32_t *>(c.chars)[j];
  uint32_t w = 0;
  for (int b = 0; b < 4; ++b)
    if (p + b < c.bytes) w |= uint32_t(c.chars[p + b]) << (8 * b);
  return w;
}

// Consecutive 4-byte chunks of one string, read as aligned words and shifted;
// the last chunk is zero-padded. The chunks depend on the bytes only, not on
// where the string sits.
struct ChunkReader {
  const StrCol *c;
  int64_t word;
  int shift;
  uint32_t lo;
  __device__ __forceinline__ ChunkReader(const StrCol &col, int64_t start)
      : c(&col), word(start >> 2), shift(int(start & 3) * 8) {
    lo = load_word(col, word);
  }
  __device__ __forceinline__ uint32_t next(int64_t remaining) {
    const uint32_t hi = load_word(*c, ++word);
    uint32_t v = shift ? (lo >> shift) | (hi << (32 - shift)) : lo;
    lo = hi;
    if (remaining < 4) v &= (uint32_t(1) << (8 * remaining)) - 1;
    return v;
  }
};

__device__ __forceinline__ uint64_t fmix64(uint64_t h) {  // MurmurHash3 finaliser
  h ^= h >> 33;
  h *= 0xff51afd7ed558ccdull;
  h ^= h >> 33;
  h *= 0xc4ceb9fe1a85ec53ull;
  h ^= h >> 33;
  return h;
}

__device__ __forceinline__ uint64_t string_hash(const StrCol &c, int64_t start, int64_t len) {
  uint64_t h = 0x243f6a8885a308d3ull ^ (uint64_t(len) * 0x9e3779b97f4a7c15ull);
  ChunkReader rd(c, start);
  for (int64_t k = 0; k < len; k += 4) {
    h = (h ^ rd.next(len - k)) * 0x100000001b3ull;
    h ^= h >> 29;
  }
  return fmix64(h);
}

__device__ __forceinline__ bool same_bytes(const StrCol &ca, int64_t a, const StrCol &cb, int64_t b,
                                           int64_t len) {
  ChunkReader ra(ca, a), rb(cb, b);
  for (int64_t k = 0; k < len; k += 4)
    if (ra.next(len - k) != rb.next(len - k)) return false;
  return true;
}

__device__ __forceinline__ uint64_t load_key(const Slot *s) {
  return __hip_atomic_load(&s->key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <bool kPaired>
__global__ __launch_bounds__(kThreads) void insert_kernel(Seq seq, int64_t n, Slot *__restrict__ table,
                                                          int64_t mask, int32_t *status) {
  const int64_t q = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (q >= n) return;
  const int col = seq_col<kPaired>(q);
  const StrCol &c = seq.col[col];
  int bad = 0;
  int64_t start, len;
  string_range(c, seq_row<kPaired>(q), start, len, bad);
  const uint64_t h = string_hash(c, start, len);
  const uint32_t tag = uint32_t(h >> 32);
  const uint64_t mine = (uint64_t(tag) << 32) | uint32_t(q);
  int64_t s = int64_t(h & uint64_t(mask));
  int64_t found = -1;
  for (int64_t probe = 0; probe <= mask; ++probe, s = (s + 1) & mask) {
    uint64_t k = load_key(table + s);
    if (k == kEmpty) {
      const uint64_t prev = atomicCAS(reinterpret_cast<unsigned long long *>(&table[s].key),
                                      static_cast<unsigned long long>(kEmpty),
                                      static_cast<unsigned long long>(mine));
      if (prev == kEmpty) {
        found = s;
        break;
      }
      k = prev;
    }
    if (uint32_t(k >> 32) != tag) continue;
    const int64_t rep = int64_t(uint32_t(k));
    const StrCol &rc = seq.col[seq_col<kPaired>(rep)];
    int rbad = 0;
    int64_t rstart, rlen;
    string_range(rc, seq_row<kPaired>(rep), rstart, rlen, rbad);
    if (rlen == len && same_bytes(c, start, rc, rstart, len)) {
      found = s;
      break;
    }
  }
  int32_t *out = seq.out[col] + seq_row<kPaired>(q);
  if (found < 0) {
    *out = -1;
    if (status != nullptr) atomicOr(status, RDF2V_STATUS_CAPACITY);
  } else {
    int32_t *mp = &table[found].minpos;
    if (int32_t(q) < __hip_atomic_load(mp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
      atomicMin(mp, int32_t(q));
    *out = int32_t(found);
  }
  if (bad && status != nullptr) atomicOr(status, RDF2V_STATUS_BAD_LENGTH);
}

__global__ __launch_bounds__(kThreads) void init_kernel(Slot *__restrict__ table, int64_t capacity,
                                                        uint64_t *__restrict__ bits, int64_t words) {
  const int64_t stride = int64_t(gridDim.x) * kThreads;
  for (int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x; i < capacity || i < words; i += stride) {
    if (i < capacity) table[i] = Slot{kEmpty, INT32_MAX, -1};
    if (i < words) bits[i] = 0;
  }
}

// Every used slot's minpos was lowered by the thread that claimed it, so it is
// an occurrence in [0, n); the range check only guards the bitset.
__global__ __launch_bounds__(kThreads) void mark_kernel(const Slot *__restrict__ table, int64_t capacity,
                                                        int64_t n, unsigned long long *__restrict__ bits) {
  const int64_t s = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (s >= capacity) return;
  const Slot t = table[s];
  if (t.key == kEmpty || t.minpos < 0 || t.minpos >= n) return;
  atomicOr(bits + (t.minpos >> 6), 1ull << (t.minpos & 63));
}

__global__ __launch_bounds__(kThreads) void popc_count_kernel(const uint64_t *__restrict__ bits, int64_t words,
                                                              int64_t *__restrict__ partials) {
  __shared__ int64_t scratch[kThreads / kWave];
  const int64_t base = int64_t(blockIdx.x) * kWordTile;
  int64_t s = 0;
#pragma unroll 4
  for (int i = 0; i < kWordsPerThread; ++i) {
    const int64_t w = base + int64_t(i) * kThreads + threadIdx.x;
    if (w < words) s += __popcll(bits[w]);
  }
  const int64_t total = block_sum<kThreads, int64_t>(s, scratch);
  if (threadIdx.x == 0) partials[blockIdx.x] = total;
}

// Exclusive scan of the block partials; the total is the number of distinct
// strings, checked against the caller's bound.
__global__ __launch_bounds__(kThreads) void popc_partials_kernel(int64_t *partials, int64_t nb, int64_t max_distinct,
                                                                 int64_t *count_out, int32_t *status) {
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
    *count_out = carry;
    if (carry > max_distinct && status != nullptr) atomicOr(status, RDF2V_STATUS_CAPACITY);
  }
}

__global__ __launch_bounds__(kThreads) void word_prefix_kernel(const uint64_t *__restrict__ bits, int64_t words,
                                                               const int64_t *__restrict__ partials,
                                                               int32_t *__restrict__ prefix) {
  __shared__ int32_t scratch[kThreads / kWave];
  const int64_t base = int64_t(blockIdx.x) * kWordTile;
  int32_t carry = int32_t(partials[blockIdx.x]);
  for (int i = 0; i < kWordsPerThread; ++i) {
    const int64_t round0 = base + int64_t(i) * kThreads;
    if (round0 >= words) break;  // uniform across the block
    const int64_t w = round0 + threadIdx.x;
    const int32_t x = w < words ? __popcll(bits[w]) : 0;
    int32_t tot;
    const int32_t ex = block_exclusive_scan<kThreads, int32_t>(x, scratch, tot);
    if (w < words) prefix[w] = carry + ex;
    carry += tot;
  }
}

__global__ __launch_bounds__(kThreads) void slot_id_kernel(Slot *__restrict__ table, int64_t capacity, int64_t n,
                                                           const uint64_t *__restrict__ bits,
                                                           const int32_t *__restrict__ prefix) {
  const int64_t s = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (s >= capacity) return;
  const Slot t = table[s];
  if (t.key == kEmpty || t.minpos < 0 || t.minpos >= n) return;
  const int64_t w = t.minpos >> 6;
  const uint64_t below = (uint64_t(1) << (t.minpos & 63)) - 1;
  table[s].id = prefix[w] + __popcll(bits[w] & below);
}

template <bool kPaired>
__global__ __launch_bounds__(kThreads) void assign_kernel(Seq seq, int64_t n, const Slot *__restrict__ table) {
  const int64_t q = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (q >= n) return;
  int32_t *out = seq.out[seq_col<kPaired>(q)] + seq_row<kPaired>(q);
  const int32_t s = *out;
  if (s >= 0) *out = table[s].id;
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct SeqPlan {
  int64_t n = 0;         // occurrences
  int64_t capacity = 0;  // table slots (power of two)
  int64_t words = 0;     // bitset words
  int64_t blocks = 0;    // popcount-scan blocks
  size_t table_off = 0, bits_off = 0, prefix_off = 0, partials_off = 0, end = 0;
};

SeqPlan plan_seq(int64_t n, int64_t max_distinct, size_t at) {
  SeqPlan p;
  p.n = n;
  const int64_t want = 2 * std::max<int64_t>(std::min(max_distinct, n), 32);
  p.capacity = 1;
  while (p.capacity < want) p.capacity <<= 1;
  p.words = ceil_div(n, 64);
  p.blocks = ceil_div(p.words, kWordTile);
  p.table_off = at;
  p.bits_off = p.table_off + align_up(size_t(p.capacity) * sizeof(Slot), 256);
  p.prefix_off = p.bits_off + align_up(size_t(p.words) * 8, 256);
  p.partials_off = p.prefix_off + align_up(size_t(p.words) * 4, 256);
  p.end = p.partials_off + align_up(size_t(p.blocks + 1) * 8, 256);
  return p;
}

template <bool kPaired>
rdf2v_status run_seq(const Seq &seq, const SeqPlan &p, int64_t max_distinct, char *ws, int64_t *count_out,
                     int32_t *status, hipStream_t stream) {
  Slot *table = reinterpret_cast<Slot *>(ws + p.table_off);
  uint64_t *bits = reinterpret_cast<uint64_t *>(ws + p.bits_off);
  int32_t *prefix = reinterpret_cast<int32_t *>(ws + p.prefix_off);
  int64_t *partials = reinterpret_cast<int64_t *>(ws + p.partials_off);
  const int64_t init_items = std::max(p.capacity, p.words);
  const unsigned init_blocks = unsigned(std::min<int64_t>(ceil_div(init_items, kThreads), 8192));
  init_kernel<<<dim3(init_blocks), dim3(kThreads), 0, stream>>>(table, p.capacity, bits, p.words);
  RDF2V_LAUNCH_CHECK();
  const unsigned occ_blocks = unsigned(ceil_div(p.n, kThreads));
  const unsigned slot_blocks = unsigned(ceil_div(p.capacity, kThreads));
  if (p.n > 0) {
    insert_kernel<kPaired><<<dim3(occ_blocks), dim3(kThreads), 0, stream>>>(seq, p.n, table, p.capacity - 1,
                                                                           status);
    RDF2V_LAUNCH_CHECK();
    mark_kernel<<<dim3(slot_blocks), dim3(kThreads), 0, stream>>>(
        table, p.capacity, p.n, reinterpret_cast<unsigned long long *>(bits));
    RDF2V_LAUNCH_CHECK();
    popc_count_kernel<<<dim3(unsigned(p.blocks)), dim3(kThreads), 0, stream>>>(bits, p.words, partials);
    RDF2V_LAUNCH_CHECK();
  }
  popc_partials_kernel<<<dim3(1), dim3(kThreads), 0, stream>>>(partials, p.blocks, max_distinct, count_out,
                                                               status);
  RDF2V_LAUNCH_CHECK();
  if (p.n > 0) {
    word_prefix_kernel<<<dim3(unsigned(p.blocks)), dim3(kThreads), 0, stream>>>(bits, p.words, partials, prefix);
    RDF2V_LAUNCH_CHECK();
    slot_id_kernel<<<dim3(slot_blocks), dim3(kThreads), 0, stream>>>(table, p.capacity, p.n, bits, prefix);
    RDF2V_LAUNCH_CHECK();
    assign_kernel<kPaired><<<dim3(occ_blocks), dim3(kThreads), 0, stream>>>(seq, p.n, table);
    RDF2V_LAUNCH_CHECK();
  }
  return RDF2V_OK;
}

struct VocabPlan {
  SeqPlan ent, pred;
};

VocabPlan plan_vocab(int64_t num_triples, int64_t max_entities, int64_t max_predicates) {
  VocabPlan v;
  v.ent = plan_seq(2 * num_triples, max_entities, 0);
  v.pred = plan_seq(num_triples, max_predicates, v.ent.end);
  return v;
}

}  // namespace

size_t vocabulary_workspace_bytes(int64_t num_triples, int64_t max_entities, int64_t max_predicates) {
  return plan_vocab(num_triples, max_entities, max_predicates).pred.end;
}

rdf2v_status launch_build_vocabulary(const VocabColumns &cols, int64_t num_triples, int64_t max_entities,
                                     int64_t max_predicates, int32_t *subj_ids, int32_t *pred_ids,
                                     int32_t *obj_ids, int64_t *counts_out, void *workspace,
                                     int32_t *status_dev, hipStream_t stream) {
  const VocabPlan plan = plan_vocab(num_triples, max_entities, max_predicates);
  char *ws = static_cast<char *>(workspace);
  Seq ent{{{cols.chars[0], cols.offsets[0], cols.bytes[0]}, {cols.chars[2], cols.offsets[2], cols.bytes[2]}},
          {subj_ids, obj_ids}};
  Seq pred{{{cols.chars[1], cols.offsets[1], cols.bytes[1]}, {cols.chars[1], cols.offsets[1], cols.bytes[1]}},
           {pred_ids, pred_ids}};
  const rdf2v_status st = run_seq<true>(ent, plan.ent, max_entities, ws, counts_out, status_dev, stream);
  if (st != RDF2V_OK) return st;
  return run_seq<false>(pred, plan.pred, max_predicates, ws, counts_out + 1, status_dev, stream);
}

}  // namespace rdf2v
