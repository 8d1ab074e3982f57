// Vocabulary on gfx950 (gpuRDF2vec Sec. 3.1: entities and predicates are
// tokenised to integer ids at the start of the pipeline): string triples ->
// dense ids, numbered by first appearance (entities over s_0, o_0, s_1, o_1,
// ...; predicates over p_0, p_1, ...).
//
// Per sequence (entities, then predicates), with an open-addressing table of
// 128-byte slots (linear probing, lock-free). A slot holds a 64-bit key
// (20-bit hash tag, 12-bit length, representative occurrence) claimed by one
// compare-and-swap, minpos (the smallest occurrence of its string) and an
// inline copy of strings up to 98 bytes as 7-byte words, each with a
// "written" byte on top, written by the claiming thread after its claim.
//   1. insert_kernel (fast pass): a block stages the bytes of its strings in
//      LDS with coalesced loads and hashes each string from there, keeping its
//      first eight 7-byte words in registers. For predicates, equal strings of
//      the block are grouped first (exactly, in LDS) and only each group's
//      first occurrence looks up the table. A lookup reads the key, minpos and
//      the first eight inline words of a slot at once, with 16-byte loads (one
//      round trip for strings up to 56 bytes); equal tag and length plus equal
//      inline words means the same string. A word not yet written leaves the
//      occurrence to the general pass, as do strings that are not staged or
//      too long to inline. No thread ever waits for another.
//   2. insert_general_kernel: the deferred occurrences, one thread each, from
//      global memory; equal tags are settled against the representative's
//      bytes whenever the inline copy does not decide.
//   Either pass lowers minpos (read first, atomicMin only if smaller) and
//   parks the slot index in the id output.
//   3. mark_kernel: every used slot sets bit minpos of a bitset over the
//      occurrences (the first occurrences of all strings) and writes minpos
//      to a compact per-slot array.
//   4. popcount scan: the rank of a first occurrence among all first
//      occurrences is its id (int32 prefix per 64-bit word).
//   5. slot_id_kernel turns each used slot's first occurrence (left in a
//      compact per-slot array by step 3) into its id; assign_kernel replaces
//      the parked slot indices by ids.
// The table is sized to a power of two >= 2 * the caller's bound on distinct
// strings, so probing stays short; the result does not depend on which thread
// wins a slot, only on minpos, so it is deterministic.

#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "launch.hpp"

namespace rdf2v {
namespace {

constexpr int kThreads = 256;
constexpr int kWordsPerThread = 16;
constexpr int kWordTile = kThreads * kWordsPerThread;
constexpr uint64_t kEmpty = ~uint64_t(0);
constexpr int kInlineWords = 14;
constexpr int kInlineBytes = 7 * kInlineWords;       // strings up to this long are copied into the slot
constexpr uint64_t kWritten = uint64_t(1) << 56;      // top byte of an inline word once written
constexpr uint64_t kLow56 = (uint64_t(1) << 56) - 1;
constexpr int kStageWordsPerString = 16;              // LDS stage: 64 bytes per string of the block
constexpr int64_t kLenField = 4095;                   // key length field (saturated)

struct alignas(128) Slot {
  uint64_t key;    // kEmpty, or tag << 44 | min(len, 4095) << 32 | representative occurrence
  int32_t minpos;  // smallest occurrence of the slot's string
  int32_t spare;
  uint64_t words[kInlineWords];  // inline copy: word i = bytes [7i, 7i + 7) | kWritten; 0 until written
};
static_assert(sizeof(Slot) == 128, "one slot per 128-byte line");
static_assert(offsetof(Slot, minpos) == 8 && offsetof(Slot, words) == 16, "the slot layout the init kernel writes");

struct StrCol {
  const uint8_t *chars;
  const int64_t *off;
  int64_t bytes;
};

struct Seq {
  StrCol col[2];  // occurrence q: column (q & 1), row q >> 1 when paired; else column 0, row q
  int32_t *out[2];
};

// A value that is the same in every lane, held as such (readfirstlane), so
// that a per-lane choice between two of them stays a register select.
__device__ __forceinline__ uint64_t uniform_u64(uint64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(v));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(v >> 32));
  return (uint64_t(hi) << 32) | lo;
}
__device__ __forceinline__ StrCol uniform_col(const StrCol &c) {
  return {reinterpret_cast<const uint8_t *>(uniform_u64(reinterpret_cast<uintptr_t>(c.chars))),
          reinterpret_cast<const int64_t *>(uniform_u64(reinterpret_cast<uintptr_t>(c.off))),
          int64_t(uniform_u64(uint64_t(c.bytes)))};
}

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

// Little-endian 4-byte word j of a column's chars (bytes outside it read 0).
__device__ __forceinline__ uint32_t load_word(const StrCol &c, int64_t j) {
  const int64_t p = 4 * j;
  if (p >= 0 && p + 4 <= c.bytes) return reinterpret_cast<const uint32_t *>(c.chars)[j];
  uint32_t w = 0;
  for (int b = 0; b < 4; ++b)
    if (p + b >= 0 && p + b < c.bytes) w |= uint32_t(c.chars[p + b]) << (8 * b);
  return w;
}

__device__ __forceinline__ uint64_t low_bytes_mask(int64_t r) {  // the low min(r, 7) bytes
  return r >= 7 ? kLow56 : (r <= 0 ? 0 : (uint64_t(1) << (8 * r)) - 1);
}

// Bytes [7i, 7i + 7) of a string as the low 56 bits of a word (zero past the
// end), from global memory (the general pass) or from the LDS stage (the fast
// pass; the stage is padded, so its reads need no checks).
__device__ __forceinline__ uint64_t word7_of(uint32_t a0, uint32_t a1, uint32_t a2, uint32_t sh, int64_t r) {
  const uint64_t lo = uint64_t(a0) | (uint64_t(a1) << 32);
  // (a2 << 31) << (33 - sh) is a2 << (64 - sh), and 0 for sh == 0.
  const uint64_t v = (lo >> sh) | ((uint64_t(a2) << 31) << (33 - sh));
  return v & low_bytes_mask(r);
}

// Staged strings are at most kInlineBytes long, so their offsets and lengths
// fit 32 bits. Each half of the word is one byte-aligned funnel shift of two
// staged 4-byte words.
__device__ __forceinline__ uint64_t word7_lds(const uint32_t *lds, int32_t at, int32_t len, int i) {
  const int32_t p = at + 7 * i;
  const int32_t a = p >> 2;
  const int32_t r = len - 7 * i;
  const uint32_t sh = uint32_t(p & 3);
  const uint32_t x0 = lds[a], x1 = lds[a + 1], x2 = lds[a + 2];
  uint32_t lo = __builtin_amdgcn_alignbyte(x1, x0, sh);                // bytes [p, p + 4)
  uint32_t hi = __builtin_amdgcn_alignbyte(x2, x1, sh) & 0x00ffffffu;  // bytes [p + 4, p + 7)
  if (r < 7) {
    lo &= r >= 4 ? ~0u : (r <= 0 ? 0u : (1u << (8 * r)) - 1);
    hi &= r <= 4 ? 0u : (1u << (8 * (r - 4))) - 1;
  }
  return (uint64_t(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t word7_global(const StrCol *col, int64_t start, int64_t len, int64_t i) {
  const int64_t p = start + 7 * i;
  const int64_t a = p >> 2;
  return word7_of(load_word(*col, a), load_word(*col, a + 1), load_word(*col, a + 2), uint32_t(p & 3) * 8,
                  len - 7 * i);
}

__device__ __forceinline__ uint64_t fmix64(uint64_t h) {  // MurmurHash3 finaliser
  h ^= h >> 33;
  h *= 0xff51afd7ed558ccdull;
  h ^= h >> 33;
  h *= 0xc4ceb9fe1a85ec53ull;
  h ^= h >> 33;
  return h;
}

__device__ __forceinline__ uint64_t hash_seed(int64_t len) {
  return 0x243f6a8885a308d3ull ^ (uint64_t(len) * 0x9e3779b97f4a7c15ull);
}
__device__ __forceinline__ uint64_t hash_step(uint64_t h, uint64_t w) {
  h = (h ^ w) * 0x100000001b3ull;
  return h ^ (h >> 29);
}

template <int kScope>
__device__ __forceinline__ uint64_t load_u64(const uint64_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, kScope);
}

constexpr int32_t kDeferred = -2;  // parked in the id output: left to the general pass
constexpr int kRegWords = 8;       // words of a string kept in registers and read with the key
constexpr int kBatchPairs = 3;     // further pairs of inline words read together

// The fast pass reads slots with plain 16-byte loads (the key with minpos, and
// pairs of inline words), which go through the caches and may hit a line the
// CU's L1 or the XCD's L2 fetched earlier, rather than with device-coherent
// loads (about 20% slower on the 20M-triple power-law graph), and with one
// instruction per 16 bytes rather than one per field (the many-lines-per-wave
// loads of the lookups are what the pass spends its time on). A value read
// this way can be stale but never wrong, because every field moves one way
// during the pass: the key goes from empty to its final value once (by
// compare-and-swap), each inline word from 0 to its final value once, and
// minpos only decreases. So a stale key reads as empty and the
// compare-and-swap then returns the real one; a stale word reads as not
// written and the occurrence is left to the general pass, which reads at agent
// scope; a stale minpos is larger than the real one and at worst costs an
// atomicMin that changes nothing. The checks also hold if a load were to see
// one 4-byte half of a key or word updated and the other not: a key with
// either half all ones goes through the compare-and-swap, and a word counts as
// written only when its top byte says so and its low half is not zero (a word
// whose low four bytes are zero is left to the general pass). Values left by
// earlier kernels (a previous call on the same table) are not visible: each
// kernel starts after the table was reset by the previous one.
__device__ __forceinline__ uint4 load16(const void *p) { return *reinterpret_cast<const uint4 *>(p); }
__device__ __forceinline__ uint64_t u64_of(uint32_t lo, uint32_t hi) { return uint64_t(lo) | (uint64_t(hi) << 32); }

// A slot's inline word against the string's: 0 same, 1 different, 2 not written.
__device__ __forceinline__ int word_state(uint64_t got, uint64_t want) {
  if ((got & ~kLow56) != kWritten || uint32_t(got) == 0) return 2;
  return got != (want | kWritten) ? 1 : 0;
}

// The table slot of one string (staged in LDS, at most kInlineBytes long, its
// first kRegWords words in wr) for occurrence q: found, or claimed (then its
// inline copy is written), with minpos lowered to q where needed. Returns the
// slot, kDeferred when an equal tag and length meet an inline copy not yet
// fully written (the general pass settles it), or -1 when the table is full.
__device__ __forceinline__ int32_t find_or_claim(Slot *__restrict__ table, int64_t mask, uint64_t h, int64_t q,
                                                 const uint32_t *lds, int32_t at, int64_t len,
                                                 const uint64_t (&wr)[kRegWords]) {
  const int nw = int((len + 6) / 7);
  const uint64_t ident = ((h >> 44) << 12) | uint64_t(len);
  const uint64_t mine = (ident << 32) | uint32_t(q);
  int64_t s = int64_t(h & uint64_t(mask));
  for (int64_t probe = 0; probe <= mask; ++probe, s = (s + 1) & mask) {
    Slot *sl = table + s;
    // One round trip: the key, minpos and the first kRegWords inline words.
    const uint4 k4 = load16(&sl->key);
    uint4 pr[kRegWords / 2];
#pragma unroll
    for (int j = 0; j < kRegWords / 2; ++j) pr[j] = 2 * j < nw ? load16(&sl->words[2 * j]) : make_uint4(0, 0, 0, 0);
    uint64_t key = u64_of(k4.x, k4.y);
    const int32_t minpos = int32_t(k4.z);
    if (k4.x == 0xffffffffu || k4.y == 0xffffffffu) {  // empty, or seen while it changed
      const uint64_t prev = atomicCAS(reinterpret_cast<unsigned long long *>(&sl->key),
                                      static_cast<unsigned long long>(kEmpty),
                                      static_cast<unsigned long long>(mine));
      if (prev == kEmpty) {
#pragma unroll
        for (int i = 0; i < kRegWords; ++i)
          if (i < nw) __hip_atomic_store(&sl->words[i], wr[i] | kWritten, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        for (int i = kRegWords; i < nw; ++i)
          __hip_atomic_store(&sl->words[i], word7_lds(lds, at, len, i) | kWritten, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
        atomicMin(&sl->minpos, int32_t(q));
        return int32_t(s);
      }
      key = prev;
    }
    if ((key >> 32) != ident) continue;
    // Same tag and length: compare the inline copy.
    int seen = 0;  // bit k set: some word had state k
#pragma unroll
    for (int j = 0; j < kRegWords / 2; ++j) {
      if (2 * j < nw) seen |= 1 << word_state(u64_of(pr[j].x, pr[j].y), wr[2 * j]);
      if (2 * j + 1 < nw) seen |= 1 << word_state(u64_of(pr[j].z, pr[j].w), wr[2 * j + 1]);
    }
    // Longer strings: the other words in batches whose loads are all in flight together.
#pragma unroll 1
    for (int b = kRegWords; b < nw; b += 2 * kBatchPairs) {
      uint4 more[kBatchPairs];
#pragma unroll
      for (int j = 0; j < kBatchPairs; ++j)
        more[j] = b + 2 * j < nw ? load16(&sl->words[b + 2 * j]) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int j = 0; j < kBatchPairs; ++j) {
        const int i = b + 2 * j;
        if (i < nw) seen |= 1 << word_state(u64_of(more[j].x, more[j].y), word7_lds(lds, at, len, i));
        if (i + 1 < nw) seen |= 1 << word_state(u64_of(more[j].z, more[j].w), word7_lds(lds, at, len, i + 1));
      }
    }
    if (seen & 2) continue;  // a different string
    if (seen & 4) return kDeferred;
    if (int32_t(q) < minpos) atomicMin(&sl->minpos, int32_t(q));
    return int32_t(s);
  }
  return -1;
}

// Copies the byte span [lo, hi) of each column (the block's strings of that
// column) into its part of the LDS stage when it fits, and returns for each
// column the first staged 4-byte word (base) and the number of staged words
// (count), or count -1 when the span is not staged. Every load of every column
// is issued before the first LDS store, so the stage costs one memory round
// trip. With kWide (columns whose bytes start 16-byte aligned) the copy moves
// 16-byte groups from a 16-byte aligned base, else 4-byte words; the group or
// word holding a column's last bytes is rebuilt bytewise (nothing past a
// column's end is read).
template <int kCols, int kPerCol, int kPad, int kBlock, bool kWide>
__device__ __forceinline__ void stage_spans(const Seq &seq, const int64_t (&span)[2][2], uint32_t *stage, int tid,
                                            int64_t (&base)[kCols], int32_t (&count)[kCols]) {
  constexpr int kUnit = kWide ? 4 : 1;  // words per load
  constexpr int kUnits = kPerCol / kUnit;
  constexpr int kLoads = (kUnits + kBlock - 1) / kBlock;
  using Load = typename std::conditional<kWide, uint4, uint32_t>::type;
  int32_t nunits[kCols], nwhole[kCols];  // staged units; those wholly inside the column
  Load staged[kCols][kLoads];
#pragma unroll
  for (int cc = 0; cc < kCols; ++cc) {
    const int64_t lo = span[cc][0], hi = span[cc][1];
    const bool ok = lo >= 0 && lo <= hi && hi <= seq.col[cc].bytes;
    base[cc] = ok ? ((lo >> 2) & ~int64_t(kUnit - 1)) : 0;
    const int64_t words = ok ? ((hi + 3) >> 2) - base[cc] : -1;
    count[cc] = (words >= 0 && words <= kPerCol - kPad) ? int32_t(words) : -1;
    nunits[cc] = count[cc] < 0 ? 0 : (count[cc] + kUnit - 1) / kUnit;
    const int64_t whole = (seq.col[cc].bytes >> 2) / kUnit - base[cc] / kUnit;
    nwhole[cc] = int32_t(min(int64_t(nunits[cc]), max(whole, int64_t(0))));
    const Load *src = reinterpret_cast<const Load *>(seq.col[cc].chars) + base[cc] / kUnit;
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int32_t u = tid + j * kBlock;
      if constexpr (kWide)
        staged[cc][j] = u < nwhole[cc] ? src[u] : make_uint4(0, 0, 0, 0);
      else
        staged[cc][j] = u < nwhole[cc] ? src[u] : 0u;
    }
  }
#pragma unroll
  for (int cc = 0; cc < kCols; ++cc) {
    uint32_t *dst = stage + cc * kPerCol;
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int32_t u = tid + j * kBlock;
      if (u < nwhole[cc]) reinterpret_cast<Load *>(dst)[u] = staged[cc][j];
    }
    if (tid == 0 && nwhole[cc] < nunits[cc]) {
      for (int w = 0; w < kUnit; ++w)
        dst[kUnit * nwhole[cc] + w] = load_word(seq.col[cc], base[cc] + kUnit * nwhole[cc] + w);
    }
    if (count[cc] >= 0 && tid < kPad) dst[count[cc] + tid] = 0;  // a zero tail for reads past the last string
  }
}

// Fast pass. A block stages its strings in LDS and hashes them from there.
// With kGroupEqual, equal strings of the block are grouped first and only each
// group's first occurrence, the leader, looks up the global table: a string
// repeated within a block costs one lookup, so the slots of frequent strings
// are not hammered by every occurrence. Occurrences whose strings are not
// staged or too long for an inline copy, and lookups that were deferred, are
// parked as kDeferred for the general pass.
template <bool kPaired, int kBlock, bool kGroupEqual, bool kWide>
__global__ __launch_bounds__(kBlock) void insert_kernel(Seq seq, int64_t n, Slot *__restrict__ table,
                                                        int64_t mask, int32_t *status) {
  constexpr int kCols = kPaired ? 2 : 1;
  constexpr int kWords = kBlock * kStageWordsPerString;
  constexpr int kPerCol = kWords / kCols;  // includes kPad tail words
  constexpr int kPad = 4;
  constexpr int kLocal = 2 * kBlock;  // entries of the block's LDS table of distinct strings
  __shared__ __align__(16) uint32_t stage[kWords];
  __shared__ int64_t span[2][2];  // per column: off[first row], off[last row + 1]
  // Grouping only (kGroupEqual):
  __shared__ uint64_t blk_hash[kGroupEqual ? kBlock : 1];
  __shared__ int32_t blk_at[kGroupEqual ? kBlock : 1];  // byte offset of the string in its column's stage
  __shared__ int32_t blk_len[kGroupEqual ? kBlock : 1];
  __shared__ int32_t loc_owner[kGroupEqual ? kLocal : 1];  // 1 + thread that claimed the entry, 0 if empty
  __shared__ int32_t loc_min[kGroupEqual ? kLocal : 1];    // smallest thread of the entry's group: its leader
  __shared__ int32_t loc_slot[kGroupEqual ? kLocal : 1];   // the leader's lookup result
  const int tid = threadIdx.x;
  const int64_t q0 = int64_t(blockIdx.x) * kBlock;
  const int64_t q = q0 + tid;
  const bool active = q < n;
  const int col = seq_col<kPaired>(q);
  // Both columns' descriptors are kernel arguments: read them as wave-uniform
  // values and pick per lane, rather than loading through a per-lane address
  // (one more memory round trip before the offsets).
  const StrCol c = (kPaired && col == 1) ? uniform_col(seq.col[kCols - 1]) : uniform_col(seq.col[0]);
  if constexpr (kGroupEqual) {
    for (int i = tid; i < kLocal; i += kBlock) {
      loc_owner[i] = 0;
      loc_min[i] = INT32_MAX;
    }
  }
  int64_t start = 0, len = 0;
  bool bad = false;
  if (active) {
    const int64_t row = seq_row<kPaired>(q);
    const int64_t a = c.off[row], b = c.off[row + 1];
    // The block's strings of one column are consecutive rows, so for valid
    // offsets they span [off[first row], off[last row + 1]): the first and
    // last thread of the column know those two offsets.
    const int64_t q_last = min(q0 + kBlock, n) - 1;
    if (q - q0 < kCols) span[col][0] = a;
    if (q_last - q < kCols) span[col][1] = b;
    bad = a < 0 || b < a || b > c.bytes;
    start = a;
    len = b - a;
  }
  __syncthreads();
  int64_t base[kCols];
  int32_t count[kCols];
  stage_spans<kCols, kPerCol, kPad, kBlock, kWide>(seq, span, stage, tid, base, count);
  __syncthreads();

  const int64_t my_base = (kPaired && col == 1) ? base[kCols - 1] : base[0];
  const int32_t my_count = (kPaired && col == 1) ? count[kCols - 1] : count[0];
  const bool fast = active && !bad && len <= kInlineBytes && my_count >= 0 && start >= 4 * my_base &&
                    start + len <= 4 * (my_base + my_count);
  const uint32_t *lds = stage + col * kPerCol;
  const int32_t at = fast ? int32_t(start - 4 * my_base) : -1;
  const int nw = fast ? int((len + 6) / 7) : 0;

  // Hash over the string's 7-byte words, which also form the inline copy; the
  // first kRegWords stay in registers for the lookup.
  uint64_t h = hash_seed(len);
  uint64_t wr[kRegWords];
#pragma unroll
  for (int i = 0; i < kRegWords; ++i) {
    wr[i] = i < nw ? word7_lds(lds, at, int32_t(len), i) : 0;
    if (i < nw) h = hash_step(h, wr[i]);
  }
#pragma unroll 1
  for (int i = kRegWords; i < nw; ++i) h = hash_step(h, word7_lds(lds, at, int32_t(len), i));
  h = fmix64(h);

  int32_t *out = ((kPaired && col == 1) ? seq.out[kCols - 1] : seq.out[0]) + seq_row<kPaired>(q);
  if constexpr (!kGroupEqual) {
    if (fast) {
      const int32_t r = find_or_claim(table, mask, h, q, lds, at, len, wr);
      if (r == -1 && status != nullptr) atomicOr(status, RDF2V_STATUS_CAPACITY);
      *out = r;
    } else if (active) {
      *out = kDeferred;
    }
  } else {
    blk_hash[tid] = h;
    blk_at[tid] = at;
    blk_len[tid] = int32_t(fast ? len : -1);
    __syncthreads();
    // Group equal strings of the block: an LDS table keyed by the hash, with
    // equal hashes confirmed by length and bytes; the group's smallest thread
    // (its first occurrence) is the leader.
    int e = -1;
    if (fast) {
      e = int(h & uint64_t(kLocal - 1));
      for (;;) {  // ends: the table has more entries than the block has threads
        const int cur = atomicCAS(&loc_owner[e], 0, tid + 1);
        bool same = cur == 0;
        if (!same) {
          const int o = cur - 1;
          if (blk_hash[o] == h && blk_len[o] == int32_t(len)) {
            const uint32_t *olds = stage + seq_col<kPaired>(q0 + o) * kPerCol;
            const int32_t oat = blk_at[o];
            same = true;
#pragma unroll
            for (int i = 0; i < kRegWords; ++i)
              if (i < nw) same = same && word7_lds(olds, oat, int32_t(len), i) == wr[i];
            for (int i = kRegWords; i < nw && same; ++i)
              same = word7_lds(olds, oat, int32_t(len), i) == word7_lds(lds, at, int32_t(len), i);
          }
        }
        if (same) {
          atomicMin(&loc_min[e], tid);
          break;
        }
        e = (e + 1) & (kLocal - 1);
      }
    }
    __syncthreads();
    if (fast && loc_min[e] == tid) {
      const int32_t r = find_or_claim(table, mask, h, q, lds, at, len, wr);
      loc_slot[e] = r;
      if (r == -1 && status != nullptr) atomicOr(status, RDF2V_STATUS_CAPACITY);
    }
    __syncthreads();
    if (active) *out = fast ? loc_slot[e] : kDeferred;
  }
}

// Byte equality of two strings of the same length `len` in global memory.
__device__ __forceinline__ bool same_string_global(const StrCol *ca, int64_t sa, const StrCol *cb, int64_t sb,
                                                   int64_t len) {
  const int64_t nw = (len + 6) / 7;
  for (int64_t i = 0; i < nw; ++i)
    if (word7_global(ca, sa, len, i) != word7_global(cb, sb, len, i)) return false;
  return true;
}

// General pass over the deferred occurrences (bad offsets, strings outside
// their block's stage, strings too long for an inline copy, compares left
// undecided): the same hash and table, with strings read from global memory,
// table loads at agent scope, and equal tags settled against the
// representative's bytes whenever the inline copy does not decide.
template <bool kPaired>
__global__ __launch_bounds__(kThreads) void insert_general_kernel(Seq seq, int64_t n, Slot *__restrict__ table,
                                                                  int64_t mask, int32_t *status) {
  const int64_t q = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (q >= n) return;
  const int col = seq_col<kPaired>(q);
  int32_t *out = ((kPaired && col == 1) ? seq.out[1] : seq.out[0]) + seq_row<kPaired>(q);
  if (*out != kDeferred) return;
  const StrCol cv = (kPaired && col == 1) ? seq.col[1] : seq.col[0];
  const StrCol *c = &cv;
  int bad = 0;
  int64_t start, len;
  string_range(*c, seq_row<kPaired>(q), start, len, bad);
  const int64_t words = (len + 6) / 7;
  uint64_t h = hash_seed(len);
  for (int64_t i = 0; i < words; ++i) h = hash_step(h, word7_global(c, start, len, i));
  h = fmix64(h);
  const uint64_t ident = ((h >> 44) << 12) | uint64_t(min(len, kLenField));
  const uint64_t mine = (ident << 32) | uint32_t(q);
  const int nw = len <= kInlineBytes ? int(words) : -1;  // -1: no inline copy
  int64_t s = int64_t(h & uint64_t(mask));
  int64_t found = -1;
  for (int64_t probe = 0; probe <= mask; ++probe, s = (s + 1) & mask) {
    Slot *sl = table + s;
    uint64_t k = load_u64<__HIP_MEMORY_SCOPE_AGENT>(&sl->key);
    if (k == kEmpty) {
      const uint64_t prev = atomicCAS(reinterpret_cast<unsigned long long *>(&sl->key),
                                      static_cast<unsigned long long>(kEmpty),
                                      static_cast<unsigned long long>(mine));
      if (prev == kEmpty) {
        for (int i = 0; i < nw; ++i)
          __hip_atomic_store(&sl->words[i], word7_global(c, start, len, i) | kWritten, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
        found = s;
        break;
      }
      k = prev;
    }
    if ((k >> 32) != ident) continue;
    int same = -1;
    if (nw >= 0) {
      bool unwritten = false, differ = false;
      for (int i = 0; i < nw && !differ; ++i) {
        const uint64_t w = load_u64<__HIP_MEMORY_SCOPE_AGENT>(&sl->words[i]);
        if ((w & ~kLow56) != kWritten)
          unwritten = true;
        else if (w != (word7_global(c, start, len, i) | kWritten))
          differ = true;
      }
      same = differ ? 0 : (unwritten ? -1 : 1);
    }
    if (same < 0) {
      const int64_t rep = int64_t(uint32_t(k));
      const StrCol *rc = &seq.col[seq_col<kPaired>(rep)];
      int rbad = 0;
      int64_t rstart, rlen;
      string_range(*rc, seq_row<kPaired>(rep), rstart, rlen, rbad);
      same = (rlen == len && same_string_global(c, start, rc, rstart, len)) ? 1 : 0;
    }
    if (same == 1) {
      found = s;
      break;
    }
  }
  if (found < 0) {
    *out = -1;
    if (status != nullptr) atomicOr(status, RDF2V_STATUS_CAPACITY);
  } else {
    int32_t *mp = &table[found].minpos;
    if (int32_t(q) < __hip_atomic_load(mp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) atomicMin(mp, int32_t(q));
    *out = int32_t(found);
  }
  if (bad && status != nullptr) atomicOr(status, RDF2V_STATUS_BAD_LENGTH);
}

// One 16-byte store per thread, each workgroup writing 4 KiB: the table as 16-byte groups (a
// slot is eight of them; its first holds key, minpos and spare), then the bitset, two words per
// thread.
__global__ __launch_bounds__(kThreads) void init_kernel(Slot *__restrict__ table, int64_t capacity,
                                                        uint64_t *__restrict__ bits, int64_t words) {
  constexpr int64_t kGroups = sizeof(Slot) / 16;
  const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  const int64_t table_groups = capacity * kGroups;
  if (i < table_groups) {
    const uint4 v = (i % kGroups) == 0 ? make_uint4(0xffffffffu, 0xffffffffu, uint32_t(INT32_MAX), 0u)
                                       : make_uint4(0u, 0u, 0u, 0u);
    reinterpret_cast<uint4 *>(table)[i] = v;
    return;
  }
  const int64_t w = 2 * (i - table_groups);
  if (w < words) bits[w] = 0;
  if (w + 1 < words) bits[w + 1] = 0;
}

// Every used slot's minpos was lowered by the thread that claimed it, so it is
// an occurrence in [0, n); the range check only guards the bitset. The slot's
// first occurrence (or -1 for an unused slot) also goes to the compact id
// array, so that slot_id_kernel reads 4 bytes per slot instead of the table.
__global__ __launch_bounds__(kThreads) void mark_kernel(const Slot *__restrict__ table, int64_t capacity,
                                                        int64_t n, unsigned long long *__restrict__ bits,
                                                        int32_t *__restrict__ ids) {
  const int64_t s = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (s >= capacity) return;
  const uint4 k4 = load16(&table[s].key);
  const int32_t m = int32_t(k4.z);
  const bool used = u64_of(k4.x, k4.y) != kEmpty && m >= 0 && m < n;
  ids[s] = used ? m : -1;
  if (used) atomicOr(bits + (m >> 6), 1ull << (m & 63));
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

// The id of a used slot: the rank of its first occurrence among all first
// occurrences (the compact array holds that occurrence, or -1).
__global__ __launch_bounds__(kThreads) void slot_id_kernel(int64_t capacity, const uint64_t *__restrict__ bits,
                                                           const int32_t *__restrict__ prefix,
                                                           int32_t *__restrict__ ids) {
  const int64_t s = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (s >= capacity) return;
  const int32_t m = ids[s];
  if (m < 0) return;
  const int64_t w = m >> 6;
  const uint64_t below = (uint64_t(1) << (m & 63)) - 1;
  ids[s] = prefix[w] + __popcll(bits[w] & below);
}

template <bool kPaired>
__global__ __launch_bounds__(kThreads) void assign_kernel(Seq seq, int64_t n, const int32_t *__restrict__ ids) {
  const int64_t q = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (q >= n) return;
  int32_t *out = seq.out[seq_col<kPaired>(q)] + seq_row<kPaired>(q);
  const int32_t s = *out;
  if (s >= 0) *out = ids[s];
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Fast-pass block sizes: one-wave blocks for entities (no grouping, so no
// reason to wait on other waves), 256 strings per block for predicates (more
// repeats to group).
constexpr int kFastBlockEntities = 64;
constexpr int kFastBlockPredicates = 256;

struct SeqPlan {
  int64_t n = 0;         // occurrences
  int64_t capacity = 0;  // table slots (power of two)
  int64_t words = 0;     // bitset words
  int64_t blocks = 0;    // popcount-scan blocks
  size_t table_off = 0, ids_off = 0, bits_off = 0, prefix_off = 0, partials_off = 0, end = 0;
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
  p.ids_off = p.table_off + align_up(size_t(p.capacity) * sizeof(Slot), 256);
  p.bits_off = p.ids_off + align_up(size_t(p.capacity) * 4, 256);
  p.prefix_off = p.bits_off + align_up(size_t(p.words) * 8, 256);
  p.partials_off = p.prefix_off + align_up(size_t(p.words) * 4, 256);
  p.end = p.partials_off + align_up(size_t(p.blocks + 1) * 8, 256);
  return p;
}

template <bool kPaired>
rdf2v_status run_seq(const Seq &seq, const SeqPlan &p, int64_t max_distinct, char *ws, int64_t *count_out,
                     int32_t *status, hipStream_t stream) {
  Slot *table = reinterpret_cast<Slot *>(ws + p.table_off);
  int32_t *ids = reinterpret_cast<int32_t *>(ws + p.ids_off);
  uint64_t *bits = reinterpret_cast<uint64_t *>(ws + p.bits_off);
  int32_t *prefix = reinterpret_cast<int32_t *>(ws + p.prefix_off);
  int64_t *partials = reinterpret_cast<int64_t *>(ws + p.partials_off);
  const int64_t init_items = p.capacity * int64_t(sizeof(Slot) / 16) + ceil_div(p.words, 2);
  init_kernel<<<dim3(unsigned(ceil_div(init_items, kThreads))), dim3(kThreads), 0, stream>>>(table, p.capacity,
                                                                                            bits, p.words);
  RDF2V_LAUNCH_CHECK();
  const unsigned occ_blocks = unsigned(ceil_div(p.n, kThreads));
  const unsigned slot_blocks = unsigned(ceil_div(p.capacity, kThreads));
  if (p.n > 0) {
    // Entities are mostly distinct within a block, predicates mostly repeated:
    // group equal strings only where that saves lookups.
    constexpr int kFastBlock = kPaired ? kFastBlockEntities : kFastBlockPredicates;
    const dim3 grid(unsigned(ceil_div(p.n, kFastBlock)));
    bool wide = true;  // every column's bytes start 16-byte aligned
    for (const StrCol &c : seq.col) wide = wide && (reinterpret_cast<uintptr_t>(c.chars) & 15) == 0;
    if (wide)
      insert_kernel<kPaired, kFastBlock, !kPaired, true><<<grid, dim3(kFastBlock), 0, stream>>>(seq, p.n, table,
                                                                                             p.capacity - 1, status);
    else
      insert_kernel<kPaired, kFastBlock, !kPaired, false><<<grid, dim3(kFastBlock), 0, stream>>>(seq, p.n, table,
                                                                                              p.capacity - 1, status);
    RDF2V_LAUNCH_CHECK();
    insert_general_kernel<kPaired><<<dim3(occ_blocks), dim3(kThreads), 0, stream>>>(seq, p.n, table,
                                                                                   p.capacity - 1, status);
    RDF2V_LAUNCH_CHECK();
    mark_kernel<<<dim3(slot_blocks), dim3(kThreads), 0, stream>>>(
        table, p.capacity, p.n, reinterpret_cast<unsigned long long *>(bits), ids);
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
    slot_id_kernel<<<dim3(slot_blocks), dim3(kThreads), 0, stream>>>(p.capacity, bits, prefix, ids);
    RDF2V_LAUNCH_CHECK();
    assign_kernel<kPaired><<<dim3(occ_blocks), dim3(kThreads), 0, stream>>>(seq, p.n, ids);
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
