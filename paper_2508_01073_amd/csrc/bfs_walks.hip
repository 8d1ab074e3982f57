// BFS walks on gfx950 (gpuRDF2vec Sec. 3.1): per root, a depth-limited BFS
// tree in which every reached entity has one predecessor, and one walk per
// leaf, root to leaf.
//
// The tree is the one a queue-order BFS builds: the entities of a level are
// expanded in the order they were reached, each through its out-edge records in
// CSR order, and an entity gets as parent the first (entity, record) that
// reaches it. The kernels get the same tree level-synchronously:
//   * the (entity, record) pairs of a level are numbered q = 0, 1, ... in
//     exactly that order (a block scan of the level's degrees);
//   * every pair that reaches an entity not yet in the tree offers q to that
//     entity with an atomic minimum, so the smallest q wins;
//   * the winners, in q order (a block scan), are the next level.
// Leaves are then ranked in the order reached and the first max_walks become
// rows root, V+p_1, v_1, ..., leaf.
//
// Three LDS tiers run a root in one workgroup with all its state in LDS: the
// tree above the depth limit, the level's degree prefix and an open-addressing
// hash table of the entities reached so far (tree members and this level's
// offers). Every root starts in one tier, picked from the expected tree size; a
// root whose tree outgrows a tier is abandoned there and queued for the next.
// The last pass, a persistent grid of workgroups that each own a slice of the
// workspace (per-entity stamps and offers, the tree beyond its first kTreeLds
// positions; about 36 bytes per entity), reruns the roots no tier could hold
// from scratch. All loops are bounded by the tree and level sizes or the table
// size; a workgroup never waits for another.

#include <algorithm>

#include "common.hpp"
#include "launch.hpp"

namespace rdf2v {
namespace {

constexpr int kThreads = 256;
constexpr int kLevelLds = 1024;  // levels of at most this many entities keep their prefix and row starts in LDS

struct BfsArgs {
  const int32_t *row_ptr;
  const int32_t *edges;  // (predicate, object) pairs
  const int32_t *roots;
  int32_t *tokens;
  int32_t *lens;
  int32_t *counts;
  int32_t *status;
  int32_t *queue_counts;  // [6]: lengths of the queues below, then how far each has been taken
  int32_t *queue[3];      // roots (indices into roots) LDS tier i could not hold
  char *workspace;        // slices of the workspace pass
  size_t slice_bytes;
  int64_t num_roots;
  int64_t num_edges;
  int32_t num_entities;
  int32_t num_predicates;
  int32_t depth;
  int32_t max_walks;
};

// Workspace slice of one workgroup: mark, offer (8 B), ent, parent, pred,
// level, has_child, and the degree prefix of a level (V + 1 entries).
inline size_t slice_bytes(int64_t V) {
  return align_up(size_t(V) * 4, 256) * 6 + align_up(size_t(V) * 8, 256) + align_up(size_t(V + 1) * 4, 256);
}

// Workspace: the queue counters, three queues (one int32 per root each), the slices.
inline size_t queue_bytes(int64_t num_roots) { return 256 + 3 * align_up(size_t(num_roots) * 4, 256); }

// Scratch arrays are shared by the whole workgroup and written by atomics or by
// other lanes; agent-scope relaxed accesses keep every read at L2.
__device__ __forceinline__ int32_t ld(const int32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st(int32_t *p, int32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld64(const uint64_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The tree of the current root: positions below kTreeLds live in LDS (parent
// as int16, level and "has a child" as bytes), the rest in the workgroup's
// global slice. Positions are assigned in the order entities are reached, so
// small trees and the first levels of big ones stay in LDS.
constexpr int kTreeLds = 1024;

struct Tree {
  int32_t *ent_s;
  int16_t *par_s;
  int32_t *pred_s;
  uint8_t *lev_s;
  uint8_t *child_s;
  int32_t *ent, *parent, *pred, *level, *has_child;  // global tier
  __device__ __forceinline__ int32_t get_ent(int32_t i) const { return i < kTreeLds ? ent_s[i] : ld(ent + i); }
  __device__ __forceinline__ int32_t get_par(int32_t i) const { return i < kTreeLds ? par_s[i] : ld(parent + i); }
  __device__ __forceinline__ int32_t get_pred(int32_t i) const { return i < kTreeLds ? pred_s[i] : ld(pred + i); }
  __device__ __forceinline__ int32_t get_lev(int32_t i) const { return i < kTreeLds ? lev_s[i] : ld(level + i); }
  __device__ __forceinline__ bool leaf(int32_t i) const { return (i < kTreeLds ? child_s[i] : ld(has_child + i)) == 0; }
  __device__ __forceinline__ void add(int32_t i, int32_t x, int32_t par, int32_t p, int32_t lev) const {
    if (i < kTreeLds) {
      ent_s[i] = x;
      par_s[i] = int16_t(par);  // par < i < kTreeLds
      pred_s[i] = p;
      lev_s[i] = uint8_t(lev);
      child_s[i] = 0;
    } else {
      st(ent + i, x);
      st(parent + i, par);
      st(pred + i, p);
      st(level + i, lev);
      st(has_child + i, 0);
    }
  }
  __device__ __forceinline__ void set_child(int32_t i) const {
    if (i < kTreeLds) child_s[i] = 1;
    else st(has_child + i, 1);
  }
};

// ---------------------------------------------------------------------------
// LDS tiers: one root at a time per workgroup, all state in LDS.

// Three LDS tiers of growing capacity and LDS footprint: one wave per root
// (about 6.3 KB of LDS, 24 workgroups per CU), 256 threads (about 25 KB, 6
// per CU) and 512 threads (about 50 KB, 3 per CU). A root goes to the next
// tier when it outgrows one. All keep VGPRs <= 80 for six waves per SIMD (the
// big tier spills a few registers for its four rounds).
struct TinyTier {
  static constexpr int kThreads = 64;
  static constexpr int kRounds = 2;
  static constexpr int kLog = 9;
  static constexpr int kCap = 384;
  static constexpr int kTreeCap = 96;
  static constexpr int kWavesPerSimd = 6;
};
struct SmallTier {
  static constexpr int kThreads = 256;
  static constexpr int kRounds = 2;     // rounds of kThreads pairs whose records are loaded together
  static constexpr int kLog = 11;       // hash table of 2^kLog slots
  static constexpr int kCap = 1536;     // most entities a root may reach here
  static constexpr int kTreeCap = 384;  // most of them above the depth limit (kept as tree nodes)
  static constexpr int kWavesPerSimd = 6;
  static constexpr int kPerCu = 6;
};
struct BigTier {
  static constexpr int kThreads = 512;
  static constexpr int kRounds = 4;
  static constexpr int kLog = 12;
  static constexpr int kCap = 3072;
  static constexpr int kTreeCap = 768;
  static constexpr int kWavesPerSimd = 6;
  static constexpr int kPerCu = 3;
};
constexpr int32_t kFreeSlot = -1;
constexpr uint32_t kNoOffer = 0xFFFFFFFFu;

// Fibonacci hashing of an entity id to one of 2^kLog slots.
template <int kLog>
__device__ __forceinline__ int32_t entity_slot(int32_t x) {
  return int32_t((uint32_t(x) * 0x9E3779B1u) >> (32 - kLog));
}

// Inclusive prefix sum over the 64 lanes of a wave with DPP moves: shifts by
// 1, 2, 4 and 8 lanes inside each row of 16, then the last lane of row 0 and of
// row 2 added to rows 1 and 3, then the last lane of row 1 added to rows 2 and
// 3 (the row-broadcast scan of AMD's GCN cross-lane notes). Lanes with no
// source lane or in masked rows add 0.
__device__ __forceinline__ int32_t wave_inclusive_sum(int32_t x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15 into rows 1 and 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31 into rows 2 and 3
  return x;
}

__device__ __forceinline__ int32_t wave_sum(int32_t v) {
  return __builtin_amdgcn_readlane(wave_inclusive_sum(v), kWave - 1);
}

__device__ __forceinline__ int32_t wave_index() { return __builtin_amdgcn_readfirstlane(int32_t(threadIdx.x) / kWave); }

// Set bits of a wave-wide mask below the calling lane.
__device__ __forceinline__ int32_t lanes_below(uint64_t b) {
  return int32_t(__builtin_amdgcn_mbcnt_hi(uint32_t(b >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(b), 0u)));
}

// Exclusive prefix sum over the block (one value per thread) and its total.
// One barrier; scratch holds NT/64 ints and must not be written again before
// the next barrier (callers alternate between two scratch buffers).
template <int NT>
__device__ __forceinline__ int32_t block_scan(int32_t x, int32_t *scratch, int32_t &total) {
  constexpr int W = NT / kWave;
  const int32_t inc = wave_inclusive_sum(x);
  if constexpr (W == 1) {
    total = __builtin_amdgcn_readlane(inc, kWave - 1);
    return inc - x;
  } else {
    const int lane = lane_id();
    const int32_t w = wave_index();
    if (lane == kWave - 1) scratch[w] = inc;
    __syncthreads();
    const int32_t waves = wave_inclusive_sum(lane < W ? scratch[lane] : 0);
    total = __builtin_amdgcn_readlane(waves, W - 1);
    return (w > 0 ? __builtin_amdgcn_readlane(waves, w - 1) : 0) + inc - x;
  }
}

// Ranks, in pair order, the flagged pairs of a chunk whose round k holds pair
// c0 + k*NT + threadIdx.x: rank[k] counts the flagged pairs before it in the
// chunk; `total` is their number. One barrier; cnt_s holds R * NT/64 ints and
// is reused like the scratch of block_scan.
template <int NT, int R>
__device__ __forceinline__ void rank_chunk(uint32_t mask, int32_t (&rank)[R], int32_t &total, int32_t *cnt_s) {
  constexpr int W = NT / kWave;
  static_assert(R * W <= kWave, "one count per lane");
  const int lane = lane_id();
  const int32_t w = wave_index();
  uint64_t b[R];
#pragma unroll
  for (int k = 0; k < R; ++k) b[k] = __ballot((mask >> k) & 1u);
  // counts in pair order: round-major, then wave
  if (lane == 0) {
#pragma unroll
    for (int k = 0; k < R; ++k) cnt_s[k * W + w] = __popcll(b[k]);
  }
  __syncthreads();
  const int32_t inc = wave_inclusive_sum(lane < R * W ? cnt_s[lane] : 0);
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int32_t idx = k * W + w;
    rank[k] = (idx > 0 ? __builtin_amdgcn_readlane(inc, idx - 1) : 0) + lanes_below(b[k]);
  }
  total = __builtin_amdgcn_readlane(inc, R * W - 1);
}

// Table entries: key = entity, value = 0 for a tree member, else 1 + the
// smallest pair index of the current level that reached it. Every entity
// inserted during a level's offers has a winning pair, so after the level the
// entry count is the tree size.
//
// Entities at the depth limit are leaves: they are not stored as tree nodes.
// Their pairs are walked twice more instead, once to mark which nodes of the
// level above get a child, and once, after the stored leaves are ranked, to
// write their walks in pair order.
//
// The pairs of a level are taken in chunks of R rounds of NT consecutive
// pairs; a thread loads the records of its R pairs together. A level of at
// most one chunk keeps its records (and winners) in registers for all its
// passes.
//
// Without in_queue, workgroup b takes roots b, b + G, ...; with it, the
// workgroups take its in_count entries one at a time through the counter
// `taken`. Roots the tier cannot hold are appended to out_queue.
template <int NT, int R, int kLog, int kCap, int kTreeCap, int kWpe>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(kWpe))) void bfs_lds_kernel(
    const BfsArgs a, const int32_t *in_queue, const int32_t *in_count, int32_t *taken, int32_t *out_queue,
    int32_t *out_count) {
  constexpr int kSlots = 1 << kLog;
  constexpr int32_t kChunk = NT * R;
  static_assert(kCap < kSlots && kTreeCap <= kCap && kTreeCap <= 32767, "table and tree sizes");
  static_assert(kSlots % (4 * NT) == 0, "the table is cleared four slots per thread at a time");
  static_assert(R <= 32, "win masks are 32-bit");
  __shared__ int32_t scan_scratch[2][R * (NT / kWave)];  // alternated between block-wide scans
  __shared__ __align__(16) int32_t h_key[kSlots];
  __shared__ __align__(16) uint32_t h_val[kSlots];
  __shared__ int32_t t_ent[kTreeCap];
  __shared__ int32_t t_pred[kTreeCap];
  __shared__ int16_t t_par[kTreeCap];
  __shared__ uint8_t t_lev[kTreeCap];
  __shared__ uint8_t t_child[kTreeCap];
  __shared__ int32_t t_lo[kTreeCap];        // CSR row start of each tree node
  __shared__ int32_t t_deg[kTreeCap];       // and its out-degree (0 for a bad row)
  __shared__ int32_t dpre_s[kTreeCap + 1];  // degree prefix of the level being expanded
  __shared__ int32_t used_s;                // table entries
  __shared__ int32_t overflow_s;
  __shared__ int32_t next_s;
  const int t = threadIdx.x;
  const int32_t V = a.num_entities;
  const uint32_t E = uint32_t(a.num_edges);
  const int64_t width = 2 * int64_t(a.depth) + 1;
  const int2 *edges = reinterpret_cast<const int2 *>(a.edges);

  // Slot of x, inserting it if absent (then `inserted` is incremented); -1
  // when the table is full (the root is then left to the next tier). The
  // entry count is checked against kCap once all offers of a level are in.
  auto claim = [&](int32_t x, int32_t &inserted) -> int32_t {
    int32_t s = entity_slot<kLog>(x);
    for (int n = 0; n < kSlots; ++n) {
      const int32_t k = __hip_atomic_load(h_key + s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      if (k == x) return s;
      if (k == kFreeSlot) {
        const int32_t old = atomicCAS(h_key + s, kFreeSlot, x);
        if (old == kFreeSlot) {
          ++inserted;
          return s;
        }
        if (old == x) return s;
      }
      s = (s + 1) & (kSlots - 1);
    }
    overflow_s = 1;
    return -1;
  };
  auto find = [&](int32_t x) -> int32_t {
    int32_t s = entity_slot<kLog>(x);
    for (int n = 0; n < kSlots; ++n) {
      const int32_t k = h_key[s];
      if (k == x) return s;
      if (k == kFreeSlot) break;
      s = (s + 1) & (kSlots - 1);
    }
    return -1;
  };

  int flags = 0;
  int32_t phase = 0;
  auto scratch = [&]() -> int32_t * { return scan_scratch[phase ^= 1]; };
  const int64_t n_in = in_queue != nullptr ? int64_t(*in_count) : a.num_roots;
  if (int64_t(blockIdx.x) >= n_in) return;  // uniform; an empty queue costs one load per workgroup
  for (int64_t k_in = blockIdx.x;; k_in += gridDim.x) {
    if (in_queue != nullptr) {  // uniform
      if (t == 0) next_s = atomicAdd(taken, 1);
      __syncthreads();
      k_in = next_s;
      __syncthreads();
    }
    if (k_in >= n_in) break;
    const int64_t r = in_queue != nullptr ? int64_t(in_queue[k_in]) : k_in;
    const int32_t root = a.roots[r];
    if (uint32_t(root) >= uint32_t(V)) {
      if (t == 0) a.counts[r] = 0;
      flags |= RDF2V_STATUS_ID_OUT_OF_RANGE;
      continue;  // uniform: every lane skips the same root
    }
    for (int i = t; i < kSlots / 4; i += NT) {
      reinterpret_cast<int4 *>(h_key)[i] = make_int4(kFreeSlot, kFreeSlot, kFreeSlot, kFreeSlot);
      reinterpret_cast<uint4 *>(h_val)[i] = make_uint4(kNoOffer, kNoOffer, kNoOffer, kNoOffer);
    }
    __syncthreads();
    if (t == 0) {
      const int32_t lo = a.row_ptr[root], hi = a.row_ptr[root + 1];
      const bool ok = uint32_t(lo) <= uint32_t(hi) && uint32_t(hi) <= E;
      if (!ok) flags |= RDF2V_STATUS_BAD_CSR;
      t_lo[0] = lo;
      t_deg[0] = ok ? hi - lo : 0;
      const int32_t s0 = entity_slot<kLog>(root);
      h_key[s0] = root;
      h_val[s0] = 0;
      used_s = 1;
      overflow_s = 0;
      t_ent[0] = root;
      t_pred[0] = -1;
      t_par[0] = -1;
      t_lev[0] = 0;
      t_child[0] = 0;
    }
    __syncthreads();
    int32_t lb = 0, le = 1;      // the level being expanded: tree nodes [lb, le)
    int32_t nlev = 0, total = 0;  // its size and its number of (entity, record) pairs
    int32_t last_wins = 0;       // entities reached at the depth limit
    bool overflow = false;
    // The thread's pairs of the chunk at c0 (round k: pair c0 + k*NT + t): level
    // entity index (-1 past the end), record, and table slot of the record's
    // entity (-1 if none).
    int32_t node_k[R];
    int2 rec_k[R];
    int32_t slot_k[R];
    auto load_chunk = [&](int32_t c0) {
#pragma unroll
      for (int k = 0; k < R; ++k) {
        node_k[k] = -1;
        rec_k[k] = make_int2(0, -1);
      }
      if (c0 + wave_index() * kWave >= total) return;  // uniform: no pair of this wave in the chunk
      // largest i with dpre[i] <= q, by halving steps from the top bit of nlev
      int32_t lo[R];
#pragma unroll
      for (int k = 0; k < R; ++k) lo[k] = 0;
      for (int32_t step = int32_t(1u << (31 - __builtin_clz(uint32_t(nlev)))); step > 0; step >>= 1) {
#pragma unroll
        for (int k = 0; k < R; ++k) {
          const int32_t m = lo[k] + step;
          if (m < nlev && dpre_s[m] <= c0 + k * NT + t) lo[k] = m;
        }
      }
#pragma unroll
      for (int k = 0; k < R; ++k) {
        const int32_t q = c0 + k * NT + t;
        node_k[k] = q < total ? lo[k] : -1;
        rec_k[k] = q < total ? edges[uint32_t(t_lo[lb + lo[k]] + (q - dpre_s[lo[k]]))] : make_int2(0, -1);
      }
    };
    // Bit k set: the thread's round-k pair reaches its entity first. With
    // `known`, slot_k holds the slots from this chunk's offers; else they are
    // looked up.
    auto winners = [&](int32_t c0, bool known) -> uint32_t {
      uint32_t m = 0;
#pragma unroll
      for (int k = 0; k < R; ++k) {
        if (!known) slot_k[k] = node_k[k] >= 0 && uint32_t(rec_k[k].y) < uint32_t(V) ? find(rec_k[k].y) : -1;
        if (slot_k[k] >= 0 && h_val[slot_k[k]] == uint32_t(c0 + k * NT + t) + 1u) m |= 1u << k;
      }
      return m;
    };
    uint32_t last_mask = 0;  // winners of a one-chunk last level
    for (int32_t lev = 0; lev < a.depth && lb < le; ++lev) {
      nlev = le - lb;  // le <= kTreeCap
      // Degree prefix of the level (rows were read when its nodes were added).
      int32_t carry = 0;
      for (int32_t c0 = lb; c0 < le; c0 += NT) {
        const int32_t i = c0 + t;
        int32_t tot;
        const int32_t ex = block_scan<NT>(i < le ? t_deg[i] : 0, scratch(), tot);
        if (i < le) dpre_s[i - lb] = carry + ex;
        carry += tot;
      }
      total = carry;
      if (t == 0) dpre_s[nlev] = total;
      __syncthreads();
      const bool one_chunk = total <= kChunk;  // uniform: records stay in registers
      const bool last = lev + 1 == a.depth;
      // Offers (tree members hold 0 and ignore them).
      bool full = false;
      int32_t inserted = 0;
      for (int32_t c0 = 0; c0 < total && !full; c0 += kChunk) {
        load_chunk(c0);
#pragma unroll
        for (int k = 0; k < R; ++k) {
          slot_k[k] = -1;
          if (full || node_k[k] < 0) continue;
          const int32_t x = rec_k[k].y;
          if (uint32_t(x) >= uint32_t(V)) {
            flags |= RDF2V_STATUS_ID_OUT_OF_RANGE;
            continue;
          }
          const int32_t s = claim(x, inserted);
          if (s < 0) {
            full = true;
          } else {
            slot_k[k] = s;
            atomicMin(h_val + s, uint32_t(c0 + k * NT + t) + 1u);
          }
        }
      }
      inserted = wave_sum(inserted);
      if (lane_id() == 0 && inserted > 0) atomicAdd(&used_s, inserted);
      __syncthreads();
      if (overflow_s || used_s > (last ? kCap : kTreeCap)) {  // uniform
        overflow = true;
        break;
      }
      if (last) {
        // Nodes of this level with a winning pair are not leaves.
        int32_t n_wins = 0;
        for (int32_t c0 = 0; c0 < total; c0 += kChunk) {
          if (!one_chunk) load_chunk(c0);
          const uint32_t m = winners(c0, one_chunk);
#pragma unroll
          for (int k = 0; k < R; ++k)
            if (m & (1u << k)) t_child[lb + node_k[k]] = 1;
          n_wins += __popc(m);
          last_mask = m;
        }
        {
          int32_t all;
          (void)block_scan<NT>(n_wins, scratch(), all);
          last_wins = all;
        }
        break;  // lb, le, nlev, total (and a one-chunk level's records) stay for the rows
      }
      // Winners in pair order become the next level.
      int32_t added = 0;
      for (int32_t c0 = 0; c0 < total; c0 += kChunk) {
        if (!one_chunk) load_chunk(c0);
        int32_t rank[R], tot, row_lo_k[R], row_hi_k[R];
        const uint32_t m = winners(c0, one_chunk);
#pragma unroll
        for (int k = 0; k < R; ++k) {  // the new nodes' rows, in flight across the ranking
          row_lo_k[k] = row_hi_k[k] = 0;
          if (m & (1u << k)) {
            row_lo_k[k] = a.row_ptr[rec_k[k].y];
            row_hi_k[k] = a.row_ptr[rec_k[k].y + 1];
          }
        }
        rank_chunk<NT, R>(m, rank, tot, scratch());
#pragma unroll
        for (int k = 0; k < R; ++k) {
          if (m & (1u << k)) {
            const int32_t pos = le + added + rank[k];  // < used_s <= kTreeCap
            const int32_t node = lb + node_k[k];
            const bool ok = uint32_t(row_lo_k[k]) <= uint32_t(row_hi_k[k]) && uint32_t(row_hi_k[k]) <= E;
            if (!ok) flags |= RDF2V_STATUS_BAD_CSR;
            t_ent[pos] = rec_k[k].y;
            t_pred[pos] = rec_k[k].x;
            t_par[pos] = int16_t(node);
            t_lev[pos] = uint8_t(lev + 1);
            t_child[pos] = 0;
            t_lo[pos] = row_lo_k[k];
            t_deg[pos] = ok ? row_hi_k[k] - row_lo_k[k] : 0;
            t_child[node] = 1;
            h_val[slot_k[k]] = 0;
          }
        }
        added += tot;
      }
      lb = le;
      le += added;
      __syncthreads();
    }
    if (overflow) {
      if (t == 0) out_queue[atomicAdd(out_count, 1)] = int32_t(r);
      continue;  // the clearing loop of the next root starts after this root's last barrier
    }
    // Walk rows: root, then the tokens of `node` and its ancestors up to level h.
    auto write_path = [&](int32_t *row, int32_t node, int32_t h) {
      for (int32_t step = h; step >= 1; --step) {
        row[2 * step] = t_ent[node];
        row[2 * step - 1] = V + t_pred[node];
        node = t_par[node];
      }
      row[0] = root;
    };
    // Leaves in the order reached, the stored tree nodes first: the first
    // max_walks become walks.
    int32_t leaves = 0;
    for (int32_t c0 = 0; c0 < le; c0 += NT) {
      const int32_t i = c0 + t;
      const int32_t leaf = i < le ? int32_t(t_child[i] == 0) : 0;
      int32_t tot;
      const int32_t ex = block_scan<NT>(leaf, scratch(), tot);
      const int32_t idx = leaves + ex;
      if (leaf && idx < a.max_walks) {
        const int32_t h = t_lev[i];
        int32_t *row = a.tokens + (r * a.max_walks + idx) * width;
        write_path(row, i, h);
        for (int64_t j = 2 * int64_t(h) + 1; j < width; ++j) row[j] = -1;
        a.lens[r * a.max_walks + idx] = 2 * h + 1;
      }
      leaves += tot;
    }
    // Then the entities at the depth limit, in pair order.
    if (last_wins > 0 && leaves < a.max_walks) {
      const bool one_chunk = total <= kChunk;
      int32_t added = 0;
      for (int32_t c0 = 0; c0 < total; c0 += kChunk) {
        uint32_t m = last_mask;
        if (!one_chunk) {
          load_chunk(c0);
          m = winners(c0, false);
        }
        int32_t rank[R], tot;
        rank_chunk<NT, R>(m, rank, tot, scratch());
#pragma unroll
        for (int k = 0; k < R; ++k) {
          const int32_t idx = leaves + added + rank[k];
          if ((m & (1u << k)) && idx < a.max_walks) {
            int32_t *row = a.tokens + (r * a.max_walks + idx) * width;
            row[2 * a.depth] = rec_k[k].y;
            row[2 * a.depth - 1] = V + rec_k[k].x;
            write_path(row, lb + node_k[k], a.depth - 1);
            a.lens[r * a.max_walks + idx] = int32_t(width);
          }
        }
        added += tot;
        if (leaves + added >= a.max_walks) break;  // uniform
      }
    }
    leaves += last_wins;
    if (t == 0) {
      a.counts[r] = min(leaves, a.max_walks);
      if (leaves > a.max_walks) flags |= RDF2V_STATUS_CAPACITY;
    }
    __syncthreads();  // the LDS is reused by the next root
  }
  if (flags && a.status != nullptr) atomicOr(a.status, flags);
}

__global__ void bfs_queue_reset_kernel(int32_t *queue_counts) {
  if (threadIdx.x < 6) queue_counts[threadIdx.x] = 0;
}

// ---------------------------------------------------------------------------
// Workspace pass: the roots no tier could hold, with per-workgroup slices of
// the workspace.

__global__ __launch_bounds__(kThreads) void bfs_walks_kernel(const BfsArgs a) {
  __shared__ int32_t scan_scratch[kThreads / kWave];
  __shared__ int32_t dpre_s[kLevelLds + 1];  // degree prefix of the current level (small levels)
  __shared__ int32_t rowlo_s[kLevelLds];     // row start of each of its entities
  __shared__ int32_t t_ent[kTreeLds];
  __shared__ int32_t t_pred[kTreeLds];
  __shared__ int16_t t_par[kTreeLds];
  __shared__ uint8_t t_lev[kTreeLds];
  __shared__ uint8_t t_child[kTreeLds];
  const int t = threadIdx.x;
  const int32_t V = a.num_entities;
  const uint32_t E = uint32_t(a.num_edges);
  const int64_t width = 2 * int64_t(a.depth) + 1;
  const int2 *edges = reinterpret_cast<const int2 *>(a.edges);

  char *base = a.workspace + size_t(blockIdx.x) * a.slice_bytes;
  const size_t a4 = align_up(size_t(V) * 4, 256), a8 = align_up(size_t(V) * 8, 256);
  int32_t *mark = reinterpret_cast<int32_t *>(base);
  uint64_t *offer = reinterpret_cast<uint64_t *>(base + a4);
  int32_t *dpre = reinterpret_cast<int32_t *>(base + 6 * a4 + a8);
  const Tree tree{t_ent,
                  t_par,
                  t_pred,
                  t_lev,
                  t_child,
                  reinterpret_cast<int32_t *>(base + a4 + a8),
                  reinterpret_cast<int32_t *>(base + 2 * a4 + a8),
                  reinterpret_cast<int32_t *>(base + 3 * a4 + a8),
                  reinterpret_cast<int32_t *>(base + 4 * a4 + a8),
                  reinterpret_cast<int32_t *>(base + 5 * a4 + a8)};

  const int32_t queued = a.queue_counts[2];
  if (int32_t(blockIdx.x) >= queued) return;  // uniform, before any barrier
  // Each workgroup initialises its own slice once per call.
  for (int32_t v = t; v < V; v += kThreads) {
    st(mark + v, -1);
    __hip_atomic_store(offer + v, ~uint64_t(0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();

  uint32_t stamp = 0xFFFFFFFEu;  // falls by one per (root, level) of this workgroup
  int flags = 0;
  for (int32_t k = blockIdx.x; k < queued; k += gridDim.x) {
    const int64_t r = a.queue[2][k];
    const int32_t root = a.roots[r];
    const int32_t mark_id = int32_t(r);
    if (uint32_t(root) >= uint32_t(V)) {
      if (t == 0) a.counts[r] = 0;
      flags |= RDF2V_STATUS_ID_OUT_OF_RANGE;
      continue;  // uniform: every lane skips the same root
    }
    if (t == 0) {
      tree.add(0, root, -1, -1, 0);
      st(mark + root, mark_id);
    }
    int32_t lb = 0, le = 1;
    __syncthreads();
    for (int32_t lev = 0; lev < a.depth && lb < le; ++lev) {
      // Degree prefix of the level's entities (their (entity, record) pairs are
      // numbered in order), with the row starts, in LDS for small levels.
      const int32_t nlev = le - lb;
      const bool small = nlev <= kLevelLds;  // uniform across the block
      int32_t carry = 0;
      for (int32_t c0 = lb; c0 < le; c0 += kThreads) {
        const int32_t i = c0 + t;
        int32_t d = 0, lo = 0;
        if (i < le) {
          const int32_t u = tree.get_ent(i);
          lo = a.row_ptr[u];
          const int32_t hi = a.row_ptr[u + 1];
          if (uint32_t(lo) <= uint32_t(hi) && uint32_t(hi) <= E) d = hi - lo;
          else flags |= RDF2V_STATUS_BAD_CSR;
        }
        int32_t tot;
        const int32_t ex = block_exclusive_scan<kThreads>(d, scan_scratch, tot);
        if (i < le) {
          if (small) {
            dpre_s[i - lb] = carry + ex;
            rowlo_s[i - lb] = lo;
          } else {
            st(dpre + (i - lb), carry + ex);
          }
        }
        carry += tot;
      }
      const int32_t total = carry;
      if (t == 0) {
        if (small) dpre_s[nlev] = total;
        else st(dpre + nlev, total);
      }
      // Pair q of the level: the level entity (index lo_i) it belongs to and the
      // pair's record index.
      auto locate = [&](int32_t q, int32_t &lo_i, uint32_t &j) {
        lo_i = 0;
        int32_t hi_i = nlev;  // largest i with dpre[i] <= q
        if (small) {
          while (hi_i - lo_i > 1) {
            const int32_t mid = (lo_i + hi_i) >> 1;
            if (dpre_s[mid] <= q) lo_i = mid;
            else hi_i = mid;
          }
          j = uint32_t(rowlo_s[lo_i] + (q - dpre_s[lo_i]));
        } else {
          while (hi_i - lo_i > 1) {
            const int32_t mid = (lo_i + hi_i) >> 1;
            if (ld(dpre + mid) <= q) lo_i = mid;
            else hi_i = mid;
          }
          const int32_t u = tree.get_ent(lb + lo_i);
          j = uint32_t(a.row_ptr[u] + (q - ld(dpre + lo_i)));
        }
      };
      --stamp;
      const uint64_t hi_bits = uint64_t(stamp) << 32;
      __syncthreads();
      // Offers: pair q reaches x; entities already in this root's tree are skipped.
      for (int32_t q = t; q < total; q += kThreads) {
        int32_t lo_i;
        uint32_t j;
        locate(q, lo_i, j);
        const int32_t x = edges[j].y;
        if (uint32_t(x) >= uint32_t(V)) {
          flags |= RDF2V_STATUS_ID_OUT_OF_RANGE;
          continue;
        }
        if (ld(mark + x) != mark_id) atomicMin(reinterpret_cast<unsigned long long *>(offer + x),
                                               (unsigned long long)(hi_bits | uint32_t(q)));
      }
      __syncthreads();
      // Winners in q order become the next level.
      int32_t added = 0;
      for (int32_t c0 = 0; c0 < total; c0 += kThreads) {
        const int32_t q = c0 + t;
        int32_t win = 0, x = 0, p = 0, node = 0;
        if (q < total) {
          int32_t lo_i;
          uint32_t j;
          locate(q, lo_i, j);
          node = lb + lo_i;
          const int2 rec = edges[j];
          p = rec.x;
          x = rec.y;
          if (uint32_t(x) < uint32_t(V)) win = ld64(offer + x) == (hi_bits | uint32_t(q));
        }
        int32_t tot;
        const int32_t ex = block_exclusive_scan<kThreads>(win, scan_scratch, tot);
        if (win) {
          const int32_t pos = le + added + ex;
          tree.add(pos, x, node, p, lev + 1);
          tree.set_child(node);
          st(mark + x, mark_id);
        }
        added += tot;
      }
      lb = le;
      le += added;
      __syncthreads();
    }
    // Leaves in the order reached: the first max_walks become walks.
    int32_t leaves = 0;
    for (int32_t c0 = 0; c0 < le; c0 += kThreads) {
      const int32_t i = c0 + t;
      const int32_t leaf = i < le ? int32_t(tree.leaf(i)) : 0;
      int32_t tot;
      const int32_t ex = block_exclusive_scan<kThreads>(leaf, scan_scratch, tot);
      const int32_t idx = leaves + ex;
      if (leaf && idx < a.max_walks) {
        const int32_t h = tree.get_lev(i);
        int32_t *row = a.tokens + (r * a.max_walks + idx) * width;
        int32_t node = i;
        for (int32_t step = h; step >= 1; --step) {
          row[2 * step] = tree.get_ent(node);
          row[2 * step - 1] = V + tree.get_pred(node);
          node = tree.get_par(node);
        }
        row[0] = root;
        for (int64_t j = 2 * int64_t(h) + 1; j < width; ++j) row[j] = -1;
        a.lens[r * a.max_walks + idx] = 2 * h + 1;
      }
      leaves += tot;
    }
    if (t == 0) {
      a.counts[r] = min(leaves, a.max_walks);
      if (leaves > a.max_walks) flags |= RDF2V_STATUS_CAPACITY;
    }
    __syncthreads();
  }
  if (flags && a.status != nullptr) atomicOr(a.status, flags);
}

}  // namespace

template <class T>
void launch_tier(const BfsArgs &a, const int32_t *in_q, const int32_t *in_c, int32_t *taken, int32_t *out_q,
                 int32_t *out_c, int64_t grid, hipStream_t stream) {
  bfs_lds_kernel<T::kThreads, T::kRounds, T::kLog, T::kCap, T::kTreeCap, T::kWavesPerSimd>
      <<<dim3(unsigned(grid)), dim3(T::kThreads), 0, stream>>>(a, in_q, in_c, taken, out_q, out_c);
}

// The tier every root starts in: the smallest whose capacity is at least twice
// the expected tree size, 1 + d + ... + d^depth for the mean out-degree d
// (at most V). Only the speed depends on this choice: a root that outgrows a
// tier is rerun by the next.
int bfs_first_tier(int32_t num_entities, int64_t num_edges, int64_t num_roots, int32_t depth) {
  const double d = num_entities > 0 ? double(num_edges) / double(num_entities) : 0.0;
  double est = 1.0, level = 1.0;
  for (int32_t l = 0; l < depth && est < 1e9; ++l) {
    level *= d;
    est += level;
  }
  est = std::min(est, double(num_entities));
  int first = 2.0 * est <= TinyTier::kCap ? 0 : 2.0 * est <= SmallTier::kCap ? 1 : 2;
  // When a tier with more threads per root holds every root on the chip at
  // once, the extra threads shorten each root instead of waiting.
  int cus = 0, dev = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    cus = 0;
  if (first < 2 && num_roots <= int64_t(cus) * BigTier::kPerCu) first = 2;
  else if (first < 1 && num_roots <= int64_t(cus) * SmallTier::kPerCu) first = 1;
  return first;
}

int64_t bfs_walks_grid(int32_t num_entities, int64_t num_roots) {
  // Workspace pass: enough workgroups to fill the chip, at most ~4 GiB of slices.
  const int64_t per = int64_t(slice_bytes(num_entities));
  int64_t g = std::max<int64_t>(1, (int64_t(1) << 32) / std::max<int64_t>(per, 1));
  g = std::min<int64_t>(g, 2048);
  g = std::min<int64_t>(g, std::max<int64_t>(num_roots, 1));
  return g;
}

size_t bfs_walks_workspace_bytes(int32_t num_entities, int64_t num_roots) {
  return queue_bytes(num_roots) + size_t(bfs_walks_grid(num_entities, num_roots)) * slice_bytes(num_entities);
}

rdf2v_status launch_bfs_walks(const int32_t *row_ptr, const int32_t *edges, int64_t num_edges,
                              int32_t num_entities, int32_t num_predicates, const int32_t *roots,
                              int64_t num_roots, int32_t depth, int32_t max_walks, int32_t *tokens_out,
                              int32_t *len_out, int32_t *counts_out, void *workspace, int32_t *status_dev,
                              hipStream_t stream) {
  if (num_roots == 0) return RDF2V_OK;
  char *ws = static_cast<char *>(workspace);
  BfsArgs a;
  a.row_ptr = row_ptr;
  a.edges = edges;
  a.roots = roots;
  a.tokens = tokens_out;
  a.lens = len_out;
  a.counts = counts_out;
  a.status = status_dev;
  a.queue_counts = reinterpret_cast<int32_t *>(ws);
  for (int i = 0; i < 3; ++i) a.queue[i] = reinterpret_cast<int32_t *>(ws + 256 + i * align_up(size_t(num_roots) * 4, 256));
  a.workspace = ws + queue_bytes(num_roots);
  a.slice_bytes = slice_bytes(num_entities);
  a.num_roots = num_roots;
  a.num_edges = num_edges;
  a.num_entities = num_entities;
  a.num_predicates = num_predicates;
  a.depth = depth;
  a.max_walks = max_walks;
  bfs_queue_reset_kernel<<<1, kWave, 0, stream>>>(a.queue_counts);
  RDF2V_LAUNCH_CHECK();
  // The first tier takes every root, one per workgroup (the hardware hands
  // out roots as workgroups finish; at most 2^20 workgroups); a later tier
  // runs a grid over its input queue, whose length only the device knows, and
  // its workgroups past the end return at once.
  const int first = bfs_first_tier(num_entities, num_edges, num_roots, depth);
  for (int tier = first; tier < 3; ++tier) {
    const int32_t *in_q = tier == first ? nullptr : a.queue[tier - 1];
    const int32_t *in_c = tier == first ? nullptr : a.queue_counts + (tier - 1);
    const int64_t grid = std::min<int64_t>(num_roots, tier == first ? int64_t(1) << 20 : 2048);
    int32_t *taken = a.queue_counts + 3 + tier;
    if (tier == 0) launch_tier<TinyTier>(a, in_q, in_c, taken, a.queue[0], a.queue_counts + 0, grid, stream);
    else if (tier == 1) launch_tier<SmallTier>(a, in_q, in_c, taken, a.queue[1], a.queue_counts + 1, grid, stream);
    else launch_tier<BigTier>(a, in_q, in_c, taken, a.queue[2], a.queue_counts + 2, grid, stream);
    RDF2V_LAUNCH_CHECK();
  }
  const int64_t grid2 = bfs_walks_grid(num_entities, num_roots);
  bfs_walks_kernel<<<dim3(unsigned(grid2)), dim3(kThreads), 0, stream>>>(a);
  RDF2V_LAUNCH_CHECK();
  return RDF2V_OK;
}

}  // namespace rdf2v
