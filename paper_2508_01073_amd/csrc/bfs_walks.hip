// BFS walks on gfx950 (gpuRDF2vec Sec. 3.1): per root, a depth-limited BFS
// tree in which every reached entity has one predecessor, and one walk per
// leaf, root to leaf.
//
// The tree is the one a queue-order BFS builds: the entities of a level are
// expanded in the order they were reached, each through its out-edge records in
// CSR order, and an entity gets as parent the first (entity, record) that
// reaches it. The kernel gets the same tree level-synchronously:
//   * the (entity, record) pairs of a level are numbered q = 0, 1, ... in
//     exactly that order (a block scan of the level's degrees);
//   * every pair that reaches an entity not yet in the tree offers
//     (stamp << 32 | q) to that entity with a 64-bit atomicMin, so the smallest
//     q wins; stamps fall with every (root, level) a workgroup processes, so
//     offers left from earlier levels or roots always lose;
//   * the winners, in q order (a block scan), are the next level.
// Leaves are then ranked in the order reached and the first max_walks become
// rows root, V+p_1, v_1, ..., leaf.
//
// A persistent grid: workgroup b takes roots b, b + G, ... and owns one slice of
// the workspace (stamps, offers, tree, degree prefix; about 36 bytes per
// entity). The first kTreeLds tree positions and small levels are kept in
// LDS. All loops are bounded by the tree and level sizes; there is no waiting
// on other workgroups.

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
  char *workspace;
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

  // Each workgroup initialises its own slice once per call.
  for (int32_t v = t; v < V; v += kThreads) {
    st(mark + v, -1);
    __hip_atomic_store(offer + v, ~uint64_t(0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();

  uint32_t stamp = 0xFFFFFFFEu;  // falls by one per (root, level) of this workgroup
  int flags = 0;
  for (int64_t r = blockIdx.x; r < a.num_roots; r += gridDim.x) {
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

int64_t bfs_walks_grid(int32_t num_entities, int64_t num_roots) {
  // Enough workgroups to fill the chip, at most ~4 GiB of slices.
  const int64_t per = int64_t(slice_bytes(num_entities));
  int64_t g = std::max<int64_t>(1, (int64_t(1) << 32) / std::max<int64_t>(per, 1));
  g = std::min<int64_t>(g, 2048);
  g = std::min<int64_t>(g, std::max<int64_t>(num_roots, 1));
  return g;
}

size_t bfs_walks_workspace_bytes(int32_t num_entities, int64_t num_roots) {
  return size_t(bfs_walks_grid(num_entities, num_roots)) * slice_bytes(num_entities);
}

rdf2v_status launch_bfs_walks(const int32_t *row_ptr, const int32_t *edges, int64_t num_edges,
                              int32_t num_entities, int32_t num_predicates, const int32_t *roots,
                              int64_t num_roots, int32_t depth, int32_t max_walks, int32_t *tokens_out,
                              int32_t *len_out, int32_t *counts_out, void *workspace, int32_t *status_dev,
                              hipStream_t stream) {
  if (num_roots == 0) return RDF2V_OK;
  BfsArgs a;
  a.row_ptr = row_ptr;
  a.edges = edges;
  a.roots = roots;
  a.tokens = tokens_out;
  a.lens = len_out;
  a.counts = counts_out;
  a.status = status_dev;
  a.workspace = static_cast<char *>(workspace);
  a.slice_bytes = slice_bytes(num_entities);
  a.num_roots = num_roots;
  a.num_edges = num_edges;
  a.num_entities = num_entities;
  a.num_predicates = num_predicates;
  a.depth = depth;
  a.max_walks = max_walks;
  const int64_t grid = bfs_walks_grid(num_entities, num_roots);
  bfs_walks_kernel<<<dim3(unsigned(grid)), dim3(kThreads), 0, stream>>>(a);
  RDF2V_LAUNCH_CHECK();
  return RDF2V_OK;
}

}  // namespace rdf2v
