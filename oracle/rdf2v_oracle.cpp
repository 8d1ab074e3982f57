// RDF2vec random-walk corpus extraction: CPU oracle.
//
// TEST INFRASTRUCTURE, NOT PRODUCT CODE. This file is a plain, slow,
// single-threaded statement of what the GPU library computes. Only the test
// suite, the smoke check and the CPU-baseline leg of the benchmark load it; the
// GPU library never calls, links or includes it, and it includes nothing from
// the GPU library. It has no blocking, no fusion and no reordering beyond the
// definitions below, so that each step can be checked against its source by eye.
//
// What it computes (gpuRDF2vec, Boeckling & Paulheim, arXiv 2508.01073):
//  * Sec. 2: a random walk is the iterative random choice of the next hop.
//  * Sec. 3.1: entities and predicates are tokenised to integer ids, walks are
//    emitted as entity/predicate (triple-based) sequences, and a walk that ends
//    before the maximum depth is padded with -1.
//  * Sec. 3.3: the walk parameters are the start entities, the depth, the
//    number of walks per entity and a random seed. The paper does not fix the
//    generator; this library fixes it to Philox4x32-10 (Salmon, Moraes, Dror &
//    Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC'11), keyed on the
//    seed and counted on (walk id, hop / 4), with the next out-edge chosen as
//    floor(u * deg / 2^32) over the out-edge records of the current entity.
//
// Readings where the paper is silent (each is listed in the design notes):
//  * CSR rows keep the input order of the triples (a stable sort by subject).
//  * Depth counts hops; a walk row holds 2*depth+1 tokens.
//  * Hops are numbered from 0; walk w starts at start[w / walks_per_node].
//  * Entity token = entity id; predicate token = num_entities + predicate id.
//  * An entity with no out-edge is a sink: the walk stops there.
//  * Duplicate triples and self-loops are kept and followed like any edge.
//
// parity pinned: Philox against rocRAND's host-callable Philox4x32-10, the edge
// index against its closed form, the CSR against std::stable_sort / numpy's
// stable argsort, and the walks against chain, sink, brute-force-enumeration and
// chi-square uniformity tests (see tests/test_oracle_pins.py); skip-gram pairs,
// entity/property walks and duplicate-free walks against hand-worked examples,
// independent numpy constructions and closed-form counts
// (tests/test_oracle_pairs.py); BFS walks against scipy's breadth_first_order
// (tests/test_oracle_bfs.py); the vocabulary against pandas.factorize and the
// integer graph its strings were made from (tests/test_oracle_vocab.py).

#include <cstdint>
#include <cstddef>
#include <string>
#include <unordered_map>
#include <vector>

namespace {

// Status codes: the same numbering as the library's public header, restated
// here so that the two share no file.
enum : int {
  REF_OK = 0,
  REF_ERR_INVALID_ARGUMENT = 1,
  REF_ERR_ID_OUT_OF_RANGE = 2,
  REF_ERR_TOO_LARGE = 3,
};

constexpr int64_t kInt32Limit = int64_t(1) << 31;
constexpr int kMaxDepth = 64;

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon et al., SC'11, Sec. 4 "Philox"): a counter-based
// generator. Each of ten rounds multiplies counter words 0 and 2 by the two
// Philox multipliers, forming 32x32->64-bit products (hi, lo); the new counter
// is (hi of product 2 ^ c1 ^ k0, lo of product 2, hi of product 0 ^ c3 ^ k1,
// lo of product 0). Between rounds the key is advanced by the two Weyl
// constants (the golden ratio and sqrt(3)-1 scaled to 32 bits), mod 2^32.
// ---------------------------------------------------------------------------
constexpr uint32_t kPhiloxM0 = 0xD2511F53u;
constexpr uint32_t kPhiloxM1 = 0xCD9E8D57u;
constexpr uint32_t kPhiloxW0 = 0x9E3779B9u;
constexpr uint32_t kPhiloxW1 = 0xBB67AE85u;

void philox4x32_10(const uint32_t counter[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c0 = counter[0], c1 = counter[1], c2 = counter[2], c3 = counter[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += kPhiloxW0;
      k1 += kPhiloxW1;
    }
    const uint64_t prod0 = uint64_t(kPhiloxM0) * uint64_t(c0);
    const uint64_t prod1 = uint64_t(kPhiloxM1) * uint64_t(c2);
    const uint32_t hi0 = uint32_t(prod0 >> 32), lo0 = uint32_t(prod0);
    const uint32_t hi1 = uint32_t(prod1 >> 32), lo1 = uint32_t(prod1);
    const uint32_t n0 = hi1 ^ c1 ^ k0;
    const uint32_t n1 = lo1;
    const uint32_t n2 = hi0 ^ c3 ^ k1;
    const uint32_t n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

// The random word for hop h of walk w: block number h / 4 of the walk's stream
// (walk id in the high counter half), word h mod 4 of that block.
uint32_t philox_word(uint64_t seed, uint64_t walk, uint64_t hop) {
  const uint64_t block = hop >> 2;
  const uint32_t counter[4] = {uint32_t(block), uint32_t(block >> 32),
                               uint32_t(walk), uint32_t(walk >> 32)};
  const uint32_t key[2] = {uint32_t(seed), uint32_t(seed >> 32)};
  uint32_t out[4];
  philox4x32_10(counter, key, out);
  return out[hop & 3];
}

// Uniform choice of one of deg out-edge records from a 32-bit word:
// floor(u * deg / 2^32), always in [0, deg) for deg >= 1.
uint32_t edge_index(uint32_t u, uint32_t deg) {
  return uint32_t((uint64_t(u) * uint64_t(deg)) >> 32);
}

}  // namespace

extern "C" {

void rdf2v_ref_philox4x32_10(const uint32_t counter[4], const uint32_t key[2], uint32_t out[4]) {
  philox4x32_10(counter, key, out);
}

uint32_t rdf2v_ref_philox_word(uint64_t seed, uint64_t walk, uint64_t hop) {
  return philox_word(seed, walk, hop);
}

uint32_t rdf2v_ref_edge_index(uint32_t u, uint32_t deg) { return edge_index(u, deg); }

// Subject-indexed CSR of (predicate, object) out-edge records (Sec. 3.1: the
// triples are loaded as a graph whose traversal yields the walks).
//   row_ptr[V+1]: row_ptr[v] .. row_ptr[v+1] are the out-edges of entity v.
//   edges[T][2]:  (predicate, object) records; inside a row, input order.
int rdf2v_ref_build_csr(const int32_t *subj, const int32_t *pred, const int32_t *obj,
                        int64_t num_triples, int32_t num_entities, int32_t num_predicates,
                        int32_t *row_ptr, int32_t *edges) {
  if (num_triples < 0 || num_entities < 0 || num_predicates < 0) return REF_ERR_INVALID_ARGUMENT;
  if (row_ptr == nullptr) return REF_ERR_INVALID_ARGUMENT;
  if (num_triples > 0 && (subj == nullptr || pred == nullptr || obj == nullptr || edges == nullptr))
    return REF_ERR_INVALID_ARGUMENT;
  if (num_triples >= kInt32Limit) return REF_ERR_TOO_LARGE;
  if (int64_t(num_entities) + int64_t(num_predicates) >= kInt32Limit) return REF_ERR_TOO_LARGE;

  for (int64_t t = 0; t < num_triples; ++t) {
    if (subj[t] < 0 || subj[t] >= num_entities) return REF_ERR_ID_OUT_OF_RANGE;
    if (obj[t] < 0 || obj[t] >= num_entities) return REF_ERR_ID_OUT_OF_RANGE;
    if (pred[t] < 0 || pred[t] >= num_predicates) return REF_ERR_ID_OUT_OF_RANGE;
  }

  // Out-degree of every entity.
  std::vector<int64_t> degree(size_t(num_entities), 0);
  for (int64_t t = 0; t < num_triples; ++t) degree[size_t(subj[t])] += 1;

  // Row offsets: exclusive prefix sum of the degrees.
  row_ptr[0] = 0;
  for (int32_t v = 0; v < num_entities; ++v)
    row_ptr[v + 1] = int32_t(int64_t(row_ptr[v]) + degree[size_t(v)]);

  // Place each triple at the next free slot of its subject's row, visiting the
  // triples in input order: this keeps input order inside every row.
  std::vector<int64_t> cursor(size_t(num_entities), 0);
  for (int32_t v = 0; v < num_entities; ++v) cursor[size_t(v)] = row_ptr[v];
  for (int64_t t = 0; t < num_triples; ++t) {
    const int64_t slot = cursor[size_t(subj[t])]++;
    edges[2 * slot + 0] = pred[t];
    edges[2 * slot + 1] = obj[t];
  }
  return REF_OK;
}

// Entities with at least one out-edge, ascending: the default start set (the
// paper starts walks from every entity when no start list is given, Sec. 3.3;
// a sink start would only yield a one-token walk).
int64_t rdf2v_ref_nonsink_starts(const int32_t *row_ptr, int32_t num_entities, int32_t *starts_out) {
  int64_t n = 0;
  for (int32_t v = 0; v < num_entities; ++v)
    if (row_ptr[v + 1] > row_ptr[v]) starts_out[n++] = v;
  return n;
}

// Walks w in [walk_begin, walk_begin + walk_count) of the corpus with
// num_start * walks_per_node walks. Row r = w - walk_begin of the outputs:
//   tokens[r][0 .. 2*depth]: e0, V+p0, e1, V+p1, e2, ...; -1 after the end.
//   len[r]: number of valid tokens = 2 * hops + 1.
int rdf2v_ref_random_walks(const int32_t *row_ptr, const int32_t *edges, int32_t num_entities,
                           int32_t num_predicates, int64_t num_edges, const int32_t *start_nodes,
                           int64_t num_start, int32_t walks_per_node, int32_t depth, uint64_t seed,
                           int64_t walk_begin, int64_t walk_count, int32_t *tokens, int32_t *len) {
  if (num_entities < 0 || num_predicates < 0 || num_edges < 0 || num_start < 0) return REF_ERR_INVALID_ARGUMENT;
  if (walks_per_node < 0 || depth < 0 || depth > kMaxDepth) return REF_ERR_INVALID_ARGUMENT;
  if (walk_begin < 0 || walk_count < 0) return REF_ERR_INVALID_ARGUMENT;
  if (num_edges >= kInt32Limit) return REF_ERR_TOO_LARGE;
  if (int64_t(num_entities) + int64_t(num_predicates) >= kInt32Limit) return REF_ERR_TOO_LARGE;
  const int64_t num_walks = num_start * int64_t(walks_per_node);  // callers keep this in range
  if (walk_begin > num_walks || walk_count > num_walks - walk_begin) return REF_ERR_INVALID_ARGUMENT;
  if (walk_count == 0) return REF_OK;
  if (row_ptr == nullptr || start_nodes == nullptr || tokens == nullptr || len == nullptr)
    return REF_ERR_INVALID_ARGUMENT;

  const int64_t width = 2 * int64_t(depth) + 1;
  int status = REF_OK;
  for (int64_t r = 0; r < walk_count; ++r) {
    const int64_t w = walk_begin + r;
    int32_t *row = tokens + r * width;
    int32_t e = start_nodes[w / walks_per_node];
    row[0] = e;
    int64_t n = 1;
    if (e < 0 || e >= num_entities) status = REF_ERR_ID_OUT_OF_RANGE;
    for (int32_t h = 0; h < depth && status == REF_OK; ++h) {
      const int64_t lo = row_ptr[e];
      const int64_t hi = row_ptr[e + 1];
      if (lo < 0 || hi < lo || hi > num_edges) { status = REF_ERR_ID_OUT_OF_RANGE; break; }
      const int64_t degree = hi - lo;
      if (degree == 0) break;  // sink: the walk ends here
      const uint32_t u = philox_word(seed, uint64_t(w), uint64_t(h));
      const int64_t k = edge_index(u, uint32_t(degree));
      const int32_t p = edges[2 * (lo + k) + 0];
      const int32_t x = edges[2 * (lo + k) + 1];
      if (p < 0 || p >= num_predicates || x < 0 || x >= num_entities) { status = REF_ERR_ID_OUT_OF_RANGE; break; }
      row[2 * h + 1] = num_entities + p;
      row[2 * h + 2] = x;
      n += 2;
      e = x;
    }
    for (int64_t j = n; j < width; ++j) row[j] = -1;
    len[r] = int32_t(n);
    if (status != REF_OK) return status;
  }
  return REF_OK;
}

// Entity walks and property walks (Tab. 1 lists both among the walk kinds;
// the paper does not define them further). They are read here as projections
// of the triple-based walk on the same random stream:
//   kind 1, entity walk:   e_0, e_1, ..., e_h   (the entity tokens),
//   kind 2, property walk: e_0, V+p_0, ..., V+p_{h-1}   (the start entity and
//                          the predicate tokens),
// each padded with -1 to depth + 1 tokens; out_len = h + 1. Input rows are
// triple-based walks of 2*depth+1 tokens with len = 2h+1.
int rdf2v_ref_project_walks(const int32_t *tokens, const int32_t *len, int64_t num_walks, int32_t depth,
                            int32_t kind, int32_t *out, int32_t *out_len) {
  if (num_walks < 0 || depth < 0 || depth > kMaxDepth || (kind != 1 && kind != 2))
    return REF_ERR_INVALID_ARGUMENT;
  const int64_t in_width = 2 * int64_t(depth) + 1, out_width = int64_t(depth) + 1;
  for (int64_t r = 0; r < num_walks; ++r) {
    const int32_t *row = tokens + r * in_width;
    int32_t *dst = out + r * out_width;
    const int64_t L = len[r];
    if (L < 1 || L > in_width || L % 2 == 0) return REF_ERR_INVALID_ARGUMENT;
    const int64_t hops = (L - 1) / 2;
    dst[0] = row[0];
    for (int64_t h = 0; h < hops; ++h) dst[1 + h] = (kind == 1) ? row[2 * h + 2] : row[2 * h + 1];
    for (int64_t j = hops + 1; j < out_width; ++j) dst[j] = -1;
    out_len[r] = int32_t(hops + 1);
  }
  return REF_OK;
}

// Duplicate-free walks (Tab. 1: "random walk duplicate free"): among the walks
// of one start entity, keep only the first occurrence (in walk-id order) of
// each distinct walk. Rows come in groups of group_size consecutive rows (the
// walks_per_node walks of one start; the last group may be shorter); two rows
// are the same walk when their lengths and their first len tokens agree.
// Kept rows are copied, in order, to out / out_len; returns how many.
int64_t rdf2v_ref_unique_walks(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                               int32_t group_size, int32_t row_width, int32_t *out, int32_t *out_len) {
  if (num_walks < 0 || group_size < 1 || row_width < 1) return -REF_ERR_INVALID_ARGUMENT;
  int64_t kept = 0;
  for (int64_t r = 0; r < num_walks; ++r) {
    const int64_t g0 = r / group_size * group_size;
    const int32_t *row = tokens + r * row_width;
    bool seen = false;
    for (int64_t q = g0; q < r && !seen; ++q) {
      if (len[q] != len[r]) continue;
      const int32_t *other = tokens + q * row_width;
      bool same = true;
      for (int32_t j = 0; j < len[r] && same; ++j) same = other[j] == row[j];
      seen = same;
    }
    if (seen) continue;
    if (out != nullptr) {
      for (int32_t j = 0; j < row_width; ++j) out[kept * row_width + j] = row[j];
      out_len[kept] = len[r];
    }
    ++kept;
  }
  return kept;
}

// BFS walks (Sec. 3.1): a breadth-first search from each root gives every
// reached entity one predecessor, the first entity that reaches it, and every
// path from a leaf of that tree back to the root becomes one walk, so each
// entity appears in at most one walk per root. Read here as a queue-order BFS
// limited to `depth` hops: entities of one level are expanded in the order in
// which they were reached, each through its out-edge records in CSR order, and
// an entity not reached before gets the current entity and record as its
// parent. A tree entity with no child (including every entity at the depth
// limit) is a leaf; leaves are taken in the order they were reached, and the
// first max_walks of them give the walks root, V+p_1, v_1, ..., leaf (rows of
// 2*depth+1 tokens padded with -1). counts[r] = number of walks written for
// root r; the return value is the number of roots whose leaves did not fit.
int64_t rdf2v_ref_bfs_walks(const int32_t *row_ptr, const int32_t *edges, int32_t num_entities,
                            int32_t num_predicates, const int32_t *roots, int64_t num_roots, int32_t depth,
                            int32_t max_walks, int32_t *tokens, int32_t *len, int32_t *counts) {
  if (num_entities < 0 || num_roots < 0 || depth < 0 || depth > kMaxDepth || max_walks < 1)
    return -REF_ERR_INVALID_ARGUMENT;
  const int64_t width = 2 * int64_t(depth) + 1;
  std::vector<int32_t> seen_root(size_t(num_entities), -1);  // root index that reached the entity
  struct Node { int32_t entity, parent, pred, level; bool has_child; };
  int64_t truncated = 0;
  for (int64_t r = 0; r < num_roots; ++r) {
    const int32_t root = roots[r];
    if (root < 0 || root >= num_entities) return -REF_ERR_ID_OUT_OF_RANGE;
    std::vector<Node> tree;
    tree.push_back({root, -1, -1, 0, false});
    seen_root[size_t(root)] = int32_t(r);
    size_t level_begin = 0, level_end = 1;
    for (int32_t level = 0; level < depth && level_begin < level_end; ++level) {
      for (size_t i = level_begin; i < level_end; ++i) {
        const int32_t u = tree[i].entity;
        for (int64_t k = row_ptr[u]; k < row_ptr[u + 1]; ++k) {
          const int32_t p = edges[2 * k], x = edges[2 * k + 1];
          if (seen_root[size_t(x)] == int32_t(r)) continue;
          seen_root[size_t(x)] = int32_t(r);
          tree[i].has_child = true;
          tree.push_back({x, int32_t(i), p, level + 1, false});
        }
      }
      level_begin = level_end;
      level_end = tree.size();
    }
    int32_t written = 0;
    for (size_t i = 0; i < tree.size(); ++i) {
      if (tree[i].has_child) continue;
      if (written == max_walks) { ++truncated; break; }
      int32_t *row = tokens + (r * int64_t(max_walks) + written) * width;
      const int32_t h = tree[i].level;
      int32_t node = int32_t(i);
      for (int32_t step = h; step >= 1; --step) {  // fill from the leaf back to the root
        row[2 * step] = tree[size_t(node)].entity;
        row[2 * step - 1] = num_entities + tree[size_t(node)].pred;
        node = tree[size_t(node)].parent;
      }
      row[0] = root;
      for (int64_t j = 2 * int64_t(h) + 1; j < width; ++j) row[j] = -1;
      len[r * int64_t(max_walks) + written] = 2 * h + 1;
      ++written;
    }
    counts[r] = written;
  }
  (void)num_predicates;
  return truncated;
}

// Vocabulary (Sec. 3.1: every entity and predicate is tokenised to an integer
// id at the start of the pipeline). Strings are given as byte buffers with
// offsets (string i is chars[offsets[i] .. offsets[i+1])). Entity ids number
// the distinct subject and object strings in order of first appearance over
// s_0, o_0, s_1, o_1, ...; predicate ids number the distinct predicate strings
// in order of first appearance over p_0, p_1, .... Returns 0, or an error code.
int rdf2v_ref_build_vocabulary(const char *s_chars, const int64_t *s_off, const char *p_chars,
                               const int64_t *p_off, const char *o_chars, const int64_t *o_off,
                               int64_t num_triples, int32_t *s_ids, int32_t *p_ids, int32_t *o_ids,
                               int64_t *num_entities, int64_t *num_predicates) {
  if (num_triples < 0) return REF_ERR_INVALID_ARGUMENT;
  std::unordered_map<std::string, int32_t> entities, predicates;
  auto id_of = [](std::unordered_map<std::string, int32_t> &vocab, const char *chars, const int64_t *off,
                  int64_t i) {
    const std::string key(chars + off[i], size_t(off[i + 1] - off[i]));
    auto it = vocab.find(key);
    if (it != vocab.end()) return it->second;
    const int32_t id = int32_t(vocab.size());
    vocab.emplace(key, id);
    return id;
  };
  for (int64_t t = 0; t < num_triples; ++t) {
    s_ids[t] = id_of(entities, s_chars, s_off, t);
    o_ids[t] = id_of(entities, o_chars, o_off, t);
    p_ids[t] = id_of(predicates, p_chars, p_off, t);
  }
  *num_entities = int64_t(entities.size());
  *num_predicates = int64_t(predicates.size());
  return REF_OK;
}

// Skip-gram training pairs (Sec. 3.2: the data module turns the walk corpus
// into center-context pairs; Sec. 3.1: padding is dropped first). For walk r
// with L = len[r] valid tokens t_0 .. t_{L-1}, every center position i and
// every context position j with 1 <= |i - j| <= window and 0 <= j < L give the
// pair (t_i, t_j), in the order walk, then i, then j. Returns the number of
// pairs; writes at most `capacity` of them to pairs[][2]. A negative return is
// an argument error.
int64_t rdf2v_ref_skipgram_pairs(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                                 int32_t row_width, int32_t window, int32_t *pairs, int64_t capacity) {
  if (num_walks < 0 || row_width < 1 || window < 0 || capacity < 0) return -REF_ERR_INVALID_ARGUMENT;
  int64_t n = 0;
  for (int64_t r = 0; r < num_walks; ++r) {
    const int32_t *row = tokens + r * row_width;
    const int64_t L = len[r];
    if (L < 0 || L > row_width) return -REF_ERR_INVALID_ARGUMENT;
    for (int64_t i = 0; i < L; ++i) {
      for (int64_t j = i - window; j <= i + window; ++j) {
        if (j == i || j < 0 || j >= L) continue;
        if (n < capacity) {
          pairs[2 * n + 0] = row[i];
          pairs[2 * n + 1] = row[j];
        }
        ++n;
      }
    }
  }
  return n;
}

// CBOW training examples (Sec. 3.2: the library trains Continuous Bag of
// Words next to Skip-Gram; CBOW predicts a center token from the tokens around
// it). For walk r with L = len[r] valid tokens t_0 .. t_{L-1}, every position i
// gives one example: centers[e] = t_i and contexts[e][0 .. 2*window) = the t_j
// with 1 <= |i - j| <= window and 0 <= j < L in ascending j, then -1 up to
// 2*window entries. Examples in the order walk, then i. Returns the number of
// examples (the sum of the lengths); writes at most `capacity` of them. A
// negative return is an argument error.
int64_t rdf2v_ref_cbow_examples(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                                int32_t row_width, int32_t window, int32_t *centers, int32_t *contexts,
                                int64_t capacity) {
  if (num_walks < 0 || row_width < 1 || window < 1 || capacity < 0) return -REF_ERR_INVALID_ARGUMENT;
  const int64_t ctx_width = 2 * int64_t(window);
  int64_t e = 0;
  for (int64_t r = 0; r < num_walks; ++r) {
    const int32_t *row = tokens + r * row_width;
    const int64_t L = len[r];
    if (L < 0 || L > row_width) return -REF_ERR_INVALID_ARGUMENT;
    for (int64_t i = 0; i < L; ++i, ++e) {
      if (e >= capacity) continue;
      centers[e] = row[i];
      int32_t *ctx = contexts + e * ctx_width;
      int64_t m = 0;
      for (int64_t j = i - window; j <= i + window; ++j)
        if (j != i && j >= 0 && j < L) ctx[m++] = row[j];
      for (; m < ctx_width; ++m) ctx[m] = -1;
    }
  }
  return e;
}

}  // extern "C"
