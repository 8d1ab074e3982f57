// Runs every entry point of the CPU oracle and the input generators on small
// graphs and edge cases, for a build with AddressSanitizer and
// UndefinedBehaviorSanitizer: any out-of-bounds access, leak, overflow or other
// undefined behaviour ends the program with an error. Results are checked only
// for the few properties that need no second implementation (lengths, ranges).
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

extern "C" {
int synth_uniform(uint64_t seed, int64_t num_triples, int32_t num_entities, int32_t num_predicates,
                  int32_t *subj, int32_t *pred, int32_t *obj, int nthreads);
int synth_powerlaw(uint64_t seed, int64_t num_triples, int32_t num_entities, int32_t num_predicates,
                   double gamma, double pred_s, double sink_fraction, int32_t *subj, int32_t *pred,
                   int32_t *obj, int32_t *rank_entity, uint8_t *sink_flag, int nthreads);
int synth_label_column(const int32_t *ids, int64_t n, const int64_t *label, int64_t num_labels,
                       const char *prefix, int32_t prefix_len, int64_t *lens, const int64_t *offsets,
                       uint8_t *chars, int nthreads);
uint32_t rdf2v_ref_philox_word(uint64_t seed, uint64_t walk, uint64_t hop);
uint32_t rdf2v_ref_edge_index(uint32_t u, uint32_t deg);
int rdf2v_ref_build_csr(const int32_t *subj, const int32_t *pred, const int32_t *obj, int64_t num_triples,
                        int32_t num_entities, int32_t num_predicates, int32_t *row_ptr, int32_t *edges);
int64_t rdf2v_ref_nonsink_starts(const int32_t *row_ptr, int32_t num_entities, int32_t *starts_out);
int rdf2v_ref_random_walks(const int32_t *row_ptr, const int32_t *edges, int32_t num_entities,
                           int32_t num_predicates, int64_t num_edges, const int32_t *start_nodes,
                           int64_t num_start, int32_t walks_per_node, int32_t depth, uint64_t seed,
                           int64_t walk_begin, int64_t walk_count, int32_t *tokens, int32_t *len);
int rdf2v_ref_project_walks(const int32_t *tokens, const int32_t *len, int64_t num_walks, int32_t depth,
                            int32_t kind, int32_t *out, int32_t *out_len);
int64_t rdf2v_ref_unique_walks(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                               int32_t group_size, int32_t row_width, int32_t *out, int32_t *out_len);
int64_t rdf2v_ref_bfs_walks(const int32_t *row_ptr, const int32_t *edges, int32_t num_entities,
                            int32_t num_predicates, const int32_t *roots, int64_t num_roots, int32_t depth,
                            int32_t max_walks, int32_t *tokens, int32_t *len, int32_t *counts);
int rdf2v_ref_build_vocabulary(const char *s_chars, const int64_t *s_off, const char *p_chars,
                               const int64_t *p_off, const char *o_chars, const int64_t *o_off,
                               int64_t num_triples, int32_t *s_ids, int32_t *p_ids, int32_t *o_ids,
                               int64_t *num_entities, int64_t *num_predicates);
int64_t rdf2v_ref_skipgram_pairs(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                                 int32_t row_width, int32_t window, int32_t *pairs, int64_t capacity);
}

#define CHECK(c)                                                  \
  do {                                                            \
    if (!(c)) {                                                   \
      std::fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
      std::exit(1);                                               \
    }                                                             \
  } while (0)

using V32 = std::vector<int32_t>;

struct Graph {
  int32_t V, P;
  V32 s, p, o, row_ptr, edges, starts;
};

static Graph make(bool powerlaw, int32_t V, int32_t P, int64_t T, uint64_t seed) {
  Graph g{V, P, V32(T), V32(T), V32(T), V32(V + 1), V32(2 * T + 2), V32(V + 1)};
  if (powerlaw)
    CHECK(synth_powerlaw(seed, T, V, P, 2.1, 1.5, 0.1, g.s.data(), g.p.data(), g.o.data(), nullptr, nullptr, 3) == 0);
  else
    CHECK(synth_uniform(seed, T, V, P, g.s.data(), g.p.data(), g.o.data(), 3) == 0);
  CHECK(rdf2v_ref_build_csr(g.s.data(), g.p.data(), g.o.data(), T, V, P, g.row_ptr.data(), g.edges.data()) == 0);
  CHECK(g.row_ptr[V] == T);
  const int64_t ns = rdf2v_ref_nonsink_starts(g.row_ptr.data(), V, g.starts.data());
  CHECK(ns >= 0 && ns <= V);
  g.starts.resize(size_t(ns));
  return g;
}

static void walks_and_consumers(const Graph &g, int32_t wpn, int32_t depth) {
  const int64_t T = int64_t(g.s.size());
  const int64_t W = int64_t(g.starts.size()) * wpn;
  const int32_t width = 2 * depth + 1;
  V32 tok(size_t(W * width) + 1), len(size_t(W) + 1);
  CHECK(rdf2v_ref_random_walks(g.row_ptr.data(), g.edges.data(), g.V, g.P, T, g.starts.data(),
                               int64_t(g.starts.size()), wpn, depth, 42, 0, W, tok.data(), len.data()) == 0);
  for (int64_t w = 0; w < W; ++w) CHECK(len[w] >= 1 && len[w] <= width && len[w] % 2 == 1);
  // a batch in the middle
  if (W > 3) {
    V32 t2(size_t(2 * width)), l2(2);
    CHECK(rdf2v_ref_random_walks(g.row_ptr.data(), g.edges.data(), g.V, g.P, T, g.starts.data(),
                                 int64_t(g.starts.size()), wpn, depth, 42, W / 2, 2, t2.data(), l2.data()) == 0);
  }
  // entity and property projections
  V32 proj(size_t(W * (depth + 1)) + 1), plen(size_t(W) + 1);
  for (int kind = 1; kind <= 2; ++kind)
    CHECK(rdf2v_ref_project_walks(tok.data(), len.data(), W, depth, kind, proj.data(), plen.data()) == 0);
  // duplicate-free walks per start entity
  V32 uo(size_t(W * width) + 1), ul(size_t(W) + 1);
  const int64_t kept = rdf2v_ref_unique_walks(tok.data(), len.data(), W, wpn > 0 ? wpn : 1, width, uo.data(), ul.data());
  CHECK(kept >= 0 && kept <= W);
  // skip-gram pairs: count, then fill, then a truncated fill
  for (int32_t window : {0, 1, 5, 64}) {
    const int64_t n = rdf2v_ref_skipgram_pairs(tok.data(), len.data(), W, width, window, nullptr, 0);
    CHECK(n >= 0);
    V32 pairs(size_t(2 * n) + 2);
    CHECK(rdf2v_ref_skipgram_pairs(tok.data(), len.data(), W, width, window, pairs.data(), n) == n);
    if (n > 1) CHECK(rdf2v_ref_skipgram_pairs(tok.data(), len.data(), W, width, window, pairs.data(), n / 2) == n);
  }
  // BFS walks from every start, small cap so that some roots are truncated
  for (int32_t d : {0, 1, 2}) {
    const int32_t cap = 7;
    const int64_t R = int64_t(g.starts.size());
    const int32_t bw = 2 * d + 1;
    V32 bt(size_t(R * cap * bw) + 1), bl(size_t(R * cap) + 1), bc(size_t(R) + 1);
    const int64_t trunc = rdf2v_ref_bfs_walks(g.row_ptr.data(), g.edges.data(), g.V, g.P, g.starts.data(), R, d,
                                              cap, bt.data(), bl.data(), bc.data());
    CHECK(trunc >= 0 && trunc <= R);
  }
}

static void vocabulary() {
  // generated IRI columns
  const int64_t T = 3000;
  const int32_t V = 500, P = 9;
  V32 s(T), p(T), o(T);
  CHECK(synth_uniform(7, T, V, P, s.data(), p.data(), o.data(), 2) == 0);
  std::vector<int64_t> ent(V), prd(P);
  for (int32_t i = 0; i < V; ++i) ent[size_t(i)] = 1 + (int64_t(i) * 7919) % V;
  for (int32_t i = 0; i < P; ++i) prd[size_t(i)] = 1 + i;
  auto column = [&](const V32 &ids, const std::vector<int64_t> &label, const std::string &prefix,
                    std::vector<int64_t> &off, std::vector<uint8_t> &chars) {
    std::vector<int64_t> lens(static_cast<size_t>(T));
    CHECK(synth_label_column(ids.data(), T, label.data(), int64_t(label.size()), prefix.data(),
                             int32_t(prefix.size()), lens.data(), nullptr, nullptr, 2) == 0);
    off.assign(size_t(T) + 1, 0);
    for (int64_t t = 0; t < T; ++t) off[size_t(t) + 1] = off[size_t(t)] + lens[size_t(t)];
    chars.assign(size_t(off[size_t(T)]) + 1, 0);
    CHECK(synth_label_column(ids.data(), T, label.data(), int64_t(label.size()), prefix.data(),
                             int32_t(prefix.size()), lens.data(), off.data(), chars.data(), 2) == 0);
  };
  std::vector<int64_t> so, po, oo;
  std::vector<uint8_t> sc, pc, oc;
  column(s, ent, "http://e/", so, sc);
  column(p, prd, "http://p/", po, pc);
  column(o, ent, "http://e/", oo, oc);
  V32 si(T), pi(T), oi(T);
  int64_t ne = 0, np = 0;
  CHECK(rdf2v_ref_build_vocabulary(reinterpret_cast<const char *>(sc.data()), so.data(),
                                   reinterpret_cast<const char *>(pc.data()), po.data(),
                                   reinterpret_cast<const char *>(oc.data()), oo.data(), T, si.data(), pi.data(),
                                   oi.data(), &ne, &np) == 0);
  CHECK(ne >= 1 && ne <= V && np >= 1 && np <= P);
  // empty strings, a NUL byte, one triple; and no triples at all
  const char chars[] = {'a', '\0', 'b'};
  const int64_t off3[] = {0, 0}, offa[] = {0, 3}, offb[] = {0, 1};
  int32_t a = -1, b = -1, c = -1;
  CHECK(rdf2v_ref_build_vocabulary(chars, off3, chars, offa, chars, offb, 1, &a, &b, &c, &ne, &np) == 0);
  CHECK(a == 0 && b == 0 && c == 1 && ne == 2 && np == 1);
  CHECK(rdf2v_ref_build_vocabulary(nullptr, off3, nullptr, off3, nullptr, off3, 0, nullptr, nullptr, nullptr, &ne,
                                   &np) == 0);
}

int main() {
  for (uint64_t h : {0ull, 3ull, 4ull, (1ull << 33) + 5}) CHECK(rdf2v_ref_philox_word(42, h * 977, h) == rdf2v_ref_philox_word(42, h * 977, h));
  CHECK(rdf2v_ref_edge_index(0xFFFFFFFFu, 7) == 6 && rdf2v_ref_edge_index(0, 1) == 0);
  {
    Graph g = make(false, 300, 7, 2000, 1);
    walks_and_consumers(g, 5, 4);
    walks_and_consumers(g, 2, 0);
    walks_and_consumers(g, 1, 17);
  }
  {
    Graph g = make(true, 2000, 11, 12000, 2);  // power law with designated sinks
    walks_and_consumers(g, 3, 8);
  }
  {
    Graph g = make(false, 5, 2, 0, 3);  // no triples: every entity is a sink
    CHECK(g.starts.empty());
    V32 tok(3), len(1);
    const int32_t sink = 2;
    CHECK(rdf2v_ref_random_walks(g.row_ptr.data(), g.edges.data(), 5, 2, 0, &sink, 1, 1, 1, 42, 0, 1, tok.data(),
                                 len.data()) == 0);
    CHECK(len[0] == 1 && tok[0] == 2 && tok[1] == -1 && tok[2] == -1);
  }
  {
    // bad arguments are rejected, not read
    int32_t rp[2] = {0, 0};
    CHECK(rdf2v_ref_build_csr(nullptr, nullptr, nullptr, 1, 1, 1, rp, nullptr) != 0);
    CHECK(rdf2v_ref_random_walks(rp, nullptr, 1, 1, 0, nullptr, 1, 1, 65, 42, 0, 1, nullptr, nullptr) != 0);
    CHECK(rdf2v_ref_skipgram_pairs(nullptr, nullptr, -1, 3, 1, nullptr, 0) < 0);
    CHECK(rdf2v_ref_unique_walks(nullptr, nullptr, 1, 0, 3, nullptr, nullptr) < 0);
    CHECK(rdf2v_ref_bfs_walks(rp, nullptr, 1, 1, nullptr, 1, 70, 1, nullptr, nullptr, nullptr) < 0);
  }
  vocabulary();
  std::puts("host sanitize: ok");
  return 0;
}
