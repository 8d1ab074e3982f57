// Seeded synthetic knowledge-graph generators (inputs only).
//
// This module produces (subject, predicate, object) id triples for the tests
// and the benchmark. It holds none of the walk method's arithmetic: its random
// numbers come from SplitMix64 (Steele, Lea & Flood, "Fast splittable
// pseudorandom number generators", OOPSLA 2014) used as a counter hash, not
// from the walks' Philox stream, and it never builds a CSR or walks a graph.
//
// Every draw is a pure function of (seed, stream, index), so the output does
// not depend on the number of threads.
//
// Recipes (the paper's own graphs are not available; these stand in for them):
//  * uniform: subject, predicate and object i.i.d. uniform; duplicates and
//    self-loops kept (the Erdos-Renyi / uniform-attachment style graphs of
//    gpuRDF2vec Sec. 5.1, which also draw each edge's predicate uniformly).
//  * power law: Chung-Lu style. Entity of rank r (1-based, over a seeded
//    Fisher-Yates permutation of the ids) has weight r^(-1/(gamma-1)), which
//    gives an out- and in-degree tail with exponent gamma. Subject and object
//    are drawn i.i.d. from these weights (same permutation, so hubs are hubs in
//    both directions); predicate rank r is drawn with weight r^(-pred_s). An
//    optional fraction of entities, chosen uniformly (Knuth's selection
//    sampling), get subject weight 0: they are sinks that walks still reach.
//    Weighted draws use Vose's alias method in double precision.

#include <cmath>
#include <cstdint>
#include <thread>
#include <vector>

namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;

inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Draw number `index` of stream `stream_key` (SplitMix64's output for state
// stream_key + (index + 1) * golden).
inline uint64_t draw(uint64_t stream_key, uint64_t index) {
  return mix64(stream_key + (index + 1) * kGolden);
}

inline uint64_t stream(uint64_t seed, uint64_t tag) { return mix64(seed ^ mix64(tag + kGolden)); }

// Uniform integer in [0, n) from a 64-bit draw (128-bit multiply-shift).
inline uint64_t below(uint64_t x, uint64_t n) {
  return uint64_t((static_cast<unsigned __int128>(x) * n) >> 64);
}

// Uniform double in [0, 1) from the top 53 bits.
inline double unit(uint64_t x) { return double(x >> 11) * (1.0 / 9007199254740992.0); }

struct Alias {
  std::vector<double> prob;
  std::vector<int32_t> alias;
  int64_t n = 0;
};

// Vose's alias method ("A linear algorithm for generating random numbers with
// a given distribution", IEEE TSE 1991). Zero weights are allowed.
Alias build_alias(const std::vector<double> &weight) {
  Alias a;
  a.n = int64_t(weight.size());
  a.prob.assign(size_t(a.n), 0.0);
  a.alias.assign(size_t(a.n), 0);
  double total = 0.0;
  for (double w : weight) total += w;
  std::vector<double> scaled(static_cast<size_t>(a.n));
  std::vector<int32_t> small, large;
  small.reserve(size_t(a.n));
  large.reserve(size_t(a.n));
  for (int64_t i = 0; i < a.n; ++i) {
    scaled[size_t(i)] = weight[size_t(i)] * double(a.n) / total;
    (scaled[size_t(i)] < 1.0 ? small : large).push_back(int32_t(i));
  }
  while (!small.empty() && !large.empty()) {
    const int32_t l = small.back(); small.pop_back();
    const int32_t g = large.back(); large.pop_back();
    a.prob[size_t(l)] = scaled[size_t(l)];
    a.alias[size_t(l)] = g;
    scaled[size_t(g)] = (scaled[size_t(g)] + scaled[size_t(l)]) - 1.0;
    (scaled[size_t(g)] < 1.0 ? small : large).push_back(g);
  }
  for (int32_t g : large) { a.prob[size_t(g)] = 1.0; a.alias[size_t(g)] = g; }
  for (int32_t l : small) { a.prob[size_t(l)] = 1.0; a.alias[size_t(l)] = l; }
  return a;
}

inline int32_t sample(const Alias &a, uint64_t x_column, uint64_t x_coin) {
  const int64_t i = int64_t(below(x_column, uint64_t(a.n)));
  return unit(x_coin) < a.prob[size_t(i)] ? int32_t(i) : a.alias[size_t(i)];
}

template <class F>
void parallel_for(int64_t n, int nthreads, F fn) {
  if (nthreads < 1) nthreads = 1;
  if (n < (int64_t(1) << 16)) nthreads = 1;
  std::vector<std::thread> pool;
  const int64_t chunk = (n + nthreads - 1) / nthreads;
  for (int t = 0; t < nthreads; ++t) {
    const int64_t lo = int64_t(t) * chunk;
    const int64_t hi = lo + chunk < n ? lo + chunk : n;
    if (lo >= hi) break;
    pool.emplace_back([=] { fn(lo, hi); });
  }
  for (auto &th : pool) th.join();
}

enum : uint64_t { kTagSubject = 1, kTagPredicate = 2, kTagObject = 3, kTagPermutation = 4, kTagSinks = 5 };

}  // namespace

extern "C" {

// Uniform i.i.d. triples.
int synth_uniform(uint64_t seed, int64_t num_triples, int32_t num_entities, int32_t num_predicates,
                  int32_t *subj, int32_t *pred, int32_t *obj, int nthreads) {
  if (num_triples < 0 || num_entities <= 0 || num_predicates <= 0) return 1;
  const uint64_t ks = stream(seed, kTagSubject), kp = stream(seed, kTagPredicate),
                 ko = stream(seed, kTagObject);
  parallel_for(num_triples, nthreads, [&](int64_t lo, int64_t hi) {
    for (int64_t t = lo; t < hi; ++t) {
      subj[t] = int32_t(below(draw(ks, uint64_t(t)), uint64_t(num_entities)));
      pred[t] = int32_t(below(draw(kp, uint64_t(t)), uint64_t(num_predicates)));
      obj[t] = int32_t(below(draw(ko, uint64_t(t)), uint64_t(num_entities)));
    }
  });
  return 0;
}

// Power-law (Chung-Lu) triples; see the header comment. If rank_entity is not
// null it receives the permutation (rank r-1 -> entity id); if sink_flag is not
// null it receives 1 for designated sinks.
int synth_powerlaw(uint64_t seed, int64_t num_triples, int32_t num_entities, int32_t num_predicates,
                   double gamma, double pred_s, double sink_fraction, int32_t *subj, int32_t *pred,
                   int32_t *obj, int32_t *rank_entity, uint8_t *sink_flag, int nthreads) {
  if (num_triples < 0 || num_entities <= 0 || num_predicates <= 0) return 1;
  if (!(gamma > 1.0) || !(pred_s > 0.0) || sink_fraction < 0.0 || sink_fraction >= 1.0) return 1;
  const int64_t V = num_entities;

  // Seeded Fisher-Yates permutation: perm[r] = entity id of rank r + 1.
  std::vector<int32_t> perm(static_cast<size_t>(V));
  for (int64_t i = 0; i < V; ++i) perm[size_t(i)] = int32_t(i);
  const uint64_t kperm = stream(seed, kTagPermutation);
  for (int64_t i = V - 1; i > 0; --i) {
    const int64_t j = int64_t(below(draw(kperm, uint64_t(i)), uint64_t(i + 1)));
    const int32_t tmp = perm[size_t(i)];
    perm[size_t(i)] = perm[size_t(j)];
    perm[size_t(j)] = tmp;
  }

  // Designated sinks: exactly floor(V * sink_fraction) entities, chosen by
  // selection sampling over the ids in order.
  std::vector<uint8_t> sink(static_cast<size_t>(V), 0);
  int64_t need = int64_t(std::floor(double(V) * sink_fraction));
  const uint64_t ksink = stream(seed, kTagSinks);
  for (int64_t i = 0; i < V && need > 0; ++i) {
    const int64_t remaining = V - i;
    if (int64_t(below(draw(ksink, uint64_t(i)), uint64_t(remaining))) < need) {
      sink[size_t(i)] = 1;
      --need;
    }
  }

  const double a = 1.0 / (gamma - 1.0);
  std::vector<double> w_obj(static_cast<size_t>(V)), w_subj(static_cast<size_t>(V));
  for (int64_t r = 0; r < V; ++r) {
    const int32_t e = perm[size_t(r)];
    const double w = std::pow(double(r + 1), -a);
    w_obj[size_t(e)] = w;
    w_subj[size_t(e)] = sink[size_t(e)] ? 0.0 : w;
  }
  std::vector<double> w_pred(static_cast<size_t>(num_predicates));
  for (int32_t r = 0; r < num_predicates; ++r) w_pred[size_t(r)] = std::pow(double(r + 1), -pred_s);

  const Alias as = build_alias(w_subj), ao = build_alias(w_obj), ap = build_alias(w_pred);
  w_obj.clear(); w_obj.shrink_to_fit();
  w_subj.clear(); w_subj.shrink_to_fit();

  const uint64_t ks = stream(seed, kTagSubject), kp = stream(seed, kTagPredicate),
                 ko = stream(seed, kTagObject);
  parallel_for(num_triples, nthreads, [&](int64_t lo, int64_t hi) {
    for (int64_t t = lo; t < hi; ++t) {
      const uint64_t i = 2 * uint64_t(t);
      subj[t] = sample(as, draw(ks, i), draw(ks, i + 1));
      pred[t] = sample(ap, draw(kp, i), draw(kp, i + 1));
      obj[t] = sample(ao, draw(ko, i), draw(ko, i + 1));
    }
  });
  if (rank_entity)
    for (int64_t r = 0; r < V; ++r) rank_entity[r] = perm[size_t(r)];
  if (sink_flag)
    for (int64_t i = 0; i < V; ++i) sink_flag[i] = sink[size_t(i)];
  return 0;
}

// Text columns for the string form of a triple column: string t is prefix
// followed by the decimal digits of label[ids[t]]. With chars == nullptr only
// the byte lengths are written (to lens); otherwise offsets (n + 1 entries,
// their prefix sum) locate string t at chars[offsets[t] ..).
int synth_label_column(const int32_t *ids, int64_t n, const int64_t *label, int64_t num_labels,
                       const char *prefix, int32_t prefix_len, int64_t *lens, const int64_t *offsets,
                       uint8_t *chars, int nthreads) {
  if (n < 0 || prefix_len < 0) return 1;
  auto digits = [](int64_t x, char *buf) {
    int k = 0;
    do {
      buf[k++] = char('0' + x % 10);
      x /= 10;
    } while (x > 0);
    return k;
  };
  int bad = 0;
  parallel_for(n, nthreads, [&](int64_t lo, int64_t hi) {
    char buf[24];
    for (int64_t t = lo; t < hi; ++t) {
      const int32_t id = ids[t];
      if (id < 0 || id >= num_labels || label[id] < 0) {
        bad = 1;
        continue;
      }
      const int k = digits(label[id], buf);
      if (chars == nullptr) {
        lens[t] = prefix_len + k;
        continue;
      }
      uint8_t *dst = chars + offsets[t];
      for (int32_t j = 0; j < prefix_len; ++j) dst[j] = uint8_t(prefix[j]);
      for (int j = 0; j < k; ++j) dst[prefix_len + j] = uint8_t(buf[k - 1 - j]);
    }
  });
  return bad;
}

}  // extern "C"
