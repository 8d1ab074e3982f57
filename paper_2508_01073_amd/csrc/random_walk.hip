// Uniform random walks over the subject-indexed CSR on gfx950.
//
// One lane runs one walk (gpuRDF2vec Sec. 4.1 launches every walk of every
// start entity at once instead of looping over entities; here the start of
// walk w is start[w / walks_per_node], computed in the kernel, so nothing is
// replicated in memory). Each hop is a random gather whose address depends on
// the previous one, and out-edge records are all about equally likely to be
// read, so nearly every hop misses L2: the kernel is bound by the rate at which
// the memory system serves L2-missing random reads. There is no dense
// contraction and no use for MFMA. With walk records (predicate, object and
// the object's row bounds in one 16-byte record) a hop is a single gather;
// without them it is two (the record, then the next entity's row bounds).
//
// Layout choices for CDNA4:
//  * one Philox4x32-10 block serves four consecutive hops of a walk, so the
//    generator's ten rounds of 32x32->64 multiplies are paid once per 4 hops;
//  * a block's walk rows are contiguous in the output, so the block assembles
//    them in LDS (odd row stride 2*depth+1: conflict-free per-lane stores) and
//    writes the whole tile with 16-byte non-temporal stores, which keeps the
//    output stream from evicting the CSR from L2 and the Infinity Cache;
//  * walks of one start entity are consecutive ids and land in one workgroup,
//    so their first hops share the start's row on the same XCD.
// Every gather is bounds-checked against the CSR's sizes, so an inconsistent
// CSR or an out-of-range id raises a status bit instead of faulting.

#include "common.hpp"
#include "walk.hpp"

namespace rdf2v {
namespace {

typedef int32_t v4i32 __attribute__((ext_vector_type(4)));

// Philox4x32-10 (Salmon, Moraes, Dror & Shaw, SC'11): ten rounds of two
// 32x32->64-bit products of counter words 0 and 2 with the Philox multipliers,
// mixed with words 1 and 3 and the round key, which advances by the Weyl
// constants between rounds.
constexpr uint32_t kMulA = 0xD2511F53u;
constexpr uint32_t kMulB = 0xCD9E8D57u;
constexpr uint32_t kWeylA = 0x9E3779B9u;
constexpr uint32_t kWeylB = 0xBB67AE85u;

struct Words4 {
  uint32_t w0, w1, w2, w3;
};

// Block `hop_block` of walk `walk`'s stream: counter (hop_block, 0, walk lo, walk hi).
__device__ __forceinline__ Words4 philox_block(uint32_t hop_block, uint64_t walk, uint32_t key_lo,
                                               uint32_t key_hi) {
  uint32_t x0 = hop_block, x1 = 0u, x2 = uint32_t(walk), x3 = uint32_t(walk >> 32);
  uint32_t k0 = key_lo, k1 = key_hi;
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    const uint32_t hi_a = __umulhi(x0, kMulA), lo_a = x0 * kMulA;
    const uint32_t hi_b = __umulhi(x2, kMulB), lo_b = x2 * kMulB;
    x0 = hi_b ^ x1 ^ k0;
    x1 = lo_b;
    x2 = hi_a ^ x3 ^ k1;
    x3 = lo_a;
    k0 += kWeylA;
    k1 += kWeylB;
  }
  return {x0, x1, x2, x3};
}

// kFused: read (predicate, object, row lo, row hi) records, so each hop is one
// 16-byte gather; otherwise read (predicate, object) and then the row bounds
// of the object (two dependent gathers per hop).
// kKind selects the tokens a hop appends: RDF2V_TOKENS_TRIPLES (predicate and
// entity), RDF2V_TOKENS_ENTITIES (entity) or RDF2V_TOKENS_PROPERTIES
// (predicate). The walk itself, and its random stream, is the same for all.
template <int kBlock, bool kFused, int kKind>
__global__ __launch_bounds__(kBlock) void random_walk_kernel(const WalkArgs a) {
  extern __shared__ __align__(16) int32_t tile[];
  const int width = kKind == RDF2V_TOKENS_TRIPLES ? 2 * a.depth + 1 : a.depth + 1;
  const int64_t row0 = int64_t(blockIdx.x) * kBlock;
  const int nrows = int(min(int64_t(kBlock), a.walk_count - row0));
  const int t = threadIdx.x;
  const int2 *__restrict__ edges = reinterpret_cast<const int2 *>(a.edges);
  const v4i32 *__restrict__ walk_edges = reinterpret_cast<const v4i32 *>(a.walk_edges);
  const int32_t *__restrict__ row_ptr = a.row_ptr;
  const uint32_t V = uint32_t(a.num_entities);
  const uint32_t P = uint32_t(a.num_predicates);
  const uint32_t E = uint32_t(a.num_edges);

  int len = 0;
  int flags = 0;
  if (t < nrows) {
    int32_t *row = tile + t * width;
    const uint64_t w = uint64_t(a.walk_begin + row0 + t);
    int32_t e = a.start[w / uint64_t(a.walks_per_node)];
    row[0] = e;
    len = 1;
    bool alive = uint32_t(e) < V;
    if (!alive) flags |= RDF2V_STATUS_ID_OUT_OF_RANGE;
    int32_t lo = 0, hi = 0;
    if (alive) {
      lo = row_ptr[e];
      hi = row_ptr[e + 1];
    }
    for (int hb = 0; alive && hb < a.depth; hb += 4) {
      const Words4 r = philox_block(uint32_t(hb >> 2), w, a.key_lo, a.key_hi);
      const uint32_t words[4] = {r.w0, r.w1, r.w2, r.w3};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (hb + j >= a.depth) break;
        if (!kFused && hb + j > 0) {
          lo = row_ptr[e];
          hi = row_ptr[e + 1];
        }
        if (uint32_t(lo) > uint32_t(hi) || uint32_t(hi) > E) {
          flags |= RDF2V_STATUS_BAD_CSR;
          alive = false;
          break;
        }
        const uint32_t deg = uint32_t(hi - lo);
        if (deg == 0) {  // sink: the walk ends here
          alive = false;
          break;
        }
        const uint32_t k = __umulhi(words[j], deg);
        int32_t p, x;
        if (kFused) {
          const v4i32 rec = walk_edges[uint32_t(lo) + k];
          p = rec.x;
          x = rec.y;
          lo = rec.z;
          hi = rec.w;
        } else {
          const int2 rec = edges[uint32_t(lo) + k];
          p = rec.x;
          x = rec.y;
        }
        if (uint32_t(p) >= P || uint32_t(x) >= V) {
          flags |= RDF2V_STATUS_ID_OUT_OF_RANGE;
          alive = false;
          break;
        }
        if (kKind == RDF2V_TOKENS_TRIPLES) {
          row[len] = int32_t(V) + p;
          row[len + 1] = x;
          len += 2;
        } else {
          row[len] = kKind == RDF2V_TOKENS_ENTITIES ? x : int32_t(V) + p;
          len += 1;
        }
        e = x;
      }
    }
    for (int j = len; j < width; ++j) row[j] = -1;
  }
  __syncthreads();

  // The block's rows are one contiguous run of nrows * width tokens.
  const int64_t total = int64_t(nrows) * width;
  int32_t *dst = a.tokens + row0 * width;
  if ((reinterpret_cast<uintptr_t>(a.tokens) & 15) == 0) {
    const int64_t n4 = total >> 2;
    const v4i32 *src4 = reinterpret_cast<const v4i32 *>(tile);
    v4i32 *dst4 = reinterpret_cast<v4i32 *>(dst);
    for (int64_t i = t; i < n4; i += kBlock) __builtin_nontemporal_store(src4[i], dst4 + i);
    for (int64_t i = (n4 << 2) + t; i < total; i += kBlock) __builtin_nontemporal_store(tile[i], dst + i);
  } else {
    for (int64_t i = t; i < total; i += kBlock) __builtin_nontemporal_store(tile[i], dst + i);
  }
  if (t < nrows) __builtin_nontemporal_store(len, a.lens + row0 + t);
  if (flags != 0 && a.status != nullptr) atomicOr(a.status, flags);
}

template <int kBlock, int kKind>
void launch_kind(const WalkArgs &a, int64_t blocks, size_t lds, hipStream_t stream) {
  if (a.walk_edges != nullptr)
    random_walk_kernel<kBlock, true, kKind><<<dim3(unsigned(blocks)), dim3(kBlock), lds, stream>>>(a);
  else
    random_walk_kernel<kBlock, false, kKind><<<dim3(unsigned(blocks)), dim3(kBlock), lds, stream>>>(a);
}

template <int kBlock>
rdf2v_status launch_walk_kernel(const WalkArgs &a, hipStream_t stream) {
  const int width = a.token_kind == RDF2V_TOKENS_TRIPLES ? 2 * a.depth + 1 : a.depth + 1;
  const int64_t blocks = (a.walk_count + kBlock - 1) / kBlock;
  if (blocks >= (int64_t(1) << 31)) return RDF2V_ERR_TOO_LARGE;
  const size_t lds = size_t(kBlock) * width * 4;
  switch (a.token_kind) {
    case RDF2V_TOKENS_TRIPLES: launch_kind<kBlock, RDF2V_TOKENS_TRIPLES>(a, blocks, lds, stream); break;
    case RDF2V_TOKENS_ENTITIES: launch_kind<kBlock, RDF2V_TOKENS_ENTITIES>(a, blocks, lds, stream); break;
    case RDF2V_TOKENS_PROPERTIES: launch_kind<kBlock, RDF2V_TOKENS_PROPERTIES>(a, blocks, lds, stream); break;
    default: return RDF2V_ERR_INVALID_ARGUMENT;
  }
  RDF2V_LAUNCH_CHECK();
  return RDF2V_OK;
}

}  // namespace

rdf2v_status launch_random_walks(const WalkArgs &a, hipStream_t stream) {
  // The LDS tile holds kBlock rows of 2*depth+1 tokens: 256 rows up to depth
  // 16 (33.8 KB), 64 rows beyond (at most 33 KB at depth 64).
  return a.depth <= 16 ? launch_walk_kernel<256>(a, stream) : launch_walk_kernel<64>(a, stream);
}

}  // namespace rdf2v
