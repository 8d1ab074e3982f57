/*
 * rdf2v.h - C ABI of the MI355X (gfx950) RDF2vec random-walk corpus library.
 *
 * RDF2vec first extracts a corpus of graph walks from a knowledge graph and
 * then trains Word2Vec on it (gpuRDF2vec, Boeckling & Paulheim, arXiv
 * 2508.01073, Sec. 2). This library is the walk-extraction step for random
 * walks: it builds a subject-indexed graph from id triples and runs
 * walks_per_node uniform random walks of at most `depth` hops from each start
 * entity, emitting each walk as an entity/predicate token row padded with -1
 * (Sec. 3.1), with walks launched all at once rather than entity by entity
 * (Sec. 4.1).
 *
 * Conventions shared by every call:
 *  - Ids are int32. Entities are 0..num_entities-1, predicates are
 *    0..num_predicates-1; in walk rows an entity's token is its id and a
 *    predicate's token is num_entities + its id (Sec. 3.1: every entity and
 *    predicate is tokenised to an integer id). num_entities + num_predicates
 *    must stay below 2^31.
 *  - All array arguments are DEVICE pointers to caller-owned memory unless
 *    stated otherwise. The library never allocates, frees or keeps device
 *    memory and keeps no global state; calls on different streams may overlap.
 *    The one exception is rdf2v_skipgram_pairs_noalloc, which uses a fixed
 *    array of device memory that the library holds on each device.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream). Every
 *    call only enqueues work on it and returns without synchronising.
 *  - Errors that the host can see (null pointers, negative or oversized
 *    counts, workspace too small) are returned synchronously and nothing is
 *    enqueued. Errors that only the device can see (ids out of range, an
 *    inconsistent CSR) are ORed as RDF2V_STATUS_* bits into *status_dev, a
 *    device int32 that the caller zeroes beforehand and reads after the stream
 *    has synchronised; status_dev may be NULL, in which case such errors are
 *    not reported. After a device-side error the outputs are unspecified, but
 *    every memory access stays inside the buffers described here.
 */
#ifndef RDF2V_H_
#define RDF2V_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum rdf2v_status {
  RDF2V_OK = 0,
  RDF2V_ERR_INVALID_ARGUMENT = 1, /* null pointer, negative count, depth outside [0, RDF2V_MAX_DEPTH], walk range outside the corpus */
  RDF2V_ERR_ID_OUT_OF_RANGE = 2,  /* an id the host can already see is out of range (e.g. triples with num_entities == 0) */
  RDF2V_ERR_TOO_LARGE = 3,        /* num_triples >= 2^31, num_entities + num_predicates >= 2^31, walk counts overflowing int64 */
  RDF2V_ERR_WORKSPACE = 4,        /* workspace NULL or smaller than the matching *_workspace_size() */
  RDF2V_ERR_HIP = 5               /* a HIP launch or runtime call failed */
} rdf2v_status;

/* Bits ORed into *status_dev by the kernels. */
#define RDF2V_STATUS_ID_OUT_OF_RANGE 0x1 /* a subject/object/start id >= num_entities or < 0, or a predicate id out of range */
#define RDF2V_STATUS_BAD_CSR 0x2         /* row_ptr not non-decreasing within [0, num_edges] */
#define RDF2V_STATUS_BAD_LENGTH 0x4      /* a walk length outside [0, row_width] (treated as clamped), or a bad string offset */
#define RDF2V_STATUS_CAPACITY 0x8        /* more results than the output holds (the rest are not written), or more distinct strings than a vocabulary bound */

/* Longest walk, in hops. A walk row holds 2 * depth + 1 tokens. */
#define RDF2V_MAX_DEPTH 64

/*
 * A read-only VIEW of a subject-indexed CSR in device memory, as written by
 * rdf2v_build_csr:
 *   row_ptr[num_entities + 1]: int32, row_ptr[0] = 0, non-decreasing,
 *                              row_ptr[num_entities] = num_edges.
 *   edges[num_edges][2]:       int32 (predicate, object) out-edge records of
 *                              entity v at rows row_ptr[v] .. row_ptr[v+1]-1;
 *                              8-byte aligned.
 * Duplicate triples and self-loops are separate records.
 */
typedef struct rdf2v_csr {
  int32_t num_entities;
  int32_t num_predicates;
  int64_t num_edges;
  const int32_t *row_ptr;
  const int32_t *edges;
  /* Optional (may be NULL): the same out-edge records extended with the row
   * bounds of their object, as written by rdf2v_build_walk_edges:
   * walk_edges[num_edges][4] = (predicate, object, row_ptr[object],
   * row_ptr[object + 1]), 16-byte aligned. When present, rdf2v_random_walks
   * reads one 16-byte record per hop instead of a record plus the next
   * entity's row bounds; the walks are identical either way. */
  const int32_t *walk_edges;
} rdf2v_csr;

/*
 * Bytes of device workspace rdf2v_build_csr needs for these sizes (0 when
 * num_triples == 0). Pure host function.
 */
size_t rdf2v_build_csr_workspace_size(int64_t num_triples, int32_t num_entities);

/*
 * Triples -> subject-indexed CSR (the graph the walks traverse; gpuRDF2vec
 * Sec. 3.1 loads the tokenised triples into device memory as a graph).
 *
 *   subj, pred, obj   [num_triples] int32 ids (device).
 *   row_ptr_out       [num_entities + 1] int32 (device), written.
 *   edges_out         [num_triples][2] int32 (predicate, object) (device),
 *                     written; 8-byte aligned; must not alias the inputs.
 *   workspace         device scratch of at least
 *                     rdf2v_build_csr_workspace_size(num_triples, num_entities)
 *                     bytes, 256-byte aligned; contents clobbered.
 *   status_dev        device int32 or NULL (RDF2V_STATUS_ID_OUT_OF_RANGE).
 *
 * Inside every row the records keep the input order of their triples (a
 * stable sort by subject), so the result is deterministic and equal to a
 * sequential counting sort. Runs as histogram, scan and stable-scatter passes
 * of an LSD radix sort on the subject id followed by a row-offset kernel.
 */
rdf2v_status rdf2v_build_csr(const int32_t *subj, const int32_t *pred, const int32_t *obj,
                             int64_t num_triples, int32_t num_entities, int32_t num_predicates,
                             int32_t *row_ptr_out, int32_t *edges_out, void *workspace,
                             size_t workspace_bytes, int32_t *status_dev, void *stream);

/*
 * Walk records: for every out-edge record k of the CSR,
 *   walk_edges_out[k] = (edges[k][0], edges[k][1], row_ptr[o], row_ptr[o + 1])
 * with o = edges[k][1], so that a walk learns the row of the entity it moves
 * to from the record it has just read (one random access per hop; the walk
 * definition is unchanged).
 *
 *   csr             CSR view (row_ptr and edges are read; walk_edges ignored).
 *   walk_edges_out  [num_edges][4] int32 (device), written; 16-byte aligned.
 *   status_dev      device int32 or NULL: RDF2V_STATUS_ID_OUT_OF_RANGE if an
 *                   object id is out of range (its row bounds are written as
 *                   0, 0).
 */
rdf2v_status rdf2v_build_walk_edges(const rdf2v_csr *csr, int32_t *walk_edges_out,
                                    int32_t *status_dev, void *stream);

/*
 * Whether walk records are expected to make rdf2v_random_walks faster on a
 * CSR of this size than row_ptr and edges read directly (the walks are
 * identical either way). Pure host function; 1 = build them, 0 = do not.
 *
 * Without records a hop reads the current entity's row bounds and then one
 * 8-byte record; with them it reads one 16-byte record from a table twice as
 * large. While row_ptr (4 * (num_entities + 1) bytes) stays resident in each
 * XCD's 4 MB L2 the bound read is a cache hit and the smaller record table
 * wins; beyond that every hop pays a second cache miss. Measured crossover on
 * gfx950 (uniform and power-law graphs, mean out-degree 20, depth 8):
 * row_ptr between 1.2 and 2.0 MB, so this returns 1 when row_ptr is larger
 * than 1.5 MiB and num_edges > 0. Negative sizes return 0.
 */
int32_t rdf2v_walk_edges_recommended(int32_t num_entities, int64_t num_edges);

/* Bytes of device workspace rdf2v_nonsink_starts needs. Pure host function. */
size_t rdf2v_nonsink_starts_workspace_size(int32_t num_entities);

/*
 * The default start set: every entity with at least one out-edge, ascending
 * (the paper starts walks from all entities when no start list is given,
 * Sec. 3.3; an entity without out-edges would only give a one-token walk).
 *
 *   starts_out  [num_entities] int32 (device): the first *count_out entries
 *               are written.
 *   count_out   one int64 in device memory: the number of start entities.
 *   workspace   device scratch, rdf2v_nonsink_starts_workspace_size() bytes,
 *               256-byte aligned.
 */
rdf2v_status rdf2v_nonsink_starts(const rdf2v_csr *csr, int32_t *starts_out, int64_t *count_out,
                                  void *workspace, size_t workspace_bytes, void *stream);

/*
 * Uniform random walks (gpuRDF2vec Sec. 2: iterative random choice of the
 * next hop; Sec. 3.1: triple-based token rows padded with -1; Sec. 4.1: all
 * walks of all start entities launched together).
 *
 * The corpus has num_walks = num_start * walks_per_node walks; walk w starts
 * at start_nodes[w / walks_per_node]. This call computes walks
 * w = walk_begin .. walk_begin + walk_count - 1 into rows r = w - walk_begin,
 * so a corpus can be produced in batches and any batch recomputed on its own.
 *
 * Walk w, from entity e_0 = start_nodes[w / walks_per_node], for hops
 * h = 0 .. depth-1: if e_h has no out-edge the walk ends; otherwise with
 * u = word (h mod 4) of Philox4x32-10(key = seed, counter = (h / 4, w)) (the
 * 64-bit seed as key words lo, hi; the counter words are lo, hi of h / 4 then
 * lo, hi of w; Salmon et al., SC'11), the walk takes out-edge record
 * k = floor(u * deg(e_h) / 2^32) of e_h's row, (p, x), and appends tokens
 * num_entities + p and x; e_{h+1} = x.
 *
 *   csr           view of a CSR as rdf2v_build_csr writes it (host pointer to
 *                 the struct; the arrays it points to are device memory). If
 *                 csr->walk_edges is set it must hold rdf2v_build_walk_edges'
 *                 records for this CSR; csr->edges is then not read.
 *   start_nodes   [num_start] int32 entity ids (device); duplicates and sinks
 *                 allowed.
 *   depth         hops per walk, 0 .. RDF2V_MAX_DEPTH.
 *   tokens_out    [walk_count][2 * depth + 1] int32 (device), row-major:
 *                 e_0, V+p_0, e_1, V+p_1, ..., then -1 after the walk's end.
 *   len_out       [walk_count] int32 (device): valid tokens, 2 * hops + 1.
 *   status_dev    device int32 or NULL (RDF2V_STATUS_* bits).
 *
 * walks_per_node == 0 or walk_count == 0 enqueues nothing and returns
 * RDF2V_OK.
 */
rdf2v_status rdf2v_random_walks(const rdf2v_csr *csr, const int32_t *start_nodes, int64_t num_start,
                                int32_t walks_per_node, int32_t depth, uint64_t seed,
                                int64_t walk_begin, int64_t walk_count, int32_t *tokens_out,
                                int32_t *len_out, int32_t *status_dev, void *stream);

/* Bytes of device workspace rdf2v_skipgram_pairs needs. Pure host function;
 * 0 when num_walks is negative or above 2^46 (rdf2v_skipgram_pairs returns
 * RDF2V_ERR_TOO_LARGE for more rows). */
size_t rdf2v_skipgram_pairs_workspace_size(int64_t num_walks);

/*
 * Skip-gram training pairs from walk rows (gpuRDF2vec Sec. 3.2: the data
 * module turns the walk corpus into center-context pairs; Sec. 3.1: the -1
 * padding is dropped first).
 *
 * For walk r with L = len[r] valid tokens t_0 .. t_{L-1}, every center
 * position i and every context position j with 1 <= |i - j| <= window and
 * 0 <= j < L give the pair (t_i, t_j); pairs are ordered by walk, then i, then
 * j. A walk of L tokens gives 2 * sum_{d=1}^{min(window, L-1)} (L - d) pairs.
 *
 *   tokens          [num_walks][row_width] int32 walk rows (device), as
 *                   rdf2v_random_walks writes them.
 *   len             [num_walks] int32 valid tokens per row (device).
 *   row_width       1 .. 2 * RDF2V_MAX_DEPTH + 1.
 *   window          >= 0 (the paper's example uses 5).
 *   pairs_out       [pair_capacity][2] int32 (center, context) (device); may
 *                   be NULL when pair_capacity == 0 (count only).
 *   pair_count_out  one int64 in device memory: the total number of pairs,
 *                   also when it exceeds pair_capacity (then only the first
 *                   pair_capacity pairs are written and RDF2V_STATUS_CAPACITY
 *                   is raised).
 *   workspace       device scratch, rdf2v_skipgram_pairs_workspace_size()
 *                   bytes, 256-byte aligned.
 *   status_dev      device int32 or NULL.
 */
rdf2v_status rdf2v_skipgram_pairs(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                                  int32_t row_width, int32_t window, int32_t *pairs_out,
                                  int64_t pair_capacity, int64_t *pair_count_out, void *workspace,
                                  size_t workspace_bytes, int32_t *status_dev, void *stream);

/* Most walk rows one rdf2v_skipgram_pairs_noalloc call takes, and the size of
 * the device array it uses for its scratch on each device (32 MiB + 64 KiB). */
#define RDF2V_NOALLOC_MAX_WALKS ((int64_t)1 << 22)
#define RDF2V_NOALLOC_SCRATCH_BYTES (((size_t)32 << 20) + ((size_t)64 << 10))

/*
 * rdf2v_skipgram_pairs for callers that cannot allocate device memory (code
 * being captured into a graph, tight serving loops, harnesses that forbid
 * hipMalloc): the same pairs, count and status, with the same arguments
 * except that there is no workspace. The scratch (per-walk output offsets and
 * block sums) lives instead in a device array of RDF2V_NOALLOC_SCRATCH_BYTES
 * that the library holds on every device it runs on until the process ends;
 * the first call on a device looks its address up (making that device current
 * for the lookup and restoring the caller's current device). The call itself
 * allocates nothing.
 *
 *   num_walks   0 .. RDF2V_NOALLOC_MAX_WALKS; more returns
 *               RDF2V_ERR_TOO_LARGE and enqueues nothing (split the rows into
 *               batches, or use rdf2v_skipgram_pairs with a workspace).
 *   stream      the device whose array is used is the stream's device.
 *
 * All calls on one device share its array and its contents persist between
 * calls: calls that overlap on one device (on different streams or from
 * different threads) race and give wrong pairs. Serialise them, e.g. on one
 * stream. No part of the array needs clearing between calls.
 */
rdf2v_status rdf2v_skipgram_pairs_noalloc(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                                          int32_t row_width, int32_t window, int32_t *pairs_out,
                                          int64_t pair_capacity, int64_t *pair_count_out, int32_t *status_dev,
                                          void *stream);

/* Bytes of device workspace rdf2v_cbow_examples needs. Pure host function;
 * 0 when num_walks is negative or above 2^46 (rdf2v_cbow_examples returns
 * RDF2V_ERR_TOO_LARGE for more rows). */
size_t rdf2v_cbow_examples_workspace_size(int64_t num_walks);

/*
 * CBOW training examples from walk rows (gpuRDF2vec Sec. 3.2: the library
 * trains Continuous Bag of Words next to Skip-Gram; CBOW predicts a center
 * token from the tokens around it; Sec. 3.1: the -1 padding is dropped).
 *
 * For walk r with L = len[r] valid tokens t_0 .. t_{L-1}, every position i
 * gives one example: the center t_i and its contexts, the t_j with
 * 1 <= |i - j| <= window and 0 <= j < L in ascending j, followed by -1 up to
 * 2 * window entries. Examples are ordered by walk, then i; a walk of L tokens
 * gives L examples (a one-token walk gives one with no context). Read in order,
 * the (center, context) of the non-padding contexts are exactly the pairs of
 * rdf2v_skipgram_pairs with the same window.
 *
 *   tokens, len, row_width  as for rdf2v_skipgram_pairs.
 *   window          1 .. 2 * RDF2V_MAX_DEPTH.
 *   centers_out     [capacity] int32 (device); may be NULL when capacity == 0.
 *   contexts_out    [capacity][2 * window] int32 (device), row-major; may be
 *                   NULL when capacity == 0.
 *   count_out       one int64 in device memory: the number of examples (the sum
 *                   of the lengths), also when it exceeds capacity (then only
 *                   the first capacity examples are written and
 *                   RDF2V_STATUS_CAPACITY is raised).
 *   workspace       device scratch, rdf2v_cbow_examples_workspace_size() bytes,
 *                   256-byte aligned.
 *   status_dev      device int32 or NULL (RDF2V_STATUS_BAD_LENGTH for a length
 *                   outside [0, row_width], treated as clamped;
 *                   RDF2V_STATUS_CAPACITY).
 */
rdf2v_status rdf2v_cbow_examples(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                                 int32_t row_width, int32_t window, int32_t *centers_out, int32_t *contexts_out,
                                 int64_t capacity, int64_t *count_out, void *workspace, size_t workspace_bytes,
                                 int32_t *status_dev, void *stream);

/* Which tokens a walk row holds (Tab. 1 lists entity walks and property walks
 * beside triple-based random walks). All three follow the same walk, drawn
 * from the same random stream, so an entity or property walk is exactly the
 * projection of the triple-based walk with the same walk id. */
typedef enum rdf2v_walk_tokens {
  RDF2V_TOKENS_TRIPLES = 0,   /* e_0, V+p_0, e_1, ..., e_h: 2*depth+1 tokens per row */
  RDF2V_TOKENS_ENTITIES = 1,  /* e_0, e_1, ..., e_h: depth+1 tokens per row */
  RDF2V_TOKENS_PROPERTIES = 2 /* e_0, V+p_0, ..., V+p_{h-1}: depth+1 tokens per row */
} rdf2v_walk_tokens;

/*
 * rdf2v_random_walks with a choice of tokens: identical arguments plus
 * token_kind; tokens_out holds walk_count rows of 2*depth+1 (TRIPLES) or
 * depth+1 (ENTITIES, PROPERTIES) tokens, padded with -1, and len_out the
 * valid tokens per row (2*hops+1 or hops+1).
 */
rdf2v_status rdf2v_random_walks_tokens(const rdf2v_csr *csr, const int32_t *start_nodes,
                                       int64_t num_start, int32_t walks_per_node, int32_t depth,
                                       uint64_t seed, int64_t walk_begin, int64_t walk_count,
                                       int32_t token_kind, int32_t *tokens_out, int32_t *len_out,
                                       int32_t *status_dev, void *stream);

/* Bytes of device workspace rdf2v_unique_walks needs. Pure host function;
 * 0 when num_walks is negative or above 255 * 2^31 (rdf2v_unique_walks
 * returns RDF2V_ERR_TOO_LARGE for more rows). */
size_t rdf2v_unique_walks_workspace_size(int64_t num_walks);

/*
 * Duplicate-free walks (Tab. 1: "random walk duplicate free"): rows come in
 * groups of group_size consecutive rows (the walks of one start entity, as
 * rdf2v_random_walks writes them for walks_per_node = group_size; the last
 * group may be shorter). Within each group only the first occurrence, in row
 * order, of each distinct walk is kept; two rows are the same walk when their
 * lengths and their first len tokens agree. Kept rows are written, in order,
 * to tokens_out / len_out, and their number to *count_out (device int64).
 *
 *   tokens, len      [num_walks][row_width] and [num_walks] int32 (device).
 *   tokens_out, len_out  room for num_walks rows (device); must not alias the
 *                    inputs.
 *   workspace        rdf2v_unique_walks_workspace_size(num_walks) bytes of
 *                    device scratch, 256-byte aligned.
 */
rdf2v_status rdf2v_unique_walks(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                                int32_t group_size, int32_t row_width, int32_t *tokens_out,
                                int32_t *len_out, int64_t *count_out, void *workspace,
                                size_t workspace_bytes, int32_t *status_dev, void *stream);

/* Bytes of device workspace rdf2v_bfs_walks needs. Pure host function;
 * 0 when a size is negative or num_roots >= 2^31 (rdf2v_bfs_walks returns
 * RDF2V_ERR_TOO_LARGE for that many roots). */
size_t rdf2v_bfs_walks_workspace_size(int32_t num_entities, int64_t num_roots);

/*
 * BFS walks (gpuRDF2vec Sec. 3.1: a BFS from each root gives every reached
 * entity one predecessor, the first entity to reach it, and each leaf-to-root
 * path of that tree is one walk, so an entity appears at most once per root).
 *
 * The tree is that of a queue-order BFS limited to `depth` hops: the entities
 * of one level are expanded in the order they were reached, each through its
 * out-edge records in CSR order, and an entity not yet in the tree gets the
 * current entity and record as its parent. Tree entities without a child
 * (including every entity at the depth limit) are leaves; in the order they
 * were reached, the first max_walks of them give the walks
 * root, V+p_1, v_1, ..., leaf.
 *
 *   csr          CSR view (row_ptr and edges are read).
 *   roots        [num_roots] int32 entity ids (device).
 *   tokens_out   [num_roots][max_walks][2 * depth + 1] int32 (device): the
 *                first counts_out[r] rows of root r are written (padded with
 *                -1); the rest are left untouched.
 *   len_out      [num_roots][max_walks] int32, written like tokens_out.
 *   counts_out   [num_roots] int32: walks written per root. A root with more
 *                leaves than max_walks raises RDF2V_STATUS_CAPACITY.
 *   workspace    rdf2v_bfs_walks_workspace_size(V, num_roots) bytes (12 bytes
 *                per root plus at most about 4 GiB), 256-byte aligned.
 */
rdf2v_status rdf2v_bfs_walks(const rdf2v_csr *csr, const int32_t *roots, int64_t num_roots, int32_t depth,
                             int32_t max_walks, int32_t *tokens_out, int32_t *len_out, int32_t *counts_out,
                             void *workspace, size_t workspace_bytes, int32_t *status_dev, void *stream);

/* Largest num_triples and bound on distinct strings rdf2v_build_vocabulary takes. */
#define RDF2V_VOCAB_MAX_TRIPLES ((int64_t)1 << 30)
#define RDF2V_VOCAB_MAX_DISTINCT ((int64_t)1 << 30)

/* Bytes of device workspace rdf2v_build_vocabulary needs (0 for arguments it
 * rejects). Pure host function. */
size_t rdf2v_build_vocabulary_workspace_size(int64_t num_triples, int64_t max_entities, int64_t max_predicates);

/*
 * Vocabulary (gpuRDF2vec Sec. 3.1: every entity and predicate is tokenised to
 * an integer id at the start of the pipeline): string triples -> the int32 id
 * triples that rdf2v_build_csr takes.
 *
 * Entity ids number the distinct subject and object strings 0, 1, ... in the
 * order they first appear in s_0, o_0, s_1, o_1, ...; predicate ids number the
 * distinct predicate strings in the order they first appear in p_0, p_1, ....
 * Strings are compared as byte sequences (any bytes, NUL included; the empty
 * string is a string). The result is deterministic.
 *
 * Each column is given as
 *   X_chars     uint8 bytes of all strings of the column (device), 4-byte
 *               aligned; may be NULL when X_bytes == 0.
 *   X_offsets   [num_triples + 1] int64 (device): string t of the column is
 *               X_chars[X_offsets[t] .. X_offsets[t + 1]). Offsets outside
 *               [0, X_bytes] or decreasing raise RDF2V_STATUS_BAD_LENGTH (the
 *               string is then read as empty).
 *   X_bytes     length of X_chars in bytes (nothing past it is read).
 * for X = subj, pred, obj.
 *
 *   num_triples     0 .. RDF2V_VOCAB_MAX_TRIPLES.
 *   max_entities,   caller's upper bounds on the distinct entity and predicate
 *   max_predicates  strings, 1 .. RDF2V_VOCAB_MAX_DISTINCT; they size the hash
 *                   tables (2 to 4 slots of 132 B per bounded string). More distinct
 *                   strings than a bound raise RDF2V_STATUS_CAPACITY.
 *   subj_ids, pred_ids, obj_ids  [num_triples] int32 outputs (device).
 *   counts_out      [2] int64 (device): distinct entities, distinct predicates.
 *   workspace       rdf2v_build_vocabulary_workspace_size(num_triples,
 *                   max_entities, max_predicates) bytes, 256-byte aligned.
 *   status_dev      device int32 or NULL (RDF2V_STATUS_BAD_LENGTH,
 *                   RDF2V_STATUS_CAPACITY).
 */
rdf2v_status rdf2v_build_vocabulary(const uint8_t *subj_chars, const int64_t *subj_offsets, int64_t subj_bytes,
                                    const uint8_t *pred_chars, const int64_t *pred_offsets, int64_t pred_bytes,
                                    const uint8_t *obj_chars, const int64_t *obj_offsets, int64_t obj_bytes,
                                    int64_t num_triples, int64_t max_entities, int64_t max_predicates,
                                    int32_t *subj_ids, int32_t *pred_ids, int32_t *obj_ids, int64_t *counts_out,
                                    void *workspace, size_t workspace_bytes, int32_t *status_dev, void *stream);

/* Static, human-readable name of a status code (any int: values that are not
 * an rdf2v_status give "RDF2V_UNKNOWN_STATUS"). */
const char *rdf2v_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* RDF2V_H_ */
