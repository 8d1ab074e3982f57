"""Graphs whose few used entity ids are spread over a huge id space, and the oracle's results
for them computed on the compact graph.

The walk rule reads an entity id only as an index (its row, its degree, the edge records of
its row; the Philox counter holds the walk id and the hop, never an entity). An order-keeping
relabel of the used ids U[0] < U[1] < ... < U[n-1] to 0..n-1 therefore changes nothing but the
labels: row i of the compact CSR is row U[i] of the full one, entities between two used ids
have no edges, and predicate tokens move from n + p to V + p. So the oracle can produce the
exact CSR, start set and walks of a graph with V close to 2^31 (whose direct run would need
tens of GiB of host memory) from the compact graph. test_sparse_ids.py checks that claim
against the oracle run directly on a 2^25-id space.
"""

import numpy as np

import oracle


def sparse_graph(V: int, P: int, T: int, n_random: int, seed: int):
    """(U, s_rank, pred, o_rank): the sorted used ids U (the extremes 0 and V-1 and the 8-bit
    digit boundaries among them) and T triples over their ranks. Subjects lean towards low
    ranks (rows of many sizes), about a tenth of the ids are never subjects (sinks), and the
    largest id keeps one self-loop under predicate P-1, so its walks emit V + P - 1."""
    rng = np.random.default_rng(seed)
    fixed = [0, 1, 255, 256, 65535, 65536, (1 << 24) - 1, 1 << 24, 1 << 30, V - 2, V - 1]
    U = np.unique(np.concatenate([np.array([x for x in fixed if 0 <= x < V], np.int64),
                                  rng.integers(0, V, n_random)]))
    n = U.size
    sink = rng.random(n) < 0.1
    sink[0] = sink[n - 1] = False
    subj_ranks = np.nonzero(~sink)[0]
    subj_ranks = subj_ranks[subj_ranks != n - 1]
    s_r = subj_ranks[(subj_ranks.size * rng.random(T - 1) ** 3).astype(np.int64)]
    p = rng.integers(0, P, T - 1)
    o_r = rng.integers(0, n, T - 1)
    s_r = np.append(s_r, n - 1)
    p = np.append(p, P - 1)
    o_r = np.append(o_r, n - 1)
    return U, s_r.astype(np.int32), p.astype(np.int32), o_r.astype(np.int32)


def expected_on_sparse(U, s_r, p, o_r, V: int, P: int, wpn: int, depth: int, seed: int):
    """(row_ptr[V+1], edges[T,2], starts, tokens, lens) of the graph with subjects U[s_r] and
    objects U[o_r] over V entities, from the oracle on the compact graph of n = U.size ids."""
    n = U.size
    rp_s, ed_s = oracle.build_csr(s_r, p, o_r, n, P)
    starts_s = oracle.nonsink_starts(rp_s, n)
    tok_s, ln_s = oracle.random_walks(rp_s, ed_s, n, P, starts_s, wpn, depth, seed)
    # row_ptr[v] = rp_s[#{i : U[i] < v}]: rp_s[0] up to U[0], rp_s[i] on (U[i-1], U[i]], rp_s[n]
    # on (U[n-1], V]
    reps = np.diff(np.concatenate([[-1], U, [V]]))
    row_ptr = np.repeat(rp_s, reps)
    edges = ed_s.copy()
    edges[:, 1] = U[ed_s[:, 1]]
    starts = U[starts_s].astype(np.int32)
    tok = np.where(tok_s < 0, -1, np.where(tok_s < n, U[np.clip(tok_s, 0, n - 1)], tok_s.astype(np.int64) - n + V))
    return row_ptr, edges, starts, tok.astype(np.int32), ln_s
