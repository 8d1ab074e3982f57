"""Pins for the CPU oracle: each test ties it to something other than itself.

* Philox4x32-10 against rocRAND's host-callable implementation (a black box
  compiled here; neither the oracle nor the GPU library includes it).
* The edge-index rule floor(u * deg / 2^32) against its closed-form cases.
* The CSR against numpy's stable argsort (a library routine) and invariants.
* Walks against closed forms (chain graph, sinks, power-of-two complete graphs
  whose every hop is rocRAND's word shifted), brute-force enumeration of all
  walks on tiny graphs, and chi-square uniformity on star graphs.

A plausible slip in the oracle (a dropped Philox term, a wrong word or block
index, walk id and hop swapped in the counter, an off-by-one in the index rule,
an unstable row order, a wrong predicate offset, wrong padding or length, batch
rows keyed on the row instead of the walk id) fails at least one of these.
"""

import itertools
import math

import numpy as np
import pytest
from scipy import stats

import oracle
import synth

U64 = np.uint64


# ----------------------------------------------------------------------------
# Philox4x32-10 (Salmon et al., SC'11) against rocRAND
# ----------------------------------------------------------------------------

def _philox_cases(n, seed=1):
    rng = np.random.default_rng(seed)
    seeds = rng.integers(0, 2**63, size=n, dtype=np.int64).astype(U64) * U64(2) + U64(1)
    walks = rng.integers(0, 2**40, size=n, dtype=np.int64).astype(U64)
    hops = rng.integers(0, 2**20, size=n, dtype=np.int64).astype(U64)
    # edge cases: zero / all-ones seeds, walk ids past 2^32, hops in later blocks
    extra = [(0, 0, 0), (0, 0, 1), (0, 0, 2), (0, 0, 3), (0, 0, 4), (42, 0, 7),
             (2**64 - 1, 2**64 - 1, 0), (42, 2**32, 5), (42, 2**32 - 1, 3), (42, 2**33 + 7, 16),
             (7, 123456789, 2**35 + 3), (2**32, 5, 9), (2**32 - 1, 5, 9)]
    ex = np.array(extra, dtype=U64)
    return np.concatenate([np.stack([seeds, walks, hops], axis=1), ex])


def test_philox_words_match_rocrand(rocrand_ref):
    cases = _philox_cases(20000)
    ref = rocrand_ref(1, cases)
    got = np.array([oracle.philox_word(int(s), int(w), int(h)) for s, w, h in cases], dtype=np.uint32)
    assert np.array_equal(got, ref)


def test_philox_blocks_match_rocrand(rocrand_ref):
    rng = np.random.default_rng(2)
    n = 5000
    rec = np.stack([rng.integers(0, 2**63, n, dtype=np.int64).astype(U64),
                    rng.integers(0, 2**63, n, dtype=np.int64).astype(U64),
                    rng.integers(0, 2**40, n, dtype=np.int64).astype(U64)], axis=1)
    ref = rocrand_ref(4, rec).reshape(n, 4)
    for i in range(n):
        seed, walk, block = (int(x) for x in rec[i])
        got = oracle.philox4x32_10([block & 0xFFFFFFFF, block >> 32, walk & 0xFFFFFFFF, walk >> 32],
                                   [seed & 0xFFFFFFFF, seed >> 32])
        assert np.array_equal(got, ref[i]), i


def test_philox_word_is_word_h_mod_4_of_block():
    # The four hops of one block read the four words of one Philox block.
    for seed, walk, block in [(42, 0, 0), (42, 17, 3), (2**40 + 5, 2**35, 2**33)]:
        blk = oracle.philox4x32_10([block & 0xFFFFFFFF, block >> 32, walk & 0xFFFFFFFF, walk >> 32],
                                   [seed & 0xFFFFFFFF, seed >> 32])
        words = [oracle.philox_word(seed, walk, 4 * block + j) for j in range(4)]
        assert words == [int(x) for x in blk]


# ----------------------------------------------------------------------------
# Edge index floor(u * deg / 2^32): closed forms
# ----------------------------------------------------------------------------

def test_edge_index_closed_forms():
    rng = np.random.default_rng(3)
    us = [0, 1, 2**31 - 1, 2**31, 2**32 - 2, 2**32 - 1] + [int(x) for x in rng.integers(0, 2**32, 3000)]
    for u in us:
        assert oracle.edge_index(u, 1) == 0
        for m in (1, 2, 5, 10, 20, 31):
            assert oracle.edge_index(u, 2**m) == u >> (32 - m)
    for deg in [1, 2, 3, 7, 10, 1000, 709_921, 2**31 - 1]:
        assert oracle.edge_index(0, deg) == 0
        assert oracle.edge_index(2**32 - 1, deg) == deg - 1
        ks = [oracle.edge_index(u, deg) for u in sorted(us)]
        assert all(0 <= k < deg for k in ks)
        assert all(a <= b for a, b in zip(ks, ks[1:]))  # monotone in u


def test_edge_index_bucket_sizes():
    # For deg = 3 the preimage of each index is an interval of length
    # ceil or floor of 2^32 / 3: the boundaries are the first u with u*3 >= k*2^32.
    deg = 3
    for k in range(1, deg):
        first = -(-(k << 32) // deg)  # ceil(k * 2^32 / deg)
        assert oracle.edge_index(first - 1, deg) == k - 1
        assert oracle.edge_index(first, deg) == k


# ----------------------------------------------------------------------------
# CSR against a stable sort by subject
# ----------------------------------------------------------------------------

def _stable_sort_csr(s, p, o, V):
    order = np.argsort(s, kind="stable")
    row_ptr = np.searchsorted(s[order], np.arange(V + 1), side="left").astype(np.int32)
    edges = np.stack([p[order], o[order]], axis=1).astype(np.int32)
    return row_ptr, edges


@pytest.mark.parametrize("V,P,T,seed", [(1, 1, 10, 0), (5, 3, 0, 1), (8, 4, 50, 2), (1000, 20, 5000, 3),
                                        (100_000, 50, 200_000, 4), (37, 1, 4096 * 3 + 17, 5)])
def test_csr_matches_stable_sort(V, P, T, seed):
    rng = np.random.default_rng(seed)
    s = rng.integers(0, V, T).astype(np.int32)
    p = rng.integers(0, P, T).astype(np.int32)
    o = rng.integers(0, V, T).astype(np.int32)
    row_ptr, edges = oracle.build_csr(s, p, o, V, P)
    rp_ref, ed_ref = _stable_sort_csr(s, p, o, V)
    assert np.array_equal(row_ptr, rp_ref)
    assert np.array_equal(edges, ed_ref)
    # invariants
    assert row_ptr[0] == 0 and row_ptr[-1] == T and np.all(np.diff(row_ptr) >= 0)


def test_csr_powerlaw_rows_keep_input_order():
    s, p, o = synth.powerlaw_triples(5000, 30, 60_000)
    row_ptr, edges = oracle.build_csr(s, p, o, 5000, 30)
    rp_ref, ed_ref = _stable_sort_csr(s, p, o, 5000)
    assert np.array_equal(row_ptr, rp_ref) and np.array_equal(edges, ed_ref)
    hub = int(np.argmax(np.diff(row_ptr)))
    idx = np.nonzero(s == hub)[0]
    assert np.array_equal(edges[row_ptr[hub]:row_ptr[hub + 1], 1], o[idx])


def test_csr_rejects_bad_input():
    s = np.array([0, 1, 2], np.int32); p = np.array([0, 0, 1], np.int32); o = np.array([1, 2, 0], np.int32)
    assert oracle.build_csr_status(s, p, o, 3, 3, 2) == oracle.OK
    assert oracle.build_csr_status(s, p, o, 3, 2, 2) == oracle.ERR_ID_OUT_OF_RANGE   # s=2 >= V
    assert oracle.build_csr_status(s, p, o, 3, 3, 1) == oracle.ERR_ID_OUT_OF_RANGE   # p=1 >= P
    assert oracle.build_csr_status(np.array([0, -1, 2], np.int32), p, o, 3, 3, 2) == oracle.ERR_ID_OUT_OF_RANGE
    assert oracle.build_csr_status(s, p, o, -1, 3, 2) == oracle.ERR_INVALID_ARGUMENT
    assert oracle.build_csr_status(s, p, o, 3, 2**31 - 2, 2) == oracle.ERR_TOO_LARGE


# ----------------------------------------------------------------------------
# Walks: closed forms
# ----------------------------------------------------------------------------

def _csr(triples, V, P):
    t = np.array(triples, dtype=np.int32).reshape(-1, 3)
    return oracle.build_csr(t[:, 0], t[:, 1], t[:, 2], V, P)


def test_chain_graph_walk_is_deterministic():
    n, P = 7, 5
    preds = [3, 0, 4, 1, 2, 2]
    rp, ed = _csr([(i, preds[i], i + 1) for i in range(n - 1)], n, P)
    for depth in (0, 1, 3, 6, 9):
        for seed in (0, 42, 2**63 + 11):
            tok, ln = oracle.random_walks(rp, ed, n, P, np.array([0, 4]), 3, depth, seed)
            for r in range(6):
                start = 0 if r < 3 else 4
                hops = min(depth, n - 1 - start)
                expect = [start]
                for h in range(hops):
                    expect += [n + preds[start + h], start + h + 1]
                expect += [-1] * (2 * depth + 1 - len(expect))
                assert tok[r].tolist() == expect
                assert ln[r] == 2 * hops + 1


def test_sink_start_gives_one_token():
    rp, ed = _csr([(0, 0, 1), (1, 0, 0)], 3, 1)  # entity 2 is a sink
    tok, ln = oracle.random_walks(rp, ed, 3, 1, np.array([2, 2]), 4, 5, 42)
    assert np.all(ln == 1)
    assert np.all(tok[:, 0] == 2) and np.all(tok[:, 1:] == -1)
    tok0, ln0 = oracle.random_walks(rp, ed, 3, 1, np.array([0]), 1, 0, 42)   # depth 0
    assert tok0.tolist() == [[0]] and ln0.tolist() == [1]


def test_walks_stop_exactly_at_first_sink():
    s, p, o = synth.powerlaw_triples(3000, 10, 6000, sink_fraction=0.3)
    V, P, d = 3000, 10, 6
    rp, ed = oracle.build_csr(s, p, o, V, P)
    deg = np.diff(rp)
    starts = oracle.nonsink_starts(rp, V)
    tok, ln = oracle.random_walks(rp, ed, V, P, starts, 5, d, 42)
    assert np.all(ln % 2 == 1) and np.all((ln >= 1) & (ln <= 2 * d + 1))
    for r in range(tok.shape[0]):
        L = ln[r]
        ents = tok[r, 0:L:2]
        assert np.all(deg[ents[:-1]] > 0)            # every entity before the last has out-edges
        if L < 2 * d + 1:
            assert deg[ents[-1]] == 0                # a walk stops early only at a sink
        if deg[ents[-1]] > 0:
            assert L == 2 * d + 1                    # a walk that ends off a sink used every hop
        assert np.all(tok[r, L:] == -1)
    assert np.any(ln < 2 * d + 1) and np.any(ln == 2 * d + 1)


@pytest.mark.parametrize("m,seed", [(1, 42), (3, 42), (4, 7), (5, 2**40 + 3)])
def test_power_of_two_complete_graph_follows_rocrand(rocrand_ref, m, seed):
    # Every entity v has out-edges j = 0..2^m-1 in input order, edge j = (pred j, obj j):
    # hop h of walk w goes to entity rocrand(seed, w, h) >> (32 - m), with predicate
    # token V + that same index. Pins the keying of the walk stream end to end.
    K = 2**m
    V, P, depth, wpn = K, K, 9, 3
    rp, ed = _csr([(v, j, j) for v in range(V) for j in range(K)], V, P)
    starts = np.arange(V, dtype=np.int32)[::-1].copy()
    walk_begin = 2  # a batch that does not start at walk 0
    tok, ln = oracle.random_walks(rp, ed, V, P, starts, wpn, depth, seed, walk_begin, V * wpn - 2)
    rows = np.arange(walk_begin, V * wpn, dtype=np.uint64)
    rec = np.array([(seed, w, h) for w in rows for h in range(depth)], dtype=np.uint64)
    choice = (rocrand_ref(1, rec).reshape(len(rows), depth) >> np.uint32(32 - m)).astype(np.int64)
    for r, w in enumerate(rows):
        expect = [int(starts[int(w) // wpn])]
        for h in range(depth):
            expect += [V + int(choice[r, h]), int(choice[r, h])]
        assert tok[r].tolist() == expect
        assert ln[r] == 2 * depth + 1


# ----------------------------------------------------------------------------
# Walks: brute-force enumeration and path frequencies on tiny graphs
# ----------------------------------------------------------------------------

def _enumerate_walks(rp, ed, V, start, depth):
    """{token tuple: probability} of every walk from start (Pi 1/deg over hops)."""
    out = {}

    def rec(e, toks, prob, h):
        lo, hi = rp[e], rp[e + 1]
        if h == depth or hi == lo:
            key = tuple(toks)
            out[key] = out.get(key, 0.0) + prob
            return
        for k in range(lo, hi):
            pp, x = int(ed[k, 0]), int(ed[k, 1])
            rec(x, toks + [V + pp, x], prob / (hi - lo), h + 1)

    rec(start, [start], 1.0, 0)
    return out


@pytest.mark.parametrize("gseed", [0, 1, 2])
def test_bruteforce_enumeration_and_frequencies(gseed):
    rng = np.random.default_rng(100 + gseed)
    V, P, E, depth = 6, 3, 12, 3
    s = rng.integers(0, V, E); p = rng.integers(0, P, E); o = rng.integers(0, V, E)
    s[:3] = 0; o[0] = 0                      # a self-loop on entity 0
    s[3] = s[4]; p[3] = p[4]; o[3] = o[4]    # a duplicate record
    rp, ed = oracle.build_csr(s, p, o, V, P)
    starts = oracle.nonsink_starts(rp, V)
    wpn = 40_000
    tok, ln = oracle.random_walks(rp, ed, V, P, starts, wpn, depth, 42 + gseed)
    for i, st in enumerate(starts):
        enum = _enumerate_walks(rp, ed, V, int(st), depth)
        rows = tok[i * wpn:(i + 1) * wpn]
        lens = ln[i * wpn:(i + 1) * wpn]
        counts = {}
        for r, L in zip(rows, lens):
            key = tuple(int(x) for x in r[:L])
            assert key in enum, key       # every emitted walk is a real walk of the graph
            counts[key] = counts.get(key, 0) + 1
        keys = sorted(enum)
        f_obs = np.array([counts.get(k, 0) for k in keys], dtype=float)
        f_exp = np.array([enum[k] * wpn for k in keys])
        if len(keys) > 1:
            assert stats.chisquare(f_obs, f_exp).pvalue > 1e-3


# ----------------------------------------------------------------------------
# Walks: uniform next-hop choice (chi-square on star graphs)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("K", [16, 10, 1000])
def test_star_first_hop_uniform(K):
    V = K + 1
    rp, ed = _csr([(0, j % 3, j + 1) for j in range(K)], V, 3)
    n = 1_600_000 if K == 1000 else 200_000
    tok, ln = oracle.random_walks(rp, ed, V, 3, np.array([0]), n, 1, 42)
    assert np.all(ln == 3)
    counts = np.bincount(tok[:, 2] - 1, minlength=K)
    assert stats.chisquare(counts).pvalue > 1e-3


def test_two_level_star_joint_uniform():
    # centre 0 -> K1 middles, each middle -> K2 leaves: (hop 0, hop 1) share a Philox block.
    K1, K2 = 7, 9
    tr = [(0, 0, 1 + i) for i in range(K1)]
    leaf = 1 + K1
    for i in range(K1):
        for j in range(K2):
            tr.append((1 + i, 1, leaf + i * K2 + j))
    V = leaf + K1 * K2
    rp, ed = _csr(tr, V, 2)
    n = 300_000
    tok, _ = oracle.random_walks(rp, ed, V, 2, np.array([0]), n, 2, 42)
    cell = tok[:, 4] - leaf
    counts = np.bincount(cell, minlength=K1 * K2)
    assert stats.chisquare(counts).pvalue > 1e-3


def test_hops_independent_across_blocks():
    # Complete graph on K=6 (non-power-of-two), depth 9: each hop's choice is uniform,
    # and hop pairs inside one Philox block and across blocks are independent.
    K = 6
    rp, ed = _csr([(v, 0, j) for v in range(K) for j in range(K)], K, 1)
    n = 120_000
    tok, _ = oracle.random_walks(rp, ed, K, 1, np.array([0]), n, 9, 42)
    ents = tok[:, 0::2]
    for h in range(1, 10):
        assert stats.chisquare(np.bincount(ents[:, h], minlength=K)).pvalue > 1e-3
    for a, b in [(1, 2), (1, 4), (1, 5), (4, 5), (3, 8), (1, 9)]:
        table = np.zeros((K, K))
        np.add.at(table, (ents[:, a], ents[:, b]), 1)
        assert stats.chi2_contingency(table).pvalue > 1e-3


# ----------------------------------------------------------------------------
# Walks on a generated workload: structure and batch invariance
# ----------------------------------------------------------------------------

def test_walk_structure_tiny_uniform():
    w = synth.WORKLOADS["tiny_uniform"]
    s, p, o = synth.triples(w)
    V, P, d = w.num_entities, w.num_predicates, w.depth
    rp, ed = oracle.build_csr(s, p, o, V, P)
    starts = oracle.nonsink_starts(rp, V)
    assert np.array_equal(starts, np.unique(s))
    tok, ln = oracle.random_walks(rp, ed, V, P, starts, w.walks_per_node, d, synth.WALK_SEED)
    assert tok.shape == (len(starts) * w.walks_per_node, 2 * d + 1)
    assert np.array_equal(tok[:, 0], np.repeat(starts, w.walks_per_node))
    triple_set = set(zip(s.tolist(), p.tolist(), o.tolist()))
    for r in range(tok.shape[0]):
        L = int(ln[r])
        assert L % 2 == 1
        row = tok[r]
        assert np.all((row[0:L:2] >= 0) & (row[0:L:2] < V))
        assert np.all((row[1:L:2] >= V) & (row[1:L:2] < V + P))
        for h in range((L - 1) // 2):
            assert (int(row[2 * h]), int(row[2 * h + 1]) - V, int(row[2 * h + 2])) in triple_set
    # walks of one start differ (the stream is keyed on the walk id)
    assert len({tuple(r) for r in tok[:w.walks_per_node].tolist()}) > 1


def test_batches_concatenate_to_one_shot():
    w = synth.WORKLOADS["tiny_uniform"]
    s, p, o = synth.triples(w)
    V, P = w.num_entities, w.num_predicates
    rp, ed = oracle.build_csr(s, p, o, V, P)
    starts = oracle.nonsink_starts(rp, V)
    total = len(starts) * 10
    full_t, full_l = oracle.random_walks(rp, ed, V, P, starts, 10, 6, 42)
    parts_t, parts_l, b = [], [], 0
    for size in itertools.cycle([1, 7, 333, 64, 1000]):
        if b >= total:
            break
        c = min(size, total - b)
        t, l = oracle.random_walks(rp, ed, V, P, starts, 10, 6, 42, b, c)
        parts_t.append(t); parts_l.append(l); b += c
    assert np.array_equal(np.concatenate(parts_t), full_t)
    assert np.array_equal(np.concatenate(parts_l), full_l)


def test_seed_changes_walks():
    w = synth.WORKLOADS["tiny_uniform"]
    s, p, o = synth.triples(w)
    rp, ed = oracle.build_csr(s, p, o, w.num_entities, w.num_predicates)
    starts = oracle.nonsink_starts(rp, w.num_entities)[:50]
    a, _ = oracle.random_walks(rp, ed, w.num_entities, w.num_predicates, starts, 4, 4, 42)
    b, _ = oracle.random_walks(rp, ed, w.num_entities, w.num_predicates, starts, 4, 4, 42)
    c, _ = oracle.random_walks(rp, ed, w.num_entities, w.num_predicates, starts, 4, 4, 43)
    assert np.array_equal(a, b) and not np.array_equal(a, c)


def test_walk_argument_errors():
    rp, ed = _csr([(0, 0, 1), (1, 0, 0)], 2, 1)
    with pytest.raises(oracle.OracleError) as e:
        oracle.random_walks(rp, ed, 2, 1, np.array([0]), 1, 65, 42)
    assert e.value.status == oracle.ERR_INVALID_ARGUMENT
    with pytest.raises(oracle.OracleError) as e:
        oracle.random_walks(rp, ed, 2, 1, np.array([5]), 1, 2, 42)
    assert e.value.status == oracle.ERR_ID_OUT_OF_RANGE
    with pytest.raises(oracle.OracleError) as e:
        oracle.random_walks(rp, ed, 2, 1, np.array([0]), 2, 2, 42, 1, 5)
    assert e.value.status == oracle.ERR_INVALID_ARGUMENT
    t, l = oracle.random_walks(rp, ed, 2, 1, np.array([0]), 0, 2, 42)
    assert t.shape == (0, 5) and l.shape == (0,)
