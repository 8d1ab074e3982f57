"""Pins for the oracle's skip-gram pair generation (gpuRDF2vec Sec. 3.2: the data
module turns the walk corpus into center-context pairs; Sec. 3.1: padding is
dropped). Each test checks the oracle against something other than itself: a
hand-worked example, an independent numpy construction by offsets, the closed
form of the pair count, and structural invariants."""

import numpy as np
import pytest

import oracle
import synth


def test_hand_worked_window_1_and_2():
    # One walk a b c d (padded), worked out by hand from the definition.
    tok = np.array([[10, 20, 30, 40, -1, -1, -1]], np.int32)
    ln = np.array([4], np.int32)
    assert oracle.skipgram_pairs(tok, ln, 1).tolist() == [
        [10, 20], [20, 10], [20, 30], [30, 20], [30, 40], [40, 30]]
    assert oracle.skipgram_pairs(tok, ln, 2).tolist() == [
        [10, 20], [10, 30],
        [20, 10], [20, 30], [20, 40],
        [30, 10], [30, 20], [30, 40],
        [40, 20], [40, 30]]
    assert oracle.skipgram_pairs(tok, ln, 0).shape == (0, 2)


def _by_offsets(tok, ln, window):
    """Independent construction: for each offset d in +-1..+-window, pair position i with
    i + d over the valid prefix, then order by (walk, i, i + d)."""
    recs = []
    for r in range(tok.shape[0]):
        L = int(ln[r])
        t = tok[r, :L]
        pos = np.arange(L)
        for d in list(range(-window, 0)) + list(range(1, window + 1)):
            ok = (pos + d >= 0) & (pos + d < L)
            i = pos[ok]
            recs.append(np.stack([np.full(i.size, r), i, i + d, t[i], t[i + d]], axis=1))
    if not recs:
        return np.zeros((0, 2), np.int32)
    a = np.concatenate(recs)
    a = a[np.lexsort((a[:, 2], a[:, 1], a[:, 0]))]
    return a[:, 3:5].astype(np.int32)


@pytest.mark.parametrize("window", [1, 2, 5, 9, 40])
def test_matches_offset_construction_on_real_walks(window):
    w = synth.WORKLOADS["tiny_uniform"]
    s, p, o = synth.triples(w)
    rp, ed = oracle.build_csr(s, p, o, w.num_entities, w.num_predicates)
    st = oracle.nonsink_starts(rp, w.num_entities)[:150]
    tok, ln = oracle.random_walks(rp, ed, w.num_entities, w.num_predicates, st, 4, 6, 42)
    pairs = oracle.skipgram_pairs(tok, ln, window)
    assert np.array_equal(pairs, _by_offsets(tok, ln, window))


def _count(L, window):
    m = min(window, L - 1)
    return 0 if m <= 0 else 2 * (m * L - m * (m + 1) // 2)


def test_pair_count_closed_form_and_invariants():
    rng = np.random.default_rng(0)
    width = 17
    n = 400
    ln = rng.integers(0, width + 1, n).astype(np.int32)
    tok = np.full((n, width), -1, np.int32)
    for r in range(n):
        tok[r, :ln[r]] = rng.integers(0, 1000, ln[r])
    for window in [0, 1, 3, 5, 16, 100]:
        pairs = oracle.skipgram_pairs(tok, ln, window)
        assert pairs.shape[0] == sum(_count(int(L), window) for L in ln)
        assert not np.any(pairs == -1)                         # padding never appears
        a = pairs[np.lexsort((pairs[:, 1], pairs[:, 0]))]
        b = pairs[:, ::-1][np.lexsort((pairs[:, 0], pairs[:, 1]))]
        assert np.array_equal(a, b)                            # (x, y) and (y, x) equally often


def test_capacity_truncates_but_counts_all():
    tok = np.array([[1, 2, 3]], np.int32)
    ln = np.array([3], np.int32)
    lib = oracle._load()
    out = np.full((3, 2), -7, np.int32)
    n = lib.rdf2v_ref_skipgram_pairs(oracle._ptr(tok), oracle._ptr(ln), 1, 3, 1, oracle._ptr(out), 2)
    assert n == 4 and out[:2].tolist() == [[1, 2], [2, 1]] and out[2].tolist() == [-7, -7]


# ----------------------------------------------------------------------------
# Entity walks and property walks (projections of the triple-based walk)
# ----------------------------------------------------------------------------

def test_projection_hand_worked():
    V = 100
    # walk 7 -p3-> 8 -p1-> 9 (2 hops of depth 3), and a sink start 5
    tok = np.array([[7, V + 3, 8, V + 1, 9, -1, -1], [5, -1, -1, -1, -1, -1, -1]], np.int32)
    ln = np.array([5, 1], np.int32)
    ent, el = oracle.project_walks(tok, ln, 3, oracle.ENTITY_WALKS)
    assert ent.tolist() == [[7, 8, 9, -1], [5, -1, -1, -1]] and el.tolist() == [3, 1]
    prop, pl = oracle.project_walks(tok, ln, 3, oracle.PROPERTY_WALKS)
    assert prop.tolist() == [[7, V + 3, V + 1, -1], [5, -1, -1, -1]] and pl.tolist() == [3, 1]


def test_projection_matches_slicing_on_real_walks():
    w = synth.WORKLOADS["tiny_uniform"]
    s, p, o = synth.triples(w)
    V = w.num_entities
    rp, ed = oracle.build_csr(s, p, o, V, w.num_predicates)
    st = oracle.nonsink_starts(rp, V)
    d = 6
    tok, ln = oracle.random_walks(rp, ed, V, w.num_predicates, st, 3, d, 42)
    ent, el = oracle.project_walks(tok, ln, d, oracle.ENTITY_WALKS)
    prop, pl = oracle.project_walks(tok, ln, d, oracle.PROPERTY_WALKS)
    assert np.array_equal(el, (ln + 1) // 2) and np.array_equal(pl, (ln + 1) // 2)
    for r in range(tok.shape[0]):
        L = int(ln[r])
        assert ent[r, :el[r]].tolist() == tok[r, 0:L:2].tolist()          # even positions
        assert prop[r, :pl[r]].tolist() == [int(tok[r, 0])] + tok[r, 1:L:2].tolist()
        assert np.all(ent[r, el[r]:] == -1) and np.all(prop[r, pl[r]:] == -1)
        assert np.all(ent[r, :el[r]] < V) and np.all(prop[r, 1:pl[r]] >= V)


# ----------------------------------------------------------------------------
# Duplicate-free walks
# ----------------------------------------------------------------------------

def test_unique_walks_hand_worked():
    tok = np.array([[1, 5, 2], [1, 5, 2], [1, 6, 3], [1, -1, -1], [1, 5, 2],   # group of start 1
                    [4, 5, 2], [4, -1, -1], [4, -1, 9]], np.int32)            # group of start 4
    ln = np.array([3, 3, 3, 1, 3, 3, 1, 1], np.int32)
    rows, lens = oracle.unique_walks(tok, ln, 5)
    # rows 1 and 4 repeat row 0; row 7 equals row 6 on its valid prefix (padding ignored)
    assert rows.tolist() == [[1, 5, 2], [1, 6, 3], [1, -1, -1], [4, 5, 2], [4, -1, -1]]
    assert lens.tolist() == [3, 3, 1, 3, 1]


def test_unique_walks_match_set_construction():
    # tiny graph with few distinct walks: many duplicates per start
    rp, ed = oracle.build_csr(np.array([0, 0, 1, 1, 2], np.int32), np.array([0, 1, 0, 0, 1], np.int32),
                              np.array([1, 2, 2, 0, 0], np.int32), 3, 2)
    starts = np.array([0, 1, 2, 0], np.int32)
    wpn = 40
    tok, ln = oracle.random_walks(rp, ed, 3, 2, starts, wpn, 4, 42)
    rows, lens = oracle.unique_walks(tok, ln, wpn)
    expect = []
    for g in range(len(starts)):
        seen = set()
        for r in range(g * wpn, (g + 1) * wpn):
            key = tuple(tok[r, :ln[r]].tolist())
            if key not in seen:
                seen.add(key)
                expect.append(r)
    assert np.array_equal(rows, tok[expect]) and np.array_equal(lens, ln[expect])
    assert len(expect) < tok.shape[0]
