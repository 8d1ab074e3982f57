"""Pins for the oracle's vocabulary (gpuRDF2vec Sec. 3.1: entities and predicates
are tokenised to integer ids at the start of the pipeline).

Ids number distinct strings in order of first appearance: entities over the
sequence s_0, o_0, s_1, o_1, ..., predicates over p_0, p_1, .... The oracle is
checked against pandas.factorize (a library factorisation that numbers values
by first appearance), a hand-worked example, and the integer graph the strings
were made from (first-appearance ranks of the underlying ids)."""

import numpy as np
import pandas as pd
import pytest

import oracle
import synth


def _column(strings):
    data = [s.encode() if isinstance(s, str) else s for s in strings]
    off = np.zeros(len(data) + 1, np.int64)
    off[1:] = np.cumsum([len(d) for d in data])
    chars = np.frombuffer(b"".join(data), np.uint8) if off[-1] else np.zeros(0, np.uint8)
    return chars, off


def _vocab(S, P, O):
    (sc, so), (pc, po), (oc, oo) = _column(S), _column(P), _column(O)
    return oracle.build_vocabulary(sc, so, pc, po, oc, oo)


def test_hand_worked():
    S = ["b", "a", "b", "", "ab"]
    P = ["knows", "knows", "likes", "a", "knows"]
    O = ["a", "c", "b", "a", "a\x00"]
    s, p, o, ne, npred = _vocab(S, P, O)
    # entity sequence b a | a c | b b | "" a | ab a\0  -> b=0 a=1 c=2 ""=3 ab=4 a\0=5
    assert s.tolist() == [0, 1, 0, 3, 4] and o.tolist() == [1, 2, 0, 1, 5] and ne == 6
    # predicate sequence knows knows likes a knows; the predicate "a" is not the entity "a"
    assert p.tolist() == [0, 0, 1, 2, 0] and npred == 3


def test_empty():
    s, p, o, ne, npred = _vocab([], [], [])
    assert s.size == p.size == o.size == 0 and ne == npred == 0


def test_matches_pandas_factorize_on_near_duplicates():
    # strings that share prefixes, differ in one byte, or are prefixes of each other
    rng = np.random.default_rng(0)
    alphabet = [b"a", b"b", b"\x00", b"\xff"]
    pool = [b"".join(rng.choice(alphabet, size=int(rng.integers(0, 6)))) for _ in range(300)]
    T = 2000
    S = [pool[i] for i in rng.integers(0, len(pool), T)]
    O = [pool[i] for i in rng.integers(0, len(pool), T)]
    P = [pool[i] for i in rng.integers(0, 40, T)]
    s, p, o, ne, npred = _vocab(S, P, O)
    seq = np.empty(2 * T, dtype=object)
    seq[0::2], seq[1::2] = S, O
    codes, uniques = pd.factorize(seq)
    assert np.array_equal(s, codes[0::2]) and np.array_equal(o, codes[1::2]) and ne == len(uniques)
    pcodes, puniques = pd.factorize(np.array(P, dtype=object))
    assert np.array_equal(p, pcodes) and npred == len(puniques)


@pytest.mark.parametrize("name", ["tiny_uniform", "uniform_1m"])
def test_recovers_the_integer_graph(name):
    w = synth.WORKLOADS[name]
    S, P, O = synth.triples(w)
    (sc, so), (pc, po), (oc, oo) = synth.string_triples(S, P, O, w.num_entities, w.num_predicates)
    s, p, o, ne, npred = oracle.build_vocabulary(sc, so, pc, po, oc, oo)
    # labels are a bijection of ids, so string ids are the first-appearance ranks of the ids
    seq = np.empty(2 * len(S), np.int64)
    seq[0::2], seq[1::2] = S, O
    uniq, first = np.unique(seq, return_index=True)
    rank = np.empty(w.num_entities, np.int64)
    rank[uniq[np.argsort(first)]] = np.arange(uniq.size)
    assert np.array_equal(s, rank[S]) and np.array_equal(o, rank[O]) and ne == uniq.size
    puniq, pfirst = np.unique(P, return_index=True)
    prank = np.empty(w.num_predicates, np.int64)
    prank[puniq[np.argsort(pfirst)]] = np.arange(puniq.size)
    assert np.array_equal(p, prank[P]) and npred == puniq.size
