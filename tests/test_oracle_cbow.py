"""Pins for the oracle's CBOW examples (gpuRDF2vec Sec. 3.2: CBOW predicts a center token
from the tokens around it). Each test ties the oracle to something other than its own loop: a
hand-worked example, an independent numpy construction with a sliding window, the skip-gram
pairs (pinned on their own), the closed-form counts, and the padding rule."""

import numpy as np
import pytest

import oracle
import synth


def test_hand_worked_window_1_and_2():
    # One walk a b c d e (padded row of 7), worked out by hand from the definition.
    tok = np.array([[10, 20, 30, 40, 50, -1, -1]], np.int32)
    ln = np.array([5], np.int32)
    c, x = oracle.cbow_examples(tok, ln, 1)
    assert c.tolist() == [10, 20, 30, 40, 50]
    assert x.tolist() == [[20, -1], [10, 30], [20, 40], [30, 50], [40, -1]]
    c, x = oracle.cbow_examples(tok, ln, 2)
    assert c.tolist() == [10, 20, 30, 40, 50]
    assert x.tolist() == [[20, 30, -1, -1], [10, 30, 40, -1], [10, 20, 40, 50], [20, 30, 50, -1],
                          [30, 40, -1, -1]]
    # a one-token walk is one example with no context; an empty row gives none
    c, x = oracle.cbow_examples(np.array([[7, -1, -1], [8, 9, -1]], np.int32), np.array([1, 0], np.int32), 1)
    assert c.tolist() == [7] and x.tolist() == [[-1, -1]]


def _sliding(tok, ln, window):
    """Independent construction: pad each valid prefix with window -1s on both sides, take the
    2*window+1 wide sliding windows, drop the middle column, and move the -1s to the end."""
    centers, rows = [], []
    for r in range(tok.shape[0]):
        L = int(ln[r])
        if L == 0:
            continue
        padded = np.concatenate([np.full(window, -1), tok[r, :L], np.full(window, -1)])
        win = np.lib.stride_tricks.sliding_window_view(padded, 2 * window + 1)
        ctx = np.delete(win, window, axis=1)
        keep = ctx != -1
        # stable move of the real contexts to the front (they keep their order)
        order = np.argsort(~keep, axis=1, kind="stable")
        packed = np.take_along_axis(ctx, order, axis=1)
        packed[~np.take_along_axis(keep, order, axis=1)] = -1
        centers.append(tok[r, :L])
        rows.append(packed)
    if not centers:
        return np.zeros(0, np.int32), np.zeros((0, 2 * window), np.int32)
    return np.concatenate(centers).astype(np.int32), np.concatenate(rows).astype(np.int32)


def _walks(name, n):
    w = synth.WORKLOADS[name]
    s, p, o = synth.triples(w)
    rp, ed = oracle.build_csr(s, p, o, w.num_entities, w.num_predicates)
    starts = oracle.nonsink_starts(rp, w.num_entities)
    return oracle.random_walks(rp, ed, w.num_entities, w.num_predicates, starts, w.walks_per_node, w.depth,
                               synth.WALK_SEED, 0, n)


@pytest.mark.parametrize("window", [1, 2, 5, 9])
def test_matches_sliding_window_construction_on_real_walks(window):
    tok, ln = _walks("tiny_uniform", 3000)
    c, x = oracle.cbow_examples(tok, ln, window)
    c2, x2 = _sliding(tok, ln, window)
    assert np.array_equal(c, c2)
    assert np.array_equal(x, x2)


@pytest.mark.parametrize("window", [1, 3, 5])
def test_flattened_contexts_are_the_skipgram_pairs(window):
    # Read in order, the (center, context) of every non-padding context are the skip-gram
    # pairs, in the skip-gram order (walk, center, context).
    tok, ln = _walks("tiny_uniform", 2000)
    c, x = oracle.cbow_examples(tok, ln, window)
    rows, cols = np.nonzero(x != -1)
    flat = np.stack([c[rows], x[rows, cols]], axis=1)
    assert np.array_equal(flat, oracle.skipgram_pairs(tok, ln, window))


def test_counts_closed_form_and_padding():
    rng = np.random.default_rng(3)
    width, window = 17, 4
    ln = rng.integers(0, width + 1, 500).astype(np.int32)
    tok = rng.integers(0, 1000, (500, width)).astype(np.int32)
    c, x = oracle.cbow_examples(tok, ln, window)
    assert c.shape[0] == int(ln.sum())  # one example per valid token
    e = 0
    for L in ln:
        for i in range(L):
            real = min(i, window) + min(L - 1 - i, window)
            assert np.all(x[e, :real] != -1) and np.all(x[e, real:] == -1)
            e += 1


def test_capacity_and_bad_arguments():
    tok, ln = _walks("tiny_uniform", 200)
    lib = oracle._load()
    n = lib.rdf2v_ref_cbow_examples(oracle._ptr(tok), oracle._ptr(ln), tok.shape[0], tok.shape[1], 2,
                                    None, None, 0)
    assert n == int(ln.sum())
    cap = n // 3
    centers = np.full(n, 12345, np.int32)
    contexts = np.full((n, 4), 12345, np.int32)
    assert lib.rdf2v_ref_cbow_examples(oracle._ptr(tok), oracle._ptr(ln), tok.shape[0], tok.shape[1], 2,
                                       oracle._ptr(centers), oracle._ptr(contexts), cap) == n
    full_c, full_x = oracle.cbow_examples(tok, ln, 2)
    assert np.array_equal(centers[:cap], full_c[:cap]) and np.all(centers[cap:] == 12345)
    assert np.array_equal(contexts[:cap], full_x[:cap]) and np.all(contexts[cap:] == 12345)
    with pytest.raises(oracle.OracleError):
        oracle.cbow_examples(tok, ln, 0)
    with pytest.raises(oracle.OracleError):
        oracle.cbow_examples(tok, np.full_like(ln, tok.shape[1] + 1), 2)
