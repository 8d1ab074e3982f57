"""Element-wise parity past output index 2^31 (gpuRDF2vec Sec. 3.2: the data module turns the
whole walk corpus into training items; Sec. 3.1: padding dropped first).

One skip-gram call and one CBOW call over the whole power-law corpus (1M entities, 20M
triples, depth 8, 50 walks per start: 48.9M walks), so that the outputs hold 6.76G pairs
(13.5G int32 elements) and 822.7M examples with 8.2G context entries. Every walk of the corpus
is first compared with the oracle, so the lengths are the oracle's; the closed-form item counts
of the lengths then locate the walks whose output lands at element 2^31, 2^32, 2^33 and at the
very end, and windows of walks around each are compared element by element with the oracle's
pairs and examples of the oracle's walks. Integer work: tolerance 0."""

import numpy as np
import pytest
import torch

import oracle
import paper_2508_01073_amd as rd
import synth
from gpu_helpers import compare_all, device, gpu_csr, gpu_walks, new_status, say

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

WINDOW = 5
SPAN = 600  # walks per compared window


@pytest.fixture(scope="module")
def corpus():
    w = synth.WORKLOADS["powerlaw_20m"]
    V, P = w.num_entities, w.num_predicates
    say(f"[large outputs] {w.describe()}")
    s, p, o = synth.triples(w)
    csr = gpu_csr(s, p, o, V, P, walk_records=True)
    rp, ed = oracle.build_csr(s, p, o, V, P)
    starts = oracle.nonsink_starts(rp, V)
    starts_dev = rd.rdf2v_nonsink_starts(csr)
    assert np.array_equal(starts_dev.cpu().numpy(), starts)
    tok, ln = gpu_walks(csr, starts_dev, w.walks_per_node, w.depth, synth.WALK_SEED)
    compare_all(rp, ed, V, P, starts, w.walks_per_node, w.depth, synth.WALK_SEED, tok, ln)
    say(f"[large outputs] all {tok.shape[0]:,} walks bit-exact")
    return w, rp, ed, starts, tok, ln, ln.cpu().numpy().astype(np.int64)


def _oracle_walks(corpus, r0, k):
    w, rp, ed, starts = corpus[:4]
    return oracle.random_walks(rp, ed, w.num_entities, w.num_predicates, starts, w.walks_per_node, w.depth,
                               synth.WALK_SEED, r0, k)


def _windows(off, targets):
    """(first walk, walks) windows of SPAN walks around the walk whose items [off[r], off[r+1])
    hold each target item index."""
    n = off.shape[0] - 1
    out = []
    for t in targets:
        r = int(np.searchsorted(off, t, side="right")) - 1
        r0 = max(0, min(r - SPAN // 2, n - SPAN))
        assert off[r0] <= t < off[r0 + SPAN]
        out.append((r0, SPAN))
    return out


def test_skipgram_pairs_past_2_pow_32_elements(corpus):
    _, _, _, _, tok, ln, L = corpus
    m = np.minimum(L - 1, WINDOW)
    per_walk = np.where(m > 0, 2 * (m * L - m * (m + 1) // 2), 0)
    off = np.concatenate([[0], np.cumsum(per_walk)])
    total = int(off[-1])
    assert 2 * total > 2**33
    say(f"[large outputs] {total:,} skip-gram pairs in one call ({2 * total:,} int32 elements)")
    pairs = torch.empty((total, 2), dtype=torch.int32, device=device())
    count = torch.empty(1, dtype=torch.int64, device=device())
    st = new_status()
    rd.rdf2v_skipgram_pairs(tok, ln, WINDOW, pairs=pairs, count=count, status=st)
    torch.cuda.synchronize()
    assert int(count.item()) == total
    rd.check_device_status(st, "rdf2v_skipgram_pairs")
    # element e of the flat output is part of pair e // 2
    targets = [2**30 - 1, 2**30, 2**31, 2**32, total - 1]
    for r0, k in _windows(off, targets):
        got = pairs[int(off[r0]):int(off[r0 + k])].cpu().numpy()
        tr, lr = _oracle_walks(corpus, r0, k)
        ref = oracle.skipgram_pairs(tr, lr, WINDOW)
        assert np.array_equal(got, ref), f"pairs of walks [{r0}, {r0 + k}) (from pair {int(off[r0]):,})"
    say("[large outputs] pair windows at elements 2^31, 2^32, 2^33 and the end bit-exact")
    del pairs
    torch.cuda.empty_cache()


def test_cbow_examples_past_2_pow_32_elements(corpus):
    _, _, _, _, tok, ln, L = corpus
    off = np.concatenate([[0], np.cumsum(L)])
    total = int(off[-1])
    width = 2 * WINDOW
    assert total * width > 2**32
    say(f"[large outputs] {total:,} CBOW examples in one call ({total * width:,} context entries)")
    centers = torch.empty(total, dtype=torch.int32, device=device())
    contexts = torch.empty((total, width), dtype=torch.int32, device=device())
    count = torch.empty(1, dtype=torch.int64, device=device())
    st = new_status()
    rd.rdf2v_cbow_examples(tok, ln, WINDOW, centers=centers, contexts=contexts, count=count, status=st)
    torch.cuda.synchronize()
    assert int(count.item()) == total
    rd.check_device_status(st, "rdf2v_cbow_examples")
    # context entry e belongs to example e // (2 * window)
    targets = [(2**31 - 1) // width, 2**31 // width, 2**32 // width, total - 1]
    for r0, k in _windows(off, targets):
        a, b = int(off[r0]), int(off[r0 + k])
        got_c, got_x = centers[a:b].cpu().numpy(), contexts[a:b].cpu().numpy()
        tr, lr = _oracle_walks(corpus, r0, k)
        ref_c, ref_x = oracle.cbow_examples(tr, lr, WINDOW)
        assert np.array_equal(got_c, ref_c), f"centers of walks [{r0}, {r0 + k})"
        assert np.array_equal(got_x, ref_x), f"contexts of walks [{r0}, {r0 + k}) (from example {a:,})"
    say("[large outputs] example windows at context entries 2^31, 2^32 and the end bit-exact")
    del centers, contexts
    torch.cuda.empty_cache()
