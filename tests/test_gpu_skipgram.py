"""GPU parity for skip-gram pair generation (through the C ABI) against the
oracle, bit-exact: small rows of every length, real walk rows at several
windows, capacity truncation, and slices of the full power-law corpus."""

import numpy as np
import pytest
import torch

import oracle
import paper_2508_01073_amd as rd
import synth
from gpu_helpers import device, gpu_csr, gpu_walks, new_status, say, to_dev

pytestmark = pytest.mark.gpu


def _gpu_pairs(tok, ln, window):
    st = new_status()
    pairs = rd.rdf2v_skipgram_pairs(tok, ln, window, status=st)
    torch.cuda.synchronize()
    rd.check_device_status(st, "rdf2v_skipgram_pairs")
    return pairs.cpu().numpy()


@pytest.mark.parametrize("width", [1, 2, 9, 17, 33, 129])
@pytest.mark.parametrize("window", [0, 1, 2, 5, 64])
def test_random_rows(width, window):
    say(f"[pairs] random rows width={width} window={window}")
    rng = np.random.default_rng(width * 100 + window)
    n = 3000
    ln = rng.integers(0, width + 1, n).astype(np.int32)
    tok = np.full((n, width), -1, np.int32)
    for r in range(n):
        tok[r, :ln[r]] = rng.integers(0, 10**6, ln[r])
    got = _gpu_pairs(to_dev(tok), to_dev(ln), window)
    ref = oracle.skipgram_pairs(tok, ln, window)
    assert got.shape == ref.shape and np.array_equal(got, ref)


@pytest.mark.parametrize("window", [1, 5, 10])
def test_walk_rows_tiny_uniform(window):
    w = synth.WORKLOADS["tiny_uniform"]
    say(f"[pairs] tiny_uniform walks window={window}")
    s, p, o = synth.triples(w)
    csr = gpu_csr(s, p, o, w.num_entities, w.num_predicates, walk_records=True)
    starts = rd.rdf2v_nonsink_starts(csr)
    tok, ln = gpu_walks(csr, starts, w.walks_per_node, w.depth, synth.WALK_SEED)
    got = _gpu_pairs(tok, ln, window)
    ref = oracle.skipgram_pairs(tok.cpu().numpy(), ln.cpu().numpy(), window)
    assert np.array_equal(got, ref)


def test_capacity_and_count():
    say("[pairs] capacity truncation")
    tok = to_dev(np.arange(40, dtype=np.int32).reshape(4, 10))
    ln = to_dev(np.array([10, 3, 0, 7], np.int32))
    ref = oracle.skipgram_pairs(tok.cpu().numpy(), ln.cpu().numpy(), 3)
    out = torch.full((20, 2), -5, dtype=torch.int32, device=device())
    st = new_status()
    pairs, count = rd.rdf2v_skipgram_pairs(tok, ln, 3, pairs=out, status=st)
    torch.cuda.synchronize()
    assert int(count.item()) == ref.shape[0]
    assert np.array_equal(out.cpu().numpy(), ref[:20])
    assert int(st.item()) & rd.RDF2V_STATUS_CAPACITY


def test_bad_lengths_are_flagged():
    say("[pairs] lengths outside the row")
    tok = to_dev(np.zeros((3, 5), np.int32))
    st = new_status()
    rd.rdf2v_skipgram_pairs(tok, to_dev(np.array([2, 9, -1], np.int32)), 2, status=st)
    torch.cuda.synchronize()
    assert int(st.item()) & rd.RDF2V_STATUS_BAD_LENGTH


def test_powerlaw_corpus_slices():
    w = synth.WORKLOADS["powerlaw_20m"]
    say(f"[pairs] {w.describe()}; window 5 over slices of the corpus")
    s, p, o = synth.triples(w)
    csr = gpu_csr(s, p, o, w.num_entities, w.num_predicates, walk_records=True)
    starts = rd.rdf2v_nonsink_starts(csr)
    tok, ln = gpu_walks(csr, starts, w.walks_per_node, w.depth, synth.WALK_SEED)
    n = tok.shape[0]
    # the count over the whole corpus (count-only call) equals the closed form summed over lengths
    count = torch.empty(1, dtype=torch.int64, device=device())
    rd.rdf2v_skipgram_pairs(tok, ln, 5, pairs=torch.empty((0, 2), dtype=torch.int32, device=device()),
                            count=count)
    L = ln.to(torch.int64)
    m = torch.clamp(L - 1, max=5)
    closed = int((2 * (m * L - m * (m + 1) // 2)).clamp(min=0).sum().item())
    assert int(count.item()) == closed
    for b in (0, n // 2, n - 150_000):
        sl_t, sl_l = tok[b:b + 150_000].contiguous(), ln[b:b + 150_000].contiguous()
        got = _gpu_pairs(sl_t, sl_l, 5)
        ref = oracle.skipgram_pairs(sl_t.cpu().numpy(), sl_l.cpu().numpy(), 5)
        assert np.array_equal(got, ref), f"slice at {b}"
