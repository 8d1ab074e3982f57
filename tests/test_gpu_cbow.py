"""GPU parity for CBOW examples (rdf2v_cbow_examples, through the C ABI) against the oracle,
bit-exact: small rows of every length at windows up to the largest, real walk rows, capacity
truncation, outputs that do not start 16-byte aligned, bad lengths, and slices of the full
power-law corpus together with the skip-gram pairs they must flatten to."""

import numpy as np
import pytest
import torch

import oracle
import paper_2508_01073_amd as rd
import synth
from gpu_helpers import device, gpu_csr, gpu_walks, new_status, say, to_dev

pytestmark = pytest.mark.gpu


def _gpu_cbow(tok, ln, window):
    st = new_status()
    c, x = rd.rdf2v_cbow_examples(tok, ln, window, status=st)
    torch.cuda.synchronize()
    rd.check_device_status(st, "rdf2v_cbow_examples")
    return c.cpu().numpy(), x.cpu().numpy()


def _random_rows(width, n, seed):
    rng = np.random.default_rng(seed)
    ln = rng.integers(0, width + 1, n).astype(np.int32)
    tok = np.full((n, width), -1, np.int32)
    for r in range(n):
        tok[r, :ln[r]] = rng.integers(0, 10**6, ln[r])
    return tok, ln


@pytest.mark.parametrize("width", [1, 2, 9, 17, 33, 129])
@pytest.mark.parametrize("window", [1, 2, 5, 20, 128])
def test_random_rows(width, window):
    # windows 20 and 128 take the 128-thread, 64-thread and unstaged launches
    say(f"[cbow] random rows width={width} window={window}")
    tok, ln = _random_rows(width, 2000, width * 1000 + window)
    c, x = _gpu_cbow(to_dev(tok), to_dev(ln), window)
    rc, rx = oracle.cbow_examples(tok, ln, window)
    assert np.array_equal(c, rc) and np.array_equal(x, rx)


@pytest.mark.parametrize("window", [1, 5, 10])
def test_walk_rows_tiny_uniform(window):
    w = synth.WORKLOADS["tiny_uniform"]
    say(f"[cbow] tiny_uniform walks window={window}")
    s, p, o = synth.triples(w)
    csr = gpu_csr(s, p, o, w.num_entities, w.num_predicates)
    starts = rd.rdf2v_nonsink_starts(csr)
    tok, ln = gpu_walks(csr, starts, w.walks_per_node, w.depth, synth.WALK_SEED)
    c, x = _gpu_cbow(tok, ln, window)
    rc, rx = oracle.cbow_examples(tok.cpu().numpy(), ln.cpu().numpy(), window)
    assert np.array_equal(c, rc) and np.array_equal(x, rx)


@pytest.mark.parametrize("shift", [0, 1, 2, 3])
def test_capacity_and_unaligned_outputs(shift):
    # capacity below the count writes a prefix; outputs that start 4, 8 or 12 bytes past a
    # 16-byte boundary take the scalar head of the streamed run
    say(f"[cbow] capacity and alignment shift={shift}")
    tok, ln = _random_rows(17, 600, 7)
    window = 3
    rc, rx = oracle.cbow_examples(tok, ln, window)
    cap = rc.shape[0] - 123
    dev = device()
    cbuf = torch.full((cap + 4,), -9, dtype=torch.int32, device=dev)
    xbuf = torch.full(((cap + 4) * 2 * window,), -9, dtype=torch.int32, device=dev)
    centers = cbuf[shift:shift + cap]
    contexts = xbuf[shift:shift + cap * 2 * window].view(cap, 2 * window)
    st = new_status()
    _, _, count = rd.rdf2v_cbow_examples(to_dev(tok), to_dev(ln), window, centers=centers, contexts=contexts,
                                         status=st)
    torch.cuda.synchronize()
    assert int(count.item()) == rc.shape[0]
    assert int(st.item()) & rd.RDF2V_STATUS_CAPACITY
    assert np.array_equal(centers.cpu().numpy(), rc[:cap])
    assert np.array_equal(contexts.cpu().numpy(), rx[:cap])
    # nothing is written around the outputs
    assert np.all(cbuf[:shift].cpu().numpy() == -9) and np.all(cbuf[shift + cap:].cpu().numpy() == -9)
    xb = xbuf.cpu().numpy()
    assert np.all(xb[:shift] == -9) and np.all(xb[shift + cap * 2 * window:] == -9)


def test_bad_lengths_are_flagged():
    say("[cbow] lengths outside the row")
    tok = to_dev(np.zeros((3, 5), np.int32))
    st = new_status()
    rd.rdf2v_cbow_examples(tok, to_dev(np.array([2, 9, -1], np.int32)), 2, status=st)
    torch.cuda.synchronize()
    assert int(st.item()) & rd.RDF2V_STATUS_BAD_LENGTH


def test_powerlaw_corpus_slices_and_pairs():
    w = synth.WORKLOADS["powerlaw_20m"]
    say(f"[cbow] {w.describe()}; window 5 over slices of the corpus")
    s, p, o = synth.triples(w)
    csr = gpu_csr(s, p, o, w.num_entities, w.num_predicates, walk_records=True)
    starts = rd.rdf2v_nonsink_starts(csr)
    tok, ln = gpu_walks(csr, starts, w.walks_per_node, w.depth, synth.WALK_SEED)
    dev = device()
    count = torch.empty(1, dtype=torch.int64, device=dev)
    empty = torch.empty(0, dtype=torch.int32, device=dev)
    rd.rdf2v_cbow_examples(tok, ln, 5, centers=empty, contexts=empty.view(0, 10), count=count)
    assert int(count.item()) == int(ln.to(torch.int64).sum().item())  # one example per valid token
    n = tok.shape[0]
    for b in (0, n // 2, n - 100_000):
        sl_t, sl_l = tok[b:b + 100_000].contiguous(), ln[b:b + 100_000].contiguous()
        c, x = _gpu_cbow(sl_t, sl_l, 5)
        rc, rx = oracle.cbow_examples(sl_t.cpu().numpy(), sl_l.cpu().numpy(), 5)
        assert np.array_equal(c, rc) and np.array_equal(x, rx), f"slice at {b}"
        # the GPU's own skip-gram pairs of the slice are the flattened contexts, in order
        rows, cols = np.nonzero(x != -1)
        pairs = rd.rdf2v_skipgram_pairs(sl_t, sl_l, 5).cpu().numpy()
        assert np.array_equal(np.stack([c[rows], x[rows, cols]], axis=1), pairs)
