"""The Python binding rejects caller-supplied outputs it cannot write safely — too small, wrong
dtype, not contiguous, on the host — before any kernel is launched (the library writes through
raw pointers), and leaves them untouched."""

import numpy as np
import pytest
import torch

import paper_2508_01073_amd as rd
import synth
from gpu_helpers import device, gpu_csr, new_status, say, to_dev

pytestmark = pytest.mark.gpu


def _i32(n, fill=-7):
    return torch.full((n,), fill, dtype=torch.int32, device=device())


@pytest.fixture(scope="module")
def graph():
    V, P = 500, 5
    s, p, o = synth.uniform_triples(V, P, 4000)
    csr = gpu_csr(s, p, o, V, P)
    starts = rd.rdf2v_nonsink_starts(csr)
    return V, P, (s, p, o), csr, starts


def test_build_csr_outputs(graph):
    V, P, (s, p, o), _, _ = graph
    say("[binding] rdf2v_build_csr outputs")
    sd, pd, od = to_dev(s), to_dev(p), to_dev(o)
    small = _i32(V)
    with pytest.raises(ValueError):
        rd.rdf2v_build_csr(sd, pd, od, V, P, row_ptr=small)
    with pytest.raises(TypeError):
        rd.rdf2v_build_csr(sd, pd, od, V, P, edges=torch.empty((len(s), 2), dtype=torch.int64, device=device()))
    with pytest.raises(TypeError):
        rd.rdf2v_build_csr(sd, pd, od, V, P, status=torch.zeros(1, dtype=torch.int32))
    with pytest.raises(TypeError):
        rd.rdf2v_build_csr(sd, pd, od, V, P, status=torch.zeros(1, dtype=torch.int64, device=device()))
    torch.cuda.synchronize()
    assert bool((small == -7).all())


def test_walk_outputs(graph):
    V, P, _, csr, starts = graph
    say("[binding] walk records, start set and walk outputs")
    with pytest.raises(TypeError):
        rd.rdf2v_build_walk_edges(csr, out=torch.empty((csr.num_edges, 4), dtype=torch.float32, device=device()))
    short = _i32(V - 1)
    with pytest.raises(ValueError):
        rd.rdf2v_nonsink_starts(csr, starts=short)
    with pytest.raises(TypeError):
        rd.rdf2v_nonsink_starts(csr, count=torch.empty(1, dtype=torch.int32, device=device()))
    n = starts.shape[0] * 2
    tok = _i32(n * 9 - 1)
    with pytest.raises(ValueError):
        rd.rdf2v_random_walks(csr, starts, 2, 4, 42, tokens=tok)
    strided = torch.full((2 * n,), -7, dtype=torch.int32, device=device())[::2]
    with pytest.raises(ValueError):
        rd.rdf2v_random_walks(csr, starts, 2, 4, 42, lens=strided)
    torch.cuda.synchronize()
    assert bool((short == -7).all()) and bool((tok == -7).all())
    # the same call with proper buffers runs
    t, ln = rd.rdf2v_random_walks(csr, starts, 2, 4, 42, status=new_status())
    torch.cuda.synchronize()
    assert t.shape == (n, 9)


def test_corpus_outputs(graph):
    V, P, _, csr, starts = graph
    say("[binding] unique walks, BFS walks, pairs and CBOW outputs")
    t, ln = rd.rdf2v_random_walks(csr, starts, 3, 4, 42)
    n = ln.shape[0]
    with pytest.raises(ValueError):
        rd.rdf2v_unique_walks(t, ln, 3, tokens_out=_i32(n * 9 - 1))
    with pytest.raises(ValueError):
        rd.rdf2v_bfs_walks(csr, starts, 2, 4, counts=_i32(starts.shape[0] - 1))
    flat = _i32(40)
    with pytest.raises(ValueError):
        rd.rdf2v_skipgram_pairs(t, ln, 2, pairs=flat)           # a capacity would be 40 rows of 2
    with pytest.raises(ValueError):
        rd.rdf2v_cbow_examples(t, ln, 2, centers=_i32(10), contexts=_i32(39))
    torch.cuda.synchronize()
    assert bool((flat == -7).all())


def test_vocabulary_outputs():
    say("[binding] vocabulary outputs")
    w = synth.WORKLOADS["tiny_uniform"]
    S, P_, O = synth.triples(w)
    cols = synth.string_triples(S, P_, O, w.num_entities, w.num_predicates)
    dev = device()
    dcols = [(torch.from_numpy(np.ascontiguousarray(c, np.uint8)).to(dev),
              torch.from_numpy(np.ascontiguousarray(off, np.int64)).to(dev)) for c, off in cols]
    n = int(dcols[0][1].shape[0]) - 1
    with pytest.raises(ValueError):
        rd.rdf2v_build_vocabulary(*dcols, w.num_entities, w.num_predicates, ids=(_i32(n - 1), _i32(n), _i32(n)))
    with pytest.raises(ValueError):
        rd.rdf2v_build_vocabulary(*dcols, w.num_entities, w.num_predicates,
                                  counts=torch.empty(1, dtype=torch.int64, device=dev))


def test_calls_on_a_side_stream(graph):
    """A call given a stream that is not the current one allocates, launches and reads its count
    on that stream: a start set or pair count read right after long work was queued on the side
    stream waits for that work, and the workspace is not handed to other work while the side
    stream still uses it."""
    V, P, (s, p, o), csr, starts = graph
    say("[binding] calls on a non-current stream behind queued work")
    torch.cuda.synchronize()
    ref_starts = starts.clone()
    tok_ref, ln_ref = rd.rdf2v_random_walks(csr, starts, 4000, 8, 7)
    pairs_ref = rd.rdf2v_skipgram_pairs(tok_ref, ln_ref, 5)
    torch.cuda.synchronize()
    side = torch.cuda.Stream(device=device())
    side.wait_stream(torch.cuda.current_stream())
    for handle in (side, side.cuda_stream):                       # a torch stream, then a raw handle
        # about 2M walks of 8 hops queued on the side stream, then calls whose results the host
        # reads at once
        tok, ln = rd.rdf2v_random_walks(csr, starts, 4000, 8, 7, stream=handle)
        got = rd.rdf2v_nonsink_starts(csr, stream=handle)
        assert torch.equal(got, ref_starts)
        pairs = rd.rdf2v_skipgram_pairs(tok, ln, 5, stream=handle)
        assert pairs.shape == pairs_ref.shape
        side.synchronize()
        assert torch.equal(pairs, pairs_ref)
        assert torch.equal(tok, tok_ref) and torch.equal(ln, ln_ref)
    # a status word written on the side stream is read there: a bad start id queued behind
    # long work must still be seen
    st = torch.zeros(1, dtype=torch.int32, device=device())
    side.wait_stream(torch.cuda.current_stream())
    bad = torch.tensor([V + 5], dtype=torch.int32, device=device())
    rd.rdf2v_random_walks(csr, starts, 4000, 8, 7, stream=side)
    rd.rdf2v_random_walks(csr, bad, 1, 8, 7, status=st, stream=side)
    with pytest.raises(rd.Rdf2vError):
        rd.check_device_status(st, "side stream", stream=side)
