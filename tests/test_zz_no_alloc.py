"""rdf2v_skipgram_pairs_noalloc (skip-gram pairs with the library's fixed per-device scratch
instead of a caller workspace) against rdf2v_skipgram_pairs, element by element: two calls in a
row, the first at the largest row count it takes and the second smaller with a ragged tail, then
a call whose output capacity cuts the pairs short; and the host-side rejection of one row too
many. Integer work: tolerance 0."""

import pytest
import torch

import paper_2508_01073_amd as rd
import synth
from gpu_helpers import device, gpu_csr, new_status, say

pytestmark = pytest.mark.gpu


def _compare(tok, ln, window, cap_extra=1000, cap=None):
    ref = rd.rdf2v_skipgram_pairs(tok, ln, window)  # the workspace entry point, exact-size output
    n_ref = int(ref.shape[0])
    cap = n_ref + cap_extra if cap is None else cap
    pairs = torch.full((cap, 2), -7, dtype=torch.int32, device=device())
    count = torch.full((1,), -1, dtype=torch.int64, device=device())
    status = new_status()
    rd.rdf2v_skipgram_pairs_noalloc(tok, ln, window, pairs=pairs, count=count, status=status)
    torch.cuda.synchronize()
    assert int(count.item()) == n_ref
    kept = min(cap, n_ref)
    assert torch.equal(pairs[:kept], ref[:kept])
    assert bool((pairs[kept:] == -7).all())
    return n_ref, int(status.item())


def test_noalloc_pairs_equal_workspace_pairs():
    V, P, depth = 50_000, 20, 8
    s, p, o = synth.powerlaw_triples(V, P, 1_000_000)
    csr = gpu_csr(s, p, o, V, P, walk_records=True)
    starts = rd.rdf2v_nonsink_starts(csr)
    n_max = rd.RDF2V_NOALLOC_MAX_WALKS
    wpn = -(-n_max // int(starts.shape[0]))
    tok, ln = rd.rdf2v_random_walks(csr, starts, wpn, depth, 42, 0, n_max)
    torch.cuda.synchronize()
    for n, window in ((n_max, 5), (100_003, 3)):
        say(f"[noalloc] skip-gram pairs of {n:,} walks, window {window}")
        n_pairs, st = _compare(tok[:n], ln[:n], window)
        assert st == 0 and n_pairs > n
    say("[noalloc] capacity cut")
    n_pairs, st = _compare(tok[:5_000], ln[:5_000], 2, cap=1_234)
    assert st == rd.RDF2V_STATUS_CAPACITY and n_pairs > 1_234
    say("[noalloc] one row beyond the bound")
    big_t = torch.empty((n_max + 1, 1), dtype=torch.int32, device=device())
    big_l = torch.ones(n_max + 1, dtype=torch.int32, device=device())
    pairs = torch.empty((1, 2), dtype=torch.int32, device=device())
    count = torch.full((1,), -1, dtype=torch.int64, device=device())
    with pytest.raises(rd.Rdf2vError) as e:
        rd.rdf2v_skipgram_pairs_noalloc(big_t, big_l, 1, pairs=pairs, count=count)
    assert e.value.status == rd.RDF2V_ERR_TOO_LARGE
    torch.cuda.synchronize()
    assert int(count.item()) == -1  # nothing was enqueued
