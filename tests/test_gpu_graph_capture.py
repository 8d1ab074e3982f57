"""The whole path captured in a HIP graph: CSR build, walk records, start set, walks and
skip-gram pairs enqueue kernels only (no allocation, copy, memset or synchronisation inside a
call), so a caller can capture them once and replay. Every replay must reproduce the eager
result bit for bit; the outputs are cleared by eager work between replays, so each replay has to
write all of them again."""

import numpy as np
import pytest
import torch

import paper_2508_01073_amd as rd
import synth
from gpu_helpers import device, say

pytestmark = pytest.mark.gpu


def _inputs(walk_records):
    dev = device()
    # a graph above the walk-records threshold when they are used, a small one otherwise
    V, P, T = (450_000, 13, 1_800_000) if walk_records else (20_000, 7, 150_000)
    s, p, o = synth.powerlaw_triples(V, P, T, seed=21)
    t = lambda a: torch.from_numpy(a).to(dev)
    return V, P, t(s), t(p), t(o)


@pytest.mark.parametrize("walk_records", [False, True])
def test_replays_match_eager(walk_records):
    dev = device()
    V, P, s, p, o = _inputs(walk_records)
    T = s.shape[0]
    wpn, depth, seed, window = 4, 6, 1234567, 3
    say(f"[graph] V={V} T={T} walk_records={walk_records}")
    # every buffer is allocated before capture
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    row_ptr = torch.empty(V + 1, dtype=torch.int32, device=dev)
    edges = torch.empty((T, 2), dtype=torch.int32, device=dev)
    ws = torch.empty(rd.rdf2v_build_csr_workspace_size(T, V), dtype=torch.uint8, device=dev)
    rec = torch.empty((T, 4), dtype=torch.int32, device=dev) if walk_records else None
    starts = torch.empty(V, dtype=torch.int32, device=dev)
    count = torch.empty(1, dtype=torch.int64, device=dev)
    ws_starts = torch.empty(rd.rdf2v_nonsink_starts_workspace_size(V), dtype=torch.uint8, device=dev)

    def front(stream):
        csr = rd.rdf2v_build_csr(s, p, o, V, P, workspace=ws, status=status, row_ptr=row_ptr, edges=edges,
                                 stream=stream)
        if walk_records:
            csr = rd.rdf2v_build_walk_edges(csr, out=rec, status=status, stream=stream)
        rd.rdf2v_nonsink_starts(csr, workspace=ws_starts, starts=starts, count=count, stream=stream, sync=False)
        return csr

    # eager run: sizes the walk and pair buffers
    csr = front(None)
    torch.cuda.synchronize()
    n_start = int(count.item())
    n_walks = n_start * wpn
    tokens = torch.empty((n_walks, 2 * depth + 1), dtype=torch.int32, device=dev)
    lens = torch.empty(n_walks, dtype=torch.int32, device=dev)
    rd.rdf2v_random_walks(csr, starts[:n_start], wpn, depth, seed, tokens=tokens, lens=lens, status=status)
    pair_count = torch.empty(1, dtype=torch.int64, device=dev)
    ws_pairs = torch.empty(rd.rdf2v_skipgram_pairs_workspace_size(n_walks), dtype=torch.uint8, device=dev)
    rd.rdf2v_skipgram_pairs(tokens, lens, window, pairs=torch.empty((0, 2), dtype=torch.int32, device=dev),
                            count=pair_count, workspace=ws_pairs, status=status)
    torch.cuda.synchronize()
    n_pairs = int(pair_count.item())
    pairs = torch.empty((n_pairs, 2), dtype=torch.int32, device=dev)
    rd.rdf2v_skipgram_pairs(tokens, lens, window, pairs=pairs, count=pair_count, workspace=ws_pairs, status=status)
    torch.cuda.synchronize()
    rd.check_device_status(status, "eager")
    ref = {k: v.clone() for k, v in dict(row_ptr=row_ptr, edges=edges, starts=starts[:n_start], count=count,
                                         tokens=tokens, lens=lens, pairs=pairs, pair_count=pair_count).items()}
    if walk_records:
        ref["rec"] = rec.clone()

    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            cur = torch.cuda.current_stream(dev)
            c = front(cur)
            rd.rdf2v_random_walks(c, starts[:n_start], wpn, depth, seed, tokens=tokens, lens=lens, status=status,
                                  stream=cur)
            rd.rdf2v_skipgram_pairs(tokens, lens, window, pairs=pairs, count=pair_count, workspace=ws_pairs,
                                    status=status, stream=cur)
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()

    outs = dict(row_ptr=row_ptr, edges=edges, starts=starts, count=count, tokens=tokens, lens=lens, pairs=pairs,
                pair_count=pair_count)
    if walk_records:
        outs["rec"] = rec
    for replay in range(3):
        for t in outs.values():  # eager work between replays: every output cleared
            t.fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        for k, want in ref.items():
            got = outs[k][:n_start] if k == "starts" else outs[k]
            assert torch.equal(got, want), f"replay {replay}: {k} differs from the eager result"
        say(f"[graph] replay {replay}: {n_walks} walks, {n_pairs} pairs equal to eager")
    del graph
    assert np.array_equal(ref["count"].cpu().numpy(), [n_start])
