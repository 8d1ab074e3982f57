"""The whole path captured in a HIP graph: CSR build, walk records, start set, walks and
skip-gram pairs enqueue kernels only (no allocation, copy, memset or synchronisation inside a
call), so a caller can capture them once and replay; so do CBOW examples, entity walks,
duplicate-free walks, BFS walks and the string vocabulary. Every replay must reproduce the eager
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


def test_next_rows_replays_match_eager():
    # The next rows' calls are capturable too: CBOW examples, entity walks, duplicate-free
    # walks, BFS walks and the string vocabulary, all with caller buffers, in one graph.
    dev = device()
    V, P, T = 20_000, 7, 150_000
    s_np, p_np, o_np = synth.powerlaw_triples(V, P, T, seed=22)
    t = lambda a: torch.from_numpy(a).to(dev)
    s, p, o = t(s_np), t(p_np), t(o_np)
    wpn, depth, seed, window = 3, 5, 99, 4
    say(f"[graph next] V={V} T={T}")
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    csr = rd.rdf2v_build_csr(s, p, o, V, P, status=status)
    starts = rd.rdf2v_nonsink_starts(csr)
    roots = starts[:500].contiguous()
    n_walks = int(starts.shape[0]) * wpn
    tokens, lens = rd.rdf2v_random_walks(csr, starts, wpn, depth, seed, status=status)
    torch.cuda.synchronize()
    # every output and workspace exists before capture; the CBOW output is sized by an eager count
    ws_cbow = torch.empty(rd.rdf2v_cbow_examples_workspace_size(n_walks), dtype=torch.uint8, device=dev)
    n_ex = int(lens.sum().item())
    centers = torch.empty(n_ex, dtype=torch.int32, device=dev)
    contexts = torch.empty((n_ex, 2 * window), dtype=torch.int32, device=dev)
    ex_count = torch.empty(1, dtype=torch.int64, device=dev)
    ent_tok = torch.empty((n_walks, depth + 1), dtype=torch.int32, device=dev)
    ent_len = torch.empty(n_walks, dtype=torch.int32, device=dev)
    uq_tok = torch.empty_like(tokens)
    uq_len = torch.empty_like(lens)
    uq_count = torch.empty(1, dtype=torch.int64, device=dev)
    ws_uq = torch.empty(rd.rdf2v_unique_walks_workspace_size(n_walks), dtype=torch.uint8, device=dev)
    max_walks = V  # a depth-2 tree has at most V leaves: no root overflows
    bfs_tok = torch.empty((roots.shape[0], max_walks, 2 * 2 + 1), dtype=torch.int32, device=dev)
    bfs_len = torch.empty((roots.shape[0], max_walks), dtype=torch.int32, device=dev)
    bfs_cnt = torch.empty(roots.shape[0], dtype=torch.int32, device=dev)
    ws_bfs = torch.empty(rd.rdf2v_bfs_walks_workspace_size(V, roots.shape[0]), dtype=torch.uint8, device=dev)
    cols = synth.string_triples(s_np, p_np, o_np, V, P)
    dcols = [(torch.from_numpy(c).to(dev), torch.from_numpy(off).to(dev)) for c, off in cols]
    ids = tuple(torch.empty(T, dtype=torch.int32, device=dev) for _ in range(3))
    vcounts = torch.empty(2, dtype=torch.int64, device=dev)
    ws_voc = torch.empty(rd.rdf2v_build_vocabulary_workspace_size(T, V, P), dtype=torch.uint8, device=dev)

    def calls(stream):
        rd.rdf2v_cbow_examples(tokens, lens, window, centers=centers, contexts=contexts, count=ex_count,
                               workspace=ws_cbow, status=status, stream=stream)
        rd.rdf2v_random_walks_tokens(csr, starts, wpn, depth, seed, token_kind=rd.RDF2V_TOKENS_ENTITIES,
                                     tokens=ent_tok, lens=ent_len, status=status, stream=stream)
        rd.rdf2v_unique_walks(tokens, lens, wpn, tokens_out=uq_tok, lens_out=uq_len, count=uq_count,
                              workspace=ws_uq, status=status, stream=stream, sync=False)
        rd.rdf2v_bfs_walks(csr, roots, 2, max_walks, tokens=bfs_tok, lens=bfs_len, counts=bfs_cnt,
                           workspace=ws_bfs, status=status, stream=stream)
        rd.rdf2v_build_vocabulary(*dcols, V, P, ids=ids, counts=vcounts, workspace=ws_voc, status=status,
                                  stream=stream)

    outs = dict(centers=centers, contexts=contexts, ex_count=ex_count, ent_tok=ent_tok, ent_len=ent_len,
                uq_tok=uq_tok, uq_len=uq_len, uq_count=uq_count, bfs_tok=bfs_tok, bfs_len=bfs_len,
                bfs_cnt=bfs_cnt, subj_ids=ids[0], pred_ids=ids[1], obj_ids=ids[2], vcounts=vcounts)
    for x in outs.values():
        x.fill_(-7)
    calls(None)
    torch.cuda.synchronize()
    rd.check_device_status(status, "eager")
    assert int(ex_count.item()) == n_ex
    ref = {k: v.clone() for k, v in outs.items()}
    kept = int(uq_count.item())

    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            calls(torch.cuda.current_stream(dev))
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()
    for replay in range(3):
        for x in outs.values():  # eager work between replays: every output cleared
            x.fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        for k, want in ref.items():
            got = outs[k]
            if k in ("uq_tok", "uq_len"):  # rows past the kept count are not written
                got, want = got[:kept], want[:kept]
            assert torch.equal(got, want), f"replay {replay}: {k} differs from the eager result"
        say(f"[graph next] replay {replay}: {n_ex} CBOW examples, {kept} kept walks, BFS and vocabulary equal")
    del graph
