"""The HIP path against the stored golden fixtures (tests/golden/, written from
the CPU oracle by tests/golden/make_golden.py): bit-exact, without running the
oracle here."""

import os

import numpy as np
import pytest
import torch

import paper_2508_01073_amd as rd
import synth
from gpu_helpers import device, gpu_csr, new_status, say, to_dev

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _read(name):
    header, rows = [], []
    for line in open(os.path.join(GOLDEN, name)):
        if line.startswith("#"):
            header.append(line[1:].strip())
        elif line.strip():
            rows.append(line.split())
    return header, rows


def _hand_graph(header):
    line = next(h for h in header if h.startswith("Triples (s, p, o)"))
    sizes, triples = line.split(": ", 1)
    V = int(sizes.split("V=")[1].split(",")[0])
    P = int(sizes.split("P=")[1])
    t = np.array([[int(x) for x in tr.split(",")] for tr in triples.split()], np.int32)
    return t, V, P


def _walk_rows(rows):
    lens = np.array([int(r[0]) for r in rows], np.int32)
    tok = np.array([[int(x) for x in r[1:]] for r in rows], np.int32)
    return tok, lens


def test_walks_hand_graph():
    say("[golden] walks on the hand graph")
    header, rows = _read("walks_hand_graph.txt")
    t, V, P = _hand_graph(header)
    csr = gpu_csr(t[:, 0], t[:, 1], t[:, 2], V, P, walk_records=True)
    tok, ln = rd.rdf2v_random_walks(csr, to_dev(np.arange(V)), 5, 6, 42)
    exp_t, exp_l = _walk_rows(rows)
    assert np.array_equal(ln.cpu().numpy(), exp_l) and np.array_equal(tok.cpu().numpy(), exp_t)


def test_walks_tiny_uniform_head():
    say("[golden] first 200 walks of tiny_uniform")
    _, rows = _read("walks_tiny_uniform_head.txt")
    w = synth.WORKLOADS["tiny_uniform"]
    s, p, o = synth.triples(w)
    csr = gpu_csr(s, p, o, w.num_entities, w.num_predicates, walk_records=True)
    starts = rd.rdf2v_nonsink_starts(csr)
    tok, ln = rd.rdf2v_random_walks(csr, starts, w.walks_per_node, w.depth, synth.WALK_SEED, 0, 200)
    exp_t, exp_l = _walk_rows(rows)
    assert np.array_equal(ln.cpu().numpy(), exp_l) and np.array_equal(tok.cpu().numpy(), exp_t)


def test_pairs_hand_graph():
    say("[golden] skip-gram pairs on the hand graph")
    walk_header, _ = _read("walks_hand_graph.txt")
    _, rows = _read("pairs_hand_graph.txt")
    t, V, P = _hand_graph(walk_header)
    csr = gpu_csr(t[:, 0], t[:, 1], t[:, 2], V, P)
    tok, ln = rd.rdf2v_random_walks(csr, to_dev([0, 3, 6]), 2, 4, 42)
    pairs = rd.rdf2v_skipgram_pairs(tok, ln, 2)
    assert np.array_equal(pairs.cpu().numpy(), np.array(rows, np.int32).reshape(-1, 2))


def test_bfs_hand_graph():
    say("[golden] BFS walks on the hand graph")
    walk_header, _ = _read("walks_hand_graph.txt")
    _, rows = _read("bfs_hand_graph.txt")
    t, V, P = _hand_graph(walk_header)
    csr = gpu_csr(t[:, 0], t[:, 1], t[:, 2], V, P)
    st = new_status()
    tok, ln, cnt = rd.rdf2v_bfs_walks(csr, to_dev(np.arange(V)), 3, 8, status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    tok, ln, cnt = tok.cpu().numpy(), ln.cpu().numpy(), cnt.cpu().numpy()
    expect_cnt = np.zeros(V, np.int64)
    for r in rows:
        root, i, L = int(r[0]), int(r[1]), int(r[2])
        expect_cnt[root] += 1
        assert ln[root, i] == L and tok[root, i].tolist() == [int(x) for x in r[3:]], (root, i)
    assert cnt.tolist() == expect_cnt.tolist()


def test_vocabulary_iri():
    say("[golden] vocabulary")
    _, rows = _read("vocabulary_iri.txt")

    def col(strings):
        data = [x.encode() for x in strings]
        off = np.zeros(len(data) + 1, np.int64)
        off[1:] = np.cumsum([len(d) for d in data])
        chars = np.frombuffer(b"".join(data), np.uint8).copy()
        return torch.from_numpy(chars).to(device()), torch.from_numpy(off).to(device())

    cols = [col([r[k] for r in rows]) for k in range(3)]
    s, p, o, counts = rd.rdf2v_build_vocabulary(*cols, 16, 16)
    got = np.stack([s.cpu().numpy(), p.cpu().numpy(), o.cpu().numpy()], axis=1)
    assert got.tolist() == [[int(x) for x in r[3:6]] for r in rows]
