"""GPU parity: the HIP path (through the C ABI) against the CPU oracle, bit-exact.

Small cases compare every output element; full-size workloads compare the
whole CSR and start set, and walk rows on sampled windows (first, last/ragged,
random, hub starts), plus properties that hold at any size on the device.
"""

import itertools

import numpy as np
import pytest
import torch

import oracle
import paper_2508_01073_amd as rd
import synth
from gpu_helpers import (assert_csr_equal, assert_rows_equal, assert_walk_records, check_walk_properties,
                         compare_all, compare_windows, device, gpu_csr, gpu_walks, new_status, plain, say, to_dev)
from sparse_ids import expected_on_sparse, sparse_graph

pytestmark = pytest.mark.gpu


# ----------------------------------------------------------------------------
# Hand-built graphs, every element
# ----------------------------------------------------------------------------

def _hand_graphs():
    g = {}
    n = 7
    g["chain"] = ([(i, i % 3, i + 1) for i in range(n - 1)], n, 3, [0, 3, 6])
    g["star10"] = ([(0, j % 4, j + 1) for j in range(10)], 11, 4, [0, 5])
    g["complete6"] = ([(v, (v + j) % 2, j) for v in range(6) for j in range(6)], 6, 2, list(range(6)))
    rng = np.random.default_rng(11)
    tr = [(int(a), int(b), int(c)) for a, b, c in zip(rng.integers(0, 8, 16), rng.integers(0, 3, 16),
                                                       rng.integers(0, 8, 16))]
    tr += [(0, 1, 0), (0, 1, 0), (3, 2, 3)]  # duplicates and self-loops
    g["multi_selfloop"] = (tr, 9, 3, [0, 3, 8, 8, 1])  # entity 8 has no out-edge
    g["sink_starts"] = ([(0, 0, 1)], 4, 1, [1, 2, 3, 0])
    return g


HAND = _hand_graphs()


@pytest.mark.parametrize("name", sorted(HAND))
@pytest.mark.parametrize("depth", [0, 1, 4, 5, 9, 17, 64])
def test_hand_graph_parity(name, depth):
    tr, V, P, starts = HAND[name]
    say(f"[hand] {name} depth={depth}")
    t = np.array(tr, dtype=np.int32)
    rp, ed = oracle.build_csr(t[:, 0], t[:, 1], t[:, 2], V, P)
    csr = gpu_csr(t[:, 0], t[:, 1], t[:, 2], V, P, walk_records=True)
    assert_csr_equal(csr, rp, ed)
    assert_walk_records(csr, rp, ed)
    wpn = 37
    for seed in (42, 2**63 + 5):
        tr_, lr_ = oracle.random_walks(rp, ed, V, P, np.array(starts), wpn, depth, seed)
        for c, what in [(csr, "walk records"), (plain(csr), "plain records")]:
            tok, ln = gpu_walks(c, to_dev(starts), wpn, depth, seed)
            assert_rows_equal(tok.cpu().numpy(), ln.cpu().numpy(), tr_, lr_, f"{name} seed {seed} {what}")


# ----------------------------------------------------------------------------
# Random graphs spanning several 4096-triple tiles with ragged tails and 1..4
# radix passes (entity id widths 1 .. 26 bits)
# ----------------------------------------------------------------------------

RANDOM_CASES = [
    (1, 1, 5000), (2, 3, 1), (37, 1, 4096 * 3 + 17), (300, 7, 50_000), (256, 5, 8192),
    (70_000, 11, 100_001), (2**25 + 3, 5, 20_000), (1_000, 20, 4095),
    (2**18, 9, 300_007), (2**18 + 1, 9, 300_007),  # two 9-bit passes; three 7-bit passes
]


@pytest.mark.parametrize("V,P,T", RANDOM_CASES)
def test_random_graph_parity(V, P, T):
    say(f"[random] V={V} P={P} T={T}")
    rng = np.random.default_rng(V * 31 + T)
    s = rng.integers(0, V, T).astype(np.int32)
    p = rng.integers(0, P, T).astype(np.int32)
    o = rng.integers(0, V, T).astype(np.int32)
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P, walk_records=True)
    assert_csr_equal(csr, rp, ed)
    assert_walk_records(csr, rp, ed)
    starts = oracle.nonsink_starts(rp, V)
    starts_gpu = rd.rdf2v_nonsink_starts(csr)
    assert np.array_equal(starts_gpu.cpu().numpy(), starts)
    for depth, wpn in [(4, 3), (8, 2), (16, 1), (33, 1)]:
        sub = starts[:20_000]
        tr_, lr_ = oracle.random_walks(rp, ed, V, P, sub, wpn, depth, 42)
        for c, what in [(csr, "walk records"), (plain(csr), "plain records")]:
            tok, ln = gpu_walks(c, to_dev(sub), wpn, depth, 42)
            assert_rows_equal(tok.cpu().numpy(), ln.cpu().numpy(), tr_, lr_, f"depth {depth} {what}")


def test_powerlaw_small_with_sinks():
    say("[powerlaw small] V=20000 T=300000 sinks 10%")
    V, P = 20_000, 40
    s, p, o = synth.powerlaw_triples(V, P, 300_000, sink_fraction=0.1)
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P, walk_records=True)
    assert_csr_equal(csr, rp, ed)
    assert_walk_records(csr, rp, ed)
    starts = oracle.nonsink_starts(rp, V)
    tr_, lr_ = oracle.random_walks(rp, ed, V, P, starts, 3, 16, 7)
    for c, what in [(csr, "walk records"), (plain(csr), "plain records")]:
        tok, ln = gpu_walks(c, to_dev(starts), 3, 16, 7)
        assert_rows_equal(tok.cpu().numpy(), ln.cpu().numpy(), tr_, lr_, f"powerlaw small {what}")


# ----------------------------------------------------------------------------
# The generated workloads
# ----------------------------------------------------------------------------

def test_tiny_uniform_full_parity():
    w = synth.WORKLOADS["tiny_uniform"]
    say(f"[workload] {w.describe()}")
    s, p, o = synth.triples(w)
    V, P = w.num_entities, w.num_predicates
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P, walk_records=True)
    assert_csr_equal(csr, rp, ed)
    assert_walk_records(csr, rp, ed)
    starts = oracle.nonsink_starts(rp, V)
    starts_dev = rd.rdf2v_nonsink_starts(csr)
    assert np.array_equal(starts_dev.cpu().numpy(), starts)
    tr_, lr_ = oracle.random_walks(rp, ed, V, P, starts, w.walks_per_node, w.depth, synth.WALK_SEED)
    for c, what in [(csr, "walk records"), (plain(csr), "plain records")]:
        tok, ln = gpu_walks(c, starts_dev, w.walks_per_node, w.depth, synth.WALK_SEED)
        assert_rows_equal(tok.cpu().numpy(), ln.cpu().numpy(), tr_, lr_, f"tiny_uniform {what}")


def _windows(num_walks, wpn, starts, deg, rng, k=24, size=1024):
    win = [(0, min(4096, num_walks)), (max(0, num_walks - 4093), min(4093, num_walks))]
    for b in rng.integers(0, max(1, num_walks - size), k):
        win.append((int(b), min(size, num_walks - int(b))))
    # walks from the highest-degree start entities
    for i in np.argsort(-deg[starts])[:4]:
        win.append((int(i) * wpn, wpn))
    return win


@pytest.mark.parametrize("name", ["uniform_1m", "powerlaw_20m", "dense_10m"])
def test_full_size_workload(name):
    w = synth.WORKLOADS[name]
    say(f"[workload] {w.describe()}")
    s, p, o = synth.triples(w)
    V, P = w.num_entities, w.num_predicates
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P, walk_records=True)
    assert_csr_equal(csr, rp, ed)
    assert_walk_records(csr, rp, ed)
    starts = oracle.nonsink_starts(rp, V)
    starts_dev = rd.rdf2v_nonsink_starts(csr)
    assert np.array_equal(starts_dev.cpu().numpy(), starts)
    num_walks = len(starts) * w.walks_per_node
    say(f"[workload] {name}: one launch of {num_walks} walks, depth {w.depth}")
    tok, ln = gpu_walks(csr, starts_dev, w.walks_per_node, w.depth, synth.WALK_SEED)
    check_walk_properties(tok, ln, starts_dev, w.walks_per_node, V, P, w.depth)
    rng = np.random.default_rng(5)
    win = _windows(num_walks, w.walks_per_node, starts, np.diff(rp), rng)
    n = compare_windows(csr, rp, ed, V, P, starts, w.walks_per_node, w.depth, synth.WALK_SEED, tok, ln, win)
    say(f"[workload] {name}: {n} sampled rows bit-exact")
    n = compare_all(rp, ed, V, P, starts, w.walks_per_node, w.depth, synth.WALK_SEED, tok, ln)
    say(f"[workload] {name}: all {n} walks bit-exact")
    # the 8-byte-record path gives the same corpus
    tok2, ln2 = gpu_walks(plain(csr), starts_dev, w.walks_per_node, w.depth, synth.WALK_SEED)
    assert torch.equal(tok2, tok) and torch.equal(ln2, ln)


# ----------------------------------------------------------------------------
# Batching, determinism, status reporting, edge cases
# ----------------------------------------------------------------------------

def test_batches_concatenate_to_one_shot():
    say("[batches] uniform 50k entities")
    V, P = 50_000, 9
    s, p, o = synth.uniform_triples(V, P, 400_000)
    csr = gpu_csr(s, p, o, V, P, walk_records=True)
    starts_dev = rd.rdf2v_nonsink_starts(csr)
    wpn, depth = 7, 6
    total = starts_dev.shape[0] * wpn
    full_t, full_l = gpu_walks(csr, starts_dev, wpn, depth, 42)
    parts_t, parts_l, b = [], [], 0
    for size in itertools.cycle([1, 255, 256, 257, 4099, 65_536, 100_003]):
        if b >= total:
            break
        c = min(size, total - b)
        t_, l_ = gpu_walks(csr, starts_dev, wpn, depth, 42, b, c)
        parts_t.append(t_); parts_l.append(l_); b += c
    assert torch.equal(torch.cat(parts_t), full_t) and torch.equal(torch.cat(parts_l), full_l)


def test_repeat_runs_identical():
    say("[repeat] powerlaw 200k entities")
    V, P = 200_000, 30
    s, p, o = synth.powerlaw_triples(V, P, 3_000_000)
    c1 = gpu_csr(s, p, o, V, P, walk_records=True)
    c2 = gpu_csr(s, p, o, V, P, walk_records=True)
    assert torch.equal(c1.row_ptr, c2.row_ptr) and torch.equal(c1.edges, c2.edges)
    assert torch.equal(c1.walk_edges, c2.walk_edges)
    st = rd.rdf2v_nonsink_starts(c1)
    a = gpu_walks(c1, st, 5, 8, 42)
    b = gpu_walks(c2, st, 5, 8, 42)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def test_status_bits_for_bad_ids():
    say("[status] out-of-range ids")
    V, P = 10, 3
    s = np.array([0, 1, 2, 3], np.int32); p = np.array([0, 1, 2, 0], np.int32)
    o = np.array([1, 2, 3, 4], np.int32)
    for bad in [("s", 10), ("o", 11), ("p", 3), ("s", -1)]:
        ss, pp, oo = s.copy(), p.copy(), o.copy()
        {"s": ss, "p": pp, "o": oo}[bad[0]][2] = bad[1]
        st = new_status()
        gpu_csr(ss, pp, oo, V, P, status=st)
        assert int(st.item()) & rd.RDF2V_STATUS_ID_OUT_OF_RANGE, bad
    csr = gpu_csr(s, p, o, V, P)
    st = new_status()
    rd.rdf2v_random_walks(csr, to_dev([0, 12]), 2, 3, 42, status=st)
    torch.cuda.synchronize()
    assert int(st.item()) & rd.RDF2V_STATUS_ID_OUT_OF_RANGE


def test_inconsistent_csr_is_flagged_not_read():
    say("[status] inconsistent CSR")
    dev = device()
    # row_ptr decreasing at entity 1 and past num_edges at entity 2: every gather is
    # bounds-checked before it is issued, so the kernel only raises the status bit.
    row_ptr = torch.tensor([0, 3, 1, 50, 4], dtype=torch.int32, device=dev)
    edges = torch.tensor([[0, 1], [0, 2], [0, 1], [0, 3]], dtype=torch.int32, device=dev)
    csr = rd.Csr(row_ptr, edges, 4, 1)
    for start in (1, 2):
        st = new_status()
        tok, ln = rd.rdf2v_random_walks(csr, to_dev([start]), 1, 4, 42, status=st)
        torch.cuda.synchronize()
        assert int(st.item()) & rd.RDF2V_STATUS_BAD_CSR
    # walk records whose row bounds run past num_edges are caught the same way
    good_rp = torch.tensor([0, 2, 3, 4, 4], dtype=torch.int32, device=dev)
    recs = torch.tensor([[0, 1, 2, 9], [0, 2, 3, 9], [0, 1, 2, 9], [0, 3, 4, 4]], dtype=torch.int32,
                        device=dev)
    csr = rd.Csr(good_rp, edges, 4, 1, recs)
    st = new_status()
    rd.rdf2v_random_walks(csr, to_dev([0, 2]), 8, 6, 42, status=st)
    torch.cuda.synchronize()
    assert int(st.item()) & rd.RDF2V_STATUS_BAD_CSR
    # building walk records over an object id out of range flags it and gives that record the
    # bounds (0, 0) of an empty row; the other records are unaffected
    bad_edges = torch.tensor([[0, 1], [0, 7], [0, 1], [0, 3]], dtype=torch.int32, device=dev)
    st = new_status()
    out = rd.rdf2v_build_walk_edges(rd.Csr(good_rp, bad_edges, 4, 1), status=st).walk_edges
    torch.cuda.synchronize()
    assert int(st.item()) & rd.RDF2V_STATUS_ID_OUT_OF_RANGE
    assert out.cpu().numpy().tolist() == [[0, 1, 2, 3], [0, 7, 0, 0], [0, 1, 2, 3], [0, 3, 4, 4]]


def test_empty_and_degenerate_inputs():
    say("[edge] empty / degenerate")
    dev = device()
    e = torch.empty(0, dtype=torch.int32, device=dev)
    csr = rd.rdf2v_build_csr(e, e, e, 5, 2)
    torch.cuda.synchronize()
    assert torch.equal(csr.row_ptr.cpu(), torch.zeros(6, dtype=torch.int32))
    assert rd.rdf2v_nonsink_starts(csr).numel() == 0
    tok, ln = gpu_walks(csr, to_dev([0, 4]), 3, 5, 42)
    assert bool((ln == 1).all()) and torch.equal(tok[:, 0].cpu(), torch.tensor([0, 0, 0, 4, 4, 4], dtype=torch.int32))
    assert bool((tok[:, 1:] == -1).all())
    tok, ln = gpu_walks(csr, to_dev([0]), 0, 5, 42)
    assert tok.shape[0] == 0 and ln.shape[0] == 0
    csr0 = rd.rdf2v_build_csr(e, e, e, 0, 0)
    torch.cuda.synchronize()
    assert csr0.row_ptr.cpu().tolist() == [0]


def test_unaligned_output_rows():
    say("[edge] output pointer not 16-byte aligned")
    V, P = 3000, 4
    s, p, o = synth.uniform_triples(V, P, 20_000)
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P)
    starts = oracle.nonsink_starts(rp, V)[:500]
    depth, wpn = 5, 3
    n = len(starts) * wpn
    buf = torch.full((n * (2 * depth + 1) + 1,), 7, dtype=torch.int32, device=device())
    tok = buf[1:].view(n, 2 * depth + 1)
    lens = torch.empty(n, dtype=torch.int32, device=device())
    gpu_walks(csr, to_dev(starts), wpn, depth, 42, tokens=tok, lens=lens)
    tr_, lr_ = oracle.random_walks(rp, ed, V, P, starts, wpn, depth, 42)
    assert_rows_equal(tok.cpu().numpy(), lens.cpu().numpy(), tr_, lr_, "unaligned")
    assert int(buf[0].item()) == 7


def test_walk_ids_beyond_2_pow_32():
    say("[edge] walk ids >= 2^32 (Philox counter high word)")
    V, P = 5000, 7
    s, p, o = synth.uniform_triples(V, P, 40_000)
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P, walk_records=True)
    starts = oracle.nonsink_starts(rp, V)[:3]
    wpn = 2**31 - 1                      # 3 * wpn walks > 2^32
    for b in (2**32 - 700, 2**32 + 5, 3 * wpn - 1000):
        tr_, lr_ = oracle.random_walks(rp, ed, V, P, starts, wpn, 9, 42, b, 1000)
        for c, what in [(csr, "walk records"), (plain(csr), "plain records")]:
            tok, ln = gpu_walks(c, to_dev(starts), wpn, 9, 42, b, 1000)
            assert_rows_equal(tok.cpu().numpy(), ln.cpu().numpy(), tr_, lr_, f"walks from {b} {what}")


def test_largest_id_space():
    # V + P = 2^31 - 1, the largest id space the token layout allows: 31-bit subject keys (four
    # 8-bit radix passes), an 8 GiB row_ptr, start-set scans over 2^31 entities, and the token
    # V + P - 1 = 2^31 - 2. The expectation is the oracle's on the compact graph, relabelled
    # (sparse_ids; the relabel is checked against the oracle itself on the CPU).
    P = 7
    V = 2**31 - 1 - P
    wpn, depth = 3, 6
    say(f"[edge] largest id space V={V} P={P}: CSR, walk records, start set, walks")
    U, s_r, p, o_r = sparse_graph(V, P, 300_000, 20_000, seed=31)
    rp_x, ed_x, starts_x, tok_x, ln_x = expected_on_sparse(U, s_r, p, o_r, V, P, wpn, depth, 42)
    assert int(tok_x.max()) == 2**31 - 2
    csr = gpu_csr(U[s_r], p, U[o_r], V, P)
    ed = csr.edges.cpu().numpy()
    assert np.array_equal(ed, ed_x), "edge records differ"
    chunk = 1 << 28
    for a in range(0, V + 1, chunk):
        got = csr.row_ptr[a:a + chunk].cpu().numpy()
        assert np.array_equal(got, rp_x[a:a + chunk]), f"row_ptr differs in [{a}, {a + chunk})"
    assert rd.rdf2v_walk_edges_recommended(V, csr.num_edges)
    csr_r = rd.rdf2v_build_walk_edges(csr)
    torch.cuda.synchronize()
    assert_walk_records(csr_r, rp_x, ed_x)
    starts = rd.rdf2v_nonsink_starts(csr)
    assert np.array_equal(starts.cpu().numpy(), starts_x)
    for c, what in [(csr_r, "walk records"), (csr, "plain records")]:
        tok, ln = gpu_walks(c, starts, wpn, depth, 42)
        assert_rows_equal(tok.cpu().numpy(), ln.cpu().numpy(), tok_x, ln_x, f"largest id space, {what}")


def test_concurrent_streams_do_not_interfere():
    say("[streams] two graphs built and walked on two streams at once")
    dev = device()
    graphs = [synth.uniform_triples(30_000, 9, 300_000, seed=1), synth.powerlaw_triples(40_000, 11, 400_000, seed=2)]
    sizes = [(30_000, 9), (40_000, 11)]
    streams = [torch.cuda.Stream(dev), torch.cuda.Stream(dev)]
    inputs = [[to_dev(a) for a in g] for g in graphs]
    torch.cuda.synchronize()
    results = []
    for (sd, pd, od), (V, P), strm in zip(inputs, sizes, streams):
        with torch.cuda.stream(strm):
            st = torch.zeros(1, dtype=torch.int32, device=dev)
            csr = rd.rdf2v_build_csr(sd, pd, od, V, P, status=st, stream=strm)
            csr = rd.rdf2v_build_walk_edges(csr, status=st, stream=strm)
            starts, cnt = rd.rdf2v_nonsink_starts(csr, stream=strm, sync=False)
            results.append((csr, starts, cnt, st, strm))
    outs = []
    for csr, starts, cnt, st, strm in results:
        strm.synchronize()
        n = int(cnt.item())
        with torch.cuda.stream(strm):
            outs.append(rd.rdf2v_random_walks(csr, starts[:n], 4, 6, 42, status=st, stream=strm))
    torch.cuda.synchronize()
    for (s, p, o), (V, P), (csr, starts, cnt, st, _), (tok, ln) in zip(graphs, sizes, results, outs):
        rd.check_device_status(st, "concurrent")
        rp, ed = oracle.build_csr(s, p, o, V, P)
        assert_csr_equal(csr, rp, ed)
        st_ref = oracle.nonsink_starts(rp, V)
        tr_, lr_ = oracle.random_walks(rp, ed, V, P, st_ref, 4, 6, 42)
        assert_rows_equal(tok.cpu().numpy(), ln.cpu().numpy(), tr_, lr_, f"stream graph V={V}")
