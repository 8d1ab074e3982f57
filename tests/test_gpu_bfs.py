"""GPU parity for BFS walks (through the C ABI) against the oracle, bit-exact:
hand-built graphs, random multigraphs and generated workloads, with depth
limits, truncation at max_walks, sink and repeated roots."""

import numpy as np
import pytest
import torch

import oracle
import paper_2508_01073_amd as rd
import synth
from gpu_helpers import device, gpu_csr, new_status, say, to_dev

pytestmark = pytest.mark.gpu


def _compare(csr, rp, ed, V, P, roots, depth, max_walks, what, expect_capacity=None):
    st = new_status()
    tok, ln, cnt = rd.rdf2v_bfs_walks(csr, to_dev(roots), depth, max_walks, status=st)
    torch.cuda.synchronize()
    flags = int(st.item())
    ref_t, ref_l, ref_c, trunc = oracle.bfs_walks(rp, ed, V, P, roots, depth, max_walks)
    cnt = cnt.cpu().numpy()
    assert np.array_equal(cnt, ref_c), f"{what}: walk counts differ"
    tok = tok.cpu().numpy()
    ln = ln.cpu().numpy()
    for r in range(len(roots)):
        k = ref_c[r]
        if not (np.array_equal(tok[r, :k], ref_t[r, :k]) and np.array_equal(ln[r, :k], ref_l[r, :k])):
            raise AssertionError(f"{what}: root {roots[r]} differs: gpu {tok[r, :k].tolist()[:3]} "
                                 f"oracle {ref_t[r, :k].tolist()[:3]}")
    assert bool(flags & rd.RDF2V_STATUS_CAPACITY) == (trunc > 0), what
    assert not flags & ~rd.RDF2V_STATUS_CAPACITY, f"{what}: status {flags}"
    return ref_c


def test_hand_graphs():
    say("[bfs] hand graphs")
    tr = [(0, 0, 1), (0, 1, 2), (1, 0, 3), (2, 1, 3), (3, 0, 0)]
    t = np.array(tr, np.int32)
    rp, ed = oracle.build_csr(t[:, 0], t[:, 1], t[:, 2], 4, 2)
    csr = gpu_csr(t[:, 0], t[:, 1], t[:, 2], 4, 2)
    for depth in (0, 1, 2, 3, 5):
        _compare(csr, rp, ed, 4, 2, np.array([0, 3, 2, 1, 0], np.int32), depth, 5, f"diamond depth {depth}")
    star = np.array([(0, j % 2, j) for j in range(1, 12)] + [(5, 1, 0)], np.int32)
    rp, ed = oracle.build_csr(star[:, 0], star[:, 1], star[:, 2], 12, 2)
    csr = gpu_csr(star[:, 0], star[:, 1], star[:, 2], 12, 2)
    _compare(csr, rp, ed, 12, 2, np.array([0, 7, 5], np.int32), 3, 4, "star truncated")
    _compare(csr, rp, ed, 12, 2, np.array([0, 7, 5], np.int32), 3, 50, "star")


@pytest.mark.parametrize("V,T,depth,seed", [(50, 150, 3, 0), (300, 1200, 4, 1), (2000, 6000, 6, 2),
                                            (5000, 60_000, 2, 3), (40, 30, 10, 4), (5000, 40_000, 3, 5)])
def test_random_multigraphs(V, T, depth, seed):
    say(f"[bfs] random multigraph V={V} T={T} depth={depth}")
    P = 7
    rng = np.random.default_rng(seed)
    s = rng.integers(0, V, T).astype(np.int32)
    p = rng.integers(0, P, T).astype(np.int32)
    o = rng.integers(0, V, T).astype(np.int32)
    s[:5] = 0; o[:2] = 0                        # self-loops and repeated edges at entity 0
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P)
    roots = np.concatenate([np.arange(min(V, 600), dtype=np.int32), np.array([0, 0, V - 1], np.int32)])
    _compare(csr, rp, ed, V, P, roots, depth, V, f"V={V} full")
    _compare(csr, rp, ed, V, P, roots, depth, 7, f"V={V} truncated")


def test_big_levels_and_trees():
    # mean out-degree 20: levels of hundreds and thousands of entities and trees
    # of up to ~20k, past the part of the tree and of a level that is kept in LDS
    say("[bfs] V=20000 T=400000 depth 4, big levels and trees")
    V, P, T = 20_000, 5, 400_000
    rng = np.random.default_rng(11)
    s = rng.integers(0, V, T).astype(np.int32)
    p = rng.integers(0, P, T).astype(np.int32)
    o = rng.integers(0, V, T).astype(np.int32)
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P)
    roots = rng.integers(0, V, 24).astype(np.int32)
    counts = _compare(csr, rp, ed, V, P, roots, 4, V, "big levels")
    assert counts.max() > 5000
    _compare(csr, rp, ed, V, P, roots, 3, 1500, "big levels truncated")


def test_tiny_uniform_all_roots():
    w = synth.WORKLOADS["tiny_uniform"]
    say("[bfs] tiny_uniform, every entity as root, depth 3")
    s, p, o = synth.triples(w)
    V, P = w.num_entities, w.num_predicates
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P)
    counts = _compare(csr, rp, ed, V, P, np.arange(V, dtype=np.int32), 3, 1000, "tiny_uniform")
    assert counts.max() > 100


def test_powerlaw_roots_with_hubs():
    say("[bfs] power law 200k entities, depth 2, hub roots")
    V, P = 200_000, 20
    s, p, o = synth.powerlaw_triples(V, P, 2_000_000, sink_fraction=0.1)
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P)
    deg = np.diff(rp)
    hubs = np.argsort(-deg)[:8].astype(np.int32)
    rng = np.random.default_rng(0)
    roots = np.concatenate([hubs, rng.integers(0, V, 300).astype(np.int32)])
    _compare(csr, rp, ed, V, P, roots, 2, 256, "power law hubs")


def test_out_of_range_root_is_flagged():
    say("[bfs] root out of range")
    t = np.array([(0, 0, 1), (1, 0, 2)], np.int32)
    csr = gpu_csr(t[:, 0], t[:, 1], t[:, 2], 3, 1)
    st = new_status()
    tok, ln, cnt = rd.rdf2v_bfs_walks(csr, to_dev([0, 9, 1]), 2, 4, status=st)
    torch.cuda.synchronize()
    assert int(st.item()) & rd.RDF2V_STATUS_ID_OUT_OF_RANGE
    assert cnt.cpu().tolist() == [1, 0, 1]


@pytest.mark.parametrize("depth,max_walks", [(2, 256), (3, 1024), (3, 40)])
def test_uniform_1m_every_start_sampled(depth, max_walks):
    # the benchmark's launch: every start entity of the 1M-triple uniform graph
    # in one call, trees of ~10^depth entities (up to ~2900 at depth 3); rows of
    # 3000 sampled roots checked against the oracle
    w = synth.WORKLOADS["uniform_1m"]
    say(f"[bfs] uniform_1m every start, depth {depth}, max_walks {max_walks}")
    s, p, o = synth.triples(w)
    V, P = w.num_entities, w.num_predicates
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P)
    roots = oracle.nonsink_starts(rp, V)
    st = new_status()
    tok, ln, cnt = rd.rdf2v_bfs_walks(csr, to_dev(roots), depth, max_walks, status=st)
    torch.cuda.synchronize()
    pick = np.sort(np.random.default_rng(depth * 7 + max_walks).choice(len(roots), 3000, replace=False))
    ref_t, ref_l, ref_c, trunc = oracle.bfs_walks(rp, ed, V, P, roots[pick], depth, max_walks)
    cnt = cnt.cpu().numpy()
    assert np.array_equal(cnt[pick], ref_c)
    tok = tok[torch.from_numpy(pick).to(device())].cpu().numpy()
    ln = ln[torch.from_numpy(pick).to(device())].cpu().numpy()
    for i in range(len(pick)):
        k = ref_c[i]
        assert np.array_equal(tok[i, :k], ref_t[i, :k]) and np.array_equal(ln[i, :k], ref_l[i, :k]), roots[pick[i]]
    flags = int(st.item())
    assert not flags & ~rd.RDF2V_STATUS_CAPACITY
    if trunc > 0:
        assert flags & rd.RDF2V_STATUS_CAPACITY
    if flags & rd.RDF2V_STATUS_CAPACITY:
        assert (cnt == max_walks).any()


def test_trees_around_storage_limits():
    # Roots whose trees have about 500 or 1000 entities above the depth limit,
    # or about 1500 or 3000 in all: on both sides of the sizes where the kernels
    # hand a root from the small on-chip tier to the big one and from there to
    # the workspace pass; children reached twice, back edges into the tree and
    # shuffled entity ids.
    say("[bfs] trees around the on-chip storage limits")
    V, P = 40_000, 3
    rng = np.random.default_rng(5)
    ids = rng.permutation(V).astype(np.int64)
    nxt = [0]

    def fresh(n):
        out = ids[nxt[0]:nxt[0] + n]
        nxt[0] += n
        return out

    trip = []
    roots = []

    def fan(root, kids, grand_per_kid):
        for c in kids:
            trip.append((root, int(rng.integers(P)), c))
        trip.append((root, 0, kids[0]))                 # reached twice
        for c in kids:
            for g in fresh(grand_per_kid):
                trip.append((c, int(rng.integers(P)), g))
            if grand_per_kid:
                trip.append((c, 1, root))               # back edge into the tree

    for n_kids in (510, 511, 512, 1022, 1023, 1024, 1534, 1535, 1536, 3071, 3072):
        r = fresh(1)[0]
        roots.append(r)
        fan(r, fresh(n_kids), 0)
    for n_grand in (1533, 1534, 1535, 3069, 3070, 3071):
        r = fresh(1)[0]
        roots.append(r)
        fan(r, fresh(1), n_grand)
    r = fresh(1)[0]
    roots.append(r)
    fan(r, fresh(40), 75)                               # 1 + 40 + 3000 entities
    t = np.array(trip, np.int64)
    rng.shuffle(t)
    s, p, o = (t[:, k].astype(np.int32) for k in range(3))
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P)
    roots = np.array(roots + roots[:3], np.int32)
    for depth in (1, 2, 3):
        _compare(csr, rp, ed, V, P, roots, depth, 4000, f"limits depth {depth}")
        _compare(csr, rp, ed, V, P, roots, depth, 1500, f"limits depth {depth} truncated")


def test_inconsistent_csr_is_flagged_not_read():
    # row_ptr decreasing at entity 1, past num_edges at entity 2 and 3: every row
    # is checked before its records are read, so BFS only raises the status bit
    say("[bfs] inconsistent CSR")
    dev = device()
    row_ptr = torch.tensor([0, 3, 1, 50, 4], dtype=torch.int32, device=dev)
    edges = torch.tensor([[0, 1], [0, 2], [0, 1], [0, 3]], dtype=torch.int32, device=dev)
    csr = rd.Csr(row_ptr, edges, 4, 1)
    for roots in ([0], [1], [2, 3], [0, 1, 2, 3] * 50):
        st = new_status()
        tok, ln, cnt = rd.rdf2v_bfs_walks(csr, to_dev(roots), 3, 8, status=st)
        torch.cuda.synchronize()
        assert int(st.item()) & rd.RDF2V_STATUS_BAD_CSR, roots
        assert bool((cnt >= 0).all()) and bool((cnt <= 8).all())
