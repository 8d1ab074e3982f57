"""Pins for the oracle's BFS walks (gpuRDF2vec Sec. 3.1: a BFS predecessor tree
per root, one walk per leaf-to-root path, each entity reached once).

The tree is checked against scipy's breadth_first_order (a library BFS that
visits a vertex's neighbours in CSR order) on graphs whose rows are sorted and
duplicate-free, so that scipy's canonical CSR has the oracle's edge order; the
walks against a hand-worked graph and structural invariants."""

import numpy as np
import pytest
from scipy.sparse import csr_matrix
from scipy.sparse.csgraph import breadth_first_order

import oracle
import synth


def _csr(triples, V, P):
    t = np.array(triples, dtype=np.int32).reshape(-1, 3)
    return oracle.build_csr(t[:, 0], t[:, 1], t[:, 2], V, P)


def test_hand_worked_diamond_with_cycle():
    # 0 -p0-> 1, 0 -p1-> 2, 1 -p0-> 3, 2 -p1-> 3, 3 -p0-> 0;  predicate tokens are 4 (p0), 5 (p1)
    rp, ed = _csr([(0, 0, 1), (0, 1, 2), (1, 0, 3), (2, 1, 3), (3, 0, 0)], 4, 2)
    tok, ln, cnt, trunc = oracle.bfs_walks(rp, ed, 4, 2, np.array([0, 3, 2]), 3, 5)
    assert cnt.tolist() == [2, 2, 1] and trunc == 0
    # root 0: 1 and 2 at level 1; 3 reached from 1 first; leaves in order reached: 2, 3
    assert tok[0, :2].tolist() == [[0, 5, 2, -1, -1, -1, -1], [0, 4, 1, 4, 3, -1, -1]]
    assert tok[1, :2].tolist() == [[3, 4, 0, 4, 1, -1, -1], [3, 4, 0, 5, 2, -1, -1]]
    # root 2: a chain 2 -> 3 -> 0 -> 1 (0 -> 2 leads back to the root); 1 is the only leaf
    assert tok[2, 0].tolist() == [2, 5, 3, 4, 0, 4, 1]
    assert ln[0, :2].tolist() == [3, 5] and ln[2, 0] == 7
    # depth 0: the root alone is the only leaf
    tok0, ln0, cnt0, _ = oracle.bfs_walks(rp, ed, 4, 2, np.array([1]), 0, 3)
    assert cnt0.tolist() == [1] and tok0[0, 0].tolist() == [1] and ln0[0, 0] == 1


def test_hand_worked_depth_limit():
    # chain 2 -> 3 -> 0 -> 1 plus 0 -> 2 back edge; from root 2 with depth 2: 2, 3, 0 (0 is at the limit)
    rp, ed = _csr([(2, 1, 3), (3, 0, 0), (0, 0, 1), (0, 1, 2)], 4, 2)
    tok, ln, cnt, _ = oracle.bfs_walks(rp, ed, 4, 2, np.array([2]), 2, 4)
    assert cnt.tolist() == [1]
    assert tok[0, 0].tolist() == [2, 5, 3, 4, 0]


def test_sink_root_and_truncation():
    rp, ed = _csr([(0, 0, j) for j in range(1, 9)], 9, 1)
    tok, ln, cnt, trunc = oracle.bfs_walks(rp, ed, 9, 1, np.array([5, 0]), 4, 3)
    assert cnt.tolist() == [1, 3] and trunc == 1              # root 0 has 8 leaves, 3 kept
    assert tok[0, 0, 0] == 5 and ln[0, 0] == 1
    assert tok[1, :3, :3].tolist() == [[0, 9, 1], [0, 9, 2], [0, 9, 3]]


def _sorted_unique_graph(V, E, P, seed):
    rng = np.random.default_rng(seed)
    s = rng.integers(0, V, E)
    o = rng.integers(0, V, E)
    so = np.unique(np.stack([s, o], axis=1), axis=0)          # sorted by (s, o), no duplicate pairs
    p = rng.integers(0, P, so.shape[0])
    return so[:, 0].astype(np.int32), p.astype(np.int32), so[:, 1].astype(np.int32)


@pytest.mark.parametrize("V,E,depth,seed", [(30, 60, 3, 0), (200, 500, 4, 1), (500, 3000, 6, 2), (50, 40, 8, 3)])
def test_tree_matches_scipy_bfs(V, E, depth, seed):
    P = 5
    s, p, o = _sorted_unique_graph(V, E, P, seed)
    rp, ed = oracle.build_csr(s, p, o, V, P)
    adj = csr_matrix((np.ones(len(s)), (s, o)), shape=(V, V))
    roots = np.arange(V, dtype=np.int32)
    tok, ln, cnt, trunc = oracle.bfs_walks(rp, ed, V, P, roots, depth, V)
    assert trunc == 0
    for r in roots:
        order, pred = breadth_first_order(adj, int(r), directed=True, return_predecessors=True)
        level = {int(r): 0}
        for v in order[1:]:
            level[int(v)] = level[int(pred[v])] + 1
        tree = [int(v) for v in order if level[int(v)] <= depth]
        parent = {v: int(pred[v]) for v in tree if v != r}
        has_child = {v: False for v in tree}
        for v, u in parent.items():
            has_child[u] = True
        leaves = [v for v in tree if not has_child[v]]           # in scipy's visiting order
        assert cnt[r] == len(leaves)
        for i, leaf in enumerate(leaves):
            path = [leaf]
            while path[-1] != r:
                path.append(parent[path[-1]])
            path = path[::-1]
            row = tok[r, i, :ln[r, i]]
            assert row[0::2].tolist() == path
            for h in range(len(path) - 1):                         # the predicate of the tree edge
                k = np.nonzero((s == path[h]) & (o == path[h + 1]))[0]
                assert row[2 * h + 1] == V + p[k[0]]


def test_invariants_on_multigraph():
    w = synth.WORKLOADS["tiny_uniform"]
    s, p, o = synth.triples(w)
    V, P = w.num_entities, w.num_predicates
    rp, ed = oracle.build_csr(s, p, o, V, P)
    triples = set(zip(s.tolist(), p.tolist(), o.tolist()))
    roots = oracle.nonsink_starts(rp, V)[:40]
    tok, ln, cnt, _ = oracle.bfs_walks(rp, ed, V, P, roots, 3, 2000)
    for r, root in enumerate(roots):
        ends = set()
        for i in range(cnt[r]):
            row = tok[r, i, :ln[r, i]]
            assert row[0] == root and ln[r, i] % 2 == 1
            for h in range((ln[r, i] - 1) // 2):
                assert (int(row[2 * h]), int(row[2 * h + 1]) - V, int(row[2 * h + 2])) in triples
            ents = row[0::2].tolist()
            assert len(set(ents)) == len(ents)                     # a walk never revisits an entity
            ends.add(int(row[-1]))
        assert len(ends) == cnt[r]                                 # each leaf ends exactly one walk
