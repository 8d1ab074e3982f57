"""Pins for the oracle's BFS walks (gpuRDF2vec Sec. 3.1: a BFS predecessor tree
per root, one walk per leaf-to-root path, each entity reached once).

The tree is checked against scipy's breadth_first_order (a library BFS that
visits a vertex's neighbours in CSR order) on graphs whose rows are sorted by
object, so that scipy's canonical CSR has the oracle's edge order: first on
duplicate-free graphs, then on multigraphs with parallel records, where the
predicate of each tree edge must be that of the input's first record from the
parent to the child. Hand-worked graphs fix the same rule in both input orders
of two parallel records, with a second parent on the same level, sinks and a
depth-limit leaf; structural invariants cover a generated multigraph."""

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


# Parallel records (Sec. 3.1 keeps one predecessor per reached entity and leaves the
# predicate to a join; here the predicate of a tree edge is that of the first record, in CSR
# order, by which the parent reaches the child). Worked by hand below on a graph where a
# parent reaches a child through two records with different predicates, a second parent of
# the same level reaches that child too, a sink hangs off level 1 and 2, and an entity with
# out-edges sits at the depth limit. Predicate tokens: V + p = 6 (p0), 7 (p1), 8 (p2).
_PARALLEL_A = [
    (0, 1, 1),  # 0 -p1-> 1: first record from 0 to 1
    (1, 2, 3),  # 1 -p2-> 3: first record from 1 to 3
    (0, 0, 2),  # 0 -p0-> 2
    (2, 0, 3),  # 2 -p0-> 3: a second parent of 3 on the same level
    (0, 2, 1),  # 0 -p2-> 1: parallel to the first record
    (1, 1, 3),  # 1 -p1-> 3: parallel to 1 -p2-> 3
    (2, 1, 4),  # 2 -p1-> 4: 4 is a sink
    (0, 0, 5),  # 0 -p0-> 5: 5 is a sink on level 1
    (3, 0, 0),  # 3 -p0-> 0: 3 has out-edges but sits at the depth limit for depth 2
    (3, 2, 4),  # 3 -p2-> 4
]
# The same triples with each pair of parallel records in the opposite input order.
_PARALLEL_B = [_PARALLEL_A[i] for i in (4, 5, 2, 3, 0, 1, 6, 7, 8, 9)]
# Order A with 0 -p0-> 2 first, so 2 is reached (and expanded) before 1 on level 1.
_PARALLEL_C = [_PARALLEL_A[i] for i in (2, 0, 1, 3, 4, 5, 6, 7, 8, 9)]


def _rows(tok, ln, cnt, r):
    return [tok[r, i, :ln[r, i]].tolist() for i in range(cnt[r])]


def test_parallel_records_first_record_labels_the_edge():
    # Order A, root 0, depth 2. Level 1 in the order reached: 1 (by p1; the later p2 record
    # is skipped), 2 (p0), 5 (p0). Level 2: 3 from 1 by 1's first record to 3 (p2, not the
    # later p1; 2's record to 3 comes after 1 was expanded), 4 from 2 (p1). Leaves in the
    # order reached: 5, 3, 4.
    rp, ed = _csr(_PARALLEL_A, 6, 3)
    tok, ln, cnt, trunc = oracle.bfs_walks(rp, ed, 6, 3, np.array([0]), 2, 8)
    assert trunc == 0 and cnt.tolist() == [3]
    assert _rows(tok, ln, cnt, 0) == [[0, 6, 5], [0, 7, 1, 8, 3], [0, 6, 2, 7, 4]]
    assert tok[0, 0].tolist() == [0, 6, 5, -1, -1]
    # Order B: the first records are now 0 -p2-> 1 and 1 -p1-> 3.
    rp, ed = _csr(_PARALLEL_B, 6, 3)
    tok, ln, cnt, _ = oracle.bfs_walks(rp, ed, 6, 3, np.array([0]), 2, 8)
    assert _rows(tok, ln, cnt, 0) == [[0, 6, 5], [0, 8, 1, 7, 3], [0, 6, 2, 7, 4]]


def test_parallel_records_second_parent_on_the_same_level():
    # Order C reaches 2 before 1, so 2 is expanded first and becomes the parent of 3 (by
    # p0); 1 reaches nothing new and is a leaf. Leaves in the order reached: 1, 5, 3, 4.
    rp, ed = _csr(_PARALLEL_C, 6, 3)
    tok, ln, cnt, _ = oracle.bfs_walks(rp, ed, 6, 3, np.array([0]), 2, 8)
    assert _rows(tok, ln, cnt, 0) == [[0, 7, 1], [0, 6, 5], [0, 6, 2, 6, 3], [0, 6, 2, 7, 4]]


def test_parallel_records_depth_and_other_roots():
    rp, ed = _csr(_PARALLEL_A, 6, 3)
    roots = np.array([0, 1, 3, 4, 1], dtype=np.int32)
    tok, ln, cnt, trunc = oracle.bfs_walks(rp, ed, 6, 3, roots, 3, 8)
    assert trunc == 0 and cnt.tolist() == [3, 3, 4, 1, 3]
    # depth 3 from 0: 3 is expanded now but reaches only 0 and 4, both already in the tree,
    # so the leaves are those of depth 2
    assert _rows(tok, ln, cnt, 0) == [[0, 6, 5], [0, 7, 1, 8, 3], [0, 6, 2, 7, 4]]
    assert tok[0, 1].tolist() == [0, 7, 1, 8, 3, -1, -1]
    # root 1: 3 by p2 (its first record to 3); from 3: 0 (p0), 4 (p2); from 0: 2 (p0, the
    # record to 1 leads back to the root), 5 (p0); depth 3 stops at 2 and 5
    assert _rows(tok, ln, cnt, 1) == [[1, 8, 3, 8, 4], [1, 8, 3, 6, 0, 6, 2], [1, 8, 3, 6, 0, 6, 5]]
    # root 3: 0 (p0), 4 (p2); from 0: 1 by p1 (its first record to 1), 2 (p0), 5 (p0)
    assert _rows(tok, ln, cnt, 2) == [[3, 8, 4], [3, 6, 0, 7, 1], [3, 6, 0, 6, 2], [3, 6, 0, 6, 5]]
    # a sink root gives the root alone; a duplicate root repeats its walks
    assert _rows(tok, ln, cnt, 3) == [[4]]
    assert _rows(tok, ln, cnt, 4) == _rows(tok, ln, cnt, 1)


def _sorted_multigraph(V, E, P, seed):
    """Rows sorted by object (so that scipy's canonical CSR visits neighbours in the oracle's
    CSR order), with parallel records: about a third of the records repeat an earlier (s, o)
    pair with their own predicate."""
    rng = np.random.default_rng(seed)
    s = rng.integers(0, V, E)
    o = rng.integers(0, V, E)
    rep = rng.integers(0, E, E // 3)
    s = np.concatenate([s, s[rep]])
    o = np.concatenate([o, o[rep]])
    order = np.lexsort((o, s))                                    # sorted by (s, o); ties keep order
    s, o = s[order], o[order]
    p = rng.integers(0, P, s.shape[0])
    return s.astype(np.int32), p.astype(np.int32), o.astype(np.int32)


@pytest.mark.parametrize("V,E,depth,seed", [(30, 90, 3, 10), (200, 700, 4, 11), (60, 400, 5, 12)])
def test_tree_matches_scipy_bfs_on_multigraph(V, E, depth, seed):
    P = 7
    s, p, o = _sorted_multigraph(V, E, P, seed)
    assert len(set(zip(s.tolist(), o.tolist()))) < len(s)          # parallel records present
    rp, ed = oracle.build_csr(s, p, o, V, P)
    adj = csr_matrix((np.ones(len(s)), (s, o)), shape=(V, V))   # parallel records merge here
    roots = np.arange(V, dtype=np.int32)
    tok, ln, cnt, trunc = oracle.bfs_walks(rp, ed, V, P, roots, depth, V)
    assert trunc == 0
    labelled = 0
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
        leaves = [v for v in tree if not has_child[v]]
        assert cnt[r] == len(leaves)
        for i, leaf in enumerate(leaves):
            path = [leaf]
            while path[-1] != r:
                path.append(parent[path[-1]])
            path = path[::-1]
            row = tok[r, i, :ln[r, i]]
            assert row[0::2].tolist() == path
            for h in range(len(path) - 1):
                # the input's first record from parent to child (rows keep input order)
                k = np.nonzero((s == path[h]) & (o == path[h + 1]))[0]
                assert row[2 * h + 1] == V + p[k[0]]
                labelled += len(set(p[k].tolist())) > 1
    assert labelled > 0                                            # some tree edge had a choice
