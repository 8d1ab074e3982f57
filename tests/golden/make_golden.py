"""Writes the golden fixtures in this folder. It calls only the CPU oracle (and the
seeded input generators), never the GPU library.

Each fixture is a small text file: a header of '#' lines (what it is, the
passage of gpuRDF2vec it follows, how it was made), then one record per line.
Run from the repository root:  python tests/golden/make_golden.py

The fixtures freeze the oracle's output on small inputs: tests/test_golden.py
regenerates them on the CPU (so any change to the oracle's arithmetic shows up
as a diff that its commit has to justify) and the GPU tests compare the HIP
path with them directly.
"""

from __future__ import annotations

import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
import synth  # noqa: E402

SEED = 42

# A hand-made multigraph with every case a walk meets: a cycle, a self-loop, a
# duplicate triple, a hub, and two sinks (entities 6 and 7 have no out-edge).
HAND_V, HAND_P = 8, 3
HAND_TRIPLES = [
    (0, 0, 1), (0, 1, 2), (0, 2, 3), (0, 0, 1),   # hub 0 with a duplicate triple
    (1, 1, 2), (2, 2, 0),                          # cycle 0 -> 1 -> 2 -> 0
    (3, 0, 3), (3, 1, 4),                          # self-loop on 3
    (4, 2, 5), (5, 0, 6), (5, 1, 7),               # chain into the sinks 6 and 7
]


def _header(lines: list[str]) -> str:
    return "".join(f"# {l}\n" for l in lines)


def hand_csr():
    t = np.array(HAND_TRIPLES, np.int32)
    return oracle.build_csr(t[:, 0], t[:, 1], t[:, 2], HAND_V, HAND_P)


def walks_text(tokens, lens) -> str:
    return "".join(f"{int(l)} " + " ".join(str(int(x)) for x in row) + "\n" for row, l in zip(tokens, lens))


def fixture_walks_hand() -> str:
    rp, ed = hand_csr()
    starts = np.arange(HAND_V, dtype=np.int32)          # every entity, sinks included
    tok, ln = oracle.random_walks(rp, ed, HAND_V, HAND_P, starts, 5, 6, SEED)
    head = _header([
        "Random walks on a hand-made multigraph (gpuRDF2vec Sec. 2: a walk chooses its next hop",
        "at random; Sec. 3.1: entity/predicate rows, padded with -1 once a walk stops).",
        f"Triples (s, p, o), V={HAND_V}, P={HAND_P}: " + " ".join(f"{s},{p},{o}" for s, p, o in HAND_TRIPLES),
        "Starts: every entity 0..7 (6 and 7 are sinks); 5 walks per start; depth 6; seed 42.",
        "Predicate token = V + p. Row: len, then the 2*depth+1 tokens of walk w = start_index*5 + j.",
        "Written by tests/golden/make_golden.py from the CPU oracle.",
    ])
    return head + walks_text(tok, ln)


def fixture_walks_tiny() -> str:
    w = synth.WORKLOADS["tiny_uniform"]
    s, p, o = synth.triples(w)
    rp, ed = oracle.build_csr(s, p, o, w.num_entities, w.num_predicates)
    starts = oracle.nonsink_starts(rp, w.num_entities)
    tok, ln = oracle.random_walks(rp, ed, w.num_entities, w.num_predicates, starts, w.walks_per_node, w.depth,
                                  synth.WALK_SEED, 0, 200)
    head = _header([
        "The first 200 walks of the tiny uniform workload (gpuRDF2vec Sec. 2, Sec. 3.1, Sec. 3.3:",
        "walks_per_node walks of at most depth hops from every start entity).",
        f"Workload: {w.describe()}; generator seed {synth.GENERATOR_SEED}; walk seed {synth.WALK_SEED};",
        "start set: entities with out-degree >= 1, ascending.",
        "Row: len, then the 2*depth+1 tokens. Written by tests/golden/make_golden.py from the CPU oracle.",
    ])
    return head + walks_text(tok, ln)


def fixture_pairs_hand() -> str:
    rp, ed = hand_csr()
    tok, ln = oracle.random_walks(rp, ed, HAND_V, HAND_P, np.array([0, 3, 6], np.int32), 2, 4, SEED)
    pairs = oracle.skipgram_pairs(tok, ln, 2)
    head = _header([
        "Skip-gram (center, context) pairs, window 2, of six walks on the hand-made graph above",
        "(gpuRDF2vec Sec. 3.2: the corpus becomes center-context pairs; Sec. 3.1: padding is dropped).",
        "Walks: starts 0, 3, 6; 2 walks each; depth 4; seed 42. Pairs in order walk, center, context.",
        "Written by tests/golden/make_golden.py from the CPU oracle.",
    ])
    return head + "".join(f"{int(a)} {int(b)}\n" for a, b in pairs)


def fixture_bfs_hand() -> str:
    rp, ed = hand_csr()
    roots = np.arange(HAND_V, dtype=np.int32)
    tok, ln, cnt, trunc = oracle.bfs_walks(rp, ed, HAND_V, HAND_P, roots, 3, 8)
    head = _header([
        "BFS walks of depth 3 from every entity of the hand-made graph above (gpuRDF2vec Sec. 3.1:",
        "a BFS predecessor tree per root, one walk per leaf-to-root path).",
        "Row: root, walk index, len, then the 2*3+1 tokens. Written by tests/golden/make_golden.py",
        "from the CPU oracle.",
    ])
    body = ""
    for r in range(HAND_V):
        for i in range(int(cnt[r])):
            body += f"{r} {i} {int(ln[r, i])} " + " ".join(str(int(x)) for x in tok[r, i]) + "\n"
    return head + body


VOCAB_TRIPLES = [
    ("http://kg.example.org/entity/Q3", "http://kg.example.org/relation/P1", "http://kg.example.org/entity/Q1"),
    ("http://kg.example.org/entity/Q1", "http://kg.example.org/relation/P2", "http://kg.example.org/entity/Q3"),
    ("http://kg.example.org/entity/Q2", "http://kg.example.org/relation/P1", "http://kg.example.org/entity/Q1"),
    ("http://kg.example.org/entity/Q1", "http://kg.example.org/relation/P3", "http://kg.example.org/entity/Q10"),
    ("http://kg.example.org/entity/Q10", "http://kg.example.org/relation/P2", "http://kg.example.org/entity/Q2"),
]


def fixture_vocab() -> str:
    def col(strings):
        data = [x.encode() for x in strings]
        off = np.zeros(len(data) + 1, np.int64)
        off[1:] = np.cumsum([len(d) for d in data])
        return np.frombuffer(b"".join(data), np.uint8), off
    S, P, O = zip(*VOCAB_TRIPLES)
    (sc, so), (pc, po), (oc, oo) = col(S), col(P), col(O)
    s, p, o, ne, npred = oracle.build_vocabulary(sc, so, pc, po, oc, oo)
    head = _header([
        "Vocabulary of five IRI triples (gpuRDF2vec Sec. 3.1: entities and predicates are tokenised",
        "to integer ids): ids by first appearance over s0, o0, s1, o1, ... and p0, p1, ....",
        f"Distinct entities {ne}, distinct predicates {npred}.",
        "Row: subject predicate object (strings), then their ids. Written by tests/golden/make_golden.py",
        "from the CPU oracle.",
    ])
    return head + "".join(f"{a} {b} {c} {int(x)} {int(y)} {int(z)}\n" for (a, b, c), x, y, z in zip(VOCAB_TRIPLES, s, p, o))


FIXTURES = {
    "walks_hand_graph.txt": fixture_walks_hand,
    "walks_tiny_uniform_head.txt": fixture_walks_tiny,
    "pairs_hand_graph.txt": fixture_pairs_hand,
    "bfs_hand_graph.txt": fixture_bfs_hand,
    "vocabulary_iri.txt": fixture_vocab,
}


def main() -> None:
    for name, make in FIXTURES.items():
        with open(os.path.join(HERE, name), "w") as f:
            f.write(make())
        print("wrote", name)


if __name__ == "__main__":
    main()
