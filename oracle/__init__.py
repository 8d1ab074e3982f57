"""CPU oracle for RDF2vec random-walk extraction: ctypes wrapper.

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this module. The GPU library in
``paper_2508_01073_amd`` never imports it and shares no code with it.

The arithmetic lives in ``rdf2v_oracle.cpp`` (plain single-threaded C++17);
this module only compiles it with g++ and marshals numpy arrays. See that file
for what each function computes and which passage of gpuRDF2vec (arXiv
2508.01073, Secs. 2, 3.1, 3.3) and of Salmon et al. (SC'11, Philox) it follows.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "rdf2v_oracle.cpp")
_LIB = os.path.join(_HERE, "librdf2v_oracle.so")

OK = 0
ERR_INVALID_ARGUMENT = 1
ERR_ID_OUT_OF_RANGE = 2
ERR_TOO_LARGE = 3

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle into ``oracle/librdf2v_oracle.so`` with g++."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.run(
            ["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-Wall", "-Wextra", _SRC, "-o", tmp],
            check=True,
        )
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build(force=True)
    lib = ctypes.CDLL(_LIB)
    u32p = ctypes.POINTER(ctypes.c_uint32)
    i32p = ctypes.c_void_p
    lib.rdf2v_ref_philox4x32_10.argtypes = [u32p, u32p, u32p]
    lib.rdf2v_ref_philox4x32_10.restype = None
    lib.rdf2v_ref_philox_word.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64]
    lib.rdf2v_ref_philox_word.restype = ctypes.c_uint32
    lib.rdf2v_ref_edge_index.argtypes = [ctypes.c_uint32, ctypes.c_uint32]
    lib.rdf2v_ref_edge_index.restype = ctypes.c_uint32
    lib.rdf2v_ref_build_csr.argtypes = [i32p, i32p, i32p, ctypes.c_int64, ctypes.c_int32,
                                        ctypes.c_int32, i32p, i32p]
    lib.rdf2v_ref_build_csr.restype = ctypes.c_int
    lib.rdf2v_ref_nonsink_starts.argtypes = [i32p, ctypes.c_int32, i32p]
    lib.rdf2v_ref_nonsink_starts.restype = ctypes.c_int64
    lib.rdf2v_ref_random_walks.argtypes = [i32p, i32p, ctypes.c_int32, ctypes.c_int32,
                                           ctypes.c_int64, i32p, ctypes.c_int64, ctypes.c_int32,
                                           ctypes.c_int32, ctypes.c_uint64, ctypes.c_int64,
                                           ctypes.c_int64, i32p, i32p]
    lib.rdf2v_ref_random_walks.restype = ctypes.c_int
    lib.rdf2v_ref_project_walks.argtypes = [i32p, i32p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                            i32p, i32p]
    lib.rdf2v_ref_project_walks.restype = ctypes.c_int
    lib.rdf2v_ref_unique_walks.argtypes = [i32p, i32p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                           i32p, i32p]
    lib.rdf2v_ref_unique_walks.restype = ctypes.c_int64
    lib.rdf2v_ref_bfs_walks.argtypes = [i32p, i32p, ctypes.c_int32, ctypes.c_int32, i32p, ctypes.c_int64,
                                        ctypes.c_int32, ctypes.c_int32, i32p, i32p, i32p]
    lib.rdf2v_ref_bfs_walks.restype = ctypes.c_int64
    lib.rdf2v_ref_build_vocabulary.argtypes = [i32p] * 6 + [ctypes.c_int64] + [i32p] * 5
    lib.rdf2v_ref_build_vocabulary.restype = ctypes.c_int
    lib.rdf2v_ref_skipgram_pairs.argtypes = [i32p, i32p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                             i32p, ctypes.c_int64]
    lib.rdf2v_ref_skipgram_pairs.restype = ctypes.c_int64
    lib.rdf2v_ref_cbow_examples.argtypes = [i32p, i32p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                            i32p, i32p, ctypes.c_int64]
    lib.rdf2v_ref_cbow_examples.restype = ctypes.c_int64
    _lib = lib
    return lib


class OracleError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: oracle status {status}")
        self.status = status


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data) if a.size else None


def philox4x32_10(counter, key) -> np.ndarray:
    """One Philox4x32-10 block: 4-word counter, 2-word key -> 4 words."""
    lib = _load()
    c = (ctypes.c_uint32 * 4)(*[int(x) & 0xFFFFFFFF for x in counter])
    k = (ctypes.c_uint32 * 2)(*[int(x) & 0xFFFFFFFF for x in key])
    out = (ctypes.c_uint32 * 4)()
    lib.rdf2v_ref_philox4x32_10(c, k, out)
    return np.array(list(out), dtype=np.uint32)


def philox_word(seed: int, walk: int, hop: int) -> int:
    return int(_load().rdf2v_ref_philox_word(seed, walk, hop))


def edge_index(u: int, deg: int) -> int:
    return int(_load().rdf2v_ref_edge_index(u, deg))


def build_csr(subj, pred, obj, num_entities: int, num_predicates: int):
    """(row_ptr[V+1], edges[T,2]) of the subject-indexed CSR, rows in input order."""
    lib = _load()
    s, p, o = _i32(subj), _i32(pred), _i32(obj)
    t = s.shape[0]
    if p.shape[0] != t or o.shape[0] != t:
        raise ValueError("subject, predicate and object arrays differ in length")
    row_ptr = np.empty(num_entities + 1, dtype=np.int32)
    edges = np.empty((t, 2), dtype=np.int32)
    st = lib.rdf2v_ref_build_csr(_ptr(s), _ptr(p), _ptr(o), t, num_entities, num_predicates,
                                 _ptr(row_ptr), _ptr(edges))
    if st != OK:
        raise OracleError(st, "rdf2v_ref_build_csr")
    return row_ptr, edges


def build_csr_status(subj, pred, obj, num_triples: int, num_entities: int, num_predicates: int) -> int:
    """Status code only (argument-validation tests)."""
    lib = _load()
    s, p, o = _i32(subj), _i32(pred), _i32(obj)
    row_ptr = np.empty(max(num_entities, 0) + 1, dtype=np.int32)
    edges = np.empty((max(s.shape[0], 1), 2), dtype=np.int32)
    return int(lib.rdf2v_ref_build_csr(_ptr(s), _ptr(p), _ptr(o), num_triples, num_entities,
                                       num_predicates, _ptr(row_ptr), _ptr(edges)))


def nonsink_starts(row_ptr, num_entities: int) -> np.ndarray:
    lib = _load()
    rp = _i32(row_ptr)
    out = np.empty(max(num_entities, 1), dtype=np.int32)
    n = lib.rdf2v_ref_nonsink_starts(_ptr(rp), num_entities, _ptr(out))
    return out[:n].copy()


def random_walks(row_ptr, edges, num_entities: int, num_predicates: int, start_nodes,
                 walks_per_node: int, depth: int, seed: int, walk_begin: int = 0,
                 walk_count: int | None = None):
    """(tokens[walk_count, 2*depth+1], len[walk_count]) for walks
    [walk_begin, walk_begin + walk_count); walk w starts at start_nodes[w // walks_per_node]."""
    lib = _load()
    rp = _i32(row_ptr)
    ed = _i32(edges).reshape(-1)
    st = _i32(start_nodes)
    num_walks = st.shape[0] * walks_per_node
    if walk_count is None:
        walk_count = num_walks - walk_begin
    width = 2 * depth + 1
    tokens = np.empty((max(walk_count, 0), width), dtype=np.int32)
    lens = np.empty(max(walk_count, 0), dtype=np.int32)
    status = lib.rdf2v_ref_random_walks(
        _ptr(rp), _ptr(ed), num_entities, num_predicates, ed.shape[0] // 2, _ptr(st), st.shape[0],
        walks_per_node, depth, seed, walk_begin, walk_count, _ptr(tokens), _ptr(lens))
    if status != OK:
        raise OracleError(status, "rdf2v_ref_random_walks")
    return tokens, lens


def skipgram_pairs(tokens, lens, window: int) -> np.ndarray:
    """(center, context) pairs [N, 2] of walk rows tokens[W, width] with lens[W] valid tokens:
    every context within `window` positions of its center, in order walk, center, context."""
    lib = _load()
    tok = _i32(tokens)
    ln = _i32(lens)
    w, width = (tok.shape[0], tok.shape[1]) if tok.ndim == 2 else (ln.shape[0], 1)
    n = lib.rdf2v_ref_skipgram_pairs(_ptr(tok), _ptr(ln), w, width, window, None, 0)
    if n < 0:
        raise OracleError(int(-n), "rdf2v_ref_skipgram_pairs")
    pairs = np.empty((n, 2), dtype=np.int32)
    lib.rdf2v_ref_skipgram_pairs(_ptr(tok), _ptr(ln), w, width, window, _ptr(pairs), n)
    return pairs


def cbow_examples(tokens, lens, window: int):
    """CBOW examples of walk rows tokens[W, width] with lens[W] valid tokens: (centers[N],
    contexts[N, 2*window]) for every valid position, contexts ascending, padded with -1."""
    lib = _load()
    tok = _i32(tokens)
    ln = _i32(lens)
    w, width = (tok.shape[0], tok.shape[1]) if tok.ndim == 2 else (ln.shape[0], 1)
    n = lib.rdf2v_ref_cbow_examples(_ptr(tok), _ptr(ln), w, width, window, None, None, 0)
    if n < 0:
        raise OracleError(int(-n), "rdf2v_ref_cbow_examples")
    centers = np.empty(n, dtype=np.int32)
    contexts = np.empty((n, 2 * window), dtype=np.int32)
    lib.rdf2v_ref_cbow_examples(_ptr(tok), _ptr(ln), w, width, window, _ptr(centers), _ptr(contexts), n)
    return centers, contexts


ENTITY_WALKS = 1
PROPERTY_WALKS = 2


def project_walks(tokens, lens, depth: int, kind: int):
    """Entity walks (kind 1: entity tokens) or property walks (kind 2: start entity, then the
    predicate tokens) of triple-based walk rows; rows of depth + 1 tokens padded with -1."""
    lib = _load()
    tok = _i32(tokens)
    ln = _i32(lens)
    n = ln.shape[0]
    out = np.empty((n, depth + 1), dtype=np.int32)
    out_len = np.empty(n, dtype=np.int32)
    st = lib.rdf2v_ref_project_walks(_ptr(tok), _ptr(ln), n, depth, kind, _ptr(out), _ptr(out_len))
    if st != OK:
        raise OracleError(st, "rdf2v_ref_project_walks")
    return out, out_len


def unique_walks(tokens, lens, group_size: int):
    """Duplicate-free walks: within each group of group_size consecutive rows (the walks of one
    start entity), the first occurrence of every distinct walk, in order -> (rows, lens)."""
    lib = _load()
    tok = _i32(tokens)
    ln = _i32(lens)
    n, width = tok.shape
    out = np.empty((n, width), dtype=np.int32)
    out_len = np.empty(n, dtype=np.int32)
    k = lib.rdf2v_ref_unique_walks(_ptr(tok), _ptr(ln), n, group_size, width, _ptr(out), _ptr(out_len))
    if k < 0:
        raise OracleError(int(-k), "rdf2v_ref_unique_walks")
    return out[:k].copy(), out_len[:k].copy()


def bfs_walks(row_ptr, edges, num_entities: int, num_predicates: int, roots, depth: int, max_walks: int):
    """BFS walks: per root, the root-to-leaf paths of its depth-limited queue-order BFS tree
    (first max_walks leaves in the order reached). Returns (tokens[R, max_walks, 2*depth+1],
    len[R, max_walks], counts[R], number of roots with more leaves than max_walks); rows past
    counts[r] are not written (filled with -1 / 0 here)."""
    lib = _load()
    rp = _i32(row_ptr)
    ed = _i32(edges).reshape(-1)
    rt = _i32(roots)
    R = rt.shape[0]
    width = 2 * depth + 1
    tokens = np.full((R, max_walks, width), -1, dtype=np.int32)
    lens = np.zeros((R, max_walks), dtype=np.int32)
    counts = np.zeros(R, dtype=np.int32)
    k = lib.rdf2v_ref_bfs_walks(_ptr(rp), _ptr(ed), num_entities, num_predicates, _ptr(rt), R, depth,
                                max_walks, _ptr(tokens), _ptr(lens), _ptr(counts))
    if k < 0:
        raise OracleError(int(-k), "rdf2v_ref_bfs_walks")
    return tokens, lens, counts, int(k)


def build_vocabulary(subj_chars, subj_off, pred_chars, pred_off, obj_chars, obj_off):
    """String triples (uint8 char buffers + int64 offsets per column) -> (subj_ids, pred_ids,
    obj_ids, num_entities, num_predicates); ids in order of first appearance (entities over
    s0, o0, s1, o1, ...; predicates over p0, p1, ...)."""
    lib = _load()
    cols = [np.ascontiguousarray(a) for a in (subj_chars, subj_off, pred_chars, pred_off, obj_chars, obj_off)]
    for c in cols[1::2]:
        assert c.dtype == np.int64
    T = cols[1].shape[0] - 1
    ids = [np.empty(T, dtype=np.int32) for _ in range(3)]
    ne = np.zeros(1, np.int64)
    npred = np.zeros(1, np.int64)
    ptr = lambda a: ctypes.c_void_p(a.ctypes.data)
    st = lib.rdf2v_ref_build_vocabulary(*[ptr(c) for c in cols], T, *[ptr(i) for i in ids], ptr(ne), ptr(npred))
    if st != OK:
        raise OracleError(st, "rdf2v_ref_build_vocabulary")
    return ids[0], ids[1], ids[2], int(ne[0]), int(npred[0])
