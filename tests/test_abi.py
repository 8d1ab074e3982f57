"""The C-ABI library loads, exports every function include/rdf2v.h declares, and
rejects bad arguments on the host before touching a GPU (no compute calls here).

Every call below fails host-side validation, which returns before any HIP API
call, so the dummy device pointers are never dereferenced.
"""

import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rdf2v.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rdf2v_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    import paper_2508_01073_amd as pkg
    return pkg._native(), pkg


def test_header_declares_the_calls():
    names = _declared_functions()
    for n in ["rdf2v_build_csr", "rdf2v_build_csr_workspace_size", "rdf2v_random_walks", "rdf2v_build_walk_edges",
              "rdf2v_nonsink_starts", "rdf2v_nonsink_starts_workspace_size", "rdf2v_status_string",
              "rdf2v_skipgram_pairs", "rdf2v_skipgram_pairs_workspace_size", "rdf2v_random_walks_tokens",
              "rdf2v_unique_walks", "rdf2v_unique_walks_workspace_size", "rdf2v_bfs_walks",
              "rdf2v_bfs_walks_workspace_size", "rdf2v_build_vocabulary",
              "rdf2v_build_vocabulary_workspace_size", "rdf2v_walk_edges_recommended",
              "rdf2v_cbow_examples", "rdf2v_cbow_examples_workspace_size", "rdf2v_skipgram_pairs_noalloc"]:
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    so, pkg = lib
    out = subprocess.run(["nm", "-D", "--defined-only", pkg.library_path()], stdout=subprocess.PIPE,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (rdf2v_\w+)", out))
    for name in _declared_functions():
        assert name in exported, name
        assert getattr(so, name) is not None
    # nothing beyond the declared C ABI is exported
    assert exported == set(_declared_functions())


def test_header_compiles_as_c():
    res = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-fsyntax-only", "-x", "c", HEADER],
                         stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert res.returncode == 0, res.stdout


def test_walk_edges_recommendation(lib):
    so, pkg = lib
    # records pay once row_ptr (4 * (V + 1) bytes) outgrows 1.5 MiB
    limit = (3 << 19) // 4 - 1  # largest V whose row_ptr fits
    assert not pkg.rdf2v_walk_edges_recommended(limit, 10**6)
    assert pkg.rdf2v_walk_edges_recommended(limit + 1, 10**6)
    assert pkg.rdf2v_walk_edges_recommended(1_000_000, 20_000_000)
    assert pkg.rdf2v_walk_edges_recommended(50_000_000, 500_000_000)
    assert not pkg.rdf2v_walk_edges_recommended(100_000, 1_000_000)
    assert not pkg.rdf2v_walk_edges_recommended(10_000, 10_000_000)
    assert not pkg.rdf2v_walk_edges_recommended(1_000_000, 0)
    assert not pkg.rdf2v_walk_edges_recommended(-1, 5)
    assert so.rdf2v_walk_edges_recommended(2**31 - 1, 2**31 - 1) == 1


def test_status_strings(lib):
    _, pkg = lib
    assert pkg.rdf2v_status_string(0) == "RDF2V_OK"
    assert pkg.rdf2v_status_string(4) == "RDF2V_ERR_WORKSPACE"
    assert pkg.rdf2v_status_string(99) == "RDF2V_UNKNOWN_STATUS"


def test_workspace_sizes(lib):
    _, pkg = lib
    assert pkg.rdf2v_build_csr_workspace_size(0, 10) == 0
    a = pkg.rdf2v_build_csr_workspace_size(5000, 1000)
    b = pkg.rdf2v_build_csr_workspace_size(20_000_000, 1_000_000)
    assert 0 < a < b and a % 256 == 0 and b % 256 == 0
    # keys x2 + payload = 16 B per triple, plus the radix count table
    assert b >= 16 * 20_000_000
    assert pkg.rdf2v_build_csr_workspace_size(2**31, 10) == 0
    assert pkg.rdf2v_nonsink_starts_workspace_size(0) >= 4


FAKE = ctypes.c_void_p(1 << 40)        # never dereferenced: validation fails first
FAKE8 = ctypes.c_void_p(1 << 40)


def _csr(pkg, V=10, P=3, E=20, row_ptr=FAKE, edges=FAKE8):
    return pkg._CsrStruct(V, P, E, row_ptr, edges)


def _walk(lib, csr, start=FAKE, S=5, wpn=2, depth=4, wb=0, wc=None, tokens=FAKE, lens=FAKE):
    so, pkg = lib
    wc = S * wpn - wb if wc is None else wc
    return so.rdf2v_random_walks(ctypes.byref(csr) if csr is not None else None, start, S, wpn, depth,
                                 42, wb, wc, tokens, lens, None, None)


def test_walk_argument_validation(lib):
    so, pkg = lib
    c = _csr(pkg)
    E_INV, E_BIG = pkg.RDF2V_ERR_INVALID_ARGUMENT, pkg.RDF2V_ERR_TOO_LARGE
    assert _walk(lib, None) == E_INV
    assert _walk(lib, c, depth=65) == E_INV
    assert _walk(lib, c, depth=-1) == E_INV
    assert _walk(lib, c, S=-1) == E_INV
    assert _walk(lib, c, wpn=-2) == E_INV
    assert _walk(lib, c, wb=-1) == E_INV
    assert _walk(lib, c, wb=3, wc=8) == E_INV           # past the end of the corpus
    assert _walk(lib, c, wb=11, wc=0) == E_INV          # begins past the end
    assert _walk(lib, c, start=None) == E_INV
    assert _walk(lib, c, tokens=None) == E_INV
    assert _walk(lib, c, lens=None) == E_INV
    assert _walk(lib, _csr(pkg, row_ptr=None)) == E_INV
    assert _walk(lib, _csr(pkg, edges=ctypes.c_void_p((1 << 40) + 4))) == E_INV   # not 8-byte aligned
    assert _walk(lib, _csr(pkg, V=-1)) == E_INV
    assert _walk(lib, _csr(pkg, E=2**31)) == E_BIG
    assert _walk(lib, _csr(pkg, V=2**30, P=2**30)) == E_BIG
    assert _walk(lib, c, S=2**62, wpn=4, wc=1) == E_BIG
    # nothing to do is not an error and launches nothing
    assert _walk(lib, c, wpn=0) == pkg.RDF2V_OK
    assert _walk(lib, c, wc=0) == pkg.RDF2V_OK
    assert _walk(lib, c, S=0) == pkg.RDF2V_OK


def test_build_argument_validation(lib):
    so, pkg = lib
    f = so.rdf2v_build_csr
    ws = pkg.rdf2v_build_csr_workspace_size(100, 10)
    WS = ctypes.c_void_p(1 << 41)
    assert f(FAKE, FAKE, FAKE, -1, 10, 3, FAKE, FAKE8, WS, ws, None, None) == pkg.RDF2V_ERR_INVALID_ARGUMENT
    assert f(FAKE, FAKE, FAKE, 100, -1, 3, FAKE, FAKE8, WS, ws, None, None) == pkg.RDF2V_ERR_INVALID_ARGUMENT
    assert f(FAKE, FAKE, FAKE, 100, 10, 3, None, FAKE8, WS, ws, None, None) == pkg.RDF2V_ERR_INVALID_ARGUMENT
    assert f(None, FAKE, FAKE, 100, 10, 3, FAKE, FAKE8, WS, ws, None, None) == pkg.RDF2V_ERR_INVALID_ARGUMENT
    assert f(FAKE, FAKE, FAKE, 100, 10, 3, FAKE, ctypes.c_void_p((1 << 40) + 4), WS, ws, None, None) \
        == pkg.RDF2V_ERR_INVALID_ARGUMENT
    assert f(FAKE, FAKE, FAKE, 2**31, 10, 3, FAKE, FAKE8, WS, ws, None, None) == pkg.RDF2V_ERR_TOO_LARGE
    assert f(FAKE, FAKE, FAKE, 100, 2**31 - 2, 3, FAKE, FAKE8, WS, ws, None, None) == pkg.RDF2V_ERR_TOO_LARGE
    assert f(FAKE, FAKE, FAKE, 100, 0, 3, FAKE, FAKE8, WS, ws, None, None) == pkg.RDF2V_ERR_ID_OUT_OF_RANGE
    assert f(FAKE, FAKE, FAKE, 100, 10, 3, FAKE, FAKE8, None, ws, None, None) == pkg.RDF2V_ERR_WORKSPACE
    assert f(FAKE, FAKE, FAKE, 100, 10, 3, FAKE, FAKE8, WS, ws - 1, None, None) == pkg.RDF2V_ERR_WORKSPACE
    assert f(FAKE, FAKE, FAKE, 100, 10, 3, FAKE, FAKE8, ctypes.c_void_p((1 << 41) + 64), ws, None, None) \
        == pkg.RDF2V_ERR_WORKSPACE


def test_walk_edges_argument_validation(lib):
    so, pkg = lib
    f = so.rdf2v_build_walk_edges
    E_INV = pkg.RDF2V_ERR_INVALID_ARGUMENT
    assert f(None, FAKE, None, None) == E_INV
    assert f(ctypes.byref(_csr(pkg, row_ptr=None)), FAKE, None, None) == E_INV
    assert f(ctypes.byref(_csr(pkg)), None, None, None) == E_INV
    assert f(ctypes.byref(_csr(pkg)), ctypes.c_void_p((1 << 40) + 8), None, None) == E_INV  # not 16-aligned
    assert f(ctypes.byref(_csr(pkg, edges=None)), FAKE, None, None) == E_INV
    assert f(ctypes.byref(_csr(pkg, E=2**31)), FAKE, None, None) == pkg.RDF2V_ERR_TOO_LARGE
    assert f(ctypes.byref(_csr(pkg, E=0, edges=None)), None, None, None) == pkg.RDF2V_OK  # nothing to do
    c0 = pkg._CsrStruct(0, 3, 20, FAKE, FAKE8, None)       # edges but no entity to point at
    assert f(ctypes.byref(c0), FAKE, None, None) == pkg.RDF2V_ERR_ID_OUT_OF_RANGE
    # walks reading walk records need them 16-byte aligned
    c = pkg._CsrStruct(10, 3, 20, FAKE, FAKE8, ctypes.c_void_p((1 << 40) + 8))
    assert _walk(lib, c) == E_INV


def test_skipgram_argument_validation(lib):
    so, pkg = lib
    f = so.rdf2v_skipgram_pairs
    need = pkg.rdf2v_skipgram_pairs_workspace_size(100)
    WS = ctypes.c_void_p(1 << 41)
    E_INV = pkg.RDF2V_ERR_INVALID_ARGUMENT
    ok_args = dict(tokens=FAKE, len=FAKE, n=100, width=9, window=5, pairs=FAKE8, cap=10, count=FAKE,
                   ws=WS, wsb=need)

    def call(**kw):
        a = dict(ok_args, **kw)
        return f(a["tokens"], a["len"], a["n"], a["width"], a["window"], a["pairs"], a["cap"], a["count"],
                 a["ws"], a["wsb"], None, None)

    assert call(n=-1) == E_INV
    assert call(window=-1) == E_INV
    assert call(cap=-1) == E_INV
    assert call(width=0) == E_INV
    assert call(width=130) == E_INV
    assert call(count=None) == E_INV
    assert call(tokens=None) == E_INV
    assert call(len=None) == E_INV
    assert call(pairs=None) == E_INV
    assert call(pairs=ctypes.c_void_p((1 << 40) + 4)) == E_INV
    assert call(ws=None) == pkg.RDF2V_ERR_WORKSPACE
    assert call(wsb=need - 1) == pkg.RDF2V_ERR_WORKSPACE
    assert pkg.rdf2v_skipgram_pairs_workspace_size(0) > 0
    assert pkg.rdf2v_skipgram_pairs_workspace_size(10**6) >= 8 * 10**6


def test_skipgram_noalloc_argument_validation(lib):
    # The same host-side checks as rdf2v_skipgram_pairs (no workspace to check), plus the fixed
    # bound on rows per call; every rejection returns before any HIP call.
    so, pkg = lib
    f = so.rdf2v_skipgram_pairs_noalloc
    E_INV = pkg.RDF2V_ERR_INVALID_ARGUMENT
    ok_args = dict(tokens=FAKE, len=FAKE, n=100, width=9, window=5, pairs=FAKE8, cap=10, count=FAKE)

    def call(**kw):
        a = dict(ok_args, **kw)
        return f(a["tokens"], a["len"], a["n"], a["width"], a["window"], a["pairs"], a["cap"], a["count"],
                 None, None)

    assert call(n=-1) == E_INV
    assert call(window=-1) == E_INV
    assert call(cap=-1) == E_INV
    assert call(width=0) == E_INV
    assert call(width=130) == E_INV
    assert call(count=None) == E_INV
    assert call(tokens=None) == E_INV
    assert call(len=None) == E_INV
    assert call(pairs=None) == E_INV
    assert call(pairs=ctypes.c_void_p((1 << 40) + 4)) == E_INV
    assert call(n=pkg.RDF2V_NOALLOC_MAX_WALKS + 1) == pkg.RDF2V_ERR_TOO_LARGE
    assert call(n=1 << 40) == pkg.RDF2V_ERR_TOO_LARGE
    # the library-held scratch holds the workspace of the largest call it takes
    assert pkg.rdf2v_skipgram_pairs_workspace_size(pkg.RDF2V_NOALLOC_MAX_WALKS) <= pkg.RDF2V_NOALLOC_SCRATCH_BYTES
    text = open(HEADER).read()
    assert "#define RDF2V_NOALLOC_MAX_WALKS ((int64_t)1 << 22)" in text
    assert "#define RDF2V_NOALLOC_SCRATCH_BYTES (((size_t)32 << 20) + ((size_t)64 << 10))" in text
    assert pkg.RDF2V_NOALLOC_MAX_WALKS == 1 << 22 and pkg.RDF2V_NOALLOC_SCRATCH_BYTES == (32 << 20) + (64 << 10)


def test_cbow_argument_validation(lib):
    so, pkg = lib
    f = so.rdf2v_cbow_examples
    need = pkg.rdf2v_cbow_examples_workspace_size(100)
    WS = ctypes.c_void_p(1 << 41)
    E_INV = pkg.RDF2V_ERR_INVALID_ARGUMENT
    ok_args = dict(tokens=FAKE, len=FAKE, n=100, width=9, window=5, centers=FAKE, contexts=FAKE8, cap=10,
                   count=FAKE, ws=WS, wsb=need)

    def call(**kw):
        a = dict(ok_args, **kw)
        return f(a["tokens"], a["len"], a["n"], a["width"], a["window"], a["centers"], a["contexts"], a["cap"],
                 a["count"], a["ws"], a["wsb"], None, None)

    assert call(n=-1) == E_INV
    assert call(window=0) == E_INV
    assert call(window=129) == E_INV
    assert call(cap=-1) == E_INV
    assert call(width=0) == E_INV
    assert call(width=130) == E_INV
    assert call(count=None) == E_INV
    assert call(tokens=None) == E_INV
    assert call(len=None) == E_INV
    assert call(centers=None) == E_INV
    assert call(contexts=None) == E_INV
    assert call(contexts=ctypes.c_void_p((1 << 40) + 2)) == E_INV
    assert call(n=2**47) == pkg.RDF2V_ERR_TOO_LARGE
    assert call(ws=None) == pkg.RDF2V_ERR_WORKSPACE
    assert call(wsb=need - 1) == pkg.RDF2V_ERR_WORKSPACE
    assert pkg.rdf2v_cbow_examples_workspace_size(10**6) >= 8 * 10**6
    assert pkg.rdf2v_cbow_examples_workspace_size(2**47) == 0


def test_token_kind_and_unique_validation(lib):
    so, pkg = lib
    c = _csr(pkg)
    f = so.rdf2v_random_walks_tokens
    for kind in (-1, 3, 7):
        assert f(ctypes.byref(c), FAKE, 5, 2, 4, 42, 0, 10, kind, FAKE, FAKE, None, None) == \
            pkg.RDF2V_ERR_INVALID_ARGUMENT
    # a valid kind still goes through the walk argument checks
    assert f(ctypes.byref(c), FAKE, 5, 2, 65, 42, 0, 10, 1, FAKE, FAKE, None, None) == pkg.RDF2V_ERR_INVALID_ARGUMENT
    u = so.rdf2v_unique_walks
    need = pkg.rdf2v_unique_walks_workspace_size(100)
    WS = ctypes.c_void_p(1 << 41)
    E_INV = pkg.RDF2V_ERR_INVALID_ARGUMENT
    assert u(FAKE, FAKE, -1, 5, 9, FAKE, FAKE, FAKE, WS, need, None, None) == E_INV
    assert u(FAKE, FAKE, 100, 0, 9, FAKE, FAKE, FAKE, WS, need, None, None) == E_INV
    assert u(FAKE, FAKE, 100, 5, 0, FAKE, FAKE, FAKE, WS, need, None, None) == E_INV
    assert u(FAKE, FAKE, 100, 5, 9, FAKE, FAKE, None, WS, need, None, None) == E_INV
    assert u(FAKE, FAKE, 100, 5, 9, None, FAKE, FAKE, WS, need, None, None) == E_INV
    assert u(FAKE, FAKE, 100, 5, 9, FAKE, FAKE, FAKE, None, need, None, None) == pkg.RDF2V_ERR_WORKSPACE
    assert u(FAKE, FAKE, 100, 5, 9, FAKE, FAKE, FAKE, WS, need - 1, None, None) == pkg.RDF2V_ERR_WORKSPACE


def test_bfs_walks_validation(lib):
    so, pkg = lib
    c = _csr(pkg)
    f = so.rdf2v_bfs_walks
    need = pkg.rdf2v_bfs_walks_workspace_size(10, 5)
    WS = ctypes.c_void_p(1 << 41)
    E_INV = pkg.RDF2V_ERR_INVALID_ARGUMENT
    assert f(None, FAKE, 5, 3, 4, FAKE, FAKE, FAKE, WS, need, None, None) == E_INV
    assert f(ctypes.byref(c), FAKE, -1, 3, 4, FAKE, FAKE, FAKE, WS, need, None, None) == E_INV
    assert f(ctypes.byref(c), FAKE, 5, 65, 4, FAKE, FAKE, FAKE, WS, need, None, None) == E_INV
    assert f(ctypes.byref(c), FAKE, 5, 3, 0, FAKE, FAKE, FAKE, WS, need, None, None) == E_INV
    assert f(ctypes.byref(c), None, 5, 3, 4, FAKE, FAKE, FAKE, WS, need, None, None) == E_INV
    assert f(ctypes.byref(c), FAKE, 5, 3, 4, FAKE, FAKE, None, WS, need, None, None) == E_INV
    assert f(ctypes.byref(c), FAKE, 5, 3, 4, FAKE, FAKE, FAKE, None, need, None, None) == pkg.RDF2V_ERR_WORKSPACE
    assert f(ctypes.byref(c), FAKE, 5, 3, 4, FAKE, FAKE, FAKE, WS, need - 1, None, None) == pkg.RDF2V_ERR_WORKSPACE
    assert f(ctypes.byref(c), FAKE, 2**40, 64, 4, FAKE, FAKE, FAKE, WS, need, None, None) == pkg.RDF2V_ERR_TOO_LARGE
    assert f(ctypes.byref(c), FAKE, 0, 3, 4, None, None, None, None, 0, None, None) == pkg.RDF2V_OK
    # the workspace is bounded (about 4 GiB) however many roots there are
    assert pkg.rdf2v_bfs_walks_workspace_size(50_000_000, 10**7) <= (1 << 32) + 3 * 10**9


def test_vocabulary_validation(lib):
    so, pkg = lib
    f = so.rdf2v_build_vocabulary
    T, ME, MP = 100, 50, 10
    need = pkg.rdf2v_build_vocabulary_workspace_size(T, ME, MP)
    assert need > 0
    WS = ctypes.c_void_p(1 << 41)
    E_INV = pkg.RDF2V_ERR_INVALID_ARGUMENT
    col = [FAKE, FAKE, 4000]

    def call(cols=None, t=T, me=ME, mp=MP, ids=(FAKE, FAKE, FAKE), counts=FAKE, ws=WS, nbytes=None):
        cols = cols or [col, col, col]
        return f(*cols[0], *cols[1], *cols[2], t, me, mp, *ids, counts, ws, need if nbytes is None else nbytes,
                 None, None)

    assert call(t=-1) == E_INV
    assert call(me=0) == E_INV and call(mp=0) == E_INV
    assert call(t=(1 << 30) + 1) == pkg.RDF2V_ERR_TOO_LARGE
    assert call(me=(1 << 30) + 1) == pkg.RDF2V_ERR_TOO_LARGE
    assert call(counts=None) == E_INV
    assert call(ids=(FAKE, None, FAKE)) == E_INV
    assert call(cols=[col, [FAKE, None, 4000], col]) == E_INV                  # offsets missing
    assert call(cols=[col, col, [None, FAKE, 4000]]) == E_INV                  # chars missing
    assert call(cols=[[ctypes.c_void_p((1 << 40) + 2), FAKE, 4000], col, col]) == E_INV  # chars unaligned
    assert call(cols=[col, [FAKE, FAKE, -1], col]) == E_INV
    assert call(ws=None) == pkg.RDF2V_ERR_WORKSPACE
    assert call(nbytes=need - 1) == pkg.RDF2V_ERR_WORKSPACE
    assert call(ws=ctypes.c_void_p((1 << 41) + 16)) == pkg.RDF2V_ERR_WORKSPACE
    # the tables are sized from the bounds: 2 to 4 slots (128 B + a 4-byte id) per bounded string
    small = pkg.rdf2v_build_vocabulary_workspace_size(10**6, 1000, 10)
    big = pkg.rdf2v_build_vocabulary_workspace_size(10**6, 10**6, 10)
    assert 2 * 132 * (10**6 - 1000) <= big - small <= 4 * 132 * 10**6
    assert pkg.rdf2v_build_vocabulary_workspace_size(-1, 1, 1) == 0


def test_nonsink_argument_validation(lib):
    so, pkg = lib
    c = _csr(pkg)
    need = pkg.rdf2v_nonsink_starts_workspace_size(10)
    f = so.rdf2v_nonsink_starts
    assert f(None, FAKE, FAKE, FAKE, need, None) == pkg.RDF2V_ERR_INVALID_ARGUMENT
    assert f(ctypes.byref(c), FAKE, None, FAKE, need, None) == pkg.RDF2V_ERR_INVALID_ARGUMENT
    assert f(ctypes.byref(c), None, FAKE, FAKE, need, None) == pkg.RDF2V_ERR_INVALID_ARGUMENT
    assert f(ctypes.byref(c), FAKE, FAKE, None, need, None) == pkg.RDF2V_ERR_WORKSPACE
    assert f(ctypes.byref(c), FAKE, FAKE, FAKE, need - 1, None) == pkg.RDF2V_ERR_WORKSPACE
    assert f(ctypes.byref(c), FAKE, FAKE, ctypes.c_void_p((1 << 41) + 4), need, None) == pkg.RDF2V_ERR_WORKSPACE


def test_binding_has_no_cpu_fallback(lib):
    # The product package never imports the oracle and has no CPU path.
    src_dir = os.path.join(ROOT, "paper_2508_01073_amd")
    for dirpath, _, files in os.walk(src_dir):
        for fn in files:
            if fn.endswith((".py", ".hip", ".hpp", ".cpp", ".h")):
                text = open(os.path.join(dirpath, fn)).read()
                assert "import oracle" not in text and "from oracle" not in text, fn
                assert "rdf2v_oracle" not in text and "rdf2v_ref_" not in text, fn


def test_binding_rejects_host_outputs():
    # Caller-supplied outputs and the status word must be device tensors of the right dtype and
    # size: the library writes through raw pointers. (Device-side cases: test_gpu_binding.py.)
    import paper_2508_01073_amd as rd
    import torch
    dev = torch.device("cuda", 0)
    with pytest.raises(TypeError):
        rd._out(torch.zeros(4, dtype=torch.int32), "x", torch.int32, 4, dev)
    with pytest.raises(TypeError):
        rd._status(torch.zeros(1, dtype=torch.int32), dev)
    assert rd._status(None, dev) is None
