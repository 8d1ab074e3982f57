"""MI355X-native RDF2vec random-walk corpus extraction.

Python binding of ``librdf2v.so`` (HIP kernels for gfx950 behind the C ABI in
``include/rdf2v.h``). The functions carry the C names and only marshal
arguments: PyTorch supplies device memory and the stream, every step of the
computation runs in the library's kernels. There is no CPU fallback: every call
raises if the library has not been built (``python -m paper_2508_01073_amd.build``),
and calls fail if no GPU is present.

Walk extraction follows gpuRDF2vec (Boeckling & Paulheim, arXiv 2508.01073):
uniform random walks (Sec. 2) emitted as entity/predicate token rows padded
with -1 (Sec. 3.1), all walks of all start entities launched together
(Sec. 4.1), with walk depth, walks per entity and seed as in Sec. 3.3.
"""

from __future__ import annotations

import contextlib
import ctypes
import os
from dataclasses import dataclass

import torch

__all__ = [
    "Csr", "Rdf2vError", "RDF2V_MAX_DEPTH", "RDF2V_STATUS_ID_OUT_OF_RANGE", "RDF2V_STATUS_BAD_CSR",
    "RDF2V_TOKENS_TRIPLES", "RDF2V_TOKENS_ENTITIES", "RDF2V_TOKENS_PROPERTIES",
    "rdf2v_build_csr_workspace_size", "rdf2v_build_csr", "rdf2v_build_walk_edges",
    "rdf2v_walk_edges_recommended",
    "rdf2v_nonsink_starts_workspace_size",
    "rdf2v_nonsink_starts", "rdf2v_random_walks", "rdf2v_random_walks_tokens",
    "rdf2v_unique_walks_workspace_size", "rdf2v_unique_walks", "rdf2v_bfs_walks_workspace_size",
    "rdf2v_bfs_walks", "rdf2v_skipgram_pairs_workspace_size",
    "rdf2v_skipgram_pairs", "rdf2v_skipgram_pairs_noalloc", "RDF2V_NOALLOC_MAX_WALKS",
    "RDF2V_NOALLOC_SCRATCH_BYTES", "rdf2v_cbow_examples_workspace_size", "rdf2v_cbow_examples",
    "rdf2v_build_vocabulary_workspace_size", "rdf2v_build_vocabulary",
    "rdf2v_status_string", "check_device_status",
    "library_path",
]

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librdf2v.so")

RDF2V_OK = 0
RDF2V_ERR_INVALID_ARGUMENT = 1
RDF2V_ERR_ID_OUT_OF_RANGE = 2
RDF2V_ERR_TOO_LARGE = 3
RDF2V_ERR_WORKSPACE = 4
RDF2V_ERR_HIP = 5
RDF2V_STATUS_ID_OUT_OF_RANGE = 0x1
RDF2V_STATUS_BAD_CSR = 0x2
RDF2V_STATUS_BAD_LENGTH = 0x4
RDF2V_STATUS_CAPACITY = 0x8
RDF2V_MAX_DEPTH = 64
RDF2V_TOKENS_TRIPLES = 0
RDF2V_TOKENS_ENTITIES = 1
RDF2V_TOKENS_PROPERTIES = 2
RDF2V_NOALLOC_MAX_WALKS = 1 << 22
RDF2V_NOALLOC_SCRATCH_BYTES = (32 << 20) + (64 << 10)

_lib = None


def library_path() -> str:
    return _LIB_PATH


class _CsrStruct(ctypes.Structure):
    _fields_ = [("num_entities", ctypes.c_int32), ("num_predicates", ctypes.c_int32),
                ("num_edges", ctypes.c_int64), ("row_ptr", ctypes.c_void_p),
                ("edges", ctypes.c_void_p), ("walk_edges", ctypes.c_void_p)]


def _native():
    """The loaded librdf2v.so; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is not built; run `python -m paper_2508_01073_amd.build`")
    lib = ctypes.CDLL(_LIB_PATH)
    vp, i32, i64, u64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_size_t
    csr_p = ctypes.POINTER(_CsrStruct)
    lib.rdf2v_build_csr_workspace_size.argtypes = [i64, i32]
    lib.rdf2v_build_csr_workspace_size.restype = sz
    lib.rdf2v_build_csr.argtypes = [vp, vp, vp, i64, i32, i32, vp, vp, vp, sz, vp, vp]
    lib.rdf2v_build_csr.restype = ctypes.c_int
    lib.rdf2v_build_walk_edges.argtypes = [csr_p, vp, vp, vp]
    lib.rdf2v_build_walk_edges.restype = ctypes.c_int
    lib.rdf2v_walk_edges_recommended.argtypes = [i32, i64]
    lib.rdf2v_walk_edges_recommended.restype = i32
    lib.rdf2v_nonsink_starts_workspace_size.argtypes = [i32]
    lib.rdf2v_nonsink_starts_workspace_size.restype = sz
    lib.rdf2v_nonsink_starts.argtypes = [csr_p, vp, vp, vp, sz, vp]
    lib.rdf2v_nonsink_starts.restype = ctypes.c_int
    lib.rdf2v_random_walks.argtypes = [csr_p, vp, i64, i32, i32, u64, i64, i64, vp, vp, vp, vp]
    lib.rdf2v_random_walks.restype = ctypes.c_int
    lib.rdf2v_random_walks_tokens.argtypes = [csr_p, vp, i64, i32, i32, u64, i64, i64, i32, vp, vp, vp, vp]
    lib.rdf2v_random_walks_tokens.restype = ctypes.c_int
    lib.rdf2v_unique_walks_workspace_size.argtypes = [i64]
    lib.rdf2v_unique_walks_workspace_size.restype = sz
    lib.rdf2v_unique_walks.argtypes = [vp, vp, i64, i32, i32, vp, vp, vp, vp, sz, vp, vp]
    lib.rdf2v_unique_walks.restype = ctypes.c_int
    lib.rdf2v_bfs_walks_workspace_size.argtypes = [i32, i64]
    lib.rdf2v_bfs_walks_workspace_size.restype = sz
    lib.rdf2v_bfs_walks.argtypes = [csr_p, vp, i64, i32, i32, vp, vp, vp, vp, sz, vp, vp]
    lib.rdf2v_bfs_walks.restype = ctypes.c_int
    lib.rdf2v_skipgram_pairs_workspace_size.argtypes = [i64]
    lib.rdf2v_skipgram_pairs_workspace_size.restype = sz
    lib.rdf2v_skipgram_pairs.argtypes = [vp, vp, i64, i32, i32, vp, i64, vp, vp, sz, vp, vp]
    lib.rdf2v_skipgram_pairs.restype = ctypes.c_int
    lib.rdf2v_skipgram_pairs_noalloc.argtypes = [vp, vp, i64, i32, i32, vp, i64, vp, vp, vp]
    lib.rdf2v_skipgram_pairs_noalloc.restype = ctypes.c_int
    lib.rdf2v_cbow_examples_workspace_size.argtypes = [i64]
    lib.rdf2v_cbow_examples_workspace_size.restype = sz
    lib.rdf2v_cbow_examples.argtypes = [vp, vp, i64, i32, i32, vp, vp, i64, vp, vp, sz, vp, vp]
    lib.rdf2v_cbow_examples.restype = ctypes.c_int
    lib.rdf2v_build_vocabulary_workspace_size.argtypes = [i64, i64, i64]
    lib.rdf2v_build_vocabulary_workspace_size.restype = sz
    lib.rdf2v_build_vocabulary.argtypes = [vp, vp, i64] * 3 + [i64, i64, i64, vp, vp, vp, vp, vp, sz, vp, vp]
    lib.rdf2v_build_vocabulary.restype = ctypes.c_int
    lib.rdf2v_status_string.argtypes = [ctypes.c_int]
    lib.rdf2v_status_string.restype = ctypes.c_char_p
    _lib = lib
    return lib


class Rdf2vError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {rdf2v_status_string(status)} ({status})")
        self.status = status


def rdf2v_status_string(status: int) -> str:
    return _native().rdf2v_status_string(int(status)).decode()


def _check(status: int, where: str) -> None:
    if status != RDF2V_OK:
        raise Rdf2vError(status, where)


def _dev_i32(t: torch.Tensor, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != torch.int32:
        raise TypeError(f"{name} must be int32, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _out(t: torch.Tensor, name: str, dtype: torch.dtype, min_numel: int, dev: torch.device) -> torch.Tensor:
    """A caller-supplied output: on the call's device, of the given dtype, contiguous, and large
    enough (the library writes through the raw pointer, so a short buffer would be overrun)."""
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda" or t.device != dev:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor on {dev}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() < min_numel:
        raise ValueError(f"{name} holds {t.numel()} elements; this call needs {min_numel}")
    return t


def _status(t: torch.Tensor | None, dev: torch.device) -> torch.Tensor | None:
    """The optional device status word (one int32 the kernels OR error bits into)."""
    return None if t is None else _out(t, "status", torch.int32, 1, dev)


def _same_device(dev: torch.device, **tensors) -> None:
    for name, t in tensors.items():
        if t is not None and t.device != dev:
            raise TypeError(f"{name} must be on {dev}, got {t.device}")


def _ws_bytes(t: torch.Tensor | None) -> int:
    """Size in bytes of a caller workspace (any dtype; contiguous device memory)."""
    if t is None:
        return 0
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda" or not t.is_contiguous():
        raise TypeError("workspace must be a contiguous CUDA (HIP) tensor")
    return t.numel() * t.element_size()


def _ptr(t: torch.Tensor | None):
    return None if t is None or t.numel() == 0 else ctypes.c_void_p(t.data_ptr())


@contextlib.contextmanager
def _on_stream(device: torch.device, stream):
    """Makes the caller's stream current for the whole call and yields its handle.

    Everything the binding does for a call then happens on that stream: tensors it allocates
    (outputs, workspaces) belong to it in torch's caching allocator, so a workspace freed when
    the call returns is reused only by work ordered after the call's kernels, and a count read
    back with ``.item()`` waits for those kernels. ``stream`` is None (the device's current
    stream), a ``torch.cuda.Stream`` or a raw hipStream_t handle (int)."""
    if stream is None:
        s = torch.cuda.current_stream(device)
    elif isinstance(stream, torch.cuda.Stream):
        s = stream
    else:
        s = torch.cuda.ExternalStream(int(stream), device=device)
    if s.device != device:
        raise TypeError(f"stream is on {s.device}, the call's tensors on {device}")
    with torch.cuda.stream(s):
        yield ctypes.c_void_p(s.cuda_stream)


@dataclass
class Csr:
    """Subject-indexed CSR in device memory (see ``rdf2v_csr`` in rdf2v.h).

    row_ptr: int32 [num_entities + 1]; edges: int32 [num_edges, 2] = (predicate, object);
    walk_edges (optional): int32 [num_edges, 4] = (predicate, object, row lo, row hi) of the
    object, from rdf2v_build_walk_edges."""
    row_ptr: torch.Tensor
    edges: torch.Tensor
    num_entities: int
    num_predicates: int
    walk_edges: torch.Tensor | None = None

    @property
    def num_edges(self) -> int:
        return int(self.edges.shape[0])

    def _c(self) -> _CsrStruct:
        we = self.walk_edges
        return _CsrStruct(self.num_entities, self.num_predicates, self.num_edges,
                          self.row_ptr.data_ptr(), self.edges.data_ptr() if self.edges.numel() else None,
                          we.data_ptr() if we is not None and we.numel() else None)


def rdf2v_build_csr_workspace_size(num_triples: int, num_entities: int) -> int:
    return int(_native().rdf2v_build_csr_workspace_size(num_triples, num_entities))


def rdf2v_build_csr(subj: torch.Tensor, pred: torch.Tensor, obj: torch.Tensor, num_entities: int,
                    num_predicates: int, *, workspace: torch.Tensor | None = None,
                    status: torch.Tensor | None = None, stream=None,
                    row_ptr: torch.Tensor | None = None, edges: torch.Tensor | None = None) -> Csr:
    """Triples (device int32 [T] each) -> Csr. Rows keep the input order of their triples."""
    _dev_i32(subj, "subj"); _dev_i32(pred, "pred"); _dev_i32(obj, "obj")
    t = subj.shape[0]
    if pred.shape[0] != t or obj.shape[0] != t:
        raise ValueError("subj, pred and obj differ in length")
    dev = subj.device
    with _on_stream(dev, stream) as h:
        _same_device(dev, pred=pred, obj=obj)
        if row_ptr is None:
            row_ptr = torch.empty(num_entities + 1, dtype=torch.int32, device=dev)
        if edges is None:
            edges = torch.empty((t, 2), dtype=torch.int32, device=dev)
        _out(row_ptr, "row_ptr", torch.int32, num_entities + 1, dev)
        _out(edges, "edges", torch.int32, 2 * t, dev)
        _status(status, dev)
        need = rdf2v_build_csr_workspace_size(t, num_entities)
        if workspace is None and need > 0:
            workspace = torch.empty(need, dtype=torch.uint8, device=dev)
        ws_bytes = _ws_bytes(workspace)
        st = _native().rdf2v_build_csr(_ptr(subj), _ptr(pred), _ptr(obj), t, num_entities, num_predicates,
                                  _ptr(row_ptr), _ptr(edges), _ptr(workspace), ws_bytes, _ptr(status),
                                  h)
        _check(st, "rdf2v_build_csr")
        return Csr(row_ptr, edges, num_entities, num_predicates)


def rdf2v_build_walk_edges(csr: Csr, *, out: torch.Tensor | None = None,
                           status: torch.Tensor | None = None, stream=None) -> Csr:
    """Returns the Csr with walk_edges [num_edges, 4] = (predicate, object, row lo, row hi)
    of the object, so the walks read one 16-byte record per hop."""
    dev = csr.row_ptr.device
    with _on_stream(dev, stream) as h:
        if out is None:
            out = torch.empty((csr.num_edges, 4), dtype=torch.int32, device=dev)
        _same_device(dev, edges=csr.edges)
        _out(out, "out", torch.int32, 4 * csr.num_edges, dev)
        _status(status, dev)
        c = csr._c()
        st = _native().rdf2v_build_walk_edges(ctypes.byref(c), _ptr(out), _ptr(status), h)
        _check(st, "rdf2v_build_walk_edges")
        return Csr(csr.row_ptr, csr.edges, csr.num_entities, csr.num_predicates, out)


def rdf2v_walk_edges_recommended(num_entities: int, num_edges: int) -> bool:
    """Whether rdf2v_build_walk_edges' records are expected to speed up the walks on a CSR of
    this size (pure host call; the walks are the same either way)."""
    return bool(_native().rdf2v_walk_edges_recommended(num_entities, num_edges))


def rdf2v_nonsink_starts_workspace_size(num_entities: int) -> int:
    return int(_native().rdf2v_nonsink_starts_workspace_size(num_entities))


def rdf2v_nonsink_starts(csr: Csr, *, workspace: torch.Tensor | None = None, stream=None,
                         starts: torch.Tensor | None = None, count: torch.Tensor | None = None,
                         sync: bool = True):
    """Entities with out-degree >= 1, ascending. With sync=True returns the int32 tensor of
    start ids (one device-to-host read of the count); else (starts, count_device_int64)."""
    dev = csr.row_ptr.device
    with _on_stream(dev, stream) as h:
        if starts is None:
            starts = torch.empty(max(csr.num_entities, 1), dtype=torch.int32, device=dev)
        if count is None:
            count = torch.empty(1, dtype=torch.int64, device=dev)
        if workspace is None:
            workspace = torch.empty(rdf2v_nonsink_starts_workspace_size(csr.num_entities),
                                    dtype=torch.uint8, device=dev)
        _out(starts, "starts", torch.int32, csr.num_entities, dev)
        _out(count, "count", torch.int64, 1, dev)
        c = csr._c()
        st = _native().rdf2v_nonsink_starts(ctypes.byref(c), _ptr(starts), _ptr(count), _ptr(workspace),
                                       _ws_bytes(workspace), h)
        _check(st, "rdf2v_nonsink_starts")
        if not sync:
            return starts, count
        return starts[: int(count.item())]


def rdf2v_random_walks(csr: Csr, start_nodes: torch.Tensor, walks_per_node: int, depth: int,
                       seed: int, walk_begin: int = 0, walk_count: int | None = None, *,
                       tokens: torch.Tensor | None = None, lens: torch.Tensor | None = None,
                       status: torch.Tensor | None = None, stream=None):
    """Walks [walk_begin, walk_begin + walk_count) -> (tokens int32 [walk_count, 2*depth+1],
    lens int32 [walk_count]). Walk w starts at start_nodes[w // walks_per_node]."""
    return _walks(csr, start_nodes, walks_per_node, depth, seed, walk_begin, walk_count,
                  RDF2V_TOKENS_TRIPLES, tokens, lens, status, stream, "rdf2v_random_walks")


def rdf2v_random_walks_tokens(csr: Csr, start_nodes: torch.Tensor, walks_per_node: int, depth: int,
                              seed: int, walk_begin: int = 0, walk_count: int | None = None,
                              token_kind: int = RDF2V_TOKENS_TRIPLES, *,
                              tokens: torch.Tensor | None = None, lens: torch.Tensor | None = None,
                              status: torch.Tensor | None = None, stream=None):
    """Like rdf2v_random_walks with a choice of tokens: RDF2V_TOKENS_TRIPLES (2*depth+1 per row),
    RDF2V_TOKENS_ENTITIES or RDF2V_TOKENS_PROPERTIES (depth+1 per row)."""
    return _walks(csr, start_nodes, walks_per_node, depth, seed, walk_begin, walk_count, token_kind,
                  tokens, lens, status, stream, "rdf2v_random_walks_tokens")


def _walks(csr, start_nodes, walks_per_node, depth, seed, walk_begin, walk_count, token_kind,
           tokens, lens, status, stream, where):
    _dev_i32(start_nodes, "start_nodes")
    dev = start_nodes.device
    with _on_stream(dev, stream) as h:
        num_walks = start_nodes.shape[0] * walks_per_node
        if walk_count is None:
            walk_count = num_walks - walk_begin
        width = 2 * depth + 1 if token_kind == RDF2V_TOKENS_TRIPLES else depth + 1
        if tokens is None:
            tokens = torch.empty((max(walk_count, 0), max(width, 1)), dtype=torch.int32, device=dev)
        if lens is None:
            lens = torch.empty(max(walk_count, 0), dtype=torch.int32, device=dev)
        rows = max(walk_count, 0)
        _out(tokens, "tokens", torch.int32, rows * width, dev)
        _out(lens, "lens", torch.int32, rows, dev)
        _status(status, dev)
        _same_device(dev, row_ptr=csr.row_ptr, edges=csr.edges, walk_edges=csr.walk_edges)
        c = csr._c()
        st = _native().rdf2v_random_walks_tokens(ctypes.byref(c), _ptr(start_nodes), start_nodes.shape[0],
                                                 walks_per_node, depth, ctypes.c_uint64(seed & (2**64 - 1)),
                                                 walk_begin, walk_count, token_kind, _ptr(tokens), _ptr(lens),
                                                 _ptr(status), h)
        _check(st, where)
        return tokens, lens


def rdf2v_unique_walks_workspace_size(num_walks: int) -> int:
    return int(_native().rdf2v_unique_walks_workspace_size(num_walks))


def rdf2v_unique_walks(tokens: torch.Tensor, lens: torch.Tensor, group_size: int, *,
                       tokens_out: torch.Tensor | None = None, lens_out: torch.Tensor | None = None,
                       count: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                       status: torch.Tensor | None = None, stream=None, sync: bool = True):
    """Duplicate-free walks: within each group of group_size consecutive rows keep the first
    occurrence of each distinct walk. With sync=True returns the kept (tokens, lens) (one
    device-to-host read of the count); else (tokens_out, lens_out, count_device_int64)."""
    _dev_i32(tokens, "tokens"); _dev_i32(lens, "lens")
    dev = tokens.device
    with _on_stream(dev, stream) as h:
        n = int(lens.shape[0])
        width = int(tokens.shape[1]) if tokens.dim() == 2 else 1
        if tokens_out is None:
            tokens_out = torch.empty((n, width), dtype=torch.int32, device=dev)
        if lens_out is None:
            lens_out = torch.empty(n, dtype=torch.int32, device=dev)
        if count is None:
            count = torch.empty(1, dtype=torch.int64, device=dev)
        if workspace is None:
            workspace = torch.empty(max(rdf2v_unique_walks_workspace_size(n), 1), dtype=torch.uint8, device=dev)
        _same_device(dev, lens=lens)
        _out(tokens_out, "tokens_out", torch.int32, n * width, dev)
        _out(lens_out, "lens_out", torch.int32, n, dev)
        _out(count, "count", torch.int64, 1, dev)
        _status(status, dev)
        st = _native().rdf2v_unique_walks(_ptr(tokens), _ptr(lens), n, group_size, width, _ptr(tokens_out),
                                          _ptr(lens_out), _ptr(count), _ptr(workspace), _ws_bytes(workspace),
                                          _ptr(status), h)
        _check(st, "rdf2v_unique_walks")
        if not sync:
            return tokens_out, lens_out, count
        k = int(count.item())
        return tokens_out[:k], lens_out[:k]


def rdf2v_bfs_walks_workspace_size(num_entities: int, num_roots: int) -> int:
    return int(_native().rdf2v_bfs_walks_workspace_size(num_entities, num_roots))


def rdf2v_bfs_walks(csr: Csr, roots: torch.Tensor, depth: int, max_walks: int, *,
                    tokens: torch.Tensor | None = None, lens: torch.Tensor | None = None,
                    counts: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                    status: torch.Tensor | None = None, stream=None):
    """BFS walks per root -> (tokens [R, max_walks, 2*depth+1], lens [R, max_walks], counts [R]);
    rows past counts[r] are left as allocated (filled with -1 / 0 when allocated here)."""
    _dev_i32(roots, "roots")
    dev = roots.device
    with _on_stream(dev, stream) as h:
        R = int(roots.shape[0])
        width = 2 * depth + 1
        if tokens is None:
            tokens = torch.full((R, max_walks, width), -1, dtype=torch.int32, device=dev)
        if lens is None:
            lens = torch.zeros((R, max_walks), dtype=torch.int32, device=dev)
        if counts is None:
            counts = torch.empty(R, dtype=torch.int32, device=dev)
        if workspace is None:
            workspace = torch.empty(max(rdf2v_bfs_walks_workspace_size(csr.num_entities, R), 1),
                                    dtype=torch.uint8, device=dev)
        _same_device(dev, row_ptr=csr.row_ptr, edges=csr.edges)
        _out(tokens, "tokens", torch.int32, R * max(max_walks, 0) * width, dev)
        _out(lens, "lens", torch.int32, R * max(max_walks, 0), dev)
        _out(counts, "counts", torch.int32, R, dev)
        _status(status, dev)
        c = csr._c()
        st = _native().rdf2v_bfs_walks(ctypes.byref(c), _ptr(roots), R, depth, max_walks, _ptr(tokens), _ptr(lens),
                                       _ptr(counts), _ptr(workspace), _ws_bytes(workspace), _ptr(status),
                                       h)
        _check(st, "rdf2v_bfs_walks")
        return tokens, lens, counts


def rdf2v_skipgram_pairs_workspace_size(num_walks: int) -> int:
    return int(_native().rdf2v_skipgram_pairs_workspace_size(num_walks))


def rdf2v_skipgram_pairs(tokens: torch.Tensor, lens: torch.Tensor, window: int, *,
                         pairs: torch.Tensor | None = None, count: torch.Tensor | None = None,
                         workspace: torch.Tensor | None = None, status: torch.Tensor | None = None,
                         stream=None):
    """Walk rows tokens [W, width] + lens [W] -> (center, context) pairs [N, 2] int32.

    With `pairs` given, writes at most pairs.shape[0] pairs and returns (pairs, count) with the
    device int64 total (no host synchronisation). Without it, a first call counts, the host reads
    the count, and a second call fills a tensor of exactly that size, which is returned."""
    _dev_i32(tokens, "tokens"); _dev_i32(lens, "lens")
    dev = tokens.device
    with _on_stream(dev, stream) as h:
        w = int(lens.shape[0])
        width = int(tokens.shape[1]) if tokens.dim() == 2 else 1
        if workspace is None:
            workspace = torch.empty(max(rdf2v_skipgram_pairs_workspace_size(w), 1), dtype=torch.uint8, device=dev)
        if count is None:
            count = torch.empty(1, dtype=torch.int64, device=dev)
        _same_device(dev, lens=lens)
        _out(count, "count", torch.int64, 1, dev)
        _status(status, dev)

        def call(out, cap):
            st = _native().rdf2v_skipgram_pairs(_ptr(tokens), _ptr(lens), w, width, window, _ptr(out), cap,
                                              _ptr(count), _ptr(workspace), _ws_bytes(workspace), _ptr(status),
                                              h)
            _check(st, "rdf2v_skipgram_pairs")

        if pairs is not None:
            if pairs.dim() != 2 or pairs.shape[1] != 2:
                raise ValueError("pairs must have shape [capacity, 2]")
            _out(pairs, "pairs", torch.int32, 0, dev)
            call(pairs, int(pairs.shape[0]))
            return pairs, count
        call(None, 0)
        n = int(count.item())
        out = torch.empty((n, 2), dtype=torch.int32, device=dev)
        call(out, n)
        return out


def rdf2v_skipgram_pairs_noalloc(tokens: torch.Tensor, lens: torch.Tensor, window: int, *, pairs: torch.Tensor,
                                 count: torch.Tensor, status: torch.Tensor | None = None, stream=None):
    """rdf2v_skipgram_pairs without a workspace, for callers that cannot allocate: the library's
    fixed per-device scratch serves instead, so this binding allocates nothing either. The caller
    supplies `pairs` [capacity, 2] and `count` (device int64 [1]); at most
    RDF2V_NOALLOC_MAX_WALKS rows per call. Calls that overlap on one device race on the shared
    scratch. Returns (pairs, count) without synchronising."""
    _dev_i32(tokens, "tokens"); _dev_i32(lens, "lens")
    dev = tokens.device
    with _on_stream(dev, stream) as h:
        w = int(lens.shape[0])
        width = int(tokens.shape[1]) if tokens.dim() == 2 else 1
        _same_device(dev, lens=lens)
        if pairs.dim() != 2 or pairs.shape[1] != 2:
            raise ValueError("pairs must have shape [capacity, 2]")
        _out(pairs, "pairs", torch.int32, 0, dev)
        _out(count, "count", torch.int64, 1, dev)
        _status(status, dev)
        st = _native().rdf2v_skipgram_pairs_noalloc(_ptr(tokens), _ptr(lens), w, width, window, _ptr(pairs),
                                                    int(pairs.shape[0]), _ptr(count), _ptr(status), h)
        _check(st, "rdf2v_skipgram_pairs_noalloc")
        return pairs, count


def rdf2v_cbow_examples_workspace_size(num_walks: int) -> int:
    return int(_native().rdf2v_cbow_examples_workspace_size(num_walks))


def rdf2v_cbow_examples(tokens: torch.Tensor, lens: torch.Tensor, window: int, *,
                        centers: torch.Tensor | None = None, contexts: torch.Tensor | None = None,
                        count: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                        status: torch.Tensor | None = None, stream=None):
    """Walk rows tokens [W, width] + lens [W] -> CBOW examples: centers [N] int32 and contexts
    [N, 2*window] int32 (ascending, padded with -1), one example per valid token.

    With `centers` and `contexts` given (capacity = their rows), writes at most that many
    examples and returns (centers, contexts, count) with the device int64 total (no host
    synchronisation). Without them, a first call counts, the host reads the count, and a second
    call fills tensors of exactly that size, which are returned as (centers, contexts)."""
    _dev_i32(tokens, "tokens"); _dev_i32(lens, "lens")
    dev = tokens.device
    with _on_stream(dev, stream) as h:
        w = int(lens.shape[0])
        width = int(tokens.shape[1]) if tokens.dim() == 2 else 1
        if workspace is None:
            workspace = torch.empty(max(rdf2v_cbow_examples_workspace_size(w), 1), dtype=torch.uint8, device=dev)
        if count is None:
            count = torch.empty(1, dtype=torch.int64, device=dev)
        _same_device(dev, lens=lens)
        _out(count, "count", torch.int64, 1, dev)
        _status(status, dev)

        def call(c, x, cap):
            st = _native().rdf2v_cbow_examples(_ptr(tokens), _ptr(lens), w, width, window, _ptr(c), _ptr(x), cap,
                                               _ptr(count), _ptr(workspace), _ws_bytes(workspace), _ptr(status),
                                               h)
            _check(st, "rdf2v_cbow_examples")

        if (centers is None) != (contexts is None):
            raise ValueError("give both centers and contexts, or neither")
        if centers is not None:
            cap = int(centers.numel())
            _out(centers, "centers", torch.int32, 0, dev)
            _out(contexts, "contexts", torch.int32, cap * 2 * max(window, 0), dev)
            call(centers, contexts, cap)
            return centers, contexts, count
        call(None, None, 0)
        n = int(count.item())
        c = torch.empty(n, dtype=torch.int32, device=dev)
        x = torch.empty((n, 2 * window), dtype=torch.int32, device=dev)
        call(c, x, n)
        return c, x


def rdf2v_build_vocabulary_workspace_size(num_triples: int, max_entities: int, max_predicates: int) -> int:
    return int(_native().rdf2v_build_vocabulary_workspace_size(num_triples, max_entities, max_predicates))


def _string_column(col, name: str, n: int):
    chars, offsets = col
    for t, dt in ((chars, torch.uint8), (offsets, torch.int64)):
        if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
            raise TypeError(f"{name} must be CUDA (HIP) tensors")
        if t.dtype != dt or not t.is_contiguous():
            raise TypeError(f"{name}: chars must be contiguous uint8 and offsets contiguous int64")
    if offsets.shape[0] != n + 1:
        raise ValueError(f"{name}: offsets must hold num_triples + 1 entries")
    return [_ptr(chars), _ptr(offsets), int(chars.numel())]


def rdf2v_build_vocabulary(subj, pred, obj, max_entities: int, max_predicates: int, *,
                           ids: tuple | None = None, counts: torch.Tensor | None = None,
                           workspace: torch.Tensor | None = None, status: torch.Tensor | None = None,
                           stream=None):
    """String triples -> id triples. subj, pred, obj are (chars uint8, offsets int64) device
    tensor pairs, string t of a column being chars[offsets[t]:offsets[t+1]].

    Returns (subj_ids, pred_ids, obj_ids, counts): int32 [T] each and a device int64 [2] of
    (distinct entities, distinct predicates); no host synchronisation."""
    offsets = subj[1]
    dev = offsets.device
    with _on_stream(dev, stream) as h:
        n = int(offsets.shape[0]) - 1
        args = (_string_column(subj, "subj", n) + _string_column(pred, "pred", n) + _string_column(obj, "obj", n))
        if ids is None:
            ids = tuple(torch.empty(n, dtype=torch.int32, device=dev) for _ in range(3))
        for i, name in zip(ids, ("subj_ids", "pred_ids", "obj_ids")):
            _out(i, name, torch.int32, n, dev)
        if counts is None:
            counts = torch.empty(2, dtype=torch.int64, device=dev)
        _out(counts, "counts", torch.int64, 2, dev)
        _status(status, dev)
        if workspace is None:
            need = rdf2v_build_vocabulary_workspace_size(n, max_entities, max_predicates)
            workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
        st = _native().rdf2v_build_vocabulary(*args, n, max_entities, max_predicates, *[_ptr(i) for i in ids],
                                              _ptr(counts), _ptr(workspace), _ws_bytes(workspace), _ptr(status),
                                              h)
        _check(st, "rdf2v_build_vocabulary")
        return ids[0], ids[1], ids[2], counts


def check_device_status(status: torch.Tensor, where: str = "device", stream=None) -> None:
    """Raise if a device status word (zeroed before the calls) has any bit set. The word is read
    on `stream` (default: the current stream), so pass the stream the calls were made on."""
    with _on_stream(status.device, stream):
        v = int(status.item())
    if v != 0:
        bits = [n for b, n in [(RDF2V_STATUS_ID_OUT_OF_RANGE, "ID_OUT_OF_RANGE"),
                               (RDF2V_STATUS_BAD_CSR, "BAD_CSR"), (RDF2V_STATUS_BAD_LENGTH, "BAD_LENGTH"),
                               (RDF2V_STATUS_CAPACITY, "CAPACITY")] if v & b]
        raise Rdf2vError(RDF2V_ERR_ID_OUT_OF_RANGE, f"{where}: status bits {'|'.join(bits) or v}")
