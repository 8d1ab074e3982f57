"""Seeded synthetic knowledge graphs and the walk workloads run on them.

Inputs only: this module generates id triples (via ``synth.cpp``) and names the
workload parameters. It holds none of the walk method's arithmetic, so both the
GPU library's tests and the CPU oracle's tests can draw their inputs from it.

The paper's own graphs (igraph Barabasi-Albert / Erdos-Renyi / uniform
attachment, FB15k-237, Wikidata5M; gpuRDF2vec Sec. 5.1, Tab. 2) are not
available; the workloads below stand in for them at the sizes and degree
shapes of that table: a sparse uniform graph for the "Random" graphs, a dense
uniform graph for the dense Erdos-Renyi ones, a power-law graph at Wikidata5M
scale, and a one-GPU share of full Wikidata.
"""

from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.cpp")
_LIB = os.path.join(_HERE, "libsynth.so")

GENERATOR_SEED = 42
WALK_SEED = 42


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    num_entities: int
    num_predicates: int
    num_triples: int
    kind: str                  # "uniform" or "powerlaw"
    depth: int                 # hops per walk
    walks_per_node: int        # walks per start entity
    gamma: float = 2.1         # power-law degree exponent (kind == "powerlaw")
    pred_s: float = 1.5        # predicate rank-frequency exponent (kind == "powerlaw")
    sink_fraction: float = 0.0 # designated sinks (kind == "powerlaw")
    batch_walks: int = 0       # >0: walks are produced in batches of this many

    def describe(self) -> str:
        shape = (f"uniform iid" if self.kind == "uniform" else
                 f"power-law gamma={self.gamma}, predicate Zipf s={self.pred_s}"
                 + (f", {self.sink_fraction:.0%} designated sinks" if self.sink_fraction else ""))
        return (f"{self.name}: V={self.num_entities:,} P={self.num_predicates:,} "
                f"T={self.num_triples:,} ({shape}); depth={self.depth}, "
                f"{self.walks_per_node} walks per non-sink entity")


WORKLOADS = {
    w.name: w for w in [
        Workload("tiny_uniform", 1_000, 20, 5_000, "uniform", depth=4, walks_per_node=10),
        Workload("uniform_1m", 100_000, 50, 1_000_000, "uniform", depth=4, walks_per_node=100),
        Workload("powerlaw_20m", 1_000_000, 200, 20_000_000, "powerlaw", depth=8, walks_per_node=50),
        Workload("dense_10m", 10_000, 100, 10_000_000, "uniform", depth=4, walks_per_node=500),
        Workload("wikidata_share_500m", 50_000_000, 5_000, 500_000_000, "powerlaw", depth=16,
                 walks_per_node=10, sink_fraction=0.10, batch_walks=50_000_000),
    ]
}
WORKLOAD_ORDER = list(WORKLOADS)

_lib = None


def build(force: bool = True) -> str:
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.run(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-pthread", "-Wall",
                        _SRC, "-o", tmp], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build(force=True)
    lib = ctypes.CDLL(_LIB)
    vp = ctypes.c_void_p
    lib.synth_uniform.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                  vp, vp, vp, ctypes.c_int]
    lib.synth_uniform.restype = ctypes.c_int
    lib.synth_powerlaw.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                   ctypes.c_double, ctypes.c_double, ctypes.c_double, vp, vp, vp,
                                   vp, vp, ctypes.c_int]
    lib.synth_powerlaw.restype = ctypes.c_int
    lib.synth_label_column.argtypes = [vp, ctypes.c_int64, vp, ctypes.c_int64, ctypes.c_char_p,
                                       ctypes.c_int32, vp, vp, vp, ctypes.c_int]
    lib.synth_label_column.restype = ctypes.c_int
    _lib = lib
    return lib


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def uniform_triples(num_entities: int, num_predicates: int, num_triples: int,
                    seed: int = GENERATOR_SEED):
    lib = _load()
    s = np.empty(num_triples, dtype=np.int32)
    p = np.empty(num_triples, dtype=np.int32)
    o = np.empty(num_triples, dtype=np.int32)
    rc = lib.synth_uniform(seed, num_triples, num_entities, num_predicates, s.ctypes.data,
                           p.ctypes.data, o.ctypes.data, _threads())
    if rc != 0:
        raise ValueError("synth_uniform: bad arguments")
    return s, p, o


def powerlaw_triples(num_entities: int, num_predicates: int, num_triples: int, gamma: float = 2.1,
                     pred_s: float = 1.5, sink_fraction: float = 0.0, seed: int = GENERATOR_SEED,
                     return_meta: bool = False):
    lib = _load()
    s = np.empty(num_triples, dtype=np.int32)
    p = np.empty(num_triples, dtype=np.int32)
    o = np.empty(num_triples, dtype=np.int32)
    perm = np.empty(num_entities, dtype=np.int32) if return_meta else None
    sinks = np.empty(num_entities, dtype=np.uint8) if return_meta else None
    rc = lib.synth_powerlaw(seed, num_triples, num_entities, num_predicates, gamma, pred_s,
                            sink_fraction, s.ctypes.data, p.ctypes.data, o.ctypes.data,
                            perm.ctypes.data if return_meta else None,
                            sinks.ctypes.data if return_meta else None, _threads())
    if rc != 0:
        raise ValueError("synth_powerlaw: bad arguments")
    if return_meta:
        return s, p, o, perm, sinks.astype(bool)
    return s, p, o


def triples(workload: Workload | str, seed: int = GENERATOR_SEED):
    """(subject, predicate, object) int32 arrays for a named workload."""
    w = WORKLOADS[workload] if isinstance(workload, str) else workload
    if w.kind == "uniform":
        return uniform_triples(w.num_entities, w.num_predicates, w.num_triples, seed)
    return powerlaw_triples(w.num_entities, w.num_predicates, w.num_triples, w.gamma, w.pred_s,
                            w.sink_fraction, seed)


# ----------------------------------------------------------------------------
# String form of a graph: IRI-like labels for entities and predicates
# ----------------------------------------------------------------------------

ENTITY_PREFIX = b"http://kg.example.org/entity/Q"
PREDICATE_PREFIX = b"http://kg.example.org/relation/P"


def label_column(ids, labels, prefix: bytes):
    """String column (chars uint8, offsets int64 with len(ids) + 1 entries): string t is
    ``prefix`` followed by the decimal digits of ``labels[ids[t]]``."""
    lib = _load()
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    labels = np.ascontiguousarray(labels, dtype=np.int64)
    n = ids.shape[0]
    lens = np.empty(n, dtype=np.int64)
    rc = lib.synth_label_column(ids.ctypes.data, n, labels.ctypes.data, labels.shape[0], prefix,
                                len(prefix), lens.ctypes.data, None, None, _threads())
    if rc != 0:
        raise ValueError("label_column: id out of range")
    offsets = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(lens, out=offsets[1:])
    del lens
    chars = np.empty(int(offsets[-1]), dtype=np.uint8)
    lib.synth_label_column(ids.ctypes.data, n, labels.ctypes.data, labels.shape[0], prefix, len(prefix),
                           None, offsets.ctypes.data, chars.ctypes.data, _threads())
    return chars, offsets


def string_triples(s, p, o, num_entities: int, num_predicates: int, seed: int = GENERATOR_SEED):
    """The string form of id triples: every entity and predicate id gets a distinct IRI-like
    label, numbered by a seeded random bijection (so label order is unrelated to id order).
    Returns ((s_chars, s_off), (p_chars, p_off), (o_chars, o_off))."""
    rng = np.random.default_rng([seed, 7])
    ent = rng.permutation(num_entities).astype(np.int64) + 1
    prd = rng.permutation(num_predicates).astype(np.int64) + 1
    return (label_column(s, ent, ENTITY_PREFIX), label_column(p, prd, PREDICATE_PREFIX),
            label_column(o, ent, ENTITY_PREFIX))
