#!/usr/bin/env python3
"""Benchmark: RDF2vec random-walk corpus extraction on one MI355X.

One step is one pass of the whole path over inputs already resident in HBM:
rdf2v_build_csr (triples -> CSR), rdf2v_build_walk_edges (16-byte walk
records, when rdf2v_walk_edges_recommended says they pay for this graph size),
rdf2v_nonsink_starts (start set) and rdf2v_random_walks (every walk of every
start entity, one launch). The default
workload is the power-law graph with 1M entities, 200 predicates and 20M
triples, depth 8, 50 walks per start entity (about 48.9M walks).

Prints ONE JSON line. `value` is valid walk tokens per second over whole steps;
`roofline` rates the walk kernel (the dominant kernel) by its useful bytes per
launch over its average launch time, measured with HIP events on the stream
the kernels run on; `cpu_baseline` times the CPU oracle on a bounded sample.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "walk tokens/sec on 1 MI355X + achieved HBM GB/s fraction of peak"
HBM_PEAK_GBS = 8000.0
PMC_FILE = os.path.join(ROOT, "profiles", "walk_kernel_pmc.json")
WALK_SOURCES = [os.path.join(ROOT, "paper_2508_01073_amd", "csrc", f)
                for f in ("random_walk.hip", "common.hpp", "walk.hpp")]


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in WALK_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def useful_bytes(lens, depth: int, num_start: int, kind: int = 0) -> tuple[int, int, int]:
    """(useful bytes, hops, valid tokens) of one walk launch.

    Gathered: 16 B per hop (the row_ptr pair and one (predicate, object) record),
    8 B more for a walk that stops at a sink (the row_ptr pair that shows it), and
    4 B per start id. Written: the padded token row (4 * width B: width = 2*depth+1
    for triple rows, depth+1 for entity or property rows) and the length (4 B)."""
    import torch
    width = 2 * depth + 1 if kind == 0 else depth + 1
    per_hop = 2 if kind == 0 else 1
    ln = lens.to(torch.int64)
    tokens = int(ln.sum().item())
    walks = int(ln.numel())
    hops = (tokens - walks) // per_hop
    early = int((lens < width).sum().item())
    gathered = 16 * hops + 8 * early + 4 * num_start
    written = walks * (4 * width + 4)
    return gathered + written, hops, tokens


def traffic_from_profile(workload: str, num_walks: int):
    """HBM bytes per walk launch from the committed rocprofv3 --pmc summary, scaled by
    the copy-kernel calibration recorded there; None when absent or taken from other
    kernel sources or another launch size."""
    try:
        with open(PMC_FILE) as fh:
            pmc = json.load(fh)
    except (OSError, ValueError):
        return None
    if (pmc.get("kernel_source_hash") != kernel_source_hash() or pmc.get("num_walks") != num_walks
            or pmc.get("workload") != workload):
        return None
    return pmc.get("hbm_bytes_per_launch")


def host_cores() -> list[int]:
    """The host cores this process may run on (its affinity set: `nproc`)."""
    if hasattr(os, "sched_getaffinity"):
        return sorted(os.sched_getaffinity(0))
    return list(range(os.cpu_count() or 1))


def cpu_baseline(w, s, p, o, target_seconds: float):
    """The CPU oracle, untuned, single-threaded and pinned to one host core, on a bounded
    sample of the workload; then the same oracle function on all host cores."""
    cores = host_cores()
    if not hasattr(os, "sched_setaffinity"):
        return _cpu_baseline(w, s, p, o, target_seconds, None, cores)
    # Pin the calling thread (the oracle runs in it through ctypes) for the one-core leg only.
    before = os.sched_getaffinity(0)
    os.sched_setaffinity(0, {cores[0]})
    try:
        out = _cpu_baseline(w, s, p, o, target_seconds, cores[0], cores)
    finally:
        os.sched_setaffinity(0, before)
    return out


def _cpu_baseline(w, s, p, o, target_seconds: float, pinned_core, cores):
    import numpy as np
    import oracle
    V, P = w.num_entities, w.num_predicates
    t0 = time.perf_counter()
    rp, ed = oracle.build_csr(s, p, o, V, P)
    t_build = time.perf_counter() - t0
    starts = oracle.nonsink_starts(rp, V)
    num_walks = len(starts) * w.walks_per_node
    # size the sample from a short probe so the whole leg takes about target_seconds
    probe = min(num_walks, 20_000)
    t0 = time.perf_counter()
    oracle.random_walks(rp, ed, V, P, starts, w.walks_per_node, w.depth, 42, 0, probe)
    rate = probe / max(time.perf_counter() - t0, 1e-9)
    sample = int(min(num_walks, max(probe, rate * target_seconds)))
    t0 = time.perf_counter()
    tokens = oracle_walk_tokens(oracle, rp, ed, V, P, starts, w, 0, sample)
    t_walk = time.perf_counter() - t0
    # the CSR build is charged in proportion to the sampled share of the walks
    t_step_share = t_walk + t_build * sample / num_walks
    out = {
        "value": tokens / t_step_share,
        "unit": "tokens/s",
        "cores": 1,
        "kind": "oracle",
        "sample": (f"oracle CSR build over all {w.num_triples:,} triples ({t_build:.2f} s, charged "
                   f"pro rata) + the first {sample:,} of {num_walks:,} walks ({t_walk:.2f} s), "
                   f"single thread pinned to host core {pinned_core} of {len(cores)}"),
        "pinned_core": pinned_core,
        "nproc": len(cores),
        "cpu_model": cpu_model(),
        "cpu_mhz": cpu_mhz(pinned_core),
    }
    # the all-core leg runs unpinned again (the caller restores the affinity set after this
    # function returns, so restore it here for the worker threads first)
    if pinned_core is not None:
        os.sched_setaffinity(0, set(cores))
    out["all_cores"] = cpu_baseline_threads(oracle, rp, ed, V, P, starts, w, rate, target_seconds / 2, cores)
    return out


def oracle_walk_tokens(oracle, rp, ed, V, P, starts, w, lo: int, hi: int, piece: int = 500_000) -> int:
    """Valid tokens of the oracle's walks [lo, hi), produced piece by piece to bound host memory."""
    import numpy as np
    toks = 0
    for b in range(lo, hi, piece):
        _, ln = oracle.random_walks(rp, ed, V, P, starts, w.walks_per_node, w.depth, 42, b, min(piece, hi - b))
        toks += int(ln.astype(np.int64).sum())
    return toks


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_mhz(core: int | None) -> float | None:
    """Current clock of a host core (MHz) as /proc/cpuinfo reports it, or None."""
    try:
        mhz = {}
        proc = None
        for line in open("/proc/cpuinfo"):
            if line.startswith("processor"):
                proc = int(line.split(":", 1)[1])
            elif line.startswith("cpu MHz") and proc is not None:
                mhz[proc] = float(line.split(":", 1)[1])
        if not mhz:
            return None
        return mhz.get(core, next(iter(mhz.values())))
    except (OSError, ValueError):
        return None


def cpu_baseline_threads(oracle, rp, ed, V, P, starts, w, rate_1t: float, seconds: float, cores):
    """The same oracle function in N threads over disjoint walk ranges (each ctypes call runs
    without the GIL), N = the host cores this process may run on (`nproc`), or OMP_NUM_THREADS
    where the host sets a smaller thread budget; walks only, about `seconds` of wall time."""
    import concurrent.futures
    n = len(cores)
    budget = os.environ.get("OMP_NUM_THREADS", "")
    if budget.isdigit() and 0 < int(budget) < n:
        n = int(budget)
    num_walks = len(starts) * w.walks_per_node
    per_thread = int(min(num_walks // n, max(1000, rate_1t * seconds)))

    def run(i):
        return oracle_walk_tokens(oracle, rp, ed, V, P, starts, w, i * per_thread, (i + 1) * per_thread)

    t0 = time.perf_counter()
    with concurrent.futures.ThreadPoolExecutor(max_workers=n) as pool:
        tokens = sum(pool.map(run, range(n)))
    elapsed = time.perf_counter() - t0
    return {"value": tokens / elapsed, "unit": "tokens/s", "threads": n, "nproc": len(cores),
            "sample": f"walks [0, {n * per_thread:,}) in {n} disjoint ranges, {elapsed:.2f} s wall (walks only)"}


def time_cbow(rd, torch, tokens, lens, n_walks, batch_cap, width, window, batch, stream, ev):
    """Time rdf2v_cbow_examples over the walk rows left in the output buffer, in batches of
    `batch` walks into one reused pair of output buffers.

    Algorithmic bytes: each walk row and its length are read once (4 * width + 4 B) and every
    example is written once (a 4-byte center and 2 * window 4-byte contexts)."""
    dev = tokens.device
    rows = min(n_walks, batch_cap)
    batch = min(batch, rows)
    cap = batch * width  # at most one example per token
    centers = torch.empty(cap, dtype=torch.int32, device=dev)
    contexts = torch.empty((cap, 2 * window), dtype=torch.int32, device=dev)
    ws = torch.empty(rd.rdf2v_cbow_examples_workspace_size(batch), dtype=torch.uint8, device=dev)
    count = torch.empty(1, dtype=torch.int64, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    total = 0
    for b0 in range(0, rows, batch):  # warm-up pass that also counts
        c = min(batch, rows - b0)
        rd.rdf2v_cbow_examples(tokens[b0:b0 + c], lens[b0:b0 + c], window, centers=centers, contexts=contexts,
                               count=count, workspace=ws, status=status, stream=stream)
        torch.cuda.synchronize()
        total += int(count.item())
    rd.check_device_status(status, "cbow examples")
    e0, e1 = ev(), ev()
    e0.record(stream)
    for b0 in range(0, rows, batch):
        c = min(batch, rows - b0)
        rd.rdf2v_cbow_examples(tokens[b0:b0 + c], lens[b0:b0 + c], window, centers=centers, contexts=contexts,
                               count=count, workspace=ws, status=status, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    useful = rows * (4 * width + 4) + total * (4 + 8 * window)
    return {
        "window": window, "walks": rows, "examples": total, "batch_walks": batch,
        "ms": ms, "examples_per_s": total / (ms * 1e-3),
        "useful_bytes": useful, "achieved_GBps": useful / (ms * 1e-3) / 1e9,
        "frac_of_hbm_peak": useful / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
    }


def time_pairs(rd, torch, tokens, lens, n_walks, batch_cap, width, window, pair_batch, stream, ev):
    """Time rdf2v_skipgram_pairs over the walk rows left in the output buffer (the whole corpus
    when it was produced in one launch), in batches of `pair_batch` walks.

    Algorithmic bytes: each walk row and its length are read once (4 * width + 4 B) and every
    pair is written once (8 B)."""
    dev = tokens.device
    rows = min(n_walks, batch_cap)
    pair_batch = min(pair_batch, rows)
    # the largest batch bounds the pair count: 2 * window * width pairs per walk at most
    cap = pair_batch * 2 * min(window, width) * width
    pairs = torch.empty((cap, 2), dtype=torch.int32, device=dev)
    ws = torch.empty(rd.rdf2v_skipgram_pairs_workspace_size(pair_batch), dtype=torch.uint8, device=dev)
    count = torch.empty(1, dtype=torch.int64, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    total_pairs = 0
    for b0 in range(0, rows, pair_batch):  # warm-up pass that also counts
        c = min(pair_batch, rows - b0)
        rd.rdf2v_skipgram_pairs(tokens[b0:b0 + c], lens[b0:b0 + c], window, pairs=pairs, count=count,
                                workspace=ws, status=status, stream=stream)
        torch.cuda.synchronize()
        total_pairs += int(count.item())
    rd.check_device_status(status, "skipgram pairs")
    e0, e1 = ev(), ev()
    e0.record(stream)
    for b0 in range(0, rows, pair_batch):
        c = min(pair_batch, rows - b0)
        rd.rdf2v_skipgram_pairs(tokens[b0:b0 + c], lens[b0:b0 + c], window, pairs=pairs, count=count,
                                workspace=ws, status=status, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    useful = rows * (4 * width + 4) + 8 * total_pairs
    return {
        "window": window, "walks": rows, "pairs": total_pairs, "batch_walks": pair_batch,
        "ms": ms, "pairs_per_s": total_pairs / (ms * 1e-3),
        "useful_bytes": useful, "achieved_GBps": useful / (ms * 1e-3) / 1e9,
        "frac_of_hbm_peak": useful / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
    }


def csr_for_bfs(rd, row_ptr, edges, V, P):
    return rd.Csr(row_ptr, edges, V, P)


def time_bfs(rd, torch, csr, roots, depth, max_walks, stream, ev):
    """Time rdf2v_bfs_walks from every start entity. Bytes: the walk rows written (the
    traversal's own reads depend on the trees and are not counted)."""
    dev = roots.device
    R = int(roots.shape[0])
    width = 2 * depth + 1
    tok = torch.empty((R, max_walks, width), dtype=torch.int32, device=dev)
    ln = torch.empty((R, max_walks), dtype=torch.int32, device=dev)
    cnt = torch.empty(R, dtype=torch.int32, device=dev)
    ws = torch.empty(rd.rdf2v_bfs_walks_workspace_size(csr.num_entities, R), dtype=torch.uint8, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    call = lambda: rd.rdf2v_bfs_walks(csr, roots, depth, max_walks, tokens=tok, lens=ln, counts=cnt,
                                      workspace=ws, status=status, stream=stream)
    call()
    torch.cuda.synchronize()
    walks = int(cnt.to(torch.int64).sum().item())
    truncated = bool(int(status.item()) & rd.RDF2V_STATUS_CAPACITY)
    e0, e1 = ev(), ev()
    e0.record(stream)
    for _ in range(3):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / 3
    return {"depth": depth, "roots": R, "max_walks_per_root": max_walks, "walks": walks,
            "some_roots_truncated": truncated, "ms": ms, "roots_per_s": R / (ms * 1e-3),
            "walks_per_s": walks / (ms * 1e-3)}


def time_unique(rd, torch, tokens, lens, n_walks, batch_cap, wpn, stream, ev):
    """Time rdf2v_unique_walks over the walk rows left in the output buffer (groups of
    walks_per_node rows). Algorithmic bytes: rows and lengths read once, kept rows written."""
    dev = tokens.device
    rows = min(n_walks, batch_cap) // wpn * wpn
    tok, ln = tokens[:rows], lens[:rows]
    out_t = torch.empty_like(tok)
    out_l = torch.empty_like(ln)
    count = torch.empty(1, dtype=torch.int64, device=dev)
    ws = torch.empty(rd.rdf2v_unique_walks_workspace_size(rows), dtype=torch.uint8, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    call = lambda: rd.rdf2v_unique_walks(tok, ln, wpn, tokens_out=out_t, lens_out=out_l, count=count,
                                         workspace=ws, status=status, stream=stream, sync=False)
    call()
    torch.cuda.synchronize()
    rd.check_device_status(status, "unique walks")
    kept = int(count.item())
    e0, e1 = ev(), ev()
    e0.record(stream)
    for _ in range(3):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / 3
    width = tok.shape[1]
    useful = rows * (4 * width + 4) + kept * (4 * width + 4)
    return {"walks": rows, "kept": kept, "ms": ms, "walks_per_s": rows / (ms * 1e-3),
            "achieved_GBps": useful / (ms * 1e-3) / 1e9,
            "frac_of_hbm_peak": useful / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}


def time_vocab(rd, torch, synth, w, s, p, o, stream, ev):
    """Time rdf2v_build_vocabulary on the string form of the workload's triples (IRI-like
    labels, a seeded bijection of the ids). Streaming bytes: every string byte and offset
    read once and every id written once (the hash-table probes are not counted)."""
    import numpy as np
    dev = torch.device("cuda:0")
    cols = synth.string_triples(s, p, o, w.num_entities, w.num_predicates)
    dcols = [(torch.from_numpy(c).to(dev), torch.from_numpy(off).to(dev)) for c, off in cols]
    T = int(s.shape[0])
    ids = tuple(torch.empty(T, dtype=torch.int32, device=dev) for _ in range(3))
    counts = torch.empty(2, dtype=torch.int64, device=dev)
    ws = torch.empty(rd.rdf2v_build_vocabulary_workspace_size(T, w.num_entities, w.num_predicates),
                     dtype=torch.uint8, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    call = lambda: rd.rdf2v_build_vocabulary(*dcols, w.num_entities, w.num_predicates, ids=ids, counts=counts,
                                             workspace=ws, status=status, stream=stream)
    call()
    torch.cuda.synchronize()
    rd.check_device_status(status, "vocabulary")
    e0, e1 = ev(), ev()
    e0.record(stream)
    for _ in range(3):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / 3
    chars = sum(int(c.nbytes) for c, _ in cols)
    streamed = chars + 3 * 8 * (T + 1) + 3 * 4 * T
    ne, npred = [int(x) for x in counts.cpu()]
    return {"triples": T, "string_bytes": chars, "distinct_entities": ne, "distinct_predicates": npred,
            "ms": ms, "triples_per_s": T / (ms * 1e-3), "string_GBps": chars / (ms * 1e-3) / 1e9,
            "streamed_GBps": streamed / (ms * 1e-3) / 1e9,
            "frac_of_hbm_peak": streamed / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}


def oracle_sample(run, probe_n: int, max_n: int, seconds: float, max_units: int | None = None):
    """Time `run(n)` -> (units, seconds) on a small probe, then on samples grown at most tenfold
    at a time towards `seconds` of oracle time (at most max_n inputs and, judging by the last
    run, about max_units outputs), until one takes at least half of it (the oracle's cost per
    item grows once its outputs leave the caches). Returns (n, units, seconds) of the last run."""
    n = max(1, min(probe_n, max_n))
    units, dt = run(n)
    while dt < 0.5 * seconds and n < max_n:
        cap = max_n if not max_units or units == 0 else min(max_n, int(max_units * n / units))
        if cap <= n:
            break
        n = min(cap, max(n + 1, int(n * min(10.0, 0.8 * seconds / max(dt, 1e-4)))))
        units, dt = run(n)
    return n, units, dt


def cpu_oracle_legs(out, args, w, s, p, o, n_start: int, seconds: float) -> None:
    """The oracle (untuned, one thread) beside every extra leg that ran, each on a bounded sample
    of the same workload: the duplicate-free walks, BFS walks, skip-gram pairs and CBOW examples
    of the oracle's own walks and CSR, and the vocabulary of a prefix of the string triples."""
    import numpy as np

    import oracle
    import synth
    legs = [k for k in ("unique_walks", "bfs_walks", "skipgram_pairs", "cbow_examples", "vocabulary") if k in out]
    if not legs:
        return
    V, P, d, wpn = w.num_entities, w.num_predicates, w.depth, w.walks_per_node
    rp, ed = oracle.build_csr(s, p, o, V, P)
    starts = oracle.nonsink_starts(rp, V)
    kind = {"triples": 0, "entities": oracle.ENTITY_WALKS, "properties": oracle.PROPERTY_WALKS}[args.tokens]
    n_walks = n_start * wpn

    def walk_rows(n):
        tok, ln = oracle.random_walks(rp, ed, V, P, starts, wpn, d, 42, 0, n)
        return (tok, ln) if kind == 0 else oracle.project_walks(tok, ln, d, kind)

    def timed(fn):
        t0 = time.perf_counter()
        r = fn()
        return r, time.perf_counter() - t0

    def record(leg, unit, what, n, units, dt):
        out[leg]["cpu_oracle"] = {"value": units / dt, "unit": unit, "cores": 1, "kind": "oracle",
                                  "sample": f"{what} ({units:,} {unit[:-2]} in {dt:.2f} s), single thread"}

    if "unique_walks" in out:
        def run(n):
            tok, ln = walk_rows(n)
            _, dt = timed(lambda: oracle.unique_walks(tok, ln, wpn))
            return n, dt
        n, u, dt = oracle_sample(run, 20 * wpn, n_walks // wpn * wpn, seconds)
        record("unique_walks", "walks/s", f"oracle duplicate-free walks of its walks [0, {n:,})", n, u, dt)
    if "bfs_walks" in out:
        bw = out["bfs_walks"]

        def run(n):
            _, dt = timed(lambda: oracle.bfs_walks(rp, ed, V, P, starts[:n], bw["depth"], bw["max_walks_per_root"]))
            return n, dt
        n, u, dt = oracle_sample(run, 200, n_start, seconds)
        record("bfs_walks", "roots/s", f"oracle BFS walks from the first {n:,} start entities", n, u, dt)
    # outputs capped at ~1.6 / 2.6 GB of oracle memory
    for leg, fn, unit, max_units in (("skipgram_pairs", oracle.skipgram_pairs, "pairs/s", 200_000_000),
                                     ("cbow_examples", oracle.cbow_examples, "examples/s", 60_000_000)):
        if leg in out:
            window = out[leg]["window"]

            def run(n, fn=fn, window=window):
                tok, ln = walk_rows(n)
                r, dt = timed(lambda: fn(tok, ln, window))
                return int(r.shape[0] if isinstance(r, np.ndarray) else r[0].shape[0]), dt
            n, u, dt = oracle_sample(run, 20_000, n_walks, seconds, max_units)
            record(leg, unit, f"oracle {leg.replace('_', ' ')} of its walks [0, {n:,}), window {window}",
                   n, u, dt)
    if "vocabulary" in out:
        def run(n):
            cols = synth.string_triples(s[:n], p[:n], o[:n], V, P)
            _, dt = timed(lambda: oracle.build_vocabulary(cols[0][0], cols[0][1], cols[1][0], cols[1][1],
                                                          cols[2][0], cols[2][1]))
            return n, dt
        n, u, dt = oracle_sample(run, 100_000, int(s.shape[0]), seconds)
        record("vocabulary", "triples/s", f"oracle vocabulary of the first {n:,} string triples", n, u, dt)


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="powerlaw_20m")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--walk-records", choices=["auto", "on", "off"], default="auto",
                    help="build 16-byte walk records in the step: as rdf2v_walk_edges_recommended "
                         "advises for the graph size (auto), always, or never")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--leg-cpu-seconds", type=float, default=2.0,
                    help="oracle time per extra leg (pairs, CBOW, BFS, duplicate-free walks, vocabulary)")
    ap.add_argument("--tokens", choices=["triples", "entities", "properties"], default="triples",
                    help="walk rows: entity/predicate triples (default), entity walks or property walks")
    ap.add_argument("--unique-walks", action="store_true",
                    help="also time duplicate-free filtering of the corpus (per start entity)")
    ap.add_argument("--bfs-depth", type=int, default=-1,
                    help="also time BFS walks from every start entity with this depth (-1: off)")
    ap.add_argument("--bfs-max-walks", type=int, default=256)
    ap.add_argument("--pairs-window", type=int, default=0,
                    help="also time skip-gram pair generation over the corpus with this window "
                         "(0: off)")
    ap.add_argument("--pairs-batch-walks", type=int, default=8_000_000)
    ap.add_argument("--cbow-window", type=int, default=0,
                    help="after the timed steps, also time rdf2v_cbow_examples over the corpus with this window")
    ap.add_argument("--vocab", action="store_true",
                    help="also time the vocabulary (string triples -> ids) on IRI-like labels of "
                         "the workload's triples")
    ap.add_argument("--copy-probe-mib", type=int, default=1024,
                    help="size of the plain device copy timed first (bandwidth reference, "
                         "counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the walks would shard by walk-id range over replicated CSRs with no exchange)",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2508_01073_amd as rd
    import synth

    if not torch.cuda.is_available():
        print("bench.py: no HIP device visible", file=sys.stderr)
        return 1
    dev = torch.device("cuda:0")
    w = synth.WORKLOADS[args.workload]
    V, P, d, wpn = w.num_entities, w.num_predicates, w.depth, w.walks_per_node
    s, p, o = synth.triples(w)
    T = int(s.shape[0])
    subj = torch.from_numpy(s).to(dev)
    pred = torch.from_numpy(p).to(dev)
    obj = torch.from_numpy(o).to(dev)

    # Everything the step writes is allocated once, outside the timed region.
    row_ptr = torch.empty(V + 1, dtype=torch.int32, device=dev)
    edges = torch.empty((T, 2), dtype=torch.int32, device=dev)
    ws_build = torch.empty(max(rd.rdf2v_build_csr_workspace_size(T, V), 1), dtype=torch.uint8, device=dev)
    use_records = {"auto": rd.rdf2v_walk_edges_recommended(V, T), "on": True, "off": False}[args.walk_records]
    walk_edges = torch.empty((T, 4), dtype=torch.int32, device=dev) if use_records else None
    ws_starts = torch.empty(rd.rdf2v_nonsink_starts_workspace_size(V), dtype=torch.uint8, device=dev)
    starts = torch.empty(V, dtype=torch.int32, device=dev)
    count = torch.empty(1, dtype=torch.int64, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    max_walks = V * wpn
    kind = {"triples": rd.RDF2V_TOKENS_TRIPLES, "entities": rd.RDF2V_TOKENS_ENTITIES,
            "properties": rd.RDF2V_TOKENS_PROPERTIES}[args.tokens]
    width = 2 * d + 1 if kind == rd.RDF2V_TOKENS_TRIPLES else d + 1
    # Walks are produced in batches of w.batch_walks into one reused buffer when the
    # workload asks for it (the 500M-triple share); otherwise in one launch.
    batch_cap = min(max_walks, w.batch_walks) if w.batch_walks else max_walks
    tokens = torch.empty((batch_cap, width), dtype=torch.int32, device=dev)
    lens = torch.empty(batch_cap, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    ev = lambda: torch.cuda.Event(enable_timing=True)

    # A plain device-to-device copy: its counter readings calibrate the --pmc runs,
    # and its rate is a measured bandwidth reference next to the 8 TB/s peak.
    copy_mib = args.copy_probe_mib
    a = torch.ones(copy_mib << 18, dtype=torch.int32, device=dev)
    b = torch.empty_like(a)
    b.copy_(a)
    c0, c1 = ev(), ev()
    c0.record(stream)
    for _ in range(3):
        b.copy_(a)
    c1.record(stream)
    torch.cuda.synchronize()
    copy_gbs = 3 * 2 * (copy_mib << 20) / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del a, b

    def step(record, measure=None):
        e0, e1, e2 = ev(), ev(), ev()
        e0.record(stream)
        csr = rd.rdf2v_build_csr(subj, pred, obj, V, P, workspace=ws_build, status=status,
                                 row_ptr=row_ptr, edges=edges, stream=stream)
        if use_records:
            csr = rd.rdf2v_build_walk_edges(csr, out=walk_edges, status=status, stream=stream)
        e1.record(stream)
        st, cnt = rd.rdf2v_nonsink_starts(csr, workspace=ws_starts, starts=starts, count=count,
                                          stream=stream, sync=False)
        n_start = int(cnt.item())
        e2.record(stream)
        n_walks = n_start * wpn
        launches = 0
        batch_events = []  # one event after each walk launch (batches of the 500M-triple share)
        for b0 in range(0, n_walks, batch_cap):
            c = min(batch_cap, n_walks - b0)
            rd.rdf2v_random_walks_tokens(csr, st[:n_start], wpn, d, 42, b0, c, kind, tokens=tokens[:c],
                                         lens=lens[:c], status=status, stream=stream)
            launches += 1
            eb = ev()
            eb.record(stream)
            batch_events.append(eb)
            if measure is not None:
                starts_read = (b0 + c + wpn - 1) // wpn - b0 // wpn
                measure.append(useful_bytes(lens[:c], d, starts_read, kind))
        e3 = batch_events[-1] if batch_events else e2
        record.append((e0, e1, e2, e3, n_start, launches, batch_events))

    warm = []
    for _ in range(max(args.warmup, 1) - 1):
        step(warm)
    per_batch = []
    step(warm, measure=per_batch)  # the last warm-up step also measures the useful bytes
    torch.cuda.synchronize()
    rd.check_device_status(status, "warmup")
    n_start, launches = warm[-1][4], warm[-1][5]
    n_walks = n_start * wpn
    ub = sum(x[0] for x in per_batch)
    hops = sum(x[1] for x in per_batch)
    ntok = sum(x[2] for x in per_batch)

    rec = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(rec)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    rd.check_device_status(status, "timed steps")

    elapsed = t1 - t0
    ms_step = 1e3 * elapsed / args.steps
    # HIP-event times of every timed step: the CSR build (+ walk records), the start set, all
    # walk launches of the step, and the whole step on the GPU; means and medians of these
    build_t = [r[0].elapsed_time(r[1]) for r in rec]
    starts_t = [r[1].elapsed_time(r[2]) for r in rec]
    walk_t = [r[2].elapsed_time(r[3]) for r in rec]
    step_t = [r[0].elapsed_time(r[3]) for r in rec]
    build_ms, starts_ms, walk_ms = float(np.mean(build_t)), float(np.mean(starts_t)), float(np.mean(walk_t))
    walk_med = float(np.median(walk_t))
    # per-batch walk times (one entry per launch of a step), median over the timed steps
    batch_ms = [float(np.median([(r[2] if i == 0 else r[6][i - 1]).elapsed_time(r[6][i]) for r in rec]))
                for i in range(launches)]
    achieved = ub / (walk_ms * 1e-3) / 1e9
    traffic = traffic_from_profile(w.name, n_walks) if launches == 1 else None

    out = {
        "metric": METRIC,
        "value": ntok * args.steps / elapsed,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {
            "workload": w.name, "num_entities": V, "num_predicates": P, "num_triples": T,
            "graph": w.kind, "depth": d, "walks_per_node": wpn, "num_start": n_start,
            "num_walks": n_walks, "seed": 42, "batch_walks": batch_cap if launches > 1 else None,
            "walk_records": use_records,
        },
        "roofline": {
            "kernel": "random_walk_kernel",
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
            "traffic_source": (None if traffic is None else
                               "profiles/walk_kernel_pmc.json: rocprofv3 --pmc FETCH_SIZE and WRITE_SIZE "
                               "of this bench on the same workload, each scaled by its reading for a 1 GiB "
                               "device copy; a committed profile matched by a hash of the walk kernel's "
                               "sources, not read in this run"),
            "achieved_median": ub / (walk_med * 1e-3) / 1e9,
            "frac_median": ub / (walk_med * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "useful_bytes_per_launch": ub if launches == 1 else None,
            "useful_bytes_per_step": ub,
            "launches_per_step": launches,
        },
        "copy_reference_GBps": copy_gbs,
        "walk_kernel_ms": walk_ms,
        "walk_kernel_ms_median": walk_med,
        "walk_kernel_ms_min_max": [float(np.min(walk_t)), float(np.max(walk_t))],
        "walk_batch_ms_median": batch_ms if launches > 1 else None,
        "build_csr_ms": build_ms,
        "build_csr_ms_median": float(np.median(build_t)),
        "nonsink_starts_ms": starts_ms,
        "nonsink_starts_ms_median": float(np.median(starts_t)),
        "step_gpu_ms_median": float(np.median(step_t)),
        "step_gpu_ms_min_max": [float(np.min(step_t)), float(np.max(step_t))],
        "valid_tokens_per_step": ntok,
        "hops_per_step": hops,
        "walk_kernel_tokens_per_s": ntok / (walk_ms * 1e-3),
        "walk_kernel_hops_per_s": hops / (walk_ms * 1e-3),
        "padded_token_slots_per_s": n_walks * width / (walk_ms * 1e-3),
    }
    out["config"]["tokens"] = args.tokens
    if args.unique_walks:
        out["unique_walks"] = time_unique(rd, torch, tokens, lens, n_walks, batch_cap, wpn, stream, ev)
    if args.bfs_depth >= 0:
        out["bfs_walks"] = time_bfs(rd, torch, csr_for_bfs(rd, row_ptr, edges, V, P), starts[:n_start],
                                    args.bfs_depth, args.bfs_max_walks, stream, ev)
    if args.pairs_window > 0:
        out["skipgram_pairs"] = time_pairs(rd, torch, tokens, lens, n_walks, batch_cap, width,
                                           args.pairs_window, args.pairs_batch_walks, stream, ev)
    if args.cbow_window > 0:
        out["cbow_examples"] = time_cbow(rd, torch, tokens, lens, n_walks, batch_cap, width, args.cbow_window,
                                         args.pairs_batch_walks, stream, ev)
    if args.vocab:
        out["vocabulary"] = time_vocab(rd, torch, synth, w, s, p, o, stream, ev)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, s, p, o, args.cpu_seconds)
        cpu_oracle_legs(out, args, w, s, p, o, n_start, args.leg_cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
