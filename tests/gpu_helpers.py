"""Helpers for the GPU parity tests: run the HIP path through the C ABI and
compare it with the CPU oracle on the same seeded inputs (tolerance 0: all of
this is integer and index work)."""

import sys

import numpy as np
import torch

import oracle
import paper_2508_01073_amd as rd


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def device() -> torch.device:
    if not torch.cuda.is_available():
        raise RuntimeError("GPU parity tests need a HIP device")
    return torch.device("cuda:0")


def to_dev(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(device())


def new_status() -> torch.Tensor:
    return torch.zeros(1, dtype=torch.int32, device=device())


def gpu_csr(s, p, o, V, P, status=None, walk_records=False) -> rd.Csr:
    st = new_status() if status is None else status
    csr = rd.rdf2v_build_csr(to_dev(s), to_dev(p), to_dev(o), V, P, status=st)
    if walk_records:
        csr = rd.rdf2v_build_walk_edges(csr, status=st)
    torch.cuda.synchronize()
    if status is None:
        rd.check_device_status(st, "rdf2v_build_csr")
    return csr


def plain(csr: rd.Csr) -> rd.Csr:
    """The same CSR without walk records (walks read the 8-byte records)."""
    return rd.Csr(csr.row_ptr, csr.edges, csr.num_entities, csr.num_predicates, None)


def assert_walk_records(csr: rd.Csr, rp_ref: np.ndarray, ed_ref: np.ndarray) -> None:
    """walk_edges[k] = (predicate, object, row_ptr[object], row_ptr[object + 1])."""
    we = csr.walk_edges.cpu().numpy().reshape(-1, 4)
    o = ed_ref[:, 1].astype(np.int64)
    expect = np.stack([ed_ref[:, 0], ed_ref[:, 1], rp_ref[o], rp_ref[o + 1]], axis=1)
    assert np.array_equal(we, expect), "walk records differ from (p, o, row_ptr[o], row_ptr[o+1])"


def gpu_walks(csr, starts_dev, wpn, depth, seed, walk_begin=0, walk_count=None, **kw):
    st = new_status()
    tok, ln = rd.rdf2v_random_walks(csr, starts_dev, wpn, depth, seed, walk_begin, walk_count,
                                    status=st, **kw)
    torch.cuda.synchronize()
    rd.check_device_status(st, "rdf2v_random_walks")
    return tok, ln


def assert_csr_equal(csr: rd.Csr, rp_ref: np.ndarray, ed_ref: np.ndarray) -> None:
    rp = csr.row_ptr.cpu().numpy()
    ed = csr.edges.cpu().numpy().reshape(-1, 2)
    assert rp.shape == rp_ref.shape and np.array_equal(rp, rp_ref), "row_ptr differs from the oracle"
    assert ed.shape == ed_ref.shape
    if not np.array_equal(ed, ed_ref):
        bad = np.nonzero(np.any(ed != ed_ref, axis=1))[0]
        raise AssertionError(f"{bad.size} edge records differ; first at {bad[:5].tolist()}")


def assert_rows_equal(tok_gpu: np.ndarray, len_gpu: np.ndarray, tok_ref: np.ndarray,
                      len_ref: np.ndarray, what: str) -> None:
    assert tok_gpu.shape == tok_ref.shape, (what, tok_gpu.shape, tok_ref.shape)
    if not np.array_equal(len_gpu, len_ref):
        bad = np.nonzero(len_gpu != len_ref)[0]
        raise AssertionError(f"{what}: {bad.size} lengths differ; first rows {bad[:5].tolist()}")
    if not np.array_equal(tok_gpu, tok_ref):
        bad = np.nonzero(np.any(tok_gpu != tok_ref, axis=1))[0]
        r = bad[0]
        raise AssertionError(f"{what}: {bad.size} rows differ; row {r}: gpu {tok_gpu[r].tolist()} "
                             f"oracle {tok_ref[r].tolist()}")


def compare_windows(csr, rp, ed, V, P, starts_np, wpn, depth, seed, tok_dev, len_dev,
                    windows, walk_base=0) -> int:
    """Compare rows of a device walk batch (covering walks walk_base..) with the
    oracle on each (begin, count) window of global walk ids. Returns rows checked."""
    n = 0
    for b, c in windows:
        r0 = b - walk_base
        tg = tok_dev[r0:r0 + c].cpu().numpy()
        lg = len_dev[r0:r0 + c].cpu().numpy()
        tr, lr = oracle.random_walks(rp, ed, V, P, starts_np, wpn, depth, seed, b, c)
        assert_rows_equal(tg, lg, tr, lr, f"walks [{b}, {b + c})")
        n += c
    return n


def compare_all(rp, ed, V, P, starts_np, wpn, depth, seed, tok_dev, len_dev, walk_base=0,
                piece: int = 1_000_000) -> int:
    """Compare every row of a device walk batch (walks walk_base ..) with the oracle,
    which runs in one thread per host core (at most 16) over disjoint walk ranges
    (each ctypes call runs without the GIL). Returns rows checked."""
    import concurrent.futures
    import os
    tok_h, len_h = tok_dev.cpu().numpy(), len_dev.cpu().numpy()
    n = len_h.shape[0]
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    chunk = (n + threads - 1) // threads

    def first_bad(lo, hi):
        for b in range(lo, hi, piece):
            c = min(piece, hi - b)
            rt, rl = oracle.random_walks(rp, ed, V, P, starts_np, wpn, depth, seed, walk_base + b, c)
            if not (np.array_equal(rl, len_h[b:b + c]) and np.array_equal(rt, tok_h[b:b + c])):
                bad = np.nonzero((rl != len_h[b:b + c]) | np.any(rt != tok_h[b:b + c], axis=1))[0]
                return b + int(bad[0])
        return -1

    with concurrent.futures.ThreadPoolExecutor(max_workers=threads) as pool:
        firsts = list(pool.map(lambda i: first_bad(i * chunk, min(n, (i + 1) * chunk)), range(threads)))
    bad = [x for x in firsts if x >= 0]
    assert not bad, f"walk {walk_base + min(bad)} differs from the oracle"
    return n


def check_walk_properties(tok: torch.Tensor, ln: torch.Tensor, starts_dev: torch.Tensor, wpn: int,
                          V: int, P: int, depth: int, walk_begin: int = 0) -> None:
    """Properties every walk row has at any size, checked on the device."""
    width = 2 * depth + 1
    w = tok.shape[0]
    assert tok.shape == (w, width)
    assert bool(((ln % 2) == 1).all()) and int(ln.min()) >= 1 and int(ln.max()) <= width
    walk_ids = torch.arange(walk_begin, walk_begin + w, device=tok.device, dtype=torch.int64)
    assert torch.equal(tok[:, 0], starts_dev[walk_ids // wpn])
    col = torch.arange(width, device=tok.device, dtype=torch.int32)
    chunk = 1 << 22
    for r0 in range(0, w, chunk):
        t = tok[r0:r0 + chunk]
        valid = col[None, :] < ln[r0:r0 + chunk, None]
        assert bool((t[~valid] == -1).all()), "padding after the walk's end must be -1"
        ent = valid & ((col % 2) == 0)[None, :]
        prd = valid & ((col % 2) == 1)[None, :]
        assert bool(((t[ent] >= 0) & (t[ent] < V)).all()), "entity token out of range"
        assert bool(((t[prd] >= V) & (t[prd] < V + P)).all()), "predicate token out of range"
