"""GPU parity on the largest workload: a one-GPU share of Wikidata (50M
entities, 5,000 predicates, 500M power-law triples, 10% designated sinks,
depth 16, 10 walks per start), with the walks produced in 50M-walk batches
into one reused device buffer.

The whole CSR and start set are compared with the oracle; every batch is
checked for the at-any-size properties on the device and then compared
bit-exactly with the oracle over all of its walks (the oracle runs on all
host cores, over disjoint walk ranges; each ctypes call runs without the
GIL), and windows across batch boundaries are recomputed by separate calls.
Then all walks run in one call (13.2G output elements), compared with the oracle
on windows past element 2^31, 2^32 and 2^33 and at the end.
Takes a few minutes, most of it the oracle.
"""

import time

import numpy as np
import pytest
import torch

import oracle
import paper_2508_01073_amd as rd
import synth
from gpu_helpers import (assert_csr_equal, assert_walk_records, check_walk_properties, compare_all,
                         compare_windows, gpu_csr, gpu_walks, say)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


@pytest.mark.timeout(1100)
def test_wikidata_share_batched_parity():
    w = synth.WORKLOADS["wikidata_share_500m"]
    V, P, d, wpn = w.num_entities, w.num_predicates, w.depth, w.walks_per_node
    say(f"[wikidata share] {w.describe()}")
    t0 = time.time()
    s, p, o = synth.triples(w)
    say(f"[wikidata share] generated in {time.time() - t0:.1f}s")
    csr = gpu_csr(s, p, o, V, P, walk_records=True)
    say("[wikidata share] GPU CSR and walk records built")
    t0 = time.time()
    rp, ed = oracle.build_csr(s, p, o, V, P)
    say(f"[wikidata share] oracle CSR in {time.time() - t0:.1f}s")
    del s, p, o
    assert_csr_equal(csr, rp, ed)
    assert_walk_records(csr, rp, ed)
    say("[wikidata share] CSR and walk records bit-exact")
    starts = oracle.nonsink_starts(rp, V)
    starts_dev = rd.rdf2v_nonsink_starts(csr)
    assert np.array_equal(starts_dev.cpu().numpy(), starts)
    num_walks = len(starts) * wpn
    batch = w.batch_walks
    width = 2 * d + 1
    tok_buf = torch.empty((batch, width), dtype=torch.int32, device=starts_dev.device)
    len_buf = torch.empty(batch, dtype=torch.int32, device=starts_dev.device)
    checked, early = 0, 0
    for b0 in range(0, num_walks, batch):
        c = min(batch, num_walks - b0)
        say(f"[wikidata share] batch [{b0}, {b0 + c})")
        tok, ln = gpu_walks(csr, starts_dev, wpn, d, synth.WALK_SEED, b0, c,
                            tokens=tok_buf[:c], lens=len_buf[:c])
        check_walk_properties(tok, ln, starts_dev, wpn, V, P, d, walk_begin=b0)
        early += int((ln < width).sum().item())
        t0 = time.time()
        checked += compare_all(rp, ed, V, P, starts, wpn, d, synth.WALK_SEED, tok, ln, walk_base=b0)
        say(f"[wikidata share]   all {c} walks bit-exact ({time.time() - t0:.1f}s)")
        if b0 > 0:
            # a window across the boundary with the previous batch, as its own call
            tb, lb = gpu_walks(csr, starts_dev, wpn, d, synth.WALK_SEED, b0 - 100, 200)
            assert torch.equal(tb[100:], tok[:100]) and torch.equal(lb[100:], ln[:100])
            checked += compare_windows(csr, rp, ed, V, P, starts, wpn, d, synth.WALK_SEED, tb, lb,
                                       [(b0 - 100, 200)], walk_base=b0 - 100)
    say(f"[wikidata share] {num_walks} walks, {early / num_walks:.1%} stopped early, "
        f"{checked} rows compared bit-exact")
    assert 0.5 < early / num_walks < 0.99

    # The whole corpus in one call: 13.2G output elements, so rows past element 2^31, 2^32 and
    # 2^33 are written through the kernel's 64-bit row offsets; windows there and at the end are
    # compared with the oracle, and the at-any-size properties hold for every row.
    del tok_buf, len_buf, tok, ln
    torch.cuda.empty_cache()
    say("[wikidata share] all walks in one call")
    tok1, ln1 = gpu_walks(csr, starts_dev, wpn, d, synth.WALK_SEED)
    assert tok1.numel() > 2**33
    rows = [(2**31 - 1) // width, 2**31 // width, 2**32 // width, 2**33 // width, num_walks - 1]
    windows = [(max(0, min(r - 100, num_walks - 200)), 200) for r in rows]
    compare_windows(csr, rp, ed, V, P, starts, wpn, d, synth.WALK_SEED, tok1, ln1, windows)
    check_walk_properties(tok1, ln1, starts_dev, wpn, V, P, d)
    say(f"[wikidata share] one call of {num_walks} walks: windows at elements 2^31, 2^32, 2^33 "
        "and the end bit-exact")
