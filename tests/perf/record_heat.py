"""How much of a walk corpus's record reads the hottest few MB of edge records could serve.

Measurement, not a test. Every hop reads one 16-byte walk record of the current entity's row, at
a random slot of that row. A cache can only serve a hop whose record it holds, so the share of
hops that fall on the hottest C bytes of records bounds the hit rate of any cache of C bytes,
for any order of the records; the same share over the hottest 128-byte lines of the records in
CSR order is what that order can give. Run from the repository root (CPU only):

    python3 tests/perf/record_heat.py [--workload powerlaw_20m] [--windows 40] [--per-window 50000]

Walks come from the oracle on evenly spaced windows of walk ids over the whole corpus.
"""

import argparse
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402

RECORD = 16
LINE = 128


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--workload", default="powerlaw_20m")
    ap.add_argument("--windows", type=int, default=40)
    ap.add_argument("--per-window", type=int, default=50_000)
    args = ap.parse_args()
    w = synth.WORKLOADS[args.workload]
    s, p, o = synth.triples(w)
    rp, ed = oracle.build_csr(s, p, o, w.num_entities, w.num_predicates)
    starts = oracle.nonsink_starts(rp, w.num_entities)
    num_walks = starts.size * w.walks_per_node
    visits = np.zeros(w.num_entities, np.float64)
    hops = 0
    for b in np.linspace(0, num_walks - args.per_window, args.windows).astype(np.int64):
        tok, ln = oracle.random_walks(rp, ed, w.num_entities, w.num_predicates, starts, w.walks_per_node,
                                      w.depth, synth.WALK_SEED, int(b), args.per_window)
        for h in range(w.depth):
            m = ln > 2 * h + 1           # walks that make hop h read a record of entity tok[:, 2h]
            visits += np.bincount(tok[m, 2 * h], minlength=w.num_entities)
            hops += int(m.sum())
    deg = np.diff(rp).astype(np.int64)
    heat = np.divide(visits, deg, out=np.zeros_like(visits), where=deg > 0)
    rec = np.repeat(heat, deg)           # per-record read rate, records in CSR order
    best = np.cumsum(np.sort(rec)[::-1]) / rec.sum()
    per_line = LINE // RECORD
    lines = np.add.reduceat(rec, np.arange(0, rec.size, per_line))
    csr_order = np.cumsum(np.sort(lines)[::-1]) / lines.sum()
    print(f"{args.workload}: {hops:,} hops from {args.windows} windows of {args.per_window:,} walks; "
          f"{rec.size * RECORD / 2**20:.0f} MiB of records")
    print("| cache | best record order | CSR order (128-B lines) |")
    print("|---|---|---|")
    for mib in (4, 8, 32, 64, 256):
        r = min(rec.size, mib * 2**20 // RECORD) - 1
        l_ = min(lines.size, mib * 2**20 // LINE) - 1
        print(f"| {mib} MiB | {100 * best[r]:.1f} % | {100 * csr_order[l_]:.1f} % |")
    return 0


if __name__ == "__main__":
    sys.exit(main())
