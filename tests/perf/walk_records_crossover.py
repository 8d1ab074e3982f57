"""Walk-kernel time with and without 16-byte walk records over graph sizes on the local GPU.

Measurement infrastructure behind rdf2v_walk_edges_recommended's threshold, not a test:
`python tests/perf/walk_records_crossover.py`. Uniform and power-law graphs with mean
out-degree 20, depth 8, about 40M walks per launch; prints one markdown table row per graph.
"""

import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import torch  # noqa: E402

import paper_2508_01073_amd as rd  # noqa: E402
import synth  # noqa: E402


def timed(fn, reps=10):
    fn()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps


def main() -> int:
    dev = torch.device("cuda:0")
    print("| graph | V | T | row_ptr MB | walks ms, records | records build ms | walks ms, plain CSR | "
          "recommended |")
    print("|---|---|---|---|---|---|---|---|", flush=True)
    for kind in ("uniform", "powerlaw"):
        for V in (100_000, 200_000, 300_000, 500_000, 750_000, 1_000_000):
            T, P, depth = 20 * V, 50, 8
            gen = synth.uniform_triples if kind == "uniform" else synth.powerlaw_triples
            s, p, o = gen(V, P, T, seed=3)
            t = lambda x: torch.from_numpy(x).to(dev)
            csr = rd.rdf2v_build_csr(t(s), t(p), t(o), V, P)
            starts = rd.rdf2v_nonsink_starts(csr)
            wpn = max(1, 40_000_000 // len(starts))
            n = len(starts) * wpn
            tok = torch.empty((n, 2 * depth + 1), dtype=torch.int32, device=dev)
            ln = torch.empty(n, dtype=torch.int32, device=dev)
            rec = torch.empty((T, 4), dtype=torch.int32, device=dev)
            csr_rec = rd.rdf2v_build_walk_edges(csr, out=rec)
            t_rec = timed(lambda: rd.rdf2v_random_walks(csr_rec, starts, wpn, depth, 42, tokens=tok, lens=ln))
            t_build = timed(lambda: rd.rdf2v_build_walk_edges(csr, out=rec))
            t_plain = timed(lambda: rd.rdf2v_random_walks(csr, starts, wpn, depth, 42, tokens=tok, lens=ln))
            print(f"| {kind} | {V:,} | {T:,} | {4 * (V + 1) / 1e6:.2f} | {t_rec:.3f} | {t_build:.3f} | "
                  f"{t_plain:.3f} | {'yes' if rd.rdf2v_walk_edges_recommended(V, T) else 'no'} |", flush=True)
            del csr, csr_rec, rec, tok, ln
            torch.cuda.empty_cache()
    return 0


if __name__ == "__main__":
    sys.exit(main())
