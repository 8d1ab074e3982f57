"""HBM traffic of the walk kernel from rocprofv3 counters, calibrated on a plain copy.

Measurement infrastructure behind bench.py's `roofline.traffic`, not a test. Run from the
repository root on the GPU:

    python3 tests/perf/walk_kernel_pmc.py --out-dir <dir> [--json profiles/walk_kernel_pmc.json]

Two counter passes of the default workload's bench (one counter block each: FETCH_SIZE, then
WRITE_SIZE), each of which first copies 1 GiB device to device. Each counter is scaled by what it
reads for that copy (1 GiB read and 1 GiB written), and the walk kernel's per-launch readings are
converted to bytes with those factors. The JSON carries a hash of the walk kernel's sources, so
bench.py drops the figure once the kernel changes.
"""

import argparse
import csv
import glob
import json
import os
import re
import statistics
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import bench  # noqa: E402  (no GPU work at import)

COPY_MIB = 1024
BENCH_ARGS = ["--steps", "1", "--warmup", "1", "--no-cpu-baseline", "--copy-probe-mib", str(COPY_MIB)]


def run_pass(counter: str, out_dir: str):
    d = os.path.join(out_dir, counter.lower())
    cmd = ["timeout", "-s", "KILL", "300", "rocprofv3", "--pmc", counter, "--output-format", "csv", "-d", d,
           "-o", "bench", "--", sys.executable, "bench.py", *BENCH_ARGS]
    print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, cwd=ROOT, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stderr[-4000:])
        raise SystemExit(f"rocprofv3 --pmc {counter} failed ({res.returncode})")
    line = [l for l in res.stdout.splitlines() if l.startswith("{")][-1]
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter file under {d}")
    rows = list(csv.DictReader(open(files[0])))
    walk = [float(r["Counter_Value"]) for r in rows
            if "random_walk_kernel" in r["Kernel_Name"] and r["Counter_Name"] == counter]
    copy = [float(r["Counter_Value"]) for r in rows
            if "copyBuffer" in r["Kernel_Name"] and r["Counter_Name"] == counter]
    kernel = next(r["Kernel_Name"] for r in rows if "random_walk_kernel" in r["Kernel_Name"])
    big = [v for v in copy if v > 0.5 * max(copy)]  # the 1 GiB copies, not the small ones
    shown = ["python3" if c == sys.executable else c for c in cmd[4:]]
    return json.loads(line), statistics.mean(walk), statistics.median(big), kernel, " ".join(shown)


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--out-dir", required=True, help="where rocprofv3 writes its results")
    ap.add_argument("--json", default=os.path.join(ROOT, "profiles", "walk_kernel_pmc.json"))
    args = ap.parse_args()
    bench_f, fetch_kib, copy_fetch_kib, kernel, cmd_f = run_pass("FETCH_SIZE", args.out_dir)
    bench_w, write_kib, copy_write_kib, _, cmd_w = run_pass("WRITE_SIZE", args.out_dir)
    copy_kib = COPY_MIB * 1024
    fetch_scale = copy_kib / copy_fetch_kib
    write_scale = copy_kib / copy_write_kib
    out = {
        "workload": bench_f["config"]["workload"],
        "num_walks": bench_f["config"]["num_walks"],
        "kernel": re.search(r"random_walk_kernel<[^>]*>", kernel).group(0),
        "kernel_source_hash": bench.kernel_source_hash(),
        "fetch_size_kib_per_launch": fetch_kib,
        "write_size_kib_per_launch": write_kib,
        "copy_bytes": COPY_MIB << 20,
        "copy_fetch_size_kib": copy_fetch_kib,
        "copy_write_size_kib": copy_write_kib,
        "fetch_scale": fetch_scale,
        "write_scale": write_scale,
        "hbm_bytes_per_launch": (fetch_kib * fetch_scale + write_kib * write_scale) * 1024,
        "commands": [cmd_f, cmd_w],
    }
    assert bench_w["config"]["num_walks"] == out["num_walks"]
    with open(args.json, "w") as fh:
        json.dump(out, fh, indent=1)
        fh.write("\n")
    print(json.dumps(out, indent=1), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
