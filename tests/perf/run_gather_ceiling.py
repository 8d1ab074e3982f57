"""Compile and run tests/perf/gather_ceiling.hip on the local GPU; prints its table.

Measurement infrastructure for the walk kernel's roofline discussion, not a
test: `python tests/perf/run_gather_ceiling.py`.
"""

import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))


def main() -> int:
    src = os.path.join(HERE, "gather_ceiling.hip")
    with tempfile.TemporaryDirectory() as tmp:
        exe = os.path.join(tmp, "gather_ceiling")
        subprocess.run(["hipcc", "-O3", "--offload-arch=gfx950", "-Xclang", "-target-feature",
                        "-Xclang", "-packed-fp32-ops", src, "-o", exe], check=True,
                       stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)
        return subprocess.run([exe]).returncode


if __name__ == "__main__":
    sys.exit(main())
