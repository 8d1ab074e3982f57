import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU; parity tests proper")
    config.addinivalue_line("markers", "slow: minutes-long case (full-size workloads)")


@pytest.fixture(scope="session")
def rocrand_ref(tmp_path_factory):
    """Callable (mode, records[n,3] uint64) -> uint32 array, backed by rocRAND's
    host-callable Philox4x32-10 compiled with g++ (test-only black box)."""
    src = os.path.join(ROOT, "tests", "pins", "rocrand_philox_ref.cpp")
    inc = "/opt/rocm/include"
    if not os.path.exists(os.path.join(inc, "rocrand", "rocrand_philox4x32_10.h")):
        pytest.skip("rocRAND headers not installed")
    exe = str(tmp_path_factory.mktemp("rocrand") / "rocrand_philox_ref")
    subprocess.run(["g++", "-O1", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I", inc, src, "-o", exe],
                   check=True)

    def run(mode: int, records) -> np.ndarray:
        rec = np.ascontiguousarray(records, dtype=np.uint64).reshape(-1, 3)
        payload = np.array([mode, rec.shape[0]], dtype=np.uint64).tobytes() + rec.tobytes()
        res = subprocess.run([exe], input=payload, stdout=subprocess.PIPE, check=True)
        return np.frombuffer(res.stdout, dtype=np.uint32)

    return run
