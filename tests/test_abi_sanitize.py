"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer: the library is
rebuilt with both sanitizers on its host code only (hipcc -Xarch_host; device code unchanged)
and tests/sanitize/abi_sanitize.c, linked against it, calls every workspace-size function at
extreme sizes and every entry point with arguments the host rejects before any HIP call. No GPU
is used; any undefined behaviour in the size arithmetic or the argument checks fails the run."""

import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def test_abi_host_code_clean_under_sanitizers(tmp_path):
    hipcc = os.path.join(ROCM, "bin", "hipcc")
    clang = os.path.join(ROCM, "llvm", "bin", "clang")
    if not (os.path.exists(hipcc) and os.path.exists(clang)):
        pytest.skip("ROCm compilers not installed")
    lib = str(tmp_path / "librdf2v_san.so")
    srcs = sorted(glob.glob(os.path.join(ROOT, "paper_2508_01073_amd", "csrc", "*.hip")))
    build = subprocess.run(
        [hipcc, "-O1", "-g", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-shared", "-fvisibility=hidden",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
         "-Xarch_host", "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"), *srcs, "-o", lib],
        stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=900)
    assert build.returncode == 0, build.stdout[-4000:]
    exe = str(tmp_path / "abi_sanitize")
    link = subprocess.run(
        [clang, "-std=c99", "-Wall", "-Wextra", "-Werror", "-g", "-fsanitize=address,undefined",
         "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"),
         os.path.join(ROOT, "tests", "sanitize", "abi_sanitize.c"), "-L", str(tmp_path), "-lrdf2v_san",
         "-L", os.path.join(ROCM, "lib"), "-lamdhip64", f"-Wl,-rpath,{tmp_path}",
         f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-o", exe],
        stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=300)
    assert link.returncode == 0, link.stdout[-4000:]
    # leaks are not checked: the HIP runtime keeps its own allocations until exit
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=300, env=env)
    assert run.returncode == 0, run.stdout[-4000:]
    assert "abi sanitize: ok" in run.stdout
