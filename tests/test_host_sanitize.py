"""The CPU oracle and the input generators under AddressSanitizer and
UndefinedBehaviorSanitizer (g++, host code only): tests/sanitize/host_sanitize.cpp
drives every oracle entry point and generator on small graphs and edge cases; any
out-of-bounds access, leak or undefined behaviour fails the run."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_oracle_and_generators_clean_under_sanitizers(tmp_path):
    if shutil.which("g++") is None:
        pytest.skip("g++ not installed")
    exe = str(tmp_path / "host_sanitize")
    srcs = [os.path.join(ROOT, "tests", "sanitize", "host_sanitize.cpp"),
            os.path.join(ROOT, "oracle", "rdf2v_oracle.cpp"), os.path.join(ROOT, "synth", "synth.cpp")]
    flags = ["-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-Wall", "-Wextra", "-Werror",
             "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
    build = subprocess.run(["g++", *flags, *srcs, "-o", exe, "-lpthread"], stdout=subprocess.PIPE,
                           stderr=subprocess.STDOUT, text=True, timeout=300)
    assert build.returncode == 0, build.stdout
    # verify_asan_link_order=0: a library the environment preloads may come before the ASan runtime
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=300, env=env)
    assert run.returncode == 0, run.stdout[-4000:]
    assert "host sanitize: ok" in run.stdout
