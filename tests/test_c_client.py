"""A plain C99 program (tests/c_client/walks_client.c) drives the library through rdf2v.h
alone: HIP runtime calls for device memory, then the CSR build, start set and walks. On the CPU
it must compile and link warning-free as C; on the GPU its output must equal the oracle's."""

import os
import subprocess

import numpy as np
import pytest

import oracle
import paper_2508_01073_amd as rd
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c_client", "walks_client.c")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


@pytest.fixture(scope="module")
def client(tmp_path_factory):
    lib_dir = os.path.dirname(rd.library_path())
    if not os.path.exists(rd.library_path()):
        pytest.fail("librdf2v.so is not built")
    exe = str(tmp_path_factory.mktemp("c_client") / "walks_client")
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), SRC,
           "-L", lib_dir, "-lrdf2v", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           f"-Wl,-rpath,{lib_dir}", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-o", exe]
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert res.returncode == 0, res.stdout
    return exe


def test_client_builds_as_c(client):
    assert os.access(client, os.X_OK)


def _run(client, tmp_path, s, p, o, V, P, wpn, depth, seed):
    inp, out = tmp_path / "in.bin", tmp_path / "out.bin"
    head = np.array([s.shape[0]], np.int64).tobytes() + np.array([V, P, wpn, depth], np.int32).tobytes()
    head += np.array([seed], np.uint64).tobytes()
    inp.write_bytes(head + s.astype(np.int32).tobytes() + p.astype(np.int32).tobytes() +
                    o.astype(np.int32).tobytes())
    res = subprocess.run([client, str(inp), str(out)], stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                         text=True, timeout=120)
    assert res.returncode == 0, res.stdout
    buf = out.read_bytes()
    num_start, num_walks = np.frombuffer(buf[:16], np.int64)
    width = 2 * depth + 1
    pos = 16
    starts = np.frombuffer(buf[pos:pos + 4 * num_start], np.int32)
    pos += 4 * num_start
    tokens = np.frombuffer(buf[pos:pos + 4 * num_walks * width], np.int32).reshape(num_walks, width)
    pos += 4 * num_walks * width
    lens = np.frombuffer(buf[pos:pos + 4 * num_walks], np.int32)
    assert pos + 4 * num_walks == len(buf)
    return starts, tokens, lens


@pytest.mark.gpu
@pytest.mark.parametrize("case", ["tiny_uniform", "powerlaw_400k"])
def test_client_matches_oracle(client, tmp_path, case):
    # the second graph is large enough (row_ptr above 1.5 MiB) for the client to take walk records
    if case == "tiny_uniform":
        w = synth.WORKLOADS[case]
        s, p, o = synth.triples(w)
        V, P, wpn, depth = w.num_entities, w.num_predicates, w.walks_per_node, w.depth
    else:
        V, P, wpn, depth = 400_000, 17, 3, 6
        s, p, o = synth.powerlaw_triples(V, P, 1_200_000, seed=9)
    seed = 2**40 + 7
    assert rd.rdf2v_walk_edges_recommended(V, s.shape[0]) == (case != "tiny_uniform")
    starts, tokens, lens = _run(client, tmp_path, s, p, o, V, P, wpn, depth, seed)
    rp, ed = oracle.build_csr(s, p, o, V, P)
    st_ref = oracle.nonsink_starts(rp, V)
    tok_ref, len_ref = oracle.random_walks(rp, ed, V, P, st_ref, wpn, depth, seed)
    assert np.array_equal(starts, st_ref)
    assert np.array_equal(lens, len_ref)
    assert np.array_equal(tokens, tok_ref)
