"""Host logic of bench.py on the CPU: the useful-byte count behind the roofline figure, the
guard on the committed counter profile, and the one-GPU restriction. No GPU is touched."""

import json
import os
import subprocess
import sys

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_useful_bytes_hand_counted():
    # depth 2 (rows of 5 tokens): a full walk (2 hops), one stopped at a sink after 1 hop,
    # one whose start is a sink (0 hops); 2 start entities read
    lens = torch.tensor([5, 3, 1], dtype=torch.int32)
    ub, hops, tokens = bench.useful_bytes(lens, depth=2, num_start=2)
    assert (hops, tokens) == (3, 9)
    gathered = 16 * 3 + 8 * 2 + 4 * 2  # per hop, per early stop, per start
    written = 3 * (4 * 5 + 4)          # padded rows and lengths
    assert ub == gathered + written


def test_useful_bytes_entity_rows():
    # entity or property rows hold depth + 1 tokens and one token per hop
    lens = torch.tensor([4, 2], dtype=torch.int32)
    ub, hops, tokens = bench.useful_bytes(lens, depth=3, num_start=1, kind=1)
    assert (hops, tokens) == (4, 6)
    assert ub == 16 * 4 + 8 * 1 + 4 * 1 + 2 * (4 * 4 + 4)


def test_traffic_only_for_matching_profile():
    with open(bench.PMC_FILE) as fh:
        pmc = json.load(fh)
    got = bench.traffic_from_profile(pmc["workload"], pmc["num_walks"])
    if pmc["kernel_source_hash"] == bench.kernel_source_hash():
        assert got == pmc["hbm_bytes_per_launch"]
        # the copy calibration: each counter scaled by what it reads for a copy of known size
        assert pmc["fetch_scale"] == pytest.approx(pmc["copy_bytes"] / 1024 / pmc["copy_fetch_size_kib"])
        assert pmc["write_scale"] == pytest.approx(pmc["copy_bytes"] / 1024 / pmc["copy_write_size_kib"])
        expect = (pmc["fetch_size_kib_per_launch"] * pmc["fetch_scale"] +
                  pmc["write_size_kib_per_launch"] * pmc["write_scale"]) * 1024
        assert pmc["hbm_bytes_per_launch"] == pytest.approx(expect)
    else:
        assert got is None  # counters taken from other kernel sources are not reported
    assert bench.traffic_from_profile("uniform_1m", pmc["num_walks"]) is None
    assert bench.traffic_from_profile(pmc["workload"], pmc["num_walks"] + 1) is None


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
    assert res.stdout == ""


def test_cpu_oracle_legs_on_tiny_workload():
    # Each extra leg that ran gets the oracle's rate on a bounded sample beside it.
    import argparse

    import bench
    import oracle
    import synth
    w = synth.WORKLOADS["tiny_uniform"]
    s, p, o = synth.triples(w)
    rp, _ = oracle.build_csr(s, p, o, w.num_entities, w.num_predicates)
    n_start = oracle.nonsink_starts(rp, w.num_entities).shape[0]
    out = {"unique_walks": {}, "bfs_walks": {"depth": 2, "max_walks_per_root": 16},
           "skipgram_pairs": {"window": 2}, "cbow_examples": {"window": 3}, "vocabulary": {}}
    bench.cpu_oracle_legs(out, argparse.Namespace(tokens="triples"), w, s, p, o, n_start, 0.02)
    for leg, unit in [("unique_walks", "walks/s"), ("bfs_walks", "roots/s"), ("skipgram_pairs", "pairs/s"),
                      ("cbow_examples", "examples/s"), ("vocabulary", "triples/s")]:
        c = out[leg]["cpu_oracle"]
        assert c["kind"] == "oracle" and c["cores"] == 1 and c["unit"] == unit and c["value"] > 0, leg
    out = {}
    bench.cpu_oracle_legs(out, argparse.Namespace(tokens="triples"), w, s, p, o, n_start, 0.02)
    assert out == {}


def test_cpu_baseline_pins_one_core_and_restores_affinity():
    # The one-thread oracle leg runs pinned to one host core, the all-core leg on every core the
    # process may use (or the host's OMP_NUM_THREADS budget when smaller), and the process gets
    # its affinity set back afterwards.
    import synth
    w = synth.WORKLOADS["tiny_uniform"]
    s, p, o = synth.triples(w)
    before = os.sched_getaffinity(0)
    out = bench.cpu_baseline(w, s, p, o, 0.05)
    assert os.sched_getaffinity(0) == before
    assert out["cores"] == 1 and out["kind"] == "oracle" and out["value"] > 0
    assert out["pinned_core"] in before and out["nproc"] == len(before)
    assert f"pinned to host core {out['pinned_core']}" in out["sample"]
    budget = os.environ.get("OMP_NUM_THREADS", "")
    expect = min(len(before), int(budget)) if budget.isdigit() and int(budget) > 0 else len(before)
    assert out["all_cores"]["threads"] == expect and out["all_cores"]["nproc"] == len(before)
