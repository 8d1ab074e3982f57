"""GPU parity for the walk variants against the oracle, bit-exact: entity walks
and property walks (projections of the triple-based walk on the same random
stream) and duplicate-free walks."""

import numpy as np
import pytest
import torch

import oracle
import paper_2508_01073_amd as rd
import synth
from gpu_helpers import assert_rows_equal, device, gpu_csr, new_status, plain, say, to_dev

pytestmark = pytest.mark.gpu

KINDS = [(rd.RDF2V_TOKENS_ENTITIES, oracle.ENTITY_WALKS), (rd.RDF2V_TOKENS_PROPERTIES, oracle.PROPERTY_WALKS)]


def _walks_kind(csr, starts_dev, wpn, depth, seed, kind, b=0, c=None):
    st = new_status()
    tok, ln = rd.rdf2v_random_walks_tokens(csr, starts_dev, wpn, depth, seed, b, c, kind, status=st)
    torch.cuda.synchronize()
    rd.check_device_status(st, "rdf2v_random_walks_tokens")
    return tok.cpu().numpy(), ln.cpu().numpy()


@pytest.mark.parametrize("depth", [0, 1, 4, 8, 16, 17, 64])
def test_entity_and_property_walks_random_graph(depth):
    say(f"[kinds] random graph depth={depth}")
    V, P, T = 3000, 13, 40_000
    rng = np.random.default_rng(depth)
    s = rng.integers(0, V, T).astype(np.int32)
    p = rng.integers(0, P, T).astype(np.int32)
    o = rng.integers(0, V, T).astype(np.int32)
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P, walk_records=True)
    starts = oracle.nonsink_starts(rp, V)[:2000]
    tr_, lr_ = oracle.random_walks(rp, ed, V, P, starts, 3, depth, 42)
    for kind, okind in KINDS:
        ref_t, ref_l = oracle.project_walks(tr_, lr_, depth, okind)
        for c, what in [(csr, "walk records"), (plain(csr), "plain records")]:
            tok, ln = _walks_kind(c, to_dev(starts), 3, depth, 42, kind)
            assert_rows_equal(tok, ln, ref_t, ref_l, f"kind {kind} depth {depth} {what}")


def test_entity_walks_powerlaw_windows():
    w = synth.WORKLOADS["powerlaw_20m"]
    say(f"[kinds] {w.name}: entity and property walks over sampled windows")
    s, p, o = synth.triples(w)
    V, P = w.num_entities, w.num_predicates
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P, walk_records=True)
    starts = oracle.nonsink_starts(rp, V)
    starts_dev = to_dev(starts)
    n = len(starts) * w.walks_per_node
    for kind, okind in KINDS:
        tok_all, len_all = rd.rdf2v_random_walks_tokens(csr, starts_dev, w.walks_per_node, w.depth,
                                                        synth.WALK_SEED, 0, n, kind)
        torch.cuda.synchronize()
        for b in (0, n // 3, n - 777):
            c = min(2048, n - b)
            tr_, lr_ = oracle.random_walks(rp, ed, V, P, starts, w.walks_per_node, w.depth, synth.WALK_SEED, b, c)
            ref_t, ref_l = oracle.project_walks(tr_, lr_, w.depth, okind)
            assert_rows_equal(tok_all[b:b + c].cpu().numpy(), len_all[b:b + c].cpu().numpy(), ref_t, ref_l,
                              f"kind {kind} window {b}")


def _gpu_unique(tok, ln, group):
    st = new_status()
    t_, l_ = rd.rdf2v_unique_walks(to_dev(tok), to_dev(ln), group, status=st)
    torch.cuda.synchronize()
    rd.check_device_status(st, "rdf2v_unique_walks")
    return t_.cpu().numpy(), l_.cpu().numpy()


@pytest.mark.parametrize("wpn,depth", [(40, 4), (7, 3), (500, 2), (1, 5), (3000, 6)])
def test_unique_walks_small_graph(wpn, depth):
    say(f"[unique] small graph wpn={wpn} depth={depth}")
    rp, ed = oracle.build_csr(np.array([0, 0, 1, 1, 2, 3], np.int32), np.array([0, 1, 0, 0, 1, 1], np.int32),
                              np.array([1, 2, 2, 0, 0, 3], np.int32), 5, 2)
    starts = np.array([0, 1, 2, 0, 4, 3], np.int32)
    tok, ln = oracle.random_walks(rp, ed, 5, 2, starts, wpn, depth, 42)
    ref_t, ref_l = oracle.unique_walks(tok, ln, wpn)
    got_t, got_l = _gpu_unique(tok, ln, wpn)
    assert_rows_equal(got_t, got_l, ref_t, ref_l, f"unique wpn={wpn}")


def test_unique_walks_random_rows_and_ragged_groups():
    say("[unique] random rows, groups straddling blocks, last group short")
    rng = np.random.default_rng(3)
    n, width = 70_001, 9
    ln = rng.choice([1, 3, 5, 7, 9], n).astype(np.int32)
    tok = np.full((n, width), -1, np.int32)
    for r in range(n):
        tok[r, :ln[r]] = rng.integers(0, 3, ln[r])       # tiny alphabet: many duplicates
    for group in (1, 37, 300, 4099):
        ref_t, ref_l = oracle.unique_walks(tok, ln, group)
        got_t, got_l = _gpu_unique(tok, ln, group)
        assert_rows_equal(got_t, got_l, ref_t, ref_l, f"group {group}")


@pytest.mark.parametrize("width,group", [(9, 1), (17, 50), (33, 64), (33, 300), (9, 1000), (65, 10), (129, 3),
                                         (5, 1024), (5, 1025)])
def test_unique_walks_row_widths_and_group_sizes(width, group):
    # blocks of whole groups (256 or 1024 threads) where the rows fit the LDS
    # stage, the general path otherwise; both against the oracle
    say(f"[unique] width {width} group {group}")
    rng = np.random.default_rng(width * 7919 + group)
    n = 20_011
    ln = (2 * rng.integers(0, (width + 1) // 2, n) + 1).astype(np.int32)
    tok = np.full((n, width), -1, np.int32)
    for r in range(n):
        tok[r, :ln[r]] = rng.integers(0, 2, ln[r])
    ref_t, ref_l = oracle.unique_walks(tok, ln, group)
    got_t, got_l = _gpu_unique(tok, ln, group)
    assert_rows_equal(got_t, got_l, ref_t, ref_l, f"width {width} group {group}")


def test_unique_walks_tiny_uniform_corpus():
    w = synth.WORKLOADS["tiny_uniform"]
    say("[unique] tiny_uniform corpus")
    s, p, o = synth.triples(w)
    V, P = w.num_entities, w.num_predicates
    rp, ed = oracle.build_csr(s, p, o, V, P)
    starts = oracle.nonsink_starts(rp, V)
    tok, ln = oracle.random_walks(rp, ed, V, P, starts, w.walks_per_node, w.depth, synth.WALK_SEED)
    ref_t, ref_l = oracle.unique_walks(tok, ln, w.walks_per_node)
    got_t, got_l = _gpu_unique(tok, ln, w.walks_per_node)
    assert_rows_equal(got_t, got_l, ref_t, ref_l, "tiny_uniform unique")
    assert ref_t.shape[0] < tok.shape[0]


def _random_rows(rng, n, width, alphabet):
    ln = (2 * rng.integers(0, (width + 1) // 2, n) + 1).astype(np.int32)
    tok = rng.integers(0, alphabet, (n, width)).astype(np.int32)
    tok[np.arange(width)[None, :] >= ln[:, None]] = -1
    return tok, ln


@pytest.mark.parametrize("n,width,group", [(1_200_007, 9, 7), (17_000_003, 3, 1025)])
def test_unique_walks_many_block_counts(n, width, group):
    # enough blocks (whole-group blocks of <= 256 rows; 4096-row tiles on the
    # general path) that their kept counts are scanned in several tiles
    say(f"[unique] {n} rows, width {width}, group {group}")
    tok, ln = _random_rows(np.random.default_rng(n), n, width, 3)
    ref_t, ref_l = oracle.unique_walks(tok, ln, group)
    got_t, got_l = _gpu_unique(tok, ln, group)
    assert_rows_equal(got_t, got_l, ref_t, ref_l, f"{n} rows group {group}")
