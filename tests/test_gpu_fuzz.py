"""Seeded randomized parity: many small graphs and parameter combinations, each run through the
HIP path (C ABI) and compared element by element with the oracle — the CSR, the start set, and
a random window of walk ids with and without walk records, for all three token kinds, plus
skip-gram pairs and CBOW examples of those rows. Sizes, depths (0 and the maximum included),
walks per start, seeds (64-bit), id spaces and sink fractions are drawn per case from one master
seed, so a failure names a case that reruns exactly."""

import numpy as np
import pytest
import torch

import oracle
import paper_2508_01073_amd as rd
from gpu_helpers import assert_csr_equal, assert_rows_equal, gpu_csr, new_status, plain, say, to_dev

pytestmark = pytest.mark.gpu

MASTER_SEED = 20250801
CASES = 500


def _case(i):
    rng = np.random.default_rng([MASTER_SEED, i])
    V = int(rng.choice([1, 2, 3, 17, 255, 256, 257, 1000, 4096, 5000, 70_000]))
    P = int(rng.integers(1, 60))
    T = int(rng.choice([0, 1, 5, 100, 4095, 4096, 4097, 10_000, 50_000]))
    depth = int(rng.choice([0, 1, 2, 3, 7, 8, 15, 16, 17, 33, 64]))
    wpn = int(rng.integers(1, 6))
    seed = int(rng.integers(0, 2**63)) * 2 + int(rng.integers(0, 2))
    # subjects from a subset of the ids, so some entities are sinks
    subj_pool = max(1, int(V * rng.uniform(0.2, 1.0)))
    s = rng.integers(0, subj_pool, T).astype(np.int32)
    if rng.random() < 0.5:  # skewed subjects: long rows next to short ones
        s = (subj_pool * rng.random(T) ** 3).astype(np.int32)
    p = rng.integers(0, P, T).astype(np.int32)
    o = rng.integers(0, V, T).astype(np.int32)
    return rng, V, P, s, p, o, depth, wpn, seed


@pytest.mark.parametrize("i", range(CASES))
def test_random_case(i):
    rng, V, P, s, p, o, depth, wpn, seed = _case(i)
    say(f"[fuzz] case {i}: V={V} P={P} T={s.shape[0]} depth={depth} wpn={wpn} seed={seed}")
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P, walk_records=bool(rng.random() < 0.5) and s.shape[0] > 0)
    assert_csr_equal(csr, rp, ed)
    starts = oracle.nonsink_starts(rp, V)
    got = rd.rdf2v_nonsink_starts(csr)
    assert np.array_equal(got.cpu().numpy(), starts)
    if rng.random() < 0.3 and V > 1:  # an explicit start list with duplicates and sinks
        starts = rng.integers(0, V, int(rng.integers(1, 50))).astype(np.int32)
    n_walks = starts.shape[0] * wpn
    if n_walks == 0:
        return
    b = int(rng.integers(0, n_walks))
    c = int(rng.integers(1, min(n_walks - b, 20_000) + 1))
    tr, lr = oracle.random_walks(rp, ed, V, P, starts, wpn, depth, seed, b, c)
    sd = to_dev(starts)
    for view, what in [(csr, "as built"), (plain(csr), "plain records")]:
        st = new_status()
        tok, ln = rd.rdf2v_random_walks(view, sd, wpn, depth, seed, b, c, status=st)
        torch.cuda.synchronize()
        rd.check_device_status(st, f"case {i}")
        assert_rows_equal(tok.cpu().numpy(), ln.cpu().numpy(), tr, lr, f"case {i} walks [{b}, {b + c}) {what}")
    for kind in (oracle.ENTITY_WALKS, oracle.PROPERTY_WALKS):
        pt, pl = oracle.project_walks(tr, lr, depth, kind)
        tok, ln = rd.rdf2v_random_walks_tokens(csr, sd, wpn, depth, seed, b, c, kind)
        torch.cuda.synchronize()
        assert_rows_equal(tok.cpu().numpy(), ln.cpu().numpy(), pt, pl, f"case {i} token kind {kind}")
    window = int(rng.integers(1, 2 * depth + 2))
    pairs = rd.rdf2v_skipgram_pairs(to_dev(tr), to_dev(lr), window).cpu().numpy()
    assert np.array_equal(pairs, oracle.skipgram_pairs(tr, lr, window)), f"case {i} pairs window {window}"
    if window <= 2 * 64:
        cg, xg = rd.rdf2v_cbow_examples(to_dev(tr), to_dev(lr), window)
        cr, xr = oracle.cbow_examples(tr, lr, window)
        assert np.array_equal(cg.cpu().numpy(), cr) and np.array_equal(xg.cpu().numpy(), xr), \
            f"case {i} CBOW window {window}"


GRAPH_CASES = 200


@pytest.mark.parametrize("i", range(GRAPH_CASES))
def test_random_bfs_and_unique_case(i):
    # BFS walks from random roots (duplicates and sinks included) at caps that truncate and
    # trees of every size (one-wave LDS tier up to the workspace pass), then duplicate-free walks
    # of short walks on the same graph (many repeats) with group sizes across block boundaries.
    rng = np.random.default_rng([MASTER_SEED, 1, i])
    V = int(rng.choice([1, 2, 5, 64, 300, 2000, 20_000]))
    P = int(rng.integers(1, 20))
    T = int(V * rng.choice([0.5, 1, 2, 4, 8]))
    subj_pool = max(1, int(V * rng.uniform(0.3, 1.0)))
    s = (subj_pool * rng.random(T) ** (3 if rng.random() < 0.5 else 1)).astype(np.int32)
    p = rng.integers(0, P, T).astype(np.int32)
    o = rng.integers(0, V, T).astype(np.int32)
    depth = int(rng.choice([0, 1, 2, 3, 4, 5]))
    max_walks = int(rng.choice([1, 2, 7, 64, 256, 1025]))
    roots = rng.integers(0, V, int(rng.integers(1, 200))).astype(np.int32)
    say(f"[fuzz] graph case {i}: V={V} P={P} T={T} bfs depth={depth} max_walks={max_walks} roots={roots.size}")
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P)
    st = new_status()
    tok, ln, cnt = rd.rdf2v_bfs_walks(csr, to_dev(roots), depth, max_walks, status=st)
    torch.cuda.synchronize()
    ref_t, ref_l, ref_c, trunc = oracle.bfs_walks(rp, ed, V, P, roots, depth, max_walks)
    assert np.array_equal(cnt.cpu().numpy(), ref_c), f"case {i}: BFS walk counts"
    valid = np.arange(max_walks)[None, :] < ref_c[:, None]
    assert np.array_equal(tok.cpu().numpy()[valid], ref_t[valid]), f"case {i}: BFS rows"
    assert np.array_equal(ln.cpu().numpy()[valid], ref_l[valid]), f"case {i}: BFS lengths"
    flags = int(st.item())
    assert bool(flags & rd.RDF2V_STATUS_CAPACITY) == (trunc > 0) and not flags & ~rd.RDF2V_STATUS_CAPACITY, \
        f"case {i}: status {flags}"

    starts = oracle.nonsink_starts(rp, V)
    if starts.size == 0:
        return
    wpn = int(rng.integers(1, 9))
    n = min(starts.size * wpn, int(rng.integers(1, 6000)))
    wd = int(rng.integers(1, 5))
    tr, lr = oracle.random_walks(rp, ed, V, P, starts, wpn, wd, int(rng.integers(0, 2**62)), 0, n)
    group = int(rng.choice([1, 2, 3, wpn, 7, 64, 1025]))
    gt, gl = rd.rdf2v_unique_walks(to_dev(tr), to_dev(lr), group)
    rt, rl = oracle.unique_walks(tr, lr, group)
    assert np.array_equal(gl.cpu().numpy(), rl) and np.array_equal(gt.cpu().numpy(), rt), \
        f"case {i}: duplicate-free walks, group {group}"


VOCAB_CASES = 100


def _string_column(rng, pool, picks):
    strs = [pool[k] for k in picks]
    off = np.zeros(len(strs) + 1, np.int64)
    off[1:] = np.cumsum([len(x) for x in strs])
    chars = np.frombuffer(b"".join(strs), np.uint8) if strs and off[-1] else np.zeros(0, np.uint8)
    return chars.copy(), off


@pytest.mark.parametrize("i", range(VOCAB_CASES))
def test_random_vocabulary_case(i):
    # Byte strings from pools of near-duplicates: empty strings, NUL and 0xFF bytes, shared
    # prefixes, lengths up to 200 (past the fast pass's 98 bytes), drawn with skew so that some
    # strings repeat thousands of times and others once.
    rng = np.random.default_rng([MASTER_SEED, 2, i])
    T = int(rng.choice([0, 1, 7, 255, 256, 257, 3000, 20_000]))
    alphabet = rng.choice([2, 4, 16, 256])
    def pool(n):
        out, base = [], bytes(rng.integers(0, alphabet, int(rng.integers(0, 150)), dtype=np.uint8))
        for _ in range(n):
            L = int(rng.choice([0, 1, 2, 5, 7, 8, 31, 97, 98, 99, 150, 200]))
            body = bytes(rng.integers(0, alphabet, L, dtype=np.uint8))
            out.append(base[:int(rng.integers(0, len(base) + 1))] + body if rng.random() < 0.5 else body)
        return out
    ent, prd = pool(int(rng.integers(1, 3000))), pool(int(rng.integers(1, 300)))
    skew = lambda n, k: (k * rng.random(n) ** 3).astype(np.int64) if rng.random() < 0.5 else rng.integers(0, k, n)
    cols = [_string_column(rng, ent, skew(T, len(ent))), _string_column(rng, prd, skew(T, len(prd))),
            _string_column(rng, ent, skew(T, len(ent)))]
    say(f"[fuzz] vocabulary case {i}: T={T} alphabet={alphabet} pools={len(ent)}/{len(prd)}")
    ref = oracle.build_vocabulary(cols[0][0], cols[0][1], cols[1][0], cols[1][1], cols[2][0], cols[2][1])
    dev = torch.device("cuda:0")
    dcols = [(torch.from_numpy(c).to(dev), torch.from_numpy(o).to(dev)) for c, o in cols]
    st = new_status()
    s, p, o, counts = rd.rdf2v_build_vocabulary(*dcols, max(1, 2 * T), max(1, T), status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0, f"case {i}: status {int(st.item())}"
    assert counts.cpu().numpy().tolist() == [ref[3], ref[4]], f"case {i}: distinct counts"
    for got, want, name in zip((s, p, o), ref[:3], ("subject", "predicate", "object")):
        assert np.array_equal(got.cpu().numpy(), want), f"case {i}: {name} ids"
