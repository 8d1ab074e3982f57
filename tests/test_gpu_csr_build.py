"""GPU parity of the CSR build (rdf2v_build_csr, through the C ABI) against the oracle on graphs
made to reach the edge cases of its kernels, bit-exact (row_ptr and edges whole):

* row_ptr comes from one pass over the sorted subjects that fills at most 64 entities per
  change of subject, the rest by binary search: runs of 62 to 66 and 127 to 129 entities
  without out-edges between subjects, before the first subject and after the last;
* the digit counts add a wave's equal digits with one atomic: tiles that hold one hub's
  triples only, tiles half hub and half others, and tiles mixing many hubs;
* the radix passes spread the id bits evenly: id spaces of 1 to 31 bits, so every pass count
  and digit width is used, with tile counts below, at and above a multiple of the 8 XCDs."""

import numpy as np
import pytest

import oracle
import paper_2508_01073_amd as rd
from gpu_helpers import assert_csr_equal, gpu_csr, new_status, say, to_dev

pytestmark = pytest.mark.gpu


def _check(s, p, o, V, P, what):
    s, p, o = (np.asarray(x, dtype=np.int32) for x in (s, p, o))
    rp, ed = oracle.build_csr(s, p, o, V, P)
    csr = gpu_csr(s, p, o, V, P)
    assert_csr_equal(csr, rp, ed)
    say(f"[csr build] {what}: {len(s):,} triples, V={V:,} bit-exact")


@pytest.mark.parametrize("gap", [1, 2, 62, 63, 64, 65, 66, 127, 128, 129, 1000])
def test_runs_of_sinks_between_subjects(gap):
    # subjects every `gap + 1` ids, starting after a gap and leaving one at the end
    rng = np.random.default_rng(gap)
    subjects = np.arange(gap, 40_000, gap + 1)
    V = int(subjects[-1]) + gap + 1
    T = 60_000
    s = rng.choice(subjects, T)
    _check(s, rng.integers(0, 7, T), rng.integers(0, V, T), V, 7, f"subjects every {gap + 1}")


@pytest.mark.parametrize("V", [1, 2, 65, 66, 130, 100_000])
def test_one_subject_at_either_end(V):
    rng = np.random.default_rng(V)
    for subj in sorted({0, V - 1}):
        T = 5_000
        _check(np.full(T, subj), rng.integers(0, 3, T), rng.integers(0, V, T), V, 3, f"only subject {subj}")


def test_hub_only_and_mixed_tiles():
    rng = np.random.default_rng(3)
    V, P = 300_000, 11
    T = 2_000_000
    # 70% of the triples on one hub (whole tiles of it after the first pass), 20% on 40 other
    # hubs, 10% spread: tiles of one key, tiles split between hubs, tiles of many keys
    hubs = rng.choice(V, 41, replace=False)
    kind = rng.random(T)
    s = np.where(kind < 0.7, hubs[0], np.where(kind < 0.9, rng.choice(hubs[1:], T), rng.integers(0, V, T)))
    _check(s, rng.integers(0, P, T), rng.integers(0, V, T), V, P, "hub tiles")


@pytest.mark.parametrize("bits", [1, 2, 7, 8, 9, 13, 16, 17, 18, 19, 24, 26])
@pytest.mark.parametrize("tiles", [1, 7, 8, 9, 23])
def test_id_widths_and_tile_counts(bits, tiles):
    rng = np.random.default_rng(bits * 100 + tiles)
    V = (1 << bits) - rng.integers(0, min(1 << (bits - 1), 5))  # just below a power of two
    T = tiles * 4096 - (0 if tiles % 2 else 1000)               # whole and ragged last tiles
    s = rng.integers(0, V, T)
    s[: T // 10] = V - 1                                        # the largest id, repeated
    _check(s, rng.integers(0, 5, T), rng.integers(0, V, T), int(V), 5, f"{bits}-bit ids, {tiles} tiles")


def test_bad_ids_still_flagged_in_every_column():
    # Subjects are checked by the first count pass, predicates and objects by the first scatter.
    V, P, T = 1000, 4, 20_000
    rng = np.random.default_rng(9)
    base = [rng.integers(0, V, T).astype(np.int32), rng.integers(0, P, T).astype(np.int32),
            rng.integers(0, V, T).astype(np.int32)]
    for col, bad in [(0, V), (0, -1), (1, P), (1, -5), (2, V + 3), (2, -2)]:
        for at in (0, 4095, 4096, T - 1):                        # tile boundaries and the ragged tail
            cols = [c.copy() for c in base]
            cols[col][at] = bad
            st = new_status()
            rd.rdf2v_build_csr(*(to_dev(c) for c in cols), V, P, status=st)
            assert int(st.item()) & rd.RDF2V_STATUS_ID_OUT_OF_RANGE, (col, bad, at)
    st = new_status()
    rd.rdf2v_build_csr(*(to_dev(c) for c in base), V, P, status=st)
    assert int(st.item()) == 0
