"""GPU parity for the vocabulary (rdf2v_build_vocabulary, through the C ABI)
against the oracle, bit-exact: hand-worked strings, near-duplicate byte
strings at every alignment, strings whose hash tags collide, the generated
workloads' IRI columns, bounds, bad offsets, and the string pipeline end to
end (vocabulary -> CSR -> walks)."""

import numpy as np
import pytest
import torch

import oracle
import paper_2508_01073_amd as rd
import synth
from gpu_helpers import device, new_status, say, to_dev

pytestmark = pytest.mark.gpu


def _column(strings, lead=0):
    """(chars, offsets) for a list of byte strings; `lead` junk bytes come first, so
    that the strings start at other alignments."""
    data = [s.encode() if isinstance(s, str) else s for s in strings]
    off = np.zeros(len(data) + 1, np.int64)
    off[1:] = np.cumsum([len(d) for d in data])
    body = b"".join(data)
    chars = np.frombuffer(b"\xab" * lead + body, np.uint8).copy()
    return chars, off + lead


def _dev_col(col, shift=0):
    """Device (chars, offsets); with `shift` the chars tensor is a view that starts
    `shift` bytes into its allocation (4-byte aligned, as the ABI asks, but for
    shift 4, 8, 12 not 16-byte aligned)."""
    chars, off = col
    chars = np.ascontiguousarray(chars, np.uint8)
    buf = torch.zeros(chars.size + shift, dtype=torch.uint8, device=device())
    buf[shift:] = torch.from_numpy(chars).to(device())
    return buf[shift:], torch.from_numpy(np.ascontiguousarray(off, np.int64)).to(device())


def _run(cols, max_e, max_p, status=None, stream=None, shifts=(0, 0, 0)):
    st = new_status() if status is None else status
    dcols = [_dev_col(c, k) for c, k in zip(cols, shifts)]
    s, p, o, counts = rd.rdf2v_build_vocabulary(*dcols, max_e, max_p, status=st, stream=stream)
    torch.cuda.synchronize()
    return (s.cpu().numpy(), p.cpu().numpy(), o.cpu().numpy(), counts.cpu().numpy().tolist(),
            int(st.item()))


def _compare(cols, what, max_e=None, max_p=None, shifts=(0, 0, 0)):
    ref = oracle.build_vocabulary(cols[0][0], cols[0][1], cols[1][0], cols[1][1], cols[2][0], cols[2][1])
    T = len(cols[0][1]) - 1
    max_e = max_e or max(1, 2 * T)
    max_p = max_p or max(1, T)
    s, p, o, counts, flags = _run(cols, max_e, max_p, shifts=shifts)
    assert flags == 0, f"{what}: status {flags}"
    assert counts == [ref[3], ref[4]], f"{what}: counts {counts} vs {ref[3:]}"
    for name, got, exp in (("subj", s, ref[0]), ("pred", p, ref[1]), ("obj", o, ref[2])):
        if not np.array_equal(got, exp):
            bad = np.nonzero(got != exp)[0]
            raise AssertionError(f"{what}: {name} ids differ at {bad.size} rows, first {bad[:5].tolist()}: "
                                 f"gpu {got[bad[:5]].tolist()} oracle {exp[bad[:5]].tolist()}")
    return ref


def test_hand_worked():
    say("[vocab] hand-worked")
    S = ["b", "a", "b", "", "ab"]
    P = ["knows", "knows", "likes", "a", "knows"]
    O = ["a", "c", "b", "a", "a\x00"]
    for lead in range(4):
        ref = _compare([_column(S, lead), _column(P, 3 - lead), _column(O, lead)], f"hand lead={lead}")
    assert ref[0].tolist() == [0, 1, 0, 3, 4] and ref[2].tolist() == [1, 2, 0, 1, 5]


def test_empty_and_single():
    say("[vocab] empty and single")
    e = _column([])
    s, p, o, counts, flags = _run([e, e, e], 1, 1)
    assert s.size == 0 and counts == [0, 0] and flags == 0
    _compare([_column([""]), _column([""]), _column([""])], "single empty strings")
    _compare([_column(["x"]), _column(["x"]), _column(["x"])], "single")


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_near_duplicates_every_alignment(seed):
    say(f"[vocab] near duplicates seed={seed}")
    rng = np.random.default_rng(seed)
    alphabet = [b"a", b"b", b"\x00", b"\xff"]
    short = [b"".join(rng.choice(alphabet, size=int(rng.integers(0, 9)))) for _ in range(400)]
    stem = bytes(rng.integers(0, 256, 300, dtype=np.uint8))
    long = [stem[:int(k)] + bytes([int(b)]) for k, b in zip(rng.integers(0, 300, 200), rng.integers(0, 3, 200))]
    pool = short + long
    T = 3000
    cols = [_column([pool[i] for i in rng.integers(0, len(pool), T)], lead=int(rng.integers(0, 8)))
            for _ in range(3)]
    _compare(cols, f"near duplicates seed={seed}")
    # bounds equal to the exact distinct counts are enough
    ref = oracle.build_vocabulary(cols[0][0], cols[0][1], cols[1][0], cols[1][1], cols[2][0], cols[2][1])
    _compare(cols, "exact bounds", max_e=ref[3], max_p=ref[4])


@pytest.mark.parametrize("shifts", [(4, 4, 4), (0, 8, 0), (12, 0, 4)])
def test_columns_not_16_byte_aligned(shifts):
    # The fast pass stages 16-byte groups only when every column starts 16-byte
    # aligned; these columns start 4 bytes past such a boundary (or 8, 12), in
    # one column or all of them, so the 4-byte staging runs.
    say(f"[vocab] column starts {shifts}")
    rng = np.random.default_rng(11)
    alphabet = [b"a", b"b", b"\x00", b"\xff"]
    pool = [b"".join(rng.choice(alphabet, size=int(rng.integers(0, 12)))) for _ in range(300)]
    pool += [b"http://kg.example.org/entity/Q" + str(k).encode() for k in range(300)]
    T = 4000
    cols = [_column([pool[i] for i in rng.integers(0, len(pool), T)], lead=int(rng.integers(0, 8)))
            for _ in range(3)]
    _compare(cols, f"column starts {shifts}", shifts=shifts)


def test_long_strings_at_scale():
    # Strings longer than the 98-byte inline copy are always left to the general
    # pass: 600,000 triples of them (1.2M entity occurrences over 5,000 strings,
    # 600,000 predicate occurrences over 300) all go through it.
    say("[vocab] long strings at scale")
    rng = np.random.default_rng(17)
    stem = b"http://kg.example.org/a-rather-long-namespace/with/several/levels/of/path/segments/entity-"
    ents = [stem + b"%09d" % k + b"x" * int(k % 5) for k in range(5000)]
    preds = [stem + b"relation-" + b"%04d" % k for k in range(300)]
    assert min(len(x) for x in ents + preds) > 98
    T = 600_000
    cols = [_column([ents[i] for i in rng.integers(0, len(ents), T)]),
            _column([preds[i] for i in rng.integers(0, len(preds), T)]),
            _column([ents[i] for i in rng.integers(0, len(ents), T)])]
    ref = _compare(cols, "long strings at scale", max_e=len(ents), max_p=len(preds))
    assert ref[3] == len(ents) and ref[4] == len(preds)


def test_inline_copy_length_boundary():
    # Strings of 96..100 bytes differing only in their last byte: up to 98 bytes
    # they are compared against the slot's inline copy, beyond it against the
    # representative's bytes.
    say("[vocab] inline length boundary")
    stem = bytes(range(7, 107))
    pool = [stem[:L - 1] + bytes([b]) for L in range(96, 101) for b in range(4)]
    rng = np.random.default_rng(5)
    T = 500
    for lead in range(4):
        cols = [_column([pool[i] for i in rng.integers(0, len(pool), T)], lead=lead) for _ in range(3)]
        ref = _compare(cols, f"boundary lead={lead}", max_e=len(pool), max_p=len(pool))
        assert ref[3] == len(pool)


def _np_hash(strings):
    """The library's 64-bit string hash, restated in numpy for equal-length strings
    (used only to construct strings whose hash tags collide): the string as
    little-endian 7-byte words, zero-padded, folded in after a length-seeded start,
    then MurmurHash3's 64-bit finaliser."""
    M = (1 << 64) - 1
    n = len(strings[0])
    a = np.frombuffer(b"".join(strings), np.uint8).reshape(len(strings), n)
    nw = (n + 6) // 7
    a = np.concatenate([a, np.zeros((len(strings), 7 * nw - n), np.uint8)], axis=1).reshape(len(strings), nw, 7)
    words = np.zeros((len(strings), nw), np.uint64)
    for b in range(7):
        words |= a[:, :, b].astype(np.uint64) << np.uint64(8 * b)
    with np.errstate(over="ignore"):
        h = np.full(len(strings), np.uint64(0x243f6a8885a308d3 ^ ((n * 0x9e3779b97f4a7c15) & M)))
        for k in range(nw):
            h = (h ^ words[:, k]) * np.uint64(0x100000001b3)
            h ^= h >> np.uint64(29)
        h ^= h >> np.uint64(33)
        h *= np.uint64(0xff51afd7ed558ccd)
        h ^= h >> np.uint64(33)
        h *= np.uint64(0xc4ceb9fe1a85ec53)
        h ^= h >> np.uint64(33)
    return h


@pytest.mark.parametrize("stem", [b"k", b"long-" * 20])
def test_colliding_hash_tags_stay_distinct(stem):
    # Equal-length strings whose 20-bit hash tags and first probe slot (64-slot
    # table) agree: the second finds the first's slot with a matching tag and
    # length, so only the byte comparison keeps them apart -- against the inline
    # copy for short strings, against the representative's bytes for strings too
    # long to be copied into the slot (105 bytes).
    say(f"[vocab] colliding tags, {len(stem) + 5}-byte strings")
    n = 1 << 16
    strings = [stem + b"%05d" % i for i in range(n)]
    h = _np_hash(strings)
    key = (h >> np.uint64(44)) << np.uint64(6) | (h & np.uint64(63))
    order = np.argsort(key, kind="stable")
    ks = key[order]
    dup = np.nonzero(ks[1:] == ks[:-1])[0]
    pairs = [(strings[order[i]], strings[order[i + 1]]) for i in dup[:8]]
    assert len(pairs) >= 4, "too few colliding pairs found"
    for a, b in pairs:
        S = [a, b, a, b, b, a]
        O = [b, a, a, b, a, b]
        P = [a, b, b, a, a, b]
        ref = _compare([_column(S), _column(P), _column(O)], f"tags {a[-5:]}/{b[-5:]}", max_e=2, max_p=2)
        assert ref[3] == 2 and ref[4] == 2


@pytest.mark.parametrize("name", ["tiny_uniform", "uniform_1m", "powerlaw_20m"])
def test_workloads_against_oracle(name):
    w = synth.WORKLOADS[name]
    say(f"[vocab] {w.describe()}")
    S, P, O = synth.triples(w)
    cols = synth.string_triples(S, P, O, w.num_entities, w.num_predicates)
    _compare(cols, name, max_e=w.num_entities, max_p=w.num_predicates)


def test_dense_workload_against_integer_ranks():
    # 10M triples over 10k entities: every string recurs ~2000 times
    w = synth.WORKLOADS["dense_10m"]
    say(f"[vocab] {w.describe()}")
    S, P, O = synth.triples(w)
    cols = synth.string_triples(S, P, O, w.num_entities, w.num_predicates)
    s, p, o, counts, flags = _run(cols, w.num_entities, w.num_predicates)
    assert flags == 0
    seq = np.empty(2 * len(S), np.int64)
    seq[0::2], seq[1::2] = S, O
    uniq, first = np.unique(seq, return_index=True)
    rank = np.empty(w.num_entities, np.int64)
    rank[uniq[np.argsort(first)]] = np.arange(uniq.size)
    puniq, pfirst = np.unique(P, return_index=True)
    prank = np.empty(w.num_predicates, np.int64)
    prank[puniq[np.argsort(pfirst)]] = np.arange(puniq.size)
    assert counts == [uniq.size, puniq.size]
    assert np.array_equal(s, rank[S]) and np.array_equal(o, rank[O]) and np.array_equal(p, prank[P])


def test_bound_exceeded_raises_capacity():
    say("[vocab] capacity")
    names = [b"e%d" % i for i in range(100)]
    cols = [_column(names), _column([b"p"] * 100), _column(names[::-1])]
    _, _, _, counts, flags = _run(cols, 100, 1)
    assert flags == 0 and counts == [100, 1]
    for max_e in (99, 40, 1):
        _, _, _, counts, flags = _run(cols, max_e, 1)
        assert flags & rd.RDF2V_STATUS_CAPACITY, max_e
    _, _, _, _, flags = _run([cols[0], _column([b"p", b"q"] * 50), cols[2]], 100, 1)
    assert flags == rd.RDF2V_STATUS_CAPACITY


def test_bad_offsets_flagged():
    say("[vocab] bad offsets")
    chars, off = _column(["aa", "bb", "cc"])
    for bad in ([0, 2, 1, 6], [0, 2, 4, 99], [-3, 2, 4, 6]):
        cols = [(chars, np.array(bad, np.int64)), (chars, off), (chars, off)]
        _, _, _, _, flags = _run(cols, 10, 10)
        assert flags == rd.RDF2V_STATUS_BAD_LENGTH, bad


def test_deterministic_across_calls_and_streams():
    say("[vocab] determinism")
    w = synth.WORKLOADS["uniform_1m"]
    S, P, O = synth.triples(w)
    cols = synth.string_triples(S, P, O, w.num_entities, w.num_predicates)
    a = _run(cols, w.num_entities, w.num_predicates)
    side = torch.cuda.Stream(device())
    b = _run(cols, w.num_entities, w.num_predicates, stream=side)
    for x, y in zip(a[:3], b[:3]):
        assert np.array_equal(x, y)
    assert a[3] == b[3]


def test_reused_workspace_across_vocabularies():
    # One workspace serves two calls over the same strings in opposite triple orders, so every
    # string gets another id and another first occurrence in the second call. Each call resets the
    # table; a slot the first call claimed must read as empty again in the second, or its string
    # would be found there and never claimed (the fast pass reads slots through the caches).
    say("[vocab] reused workspace")
    w = synth.WORKLOADS["uniform_1m"]
    S, P, O = synth.triples(w)
    T = S.shape[0]
    ws = torch.empty(rd.rdf2v_build_vocabulary_workspace_size(T, w.num_entities, w.num_predicates),
                     dtype=torch.uint8, device=device())
    for order in ("forward", "reversed"):
        if order == "reversed":
            S, P, O = S[::-1].copy(), P[::-1].copy(), O[::-1].copy()
        cols = synth.string_triples(S, P, O, w.num_entities, w.num_predicates)
        ref = oracle.build_vocabulary(cols[0][0], cols[0][1], cols[1][0], cols[1][1], cols[2][0], cols[2][1])
        st = new_status()
        s, p, o, counts = rd.rdf2v_build_vocabulary(*[_dev_col(c) for c in cols], w.num_entities,
                                                    w.num_predicates, workspace=ws, status=st)
        torch.cuda.synchronize()
        assert int(st.item()) == 0
        assert counts.cpu().numpy().tolist() == [ref[3], ref[4]]
        for got, exp in ((s, ref[0]), (p, ref[1]), (o, ref[2])):
            assert np.array_equal(got.cpu().numpy(), exp), order


def test_string_pipeline_end_to_end():
    # strings -> ids on the GPU -> CSR -> walks equals the oracle pipeline from the same strings
    say("[vocab] end to end")
    w = synth.WORKLOADS["tiny_uniform"]
    S, P, O = synth.triples(w)
    cols = synth.string_triples(S, P, O, w.num_entities, w.num_predicates)
    st = new_status()
    s, p, o, counts = rd.rdf2v_build_vocabulary(*[_dev_col(c) for c in cols], w.num_entities,
                                                w.num_predicates, status=st)
    V, Pn = [int(x) for x in counts.cpu()]
    csr = rd.rdf2v_build_csr(s, p, o, V, Pn, status=st)
    starts = rd.rdf2v_nonsink_starts(csr)
    tok, ln = rd.rdf2v_random_walks(csr, starts, w.walks_per_node, w.depth, synth.WALK_SEED, status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    rs, rp_, ro, rV, rP = oracle.build_vocabulary(cols[0][0], cols[0][1], cols[1][0], cols[1][1], cols[2][0],
                                                  cols[2][1])
    assert (V, Pn) == (rV, rP)
    row_ptr, edges = oracle.build_csr(rs, rp_, ro, rV, rP)
    ref_starts = oracle.nonsink_starts(row_ptr, rV)
    ref_t, ref_l = oracle.random_walks(row_ptr, edges, rV, rP, ref_starts, w.walks_per_node, w.depth,
                                       synth.WALK_SEED)
    assert np.array_equal(starts.cpu().numpy(), ref_starts)
    assert np.array_equal(tok.cpu().numpy(), ref_t) and np.array_equal(ln.cpu().numpy(), ref_l)
