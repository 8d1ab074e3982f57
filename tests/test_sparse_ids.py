"""The relabel argument behind the largest-id-space GPU test: the oracle's CSR, start set and
walks of a graph whose used ids are spread over a 2^25-id space equal those of its compact
graph mapped back (sparse_ids.expected_on_sparse). Here the oracle also runs directly on the
large id space, so the mapping is checked against it, not assumed."""

import numpy as np

import oracle
from sparse_ids import expected_on_sparse, sparse_graph


def test_relabelled_oracle_equals_direct_oracle():
    V, P, wpn, depth, seed = (1 << 25) + 3, 5, 3, 6, 42
    U, s_r, p, o_r = sparse_graph(V, P, 40_000, 3000, seed=7)
    assert U[0] == 0 and U[-1] == V - 1
    s, o = U[s_r].astype(np.int32), U[o_r].astype(np.int32)
    rp, ed = oracle.build_csr(s, p, o, V, P)
    starts = oracle.nonsink_starts(rp, V)
    tok, ln = oracle.random_walks(rp, ed, V, P, starts, wpn, depth, seed)

    rp_x, ed_x, starts_x, tok_x, ln_x = expected_on_sparse(U, s_r, p, o_r, V, P, wpn, depth, seed)
    assert rp_x.shape == rp.shape and np.array_equal(rp_x, rp)
    assert np.array_equal(ed_x, ed)
    assert np.array_equal(starts_x, starts)
    assert np.array_equal(ln_x, ln) and np.array_equal(tok_x, tok)
    # the graph reaches what the GPU test relies on: sinks, long rows, and the largest token
    assert (np.diff(rp)[U] == 0).any() and np.diff(rp).max() > 100
    assert int(tok.max()) == V + P - 1
