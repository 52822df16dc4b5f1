"""Property-based pins of the CPU oracle (runs without a GPU): hypothesis draws
tiny forests over vocabularies of 2, 3 and 8 tokens, so partial-label
mismatches, sequences that are prefixes of others, duplicates and empty
sequences all occur, and the oracle must agree with a brute-force numpy
definition of the match (System Design: the largest prefix match over each
peer's tree; Algorithm 1: the argmax over all trees) and with the set
semantics of loads and merges (Section "Trie-broadcast loss": a snapshot
replaces the receiver's estimate; inserts only add)."""
import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
import pins

SETTINGS = settings(max_examples=150, deadline=None, derandomize=True,
                    suppress_health_check=[HealthCheck.too_slow])


@st.composite
def forests(draw):
    vocab = draw(st.sampled_from([2, 3, 8]))
    tok = st.integers(0, vocab - 1)
    seq = st.lists(tok, min_size=0, max_size=12)
    P = draw(st.integers(1, 5))
    sets = [draw(st.lists(seq, min_size=0, max_size=6)) for _ in range(P)]
    queries = draw(st.lists(st.lists(tok, min_size=0, max_size=16), min_size=1, max_size=12))
    return P, sets, queries


def _oracle(P, sets):
    o = oracle.Oracle(P)
    for p, S in enumerate(sets):
        t, off = pins._csr(S)
        o.load(p, t, off)
    return o


def _route(o, queries):
    t, off = pins._csr(queries)
    return o.route(t, off, 1)


@SETTINGS
@given(forests())
def test_route_equals_brute_force(f):
    P, sets, queries = f
    o = _oracle(P, sets)
    m, c = _route(o, queries)
    m_np, c_np = pins.reference_matrix([[np.asarray(s, np.int64) for s in S] for S in sets],
                                       [np.asarray(q, np.int64) for q in queries])
    o.close()
    assert np.array_equal(m, m_np)
    assert np.array_equal(c, c_np)


@SETTINGS
@given(forests(), st.data())
def test_merge_equals_load_of_the_union(f, data):
    """Merging a batch into the loaded sets routes like loading the unions;
    merging it again (a duplicated broadcast) changes nothing."""
    P, sets, queries = f
    tok = st.integers(0, 7)
    batch = data.draw(st.lists(st.tuples(st.integers(0, P - 1), st.lists(tok, max_size=10)), max_size=10))
    o = _oracle(P, sets)
    peers = np.array([p for p, _ in batch], np.int32)
    t, off = pins._csr([s for _, s in batch])
    o.merge(peers, t, off)
    m1, c1 = _route(o, queries)
    o.merge(peers, t, off)
    m2, c2 = _route(o, queries)
    union = [list(S) + [s for p, s in batch if p == i] for i, S in enumerate(sets)]
    u = _oracle(P, union)
    mu, cu = _route(u, queries)
    o.close()
    u.close()
    assert np.array_equal(m1, mu) and np.array_equal(c1, cu)
    assert np.array_equal(m2, mu) and np.array_equal(c2, cu)


@SETTINGS
@given(forests(), st.data())
def test_load_replaces(f, data):
    """A second load of a peer replaces its set: the result equals a fresh
    oracle loaded with the new set only."""
    P, sets, queries = f
    p = data.draw(st.integers(0, P - 1))
    new = data.draw(st.lists(st.lists(st.integers(0, 7), max_size=10), max_size=6))
    o = _oracle(P, sets)
    t, off = pins._csr(new)
    o.load(p, t, off)
    m, c = _route(o, queries)
    fresh = [new if i == p else S for i, S in enumerate(sets)]
    u = _oracle(P, fresh)
    mu, cu = _route(u, queries)
    o.close()
    u.close()
    assert np.array_equal(m, mu) and np.array_equal(c, cu)
