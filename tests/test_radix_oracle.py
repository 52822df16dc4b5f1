"""Pins of the second CPU oracle, one radix tree per peer (oracle/radix_oracle.c),
runs without a GPU.

It is checked against things other than itself:
* the hand-worked golden examples (System Design, Algorithm 1, Section
  "Trie-broadcast loss");
* the prefix-set formulation of a trie and numpy brute force of
  max_s LCP(q, s), with numpy's first-maximum argmax for the tie rule;
* the linear-scan oracle (prefix_oracle.c), an independent formulation of the
  same definition, on hypothesis-drawn forests, all of the tiny workload and
  samples of the other four;
* the closed form of a radix tree's shape: its nodes are exactly the stored
  members, the branch points, and (with split_block B) the multiples of B on
  stored paths; its label tokens are exactly the distinct non-empty prefixes;
* split_block does not change any match length (the reading of the long
  workload's 16-token blocks as structure only);
* planted mistakes in its INSERT and MATCH each fail at least one of these.
"""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
import pins
import workloads as W

SETTINGS = settings(max_examples=150, deadline=None, derandomize=True,
                    suppress_health_check=[HealthCheck.too_slow])


def make(P, split_block=0, lib_path=None):
    return oracle.RadixOracle(P, split_block=split_block, lib_path=lib_path)


def _load(o, P, sets):
    for p, S in enumerate(sets):
        t, off = pins._csr(S)
        o.load(p, t, off)
    return o


def _route(o, queries):
    t, off = pins._csr(queries)
    return o.route(t, off, 1)


def shape_closed_form(S, B=0):
    """Nodes (root excluded) and label tokens of a path-compressed radix tree
    over the member set S: a node sits at every prefix u that is a member, a
    branch point (two or more distinct next tokens among the members it
    prefixes) or, with B > 0, at a depth that is a multiple of B."""
    prefixes = {}
    members = set()
    for s in S:
        s = tuple(int(x) for x in s)
        members.add(s)
        for k in range(1, len(s) + 1):
            prefixes.setdefault(s[:k], set())
        for k in range(len(s)):
            prefixes.setdefault(s[:k], set()).add(s[k])
    nodes = 0
    for u, nxt in prefixes.items():
        if not u:
            continue
        if u in members or len(nxt) >= 2 or (B > 0 and len(u) % B == 0):
            nodes += 1
    tokens = sum(1 for u in prefixes if u)
    return nodes, tokens


def shape_failures(o, sets, B=0):
    fails = []
    for p, S in enumerate(sets):
        want_nodes, want_tokens = shape_closed_form(S, B)
        if o.check(p):
            fails.append(f"peer {p}: structure rule {o.check(p)} broken")
        if o.node_count(p) != want_nodes:
            fails.append(f"peer {p}: {o.node_count(p)} nodes, closed form {want_nodes}")
        if o.tree_tokens(p) != want_tokens:
            fails.append(f"peer {p}: {o.tree_tokens(p)} label tokens, closed form {want_tokens}")
    return fails


def check_shapes(mk, seeds, blocks=(0, 2, 3)) -> list:
    fails = []
    for B in blocks:
        for sd in seeds:
            w = W.tiny_random(sd, num_peers=3, vocab=2 + sd % 3, n_queries=1)
            o = mk(3, B)
            pins.load_all(o, w.snapshot, 3)
            fails += [f"B={B} seed={sd}: {x}" for x in shape_failures(o, pins._peer_lists(w), B)]
    return fails


def check_split_block_invariance(mk, seeds, blocks=(1, 2, 3, 5)) -> list:
    fails = []
    for sd in seeds:
        w = W.tiny_random(sd, num_peers=4, vocab=3, n_queries=40)
        o0 = mk(4, 0)
        pins.load_all(o0, w.snapshot, 4)
        m0, c0 = o0.route(w.queries.tokens, w.queries.offsets, 1)
        for B in blocks:
            o = mk(4, B)
            pins.load_all(o, w.snapshot, 4)
            m, c = o.route(w.queries.tokens, w.queries.offsets, 1)
            if not (np.array_equal(m, m0) and np.array_equal(c, c0)):
                fails.append(f"seed {sd}: split_block {B} changed a match")
    return fails


# --------------------------------------------------------------------------
def test_golden_hand_examples():
    assert pins.check_golden(make) == []


@pytest.mark.parametrize("vocab", [2, 3, 8])
def test_tiny_random_vs_prefix_set_and_numpy(vocab):
    assert pins.check_tiny_random(make, seeds=range(12), vocabs=(vocab,)) == []


def test_merge_union_order_duplicates_reload():
    assert pins.check_merge_semantics(make, seeds=range(8)) == []


def test_tree_shape_closed_form():
    assert check_shapes(lambda P, B: make(P, B), seeds=range(10)) == []


def test_split_block_does_not_change_matches():
    assert check_split_block_invariance(lambda P, B: make(P, B), seeds=range(8)) == []


def test_config1_all_rows_vs_linear_scan_oracle():
    w = W.make_config(1)
    a = oracle.Oracle(w.num_peers)
    pins.load_all(a, w.snapshot, w.num_peers)
    b = make(w.num_peers)
    b.load_seqset(w.snapshot)
    ma, ca = a.route(w.queries.tokens, w.queries.offsets, 4)
    mb, cb = b.route(w.queries.tokens, w.queries.offsets, 4)
    assert np.array_equal(ma, mb) and np.array_equal(ca, cb)
    assert pins.check_config_invariants(make, w, np.arange(len(w.queries))) == []
    assert shape_failures(b, pins._peer_lists(w)) == []


@pytest.mark.parametrize("cfg,kw", [
    (2, dict(n_queries=768, prompts_per_peer=300)),
    (3, dict(n_queries=256, prompts_per_peer=80)),
    (4, dict(n_queries=96, prompts_per_peer=24)),
])
def test_configs_vs_linear_scan_oracle(cfg, kw):
    """Reduced workloads of the medium, stale and long recipes: every row equal
    to the linear scan; the long one also with 16-token split blocks."""
    w = W.make_config(cfg, **kw)
    snaps = [w.snapshot] + ([w.true_snapshot] if cfg == 3 else [])
    for snap in snaps:
        a = oracle.Oracle(w.num_peers)
        pins.load_all(a, snap, w.num_peers)
        ma, ca = a.route(w.queries.tokens, w.queries.offsets, 4)
        for B in ((0, 16) if cfg == 4 else (0,)):
            b = make(w.num_peers, B)
            b.load_seqset(snap)
            mb, cb = b.route(w.queries.tokens, w.queries.offsets, 4)
            assert np.array_equal(ma, mb) and np.array_equal(ca, cb), (cfg, B)
            assert all(b.check(p) == 0 for p in range(w.num_peers))
            b.close()
        a.close()


def test_stream_phases_vs_linear_scan_oracle():
    """The streaming recipe at reduced size: base trees, then merge batches and
    lookups in turn, every row equal to the linear scan after every phase."""
    w = W.make_config(5, prompts_per_peer=12, rounds=2, phase_queries=300, phase_inserts=400)
    for dist in ("uniform", "zipf"):
        a = oracle.Oracle(w.num_peers)
        pins.load_all(a, w.snapshot, w.num_peers)
        b = make(w.num_peers)
        b.load_seqset(w.snapshot)
        for ph in w.phases(dist):
            a.merge(ph.inserts.peer, ph.inserts.tokens, ph.inserts.offsets)
            b.merge(ph.inserts.peer, ph.inserts.tokens, ph.inserts.offsets)
            ma, ca = a.route(ph.queries.tokens, ph.queries.offsets, 4)
            mb, cb = b.route(ph.queries.tokens, ph.queries.offsets, 4)
            assert np.array_equal(ma, mb) and np.array_equal(ca, cb), (dist, ph.round)
        assert all(b.check(p) == 0 for p in range(w.num_peers))


def test_tree_tokens_equal_linear_oracle():
    for sd in range(6):
        w = W.tiny_random(sd, num_peers=3, vocab=2 + sd % 3, n_queries=1)
        a = oracle.Oracle(3)
        pins.load_all(a, w.snapshot, 3)
        b = make(3)
        b.load_seqset(w.snapshot)
        assert [a.tree_tokens(p) for p in range(3)] == [b.tree_tokens(p) for p in range(3)]


def test_edge_cases():
    o = make(3)
    e = np.zeros(0, np.int32)
    m, c = o.route(e, np.zeros(1, np.int64))
    assert m.shape == (0, 3) and c.shape == (0,)
    m, c = o.route(e, np.zeros(2, np.int64))  # one empty query, empty forest
    assert m.tolist() == [[0, 0, 0]] and c.tolist() == [0]
    with pytest.raises(ValueError):
        o.load(3, e, np.zeros(1, np.int64))
    with pytest.raises(ValueError):
        o.load(0, np.zeros(2, np.int32), np.array([0, 2, 1], np.int64))
    with pytest.raises(ValueError):
        o.merge(np.array([-1], np.int32), np.zeros(1, np.int32), np.array([0, 1], np.int64))
    # extreme int32 tokens are ordinary keys
    big = np.array([2**31 - 1, -2**31, 0, -1], np.int32)
    o.load(1, big, np.array([0, 4], np.int64))
    assert o.prefix_match(1, big[:3]) == 3 and o.prefix_match(1, big[1:]) == 0
    with pytest.raises(ValueError):
        make(0)


# ---- property-based: against the numpy definition and the linear scan -------
@st.composite
def forests(draw):
    vocab = draw(st.sampled_from([2, 3, 8]))
    tok = st.integers(0, vocab - 1)
    seq = st.lists(tok, min_size=0, max_size=12)
    P = draw(st.integers(1, 5))
    sets = [draw(st.lists(seq, min_size=0, max_size=6)) for _ in range(P)]
    queries = draw(st.lists(st.lists(tok, min_size=0, max_size=16), min_size=1, max_size=12))
    B = draw(st.sampled_from([0, 0, 1, 2, 3, 4]))
    return P, sets, queries, B


@SETTINGS
@given(forests())
def test_hypothesis_route_equals_brute_force_and_linear_scan(f):
    P, sets, queries, B = f
    b = _load(make(P, B), P, sets)
    m, c = _route(b, queries)
    m_np, c_np = pins.reference_matrix([[np.asarray(s, np.int64) for s in S] for S in sets],
                                       [np.asarray(q, np.int64) for q in queries])
    a = _load(oracle.Oracle(P), P, sets)
    ma, ca = _route(a, queries)
    assert np.array_equal(m, m_np) and np.array_equal(c, c_np)
    assert np.array_equal(m, ma) and np.array_equal(c, ca)
    assert shape_failures(b, sets, B) == []


@SETTINGS
@given(forests(), st.data())
def test_hypothesis_merge_equals_load_of_the_union(f, data):
    P, sets, queries, B = f
    batch = data.draw(st.lists(st.tuples(st.integers(0, P - 1), st.lists(st.integers(0, 7), max_size=10)),
                               max_size=10))
    b = _load(make(P, B), P, sets)
    peers = np.array([p for p, _ in batch], np.int32)
    t, off = pins._csr([s for _, s in batch])
    b.merge(peers, t, off)
    m1, c1 = _route(b, queries)
    b.merge(peers, t, off)
    m2, c2 = _route(b, queries)
    union = [list(S) + [s for p, s in batch if p == i] for i, S in enumerate(sets)]
    u = _load(make(P, B), P, union)
    mu, cu = _route(u, queries)
    assert np.array_equal(m1, mu) and np.array_equal(c1, cu)
    assert np.array_equal(m2, mu) and np.array_equal(c2, cu)
    assert shape_failures(b, union, B) == []


# ---- planted mistakes ------------------------------------------------------
RX_PLANTS = ["PLANT_RX_CHILD_LOWER_BOUND", "PLANT_RX_LEAF_DROPS_LAST", "PLANT_RX_SPLIT_NO_ADVANCE",
             "PLANT_RX_MATCH_PAST_PARTIAL", "PLANT_RX_LOAD_APPENDS"]


@pytest.mark.parametrize("plant", RX_PLANTS)
def test_planted_mistake_is_caught(plant, tmp_path):
    path = oracle.build(plant=plant, out=str(tmp_path / f"lib_{plant}.so"))

    def mk(P, B=0):
        return make(P, B, lib_path=path)

    fails = []
    for check in (lambda: pins.check_golden(mk),
                  lambda: pins.check_tiny_random(mk, seeds=range(3), vocabs=(3,)),
                  lambda: pins.check_merge_semantics(mk, seeds=range(2)),
                  lambda: check_shapes(mk, seeds=range(3)),
                  lambda: check_split_block_invariance(mk, seeds=range(2))):
        try:
            fails += check()
        except ValueError as e:  # the insert's own guard refused a corrupt tree
            fails.append(str(e))
    assert fails, f"{plant} slipped through every pin"
