"""The CPU oracle checked against things other than itself (runs without a GPU)."""
import numpy as np
import pytest

import oracle
import pins
import workloads as W


def make(P):
    return oracle.Oracle(P)


def test_golden_hand_examples():
    assert pins.check_golden(make) == []


def test_golden_file_is_nontrivial():
    exs = pins.parse_golden()
    assert len(exs) >= 5
    nq = sum(1 for e in exs for op in e.ops if op[0] == "query")
    assert nq >= 25
    # the examples exercise a tie that is not at peer 0 and a merge
    assert any(op[0] == "merge" for e in exs for op in e.ops)


@pytest.mark.parametrize("vocab", [2, 3, 8])
def test_tiny_random_vs_prefix_set_and_numpy(vocab):
    assert pins.check_tiny_random(make, seeds=range(12), vocabs=(vocab,)) == []


def test_merge_union_order_duplicates_reload():
    assert pins.check_merge_semantics(make, seeds=range(8)) == []


def test_config1_invariants_and_closed_forms():
    w = W.make_config(1)
    idx = np.arange(len(w.queries))
    assert pins.check_config_invariants(make, w, idx) == []


def test_config2_sample_invariants_and_closed_forms():
    w = W.make_config(2, n_queries=512, prompts_per_peer=400)
    idx = np.arange(0, 512, 4)
    assert pins.check_config_invariants(make, w, idx) == []


def test_config1_full_vs_numpy_bruteforce_sample():
    """All of config 1's peers against numpy brute force on a query sample."""
    w = W.make_config(1)
    o = make(w.num_peers)
    pins.load_all(o, w.snapshot, w.num_peers)
    idx = np.arange(0, len(w.queries), 16)
    sub = w.queries.subset(idx)
    m, c = o.route(sub.tokens, sub.offsets, 4)
    sets = pins._peer_lists(w)
    m_np, c_np = pins.reference_matrix(sets, [sub.seq(i) for i in range(len(sub))])
    assert np.array_equal(m, m_np)
    assert np.array_equal(c, c_np)


def test_stale_replicas_never_exceed_true_trees():
    """Estimates hold a subset of each peer's inserts, so they never match more
    (Section "Stale trie estimates": staleness can only cost cache hits)."""
    w = W.make_config(3, n_queries=96, prompts_per_peer=60)
    est, tru = make(w.num_peers), make(w.num_peers)
    pins.load_all(est, w.snapshot, w.num_peers)
    pins.load_all(tru, w.true_snapshot, w.num_peers)
    me, _ = est.route(w.queries.tokens, w.queries.offsets, 4)
    mt, _ = tru.route(w.queries.tokens, w.queries.offsets, 4)
    assert (me <= mt).all()
    assert np.array_equal(me[:, 0], mt[:, 0])  # observer 0's own tree is exact
    assert (me < mt).any()  # the drops matter for some query


def test_edge_cases():
    o = make(3)
    e = np.zeros(0, np.int32)
    m, c = o.route(e, np.zeros(1, np.int64))  # no queries
    assert m.shape == (0, 3) and c.shape == (0,)
    m, c = o.route(e, np.zeros(2, np.int64))  # one empty query, empty forest
    assert m.tolist() == [[0, 0, 0]] and c.tolist() == [0]
    with pytest.raises(ValueError):
        o.load(3, e, np.zeros(1, np.int64))  # bad peer
    with pytest.raises(ValueError):
        o.load(0, np.zeros(2, np.int32), np.array([0, 2, 1], np.int64))  # non-monotone
    with pytest.raises(ValueError):
        o.merge(np.array([-1], np.int32), np.zeros(1, np.int32), np.array([0, 1], np.int64))


def test_select_golden_hand_examples():
    assert pins.check_select_golden(make) == []


def test_select_golden_file_is_nontrivial():
    exs = pins.parse_select_golden()
    cases = [c for e in exs for c in e[3]]
    assert len(cases) >= 10
    assert any(c[1] >= 0 and c[2] for c in cases)          # prefer-local with a local peer
    assert any(c[5] == -1 for c in cases)                   # no second choice
    assert any(not c[0].any() for c in cases)               # nothing eligible


def test_select_random_vs_sorted_order():
    assert pins.check_select_random(make, seeds=range(10)) == []


def test_select_rejects_bad_local():
    o = oracle.Oracle(3)
    t, off = np.array([1], np.int32), np.array([0, 1], np.int64)
    with pytest.raises(ValueError):
        o.route_select(t, off, None, 3, False)
    with pytest.raises(ValueError):
        o.route_select(t, off, np.ones(2, np.uint8), -1, False)


def test_export_golden_hand_examples():
    assert pins.check_export_golden(make) == []


def test_export_random_vs_bruteforce_and_round_trip():
    assert pins.check_export_random(make, seeds=range(12)) == []


def test_lru_golden_hand_examples():
    assert pins.check_lru_golden(make) == []


def test_lru_random_vs_sort_model():
    assert pins.check_lru_random(make, seeds=range(16)) == []


def test_lru_evicting_everything_empties_and_time_is_monotone():
    o = oracle.Oracle(2)
    o.set_local(1)
    o.set_time(5)
    o.load(1, np.array([1, 2, 3, 4], np.int32), np.array([0, 2, 4], np.int64))
    assert o.evict(100) == 4
    assert o.export(1)[1].tolist() == [0]
    with pytest.raises(ValueError):
        o.set_time(4)
    # other peers are unaffected by the local peer's evictions
    o.load(0, np.array([1, 2], np.int32), np.array([0, 2], np.int64))
    assert o.prefix_match(0, np.array([1, 2], np.int32)) == 2


def test_tree_tokens_vs_prefix_set():
    """Tokens a tree holds = the number of distinct non-empty prefixes."""
    for sd in range(8):
        w = W.tiny_random(sd, num_peers=3, vocab=2 + sd % 3, n_queries=1)
        o = make(3)
        pins.load_all(o, w.snapshot, 3)
        if sd % 2:
            o.set_local(sd % 3)
        for p, S in enumerate(pins._peer_lists(w)):
            prefixes = {tuple(int(x) for x in s[:k]) for s in S for k in range(1, len(s) + 1)}
            assert o.tree_tokens(p) == len(prefixes), (sd, p)


PLANTS = ["PLANT_LCP_OFF_BY_ONE", "PLANT_MIN_NOT_MAX", "PLANT_TIE_HIGHEST",
          "PLANT_LOAD_APPENDS", "PLANT_MERGE_WRONG_PEER", "PLANT_IGNORE_ELIGIBLE",
          "PLANT_LOCAL_ALWAYS_FIRST", "PLANT_EXPORT_KEEPS_PREFIXES", "PLANT_EVICT_MRU",
          "PLANT_TOUCH_NOTHING"]


@pytest.mark.parametrize("plant", PLANTS)
def test_planted_mistake_is_caught(plant, tmp_path):
    """A plausible mistake planted in the oracle fails at least one pin."""
    path = oracle.build(plant=plant, out=str(tmp_path / f"lib_{plant}.so"))

    def mk(P):
        return oracle.Oracle(P, lib_path=path)

    fails = pins.check_golden(mk) + pins.check_tiny_random(mk, seeds=range(3), vocabs=(3,)) \
        + pins.check_merge_semantics(mk, seeds=range(2)) + pins.check_select_golden(mk) \
        + pins.check_select_random(mk, seeds=range(2)) + pins.check_export_golden(mk) \
        + pins.check_export_random(mk, seeds=range(3)) + pins.check_lru_golden(mk) \
        + pins.check_lru_random(mk, seeds=range(3))
    assert fails, f"{plant} slipped through every pin"
