"""The seeded generators: deterministic, and shaped as the configurations state."""
import numpy as np

import workloads as W


def _same(a, b):
    return np.array_equal(a.tokens, b.tokens) and np.array_equal(a.offsets, b.offsets)


def test_deterministic():
    a, b = W.make_config(1), W.make_config(1)
    assert _same(a.snapshot, b.snapshot) and _same(a.queries, b.queries)
    c = W.make_config(1, seed_base=W.SEED_BASE + 1)
    assert not _same(a.queries, c.queries)


def test_tiny_shape():
    w = W.make_config(1)
    assert w.num_peers == 4 and len(w.queries) == 2048 and len(w.snapshot) == 800
    L = w.snapshot.lengths()
    assert L.min() >= 64 + 256 + 32 and L.max() <= 64 + 256 + 128
    assert np.all(np.diff(w.snapshot.peer) >= 0)
    frac_unseen = w.meta["query_unseen"].mean()
    assert 0.06 < frac_unseen < 0.14
    # round-robin homing: topic t lives on peer t mod 4
    for t in range(16):
        assert t in w.meta["homed"][t % 4]


def test_medium_shape_small():
    w = W.make_config(2, n_queries=2000, prompts_per_peer=50)
    assert w.num_peers == 16
    L = w.queries.lengths()
    assert L.min() >= 128 + 1024 + 64 and L.max() <= 128 + 1024 + 256
    # every topic homed on exactly two distinct peers
    cnt = np.zeros(64, int)
    for h in w.meta["homed"]:
        for t in h:
            cnt[t] += 1
    assert (cnt == 2).all()


def test_stale_window_drops_only_recent_inserts():
    w = W.make_config(3, n_queries=16, prompts_per_peer=40)
    keep = w.meta["stale_keep"]
    per = 40
    assert keep[:per].all()  # observer 0 exact
    for p in range(1, 64):
        seg = keep[p * per:(p + 1) * per]
        assert seg[: per - w.meta["stale_window"]].all()
    assert 0.1 < 1 - keep[per:].mean() < 0.3
    L = w.true_snapshot.lengths()
    assert L.max() <= 4096 and L.min() >= 256 + 512 + 64


def test_stream_phases_are_independent_and_deterministic():
    w = W.make_config(5, prompts_per_peer=4, rounds=2, phase_queries=64, phase_inserts=32)
    a = w.phase("zipf", 1)
    b = W.make_config(5, prompts_per_peer=4, rounds=2, phase_queries=64, phase_inserts=32).phase("zipf", 1)
    assert _same(a.queries, b.queries) and _same(a.inserts, b.inserts)
    assert (a.inserts.peer >= 1).all() and (a.inserts.peer < 128).all()


def test_tiny_random_has_sharing():
    w = W.tiny_random(3, num_peers=3, vocab=2, n_queries=20)
    assert len(w.snapshot) > 0
