"""Forest compaction on the GPU: after merges, snapshot reloads, touches and
evictions, the rebuilt device image routes, exports, counts tokens and evicts
exactly as the CPU oracle does, holds no more records than before, and takes
further updates."""
import numpy as np
import pytest

import pins
import workloads as W
from gpu_util import announce, assert_rows_equal, gpu_route, nthreads, oracle_for
from test_lru_gpu import Both, _gpu_export, _oracle_export
from test_merge_gpu import _forest, _merge

pytestmark = pytest.mark.gpu


def _compact(f, label):
    announce(f"compact {label}")
    before, after = f.compact()
    info = f.info()
    assert info["num_nodes"] == after, (label, info, after)
    assert 1 <= after <= before, (label, before, after)
    return before, after


def test_compact_fresh_upload_keeps_every_record():
    """An image built from snapshots holds no dead records: compaction keeps
    them all and changes no result."""
    w = W.make_config(1)
    f = _forest(w.snapshot, w.num_peers)
    o = oracle_for(w.snapshot, w.num_peers)
    m0, c0 = gpu_route(f, w.queries, "before compaction")
    before, after = _compact(f, "fresh upload")
    assert before == after
    m1, c1 = gpu_route(f, w.queries, "after compaction")
    assert np.array_equal(m0, m1) and np.array_equal(c0, c1)
    m_or, c_or = o.route(w.queries.tokens, w.queries.offsets, nthreads())
    assert_rows_equal(m1, c1, m_or, c_or, what="fresh upload compacted")
    f.close()
    o.close()


@pytest.mark.parametrize("seed", range(4))
def test_compact_between_random_operations(seed):
    """Local peer 1 of 3 over a small vocabulary, so merges split edges and
    rebuild child blocks often; compaction at random steps, twice in a row at
    the end (the second finds nothing to drop)."""
    rng = np.random.default_rng(9100 + seed)
    vocab = 2 + seed % 3

    def seqs(k, lo=1, hi=9):
        return [rng.integers(0, vocab, size=int(rng.integers(lo, hi))).tolist() for _ in range(k)]

    b = Both(3, 1)
    t = 0
    b.time(t)
    for p in range(3):
        b.load(p, seqs(6))
    queries = seqs(20, 0, 10)
    shrank = False
    for step in range(16):
        t += int(rng.integers(0, 3))
        b.time(t)
        kind = step % 4
        if kind == 0:
            b.merge([(int(rng.integers(0, 3)), s) for s in seqs(4)])
        elif kind == 1:
            b.touch([queries[i] for i in rng.integers(0, len(queries), size=5)])
        elif kind == 2:
            g, o = b.evict(int(rng.integers(1, 8)))
            assert g == o, (seed, step, g, o)
        else:
            b.load(int(rng.integers(0, 3)), seqs(5))
        if step % 3 == 2:
            before, after = _compact(b.f, f"seed={seed} step={step}")
            shrank |= after < before
        b.check(queries, f"seed={seed} step={step}")
    before, after = _compact(b.f, f"seed={seed} final")
    again = _compact(b.f, f"seed={seed} final again")
    assert again == (after, after)
    b.check(queries, f"seed={seed} final")
    assert shrank or before > after, "no compaction found a dead record"
    b.f.check()
    b.f.close()


def test_compact_many_peers_and_wide_blocks():
    """70 peers (two mask words) and first tokens from 300 values, so the
    root's child block is wider than 64 and needs separators."""
    rng = np.random.default_rng(77)
    P = 70

    def seqs(k):
        out = []
        for _ in range(k):
            n = int(rng.integers(1, 7))
            s = [int(rng.integers(0, 300))] + rng.integers(0, 4, size=n - 1).tolist()
            out.append(s)
        return out

    b = Both(P, 3)
    b.time(1)
    for p in range(P):
        b.load(p, seqs(4))
    queries = seqs(60) + [[q[0]] for q in seqs(20)]
    for r in range(3):
        b.time(2 + r)
        b.merge([(int(rng.integers(0, P)), s) for s in seqs(80)])
        b.touch(queries[:30])
    before, after = _compact(b.f, "wide")
    assert after < before
    b.check(queries, "wide compacted")
    g, o = b.evict(40)
    assert g == o
    b.merge([(int(rng.integers(0, P)), s) for s in seqs(50)])
    b.check(queries, "wide after further updates")
    b.f.close()


def test_compact_after_evicting_everything():
    w = W.tiny_random(5, num_peers=2, vocab=3, n_queries=40)
    b = Both(2, 0)
    b.time(1)
    for p in range(2):
        lo, hi = w.snapshot.peer_range(p)
        b.load(p, [w.snapshot.seq(i) for i in range(lo, hi)])
    b.load(1, [])
    queries = [w.queries.seq(i) for i in range(len(w.queries))]
    g, o = b.evict(10 ** 9)
    assert g == o
    before, after = _compact(b.f, "emptied")
    assert after == 1  # the root alone
    b.check(queries, "emptied and compacted")
    b.merge([(0, s) for s in queries[:10]])
    b.check(queries, "refilled after compaction")
    assert _gpu_export(b.f, 0, "refilled") == _oracle_export(b.o, 0)
    b.f.close()


def test_compact_stream_merges():
    """The streaming recipe at reduced size: merge rounds leave dead child
    blocks; after compaction every lookup is still exact and the merges that
    follow compose."""
    w = W.make_config(5, prompts_per_peer=30, rounds=3, phase_queries=2000, phase_inserts=1500)
    f = _forest(w.snapshot, 128)
    o = oracle_for(w.snapshot, 128)
    for ph in w.phases("zipf"):
        _merge(f, ph.inserts, f"stream round {ph.round}")
        o.merge(ph.inserts.peer, ph.inserts.tokens, ph.inserts.offsets)
        before, after = _compact(f, f"stream round {ph.round}")
        assert after < before
        m, c = gpu_route(f, ph.queries, f"stream round {ph.round} compacted")
        m_or, c_or = o.route(ph.queries.tokens, ph.queries.offsets, nthreads())
        assert_rows_equal(m, c, m_or, c_or, what=f"stream round {ph.round} compacted")
    for p in (0, 5, 127):
        t, off = f.export_snapshot(p)
        got = sorted(tuple(x) for x in pins.csr_to_list(t.cpu().numpy(), off.cpu().numpy()))
        assert got == sorted(tuple(x) for x in pins.csr_to_list(*o.export(p))), p
    f.close()
    o.close()
