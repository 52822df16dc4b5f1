"""Delta-merge parity on the GPU: batches of inserts applied by the HIP merge
kernels (updateTrie / updateTrieEstimate), then routed, versus the CPU oracle
given the same snapshots and inserts.  Bit-exact on every output."""
import numpy as np
import pytest

import oracle
import pins
import workloads as W
from gpu_util import (announce, assert_properties, assert_rows_equal, device, gpu_route, nthreads,
                      oracle_for, radix_for, to_dev)

pytestmark = pytest.mark.gpu


def _merge(f, ins, label=""):
    import torch
    dev = device()
    announce(f"merge {label}: {len(ins)} inserts")
    peer = torch.from_numpy(np.ascontiguousarray(ins.peer, dtype=np.int32)).to(dev)
    t, o = to_dev(ins)
    f.merge(peer, t, o)
    torch.cuda.synchronize()


def _forest(snapshot, P):
    from paper_2606_17059_amd import Forest
    f = Forest(P)
    if snapshot is not None:
        f.load_seqset(snapshot)
    return f


def test_golden_examples_with_merges():
    from paper_2606_17059_amd import Forest
    import torch
    dev = device()
    for ex in pins.parse_golden():
        f = Forest(ex.peers)
        for op in ex.ops:
            if op[0] == "load":
                t, o = pins._csr(op[2])
                f.load_snapshot(op[1], t, o)
            elif op[0] == "merge":
                t, o = pins._csr([s for _, s in op[1]])
                ins = W.SeqSet(t, o, np.array([p for p, _ in op[1]], np.int32))
                _merge(f, ins, ex.name)
            else:
                _, q, m_exp, c_exp = op
                t, o = pins._csr([q])
                announce(f"golden {ex.name} q={q}")
                m, c = f.route(torch.from_numpy(t).to(dev), torch.from_numpy(o).to(dev))
                assert m.cpu().numpy()[0].tolist() == m_exp and int(c.cpu()[0]) == c_exp, (ex.name, q)
        f.close()


def _random_batch(seed, P, vocab, n):
    w = W.tiny_random(seed, num_peers=P, vocab=vocab, max_seqs=max(1, n // P), n_queries=1)
    return w.snapshot


@pytest.mark.parametrize("vocab", [2, 3, 8])
def test_tiny_random_merge_sequences(vocab):
    """Snapshots, then three merge batches; every route compared with the oracle."""
    for sd in range(12):
        P = [1, 3, 5, 64, 65, 130][sd % 6]
        base = W.tiny_random(sd, num_peers=P, vocab=vocab, max_seqs=8 if P < 10 else 2, n_queries=60)
        f = _forest(base.snapshot if sd % 3 else None, P)  # every third case starts empty
        o = oracle.Oracle(P)
        if sd % 3:
            pins.load_all(o, base.snapshot, P)
        for r in range(3):
            ins = _random_batch(1000 * sd + r, P, vocab, 24)
            if len(ins) == 0:
                continue
            _merge(f, ins, f"vocab={vocab} seed={sd} batch={r}")
            o.merge(ins.peer, ins.tokens, ins.offsets)
            m, c = gpu_route(f, base.queries, f"after batch {r}")
            m_or, c_or = o.route(base.queries.tokens, base.queries.offsets, 2)
            assert_rows_equal(m, c, m_or, c_or, what=f"vocab={vocab} seed={sd} batch={r}")
            # cached prompts as queries: every inserted sequence matches its owner in full
            mi, _ = gpu_route(f, ins, "inserted sequences as queries")
            assert np.array_equal(mi[np.arange(len(ins)), ins.peer], ins.lengths())
        f.check()
        f.close()


def test_duplicates_prefixes_and_shared_new_prefixes_in_one_batch():
    """Inserts that duplicate each other, are prefixes of each other, or share a
    long new prefix, all in one batch (several rounds of splits and adds)."""
    rng = np.random.default_rng(5)
    P = 4
    shared = rng.integers(0, 50, 300).astype(np.int32)
    seqs, owners = [], []
    for i in range(200):
        k = int(rng.integers(0, 300))
        tail = rng.integers(0, 50, int(rng.integers(0, 40))).astype(np.int32)
        seqs.append(np.concatenate([shared[:k], tail]))
        owners.append(int(rng.integers(0, P)))
    seqs += [shared.copy(), shared[:10].copy(), shared[:10].copy(), np.zeros(0, np.int32)]
    owners += [0, 1, 1, 2]
    ins = W.from_lists(seqs, owners)
    qs = W.from_lists([s for s in seqs] + [shared[:k] for k in range(0, 300, 7)])
    f = _forest(None, P)
    _merge(f, ins, "shared prefixes")
    o = oracle.Oracle(P)
    o.merge(ins.peer, ins.tokens, ins.offsets)
    m, c = gpu_route(f, qs, "shared prefixes")
    m_or, c_or = o.route(qs.tokens, qs.offsets, 2)
    assert_rows_equal(m, c, m_or, c_or, what="shared prefixes")


def test_batch_order_does_not_matter():
    w = W.make_config(1, n_queries=400, prompts_per_peer=60)
    extra = W.make_config(1, seed_base=W.SEED_BASE + 9, n_queries=1, prompts_per_peer=60).snapshot
    perm = np.random.default_rng(3).permutation(len(extra))
    f1, f2 = _forest(w.snapshot, 4), _forest(w.snapshot, 4)
    _merge(f1, extra, "in order")
    _merge(f2, extra.subset(perm), "shuffled")
    m1, c1 = gpu_route(f1, w.queries, "in order")
    m2, c2 = gpu_route(f2, w.queries, "shuffled")
    assert np.array_equal(m1, m2) and np.array_equal(c1, c2)
    o = oracle_for(w.snapshot, 4)
    o.merge(extra.peer, extra.tokens, extra.offsets)
    m_or, c_or = o.route(w.queries.tokens, w.queries.offsets, nthreads())
    assert_rows_equal(m1, c1, m_or, c_or, what="merged config 1")


def test_round_out_of_capacity_is_refused_and_repeated():
    """A merge round whose allocations do not fit the forest's spare capacity
    is refused (nothing written), the forest grows, and the round runs again.
    Compaction leaves a forest with 1/8 spare records; a fresh forest has no
    merge history to size its spare by, so one insert that rebuilds a block of
    20,000 children cannot fit.  The same batch also adds a second child to a
    small node and splits edges, whose allocations come after the refused one
    on the device counters and are refused too.  Every row against the oracle
    after each merge; the refusals show in the forest info."""
    import torch
    rng = np.random.default_rng(31)
    P = 3
    kids = np.sort(rng.choice(np.arange(0, 200000, 2), 20000, replace=False))
    seqs = [[7, int(t), 1, 2, 3] for t in kids] + [[9, 9, 9, 9, 9, 9]]
    owners = [i % P for i in range(len(seqs))]
    snap = W.from_lists(seqs, owners)
    f = _forest(snap, P)
    o = oracle_for(snap, P)
    qs = W.from_lists([list(s) for s in seqs[::97]] + [[7, int(kids[5]), 1, 2, 9], [7, 1], [9, 9, 9, 4], [9, 9]])
    gpu_route(f, qs, "refusal: upload")
    before, after = f.compact()
    assert after == before
    batches = [
        [(0, [7, 1, 5]), (1, [9, 9, 9, 4, 4]), (2, [7, int(kids[5]), 1, 2, 8, 8]), (1, [9, 9, 2])],
        [(2, [7, 3, 3]), (0, [7, int(kids[7]), 4]), (1, [9, 9, 9, 9, 9, 9, 9])],
    ]
    for k, items in enumerate(batches):
        peers = np.array([p for p, _ in items], np.int32)
        t, off = pins._csr([s for _, s in items])
        announce(f"refusal: merge batch {k}")
        f.merge(torch.from_numpy(peers).to(device()), torch.from_numpy(t).to(device()),
                torch.from_numpy(off).to(device()))
        o.merge(peers, t, off)
        torch.cuda.synchronize()
        q2 = W.from_lists([qs.seq(i).tolist() for i in range(len(qs))] + [s for _, s in items])
        m, c = gpu_route(f, q2, f"refusal: after batch {k}")
        m_or, c_or = o.route(q2.tokens, q2.offsets, nthreads())
        assert_rows_equal(m, c, m_or, c_or, what=f"refusal batch {k}")
        if k == 0:
            assert f.info()["merge_refusals"] >= 1, f.info()
    f.check()
    f.close()
    o.close()


def _merge_lists(f, o, items, label):
    """Merge (peer, sequence) pairs into the GPU forest and the oracle."""
    import torch
    peers = np.array([p for p, _ in items], np.int32)
    t, off = pins._csr([s for _, s in items])
    announce(f"{label}: merge of {len(items)} inserts")
    f.merge(torch.from_numpy(peers).to(device()), torch.from_numpy(t).to(device()),
            torch.from_numpy(off).to(device()))
    o.merge(peers, t, off)
    torch.cuda.synchronize()


def test_device_driven_rounds_hand_over_to_host_rounds():
    """After a forest's first merge, a merge runs two rounds sized on the
    device before it reads anything back; what they leave goes on in rounds
    the host reads back after every walk.  Three batches force each hand-over:
    a chain of inserts that share a new prefix and part from it one token
    after another (a slot, then the same edge over and over: more rounds than
    the device runs); more ADD entries in one round than the one-workgroup
    plan takes (the multi-launch path); and label tokens far beyond the pool's
    spare room after compaction (the device round's allocation is refused,
    the host grows the forest and repeats it).  Every row against the oracle
    after each merge; refusals show in the forest info."""
    rng = np.random.default_rng(41)
    P = 5
    seqs = [[3, 1, 4, 1, 5, 9, 2, 6][: 2 + i % 6] + [100 + i] for i in range(40)]
    owners = [i % P for i in range(len(seqs))]
    snap = W.from_lists(seqs, owners)
    f = _forest(snap, P)
    o = oracle_for(snap, P)

    def check(extra, label):
        q = W.from_lists([list(s) for s in seqs] + [list(s) for s in extra])
        m, c = gpu_route(f, q, label)
        m_or, c_or = o.route(q.tokens, q.offsets, nthreads())
        assert_rows_equal(m, c, m_or, c_or, what=label)

    first = [(1, [3, 1, 4, 7]), (2, [8, 8])]
    _merge_lists(f, o, first, "hand-over: first merge (host rounds)")
    check([s for _, s in first], "hand-over: after the first merge")
    chain = [(0, [50, 1, 2, 3, 4]), (1, [50, 1, 2, 3, 5]), (2, [50, 1, 2, 6]), (3, [50, 1, 7]),
             (4, [50, 1, 2, 3, 4, 8]), (0, [50, 1, 2, 9]), (1, [50, 2]), (2, [50, 1, 2, 3, 5, 5])]
    _merge_lists(f, o, chain, "hand-over: chain of cuts")
    check([s for _, s in chain] + [[50, 1, 2, 3], [50, 1, 2, 3, 4, 8, 1], [50]], "hand-over: after the chain")
    wide = [(int(i % P), [60000 + i, 7, 7]) for i in range(11000)]  # 11,000 ADD entries at the root
    _merge_lists(f, o, wide, "hand-over: round over the plan's size")
    check([s for _, s in wide[::50]] + [[60000 + 11000, 7]], "hand-over: after the wide round")
    refusals = f.info()["merge_refusals"]
    before, after = f.compact()
    long_rest = [(int(i % P), [70000 + i] + rng.integers(0, 1000, 300).tolist()) for i in range(600)]
    _merge_lists(f, o, long_rest, "hand-over: labels past the spare pool")
    check([s for _, s in long_rest[::13]], "hand-over: after the refused round")
    assert f.info()["merge_refusals"] > refusals, f.info()
    f.check()
    f.close()
    o.close()


def test_invalid_inserts_are_skipped_and_reported():
    import torch
    from paper_2606_17059_amd import RouterError
    dev = device()
    f = _forest(None, 3)
    toks = torch.tensor([1, 2, 3, 4, 5], dtype=torch.int32, device=dev)
    offs = torch.tensor([0, 2, 5, 4, 9, 5], dtype=torch.int64, device=dev)  # [0,2) [2,5) bad bad [9,5)bad
    peer = torch.tensor([0, 7, 1, 2, 0], dtype=torch.int32, device=dev)  # peer 7 out of range
    announce("invalid inserts")
    f.merge(peer, toks, offs)
    with pytest.raises(RouterError):
        f.check()
    f.check()  # the count was reset
    qs = W.from_lists([[1, 2, 3], [3, 4, 5]])
    m, c = gpu_route(f, qs, "after invalid inserts")
    assert m.tolist() == [[2, 0, 0], [0, 0, 0]]


def test_snapshot_load_after_merges():
    """Once merges ran, a snapshot load replaces the peer's tree on the device."""
    w = W.make_config(1, n_queries=300, prompts_per_peer=40)
    extra = W.make_config(1, seed_base=W.SEED_BASE + 4, n_queries=1, prompts_per_peer=30).snapshot
    f = _forest(w.snapshot, 4)
    o = oracle_for(w.snapshot, 4)
    _merge(f, extra, "before reload")
    o.merge(extra.peer, extra.tokens, extra.offsets)
    # peer 2 receives a new snapshot (the extra prompts of peer 3), peer 1 crashes
    lo, hi = extra.peer_range(3)
    t = extra.tokens[extra.offsets[lo]:extra.offsets[hi]]
    off = extra.offsets[lo:hi + 1] - extra.offsets[lo]
    for peer, tt, oo in ((2, t, off), (1, np.zeros(0, np.int32), np.zeros(1, np.int64))):
        announce(f"device load peer {peer}")
        f.load_snapshot(peer, tt, oo)
        o.load(peer, tt, oo)
        m, c = gpu_route(f, w.queries, f"after load of peer {peer}")
        m_or, c_or = o.route(w.queries.tokens, w.queries.offsets, nthreads())
        assert_rows_equal(m, c, m_or, c_or, what=f"load after merge, peer {peer}")
    # a merge after the reload still composes
    _merge(f, extra, "after reload")
    o.merge(extra.peer, extra.tokens, extra.offsets)
    m, c = gpu_route(f, w.queries, "after reload + merge")
    m_or, c_or = o.route(w.queries.tokens, w.queries.offsets, nthreads())
    assert_rows_equal(m, c, m_or, c_or, what="merge after reload")


def _stream_phases(w, dist, f, o, label, linear=None, linear_sample=0):
    """Each round: the merge batch into the GPU forest and into the oracle,
    then the round's lookups, every row compared; with ``linear`` also a
    sample against the linear-scan oracle."""
    for ph in w.phases(dist):
        _merge(f, ph.inserts, f"{label} {dist} round {ph.round}")
        o.merge(ph.inserts.peer, ph.inserts.tokens, ph.inserts.offsets)
        m, c = gpu_route(f, ph.queries, f"{label} {dist} round {ph.round}")
        assert_properties(m, c, ph.queries, f"{label} {dist} {ph.round}")
        announce(f"{label} {dist} round {ph.round}: oracle, every row")
        m_or, c_or = o.route(ph.queries.tokens, ph.queries.offsets, nthreads())
        assert_rows_equal(m, c, m_or, c_or, what=f"{label} {dist} {ph.round} every row")
        if linear is not None:
            linear.merge(ph.inserts.peer, ph.inserts.tokens, ph.inserts.offsets)
            idx = np.unique(np.random.default_rng(ph.round).choice(len(ph.queries), linear_sample, replace=False))
            m_ls, c_ls = linear.route_seqset(ph.queries, idx, nthreads())
            assert_rows_equal(m, c, m_ls, c_ls, idx, f"{label} {dist} {ph.round} linear-scan sample")
        # the inserted prompts now match their replicas in full
        k = min(64, len(ph.inserts))
        sub = ph.inserts.subset(np.arange(k))
        mi, _ = gpu_route(f, sub, "inserts as queries")
        assert np.array_equal(mi[np.arange(k), sub.peer], sub.lengths())


def test_stream_config_small():
    w = W.make_config(5, prompts_per_peer=30, rounds=2, phase_queries=3000, phase_inserts=1500)
    for dist in ("uniform", "zipf"):
        f = _forest(w.snapshot, 128)
        o = oracle_for(w.snapshot, 128)
        _stream_phases(w, dist, f, o, "stream small")
        f.close()
        o.close()


@pytest.mark.timeout(1500)
def test_stream_config_full():
    """128 peers x 2,000 prompts; 4 rounds of (10,000 inserts, 1,048,576 lookups)
    per topic distribution; every lookup of every phase against the radix-tree
    oracle, 48 per phase against the linear scan."""
    announce("stream full: generating")
    w = W.make_config(5)
    for dist in ("uniform", "zipf"):
        f = _forest(w.snapshot, 128)
        r = radix_for(w.snapshot, 128)
        lin = oracle_for(w.snapshot, 128)
        _stream_phases(w, dist, f, r, "stream full", linear=lin, linear_sample=48)
        f.close()
        r.close()
        lin.close()
