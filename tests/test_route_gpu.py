"""Route parity on the GPU: the HIP path through the C ABI versus the CPU oracle.

Integer outputs, so the bar is bit-exact: every match length and every chosen
peer, on every row.  Small cases compare with the linear-scan oracle;
full-size workloads with the per-peer radix-tree oracle (itself pinned to the
linear scan), plus a sample with the linear scan so the two oracles agree at
full size too.
"""
import numpy as np
import pytest

import oracle
import pins
import workloads as W
from gpu_util import (announce, assert_properties, assert_rows_equal, device, gpu_route, nthreads,
                      oracle_for, radix_for, to_dev)

pytestmark = pytest.mark.gpu


def _forest(snapshot, P):
    from paper_2606_17059_amd import Forest
    f = Forest(P)
    f.load_seqset(snapshot)
    return f


def test_golden_examples_on_gpu():
    from paper_2606_17059_amd import Forest
    import torch
    dev = device()
    for ex in pins.parse_golden():
        if any(op[0] == "merge" for op in ex.ops):
            continue  # examples with merges run in the merge tests
        f = Forest(ex.peers)
        for op in ex.ops:
            if op[0] == "load":
                t, o = pins._csr(op[2])
                f.load_snapshot(op[1], t, o)
            else:
                _, q, m_exp, c_exp = op
                t, o = pins._csr([q])
                announce(f"golden {ex.name} q={q}")
                m, c = f.route(torch.from_numpy(t).to(dev), torch.from_numpy(o).to(dev))
                assert m.cpu().numpy()[0].tolist() == m_exp and int(c.cpu()[0]) == c_exp, (ex.name, q)
        f.close()


@pytest.mark.parametrize("vocab", [2, 3, 8])
def test_tiny_random_all_rows(vocab):
    for sd in range(16):
        P = [1, 2, 3, 5, 64, 65, 130][sd % 7]
        w = W.tiny_random(sd, num_peers=P, vocab=vocab, max_seqs=6 if P > 10 else 12, n_queries=67)
        f = _forest(w.snapshot, P)
        m, c = gpu_route(f, w.queries, f"tiny vocab={vocab} seed={sd} P={P}")
        o = oracle_for(w.snapshot, P)
        m_or, c_or = o.route(w.queries.tokens, w.queries.offsets, 2)
        assert_rows_equal(m, c, m_or, c_or, what=f"tiny vocab={vocab} seed={sd}")
        f.close()


def test_max_peers_1024():
    w = W.tiny_random(77, num_peers=1024, vocab=3, max_seqs=2, n_queries=40)
    f = _forest(w.snapshot, 1024)
    m, c = gpu_route(f, w.queries, "P=1024")
    o = oracle_for(w.snapshot, 1024)
    m_or, c_or = o.route(w.queries.tokens, w.queries.offsets, 2)
    assert_rows_equal(m, c, m_or, c_or, what="P=1024")


def test_config1_tiny_all_rows():
    w = W.make_config(1)
    f = _forest(w.snapshot, w.num_peers)
    m, c = gpu_route(f, w.queries, "config 1 tiny")
    o = oracle_for(w.snapshot, w.num_peers)
    m_or, c_or = o.route(w.queries.tokens, w.queries.offsets, nthreads())
    assert_rows_equal(m, c, m_or, c_or, what="config 1")


@pytest.mark.timeout(900)
def test_config2_medium_full_batch():
    """The medium workload's full batch (65,536 queries, 16 peers): every row
    against the radix-tree oracle, a sample and the ragged tail against the
    linear scan too."""
    w = W.make_config(2)
    f = _forest(w.snapshot, w.num_peers)
    m, c = gpu_route(f, w.queries, "config 2 medium full")
    assert_properties(m, c, w.queries, "config 2")
    r = radix_for(w.snapshot, w.num_peers)
    m_rx, c_rx = r.route(w.queries.tokens, w.queries.offsets, nthreads())
    r.close()
    assert_rows_equal(m, c, m_rx, c_rx, what="config 2 every row")
    rng = np.random.default_rng(2)
    idx = np.unique(np.concatenate([rng.choice(len(w.queries), 512, replace=False),
                                    np.arange(len(w.queries) - 37, len(w.queries))]))
    o = oracle_for(w.snapshot, w.num_peers)
    m_or, c_or = o.route_seqset(w.queries, idx, nthreads())
    assert_rows_equal(m, c, m_or, c_or, idx, "config 2 linear-scan sample")
    # determinism: a second launch gives identical bytes
    m2, c2 = gpu_route(f, w.queries, "config 2 medium repeat")
    assert np.array_equal(m, m2) and np.array_equal(c, c2)


def test_small_batches_ragged():
    """Batch sizes around the 4-waves-per-block boundary, several tiles."""
    w = W.make_config(2, n_queries=1031, prompts_per_peer=150)
    f = _forest(w.snapshot, w.num_peers)
    o = oracle_for(w.snapshot, w.num_peers)
    for n in (1, 2, 3, 4, 5, 7, 8, 9, 63, 64, 65, 1031):
        sub = w.queries.subset(np.arange(n))
        m, c = gpu_route(f, sub, f"ragged n={n}")
        m_or, c_or = o.route(sub.tokens, sub.offsets, nthreads())
        assert_rows_equal(m, c, m_or, c_or, what=f"ragged n={n}")


def test_edge_cases():
    import torch
    from paper_2606_17059_amd import Forest
    dev = device()
    f = Forest(5)
    # empty forest, empty query, ordinary query
    qs = W.from_lists([[], [1, 2, 3], [7]])
    m, c = gpu_route(f, qs, "empty forest")
    assert m.tolist() == [[0] * 5] * 3 and c.tolist() == [0, 0, 0]
    f.load_snapshot(3, np.array([1, 2, 3, 4], np.int32), np.array([0, 4]))
    f.load_snapshot(1, np.array([1, 2], np.int32), np.array([0, 2]))
    m, c = gpu_route(f, qs, "two peers loaded")
    assert m.tolist() == [[0] * 5, [0, 2, 0, 3, 0], [0] * 5] and c.tolist() == [0, 3, 0]
    # zero queries is a no-op
    e = torch.zeros(0, dtype=torch.int32, device=dev)
    mo, co = f.route(e, torch.zeros(1, dtype=torch.int64, device=dev))
    assert mo.shape == (0, 5)
    # offsets outside the token buffer or decreasing: row of -1, nothing read
    toks = torch.tensor([1, 2, 3], dtype=torch.int32, device=dev)
    offs = torch.tensor([0, 3, 2, 9, -1, 3], dtype=torch.int64, device=dev)
    announce("invalid offsets")
    m, c = f.route(toks, offs)
    m, c = m.cpu().numpy(), c.cpu().numpy()
    assert m[0].tolist() == [0, 2, 0, 3, 0] and c[0] == 3
    assert (m[1:] == -1).all() and (c[1:] == -1).all()
    f.close()


def test_reload_replaces_on_device():
    """A new snapshot replaces a peer's tree for the next route (the device
    image is rebuilt), and a duplicate load changes nothing."""
    w = W.make_config(1, n_queries=300, prompts_per_peer=50)
    f = _forest(w.snapshot, w.num_peers)
    m1, c1 = gpu_route(f, w.queries, "before reload")
    f.load_snapshot(1, np.zeros(0, np.int32), np.zeros(1, np.int64))  # peer 1 crashed
    m2, c2 = gpu_route(f, w.queries, "peer 1 emptied")
    assert (m2[:, 1] == 0).all()
    lo, hi = w.snapshot.peer_range(1)
    for _ in range(2):  # recovered, and the broadcast duplicated
        f.load_snapshot(1, w.snapshot.tokens[w.snapshot.offsets[lo]:w.snapshot.offsets[hi]],
                        w.snapshot.offsets[lo:hi + 1] - w.snapshot.offsets[lo])
    m3, c3 = gpu_route(f, w.queries, "peer 1 reloaded")
    assert np.array_equal(m1, m3) and np.array_equal(c1, c3)


def _sample(n, k, seed):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([rng.choice(n, min(k, n), replace=False), np.arange(max(0, n - 13), n)]))


@pytest.mark.timeout(1200)
def test_config3_stale_estimates_and_truth_full_batch():
    """64 peers, 262,144 queries: the estimated forest (stale replicas) and the
    true forest, every row of each against the radix-tree oracle; estimates
    never match more than the truth (Section "Stale trie estimates")."""
    announce("config 3: generating")
    w = W.make_config(3)
    out = {}
    for snap, what in ((w.snapshot, "est"), (w.true_snapshot, "true")):
        f = _forest(snap, w.num_peers)
        m, c = gpu_route(f, w.queries, f"config 3 {what} forest")
        f.close()
        assert_properties(m, c, w.queries, f"config 3 {what}")
        announce(f"config 3 {what}: radix oracle, every row")
        r = radix_for(snap, w.num_peers)
        m_rx, c_rx = r.route(w.queries.tokens, w.queries.offsets, nthreads())
        r.close()
        assert_rows_equal(m, c, m_rx, c_rx, what=f"config 3 {what} every row")
        out[what] = (m, c)
    (me, ce), (mt, _) = out["est"], out["true"]
    assert (me <= mt).all() and np.array_equal(me[:, 0], mt[:, 0])
    idx = _sample(len(w.queries), 64, 3)
    o = oracle_for(w.snapshot, w.num_peers)
    m_or, c_or = o.route_seqset(w.queries, idx, nthreads())
    o.close()
    assert_rows_equal(me, ce, m_or, c_or, idx, "config 3 est linear-scan sample")


@pytest.mark.timeout(900)
def test_config4_long_context_full_batch():
    """32 peers, 8K-33K-token shared prefixes, 32,768 queries: every row
    against the radix-tree oracle with nodes forced at every 16-token block
    (the workload's split granularity), a sample against the linear scan."""
    announce("config 4: generating")
    w = W.make_config(4)
    f = _forest(w.snapshot, w.num_peers)
    m, c = gpu_route(f, w.queries, "config 4 long")
    assert_properties(m, c, w.queries, "config 4")
    r = radix_for(w.snapshot, w.num_peers, split_block=16)
    m_rx, c_rx = r.route(w.queries.tokens, w.queries.offsets, nthreads())
    r.close()
    assert_rows_equal(m, c, m_rx, c_rx, what="config 4 every row")
    idx = _sample(len(w.queries), 256, 4)
    o = oracle_for(w.snapshot, w.num_peers)
    m_or, c_or = o.route_seqset(w.queries, idx, nthreads())
    assert_rows_equal(m, c, m_or, c_or, idx, "config 4 linear-scan sample")


def test_route_launcher_matches_oracle():
    """The pre-checked launcher (the timed loop's launch path) writes the same
    outputs as the oracle, call after call, on two query batches."""
    import torch
    w = W.make_config(1)
    P = w.num_peers
    f = _forest(w.snapshot, P)
    o = oracle_for(w.snapshot, P)
    m_or, c_or = o.route(w.queries.tokens, w.queries.offsets, nthreads())
    qt, qo = to_dev(w.queries)
    half = w.queries.subset(np.arange(len(w.queries) // 2))
    ht, ho = to_dev(half)
    nq, nh = len(w.queries), len(half)
    ml = torch.full((nq, P), -7, dtype=torch.int32, device=device())
    ch = torch.full((nq,), -7, dtype=torch.int32, device=device())
    mh = torch.full((nh, P), -7, dtype=torch.int32, device=device())
    chh = torch.full((nh,), -7, dtype=torch.int32, device=device())
    la = f.route_launcher(qt, qo, ml, ch)
    lb = f.route_launcher(ht, ho, mh, chh)
    announce("route launcher")
    for _ in range(3):
        la()
        lb()
    torch.cuda.synchronize()
    assert_rows_equal(ml.cpu().numpy(), ch.cpu().numpy(), m_or, c_or, what="launcher full batch")
    assert_rows_equal(mh.cpu().numpy(), chh.cpu().numpy(), m_or[:nh], c_or[:nh], what="launcher half batch")
    with pytest.raises(ValueError):
        f.route_launcher(qt, qo, mh, ch)
    f.close()
    o.close()


def test_deep_paths():
    """Every prefix of a 300-token sequence ends a stored sequence of some peer,
    so a walk passes 300 one-token edges whose peer sets change along the way;
    queries stop at every kind of point along it."""
    rng = np.random.default_rng(7)
    s = rng.integers(0, 5, 300).astype(np.int32)
    P = 4
    seqs, owners = [], []
    for L in range(1, 301):
        seqs.append(s[:L].tolist())
        owners.append(L % P if L % 7 else 0)
    snap = W.from_lists(seqs, owners)
    qs = [s.tolist(), s[:150].tolist(), s[:8].tolist(), s[:9].tolist(), []]
    for cut in (1, 7, 8, 9, 16, 17, 64, 65, 299):
        q = s.copy()
        q[cut] = (q[cut] + 1) % 5  # mismatch inside the walk
        qs.append(q.tolist())
    qs.append(s.tolist() + [1, 2, 3])  # longer than every stored sequence
    queries = W.from_lists(qs)
    f = _forest(snap, P)
    o = oracle_for(snap, P)
    m_or, c_or = o.route(queries.tokens, queries.offsets, 2)
    m, c = gpu_route(f, queries, "deep path")
    assert_rows_equal(m, c, m_or, c_or, what="deep path")
    f.close()


def test_invalid_offsets_between_valid_queries():
    """Queries with bad offsets get rows of -1 wherever they sit in a batch;
    their neighbours are routed normally."""
    import torch
    from paper_2606_17059_amd import Forest
    dev = device()
    f = Forest(3)
    f.load_snapshot(0, np.array([1, 2, 3, 4, 5], np.int32), np.array([0, 5]))
    f.load_snapshot(2, np.array([1, 2, 9], np.int32), np.array([0, 3]))
    toks = torch.tensor([1, 2, 3, 4, 1, 2, 9, 9], dtype=torch.int32, device=dev)
    # offsets 0,4,2,7,99 and 99,-1,3,8 give the queries [0,4) ok, [4,2) bad,
    # [2,7) ok, [7,99) bad, then [99,-1) bad, [-1,3) bad, [3,8) ok
    offs = [0, 4, 2, 7, 99, -1, 3, 8]
    exp_m = [[4, 0, 2], [-1] * 3, [0, 0, 0], [-1] * 3, [-1] * 3, [-1] * 3, [0, 0, 0]]
    exp_c = [0, -1, 0, -1, -1, -1, 0]
    o = torch.tensor(offs, dtype=torch.int64, device=dev)
    announce("invalid offsets between valid queries")
    m, c = f.route(toks, o)
    assert m.cpu().numpy().tolist() == exp_m and c.cpu().numpy().tolist() == exp_c
    f.close()


_LONG_VOCAB = 50000


def _long_forest(rng, P):
    """Six shared prefixes of 3,000-7,000 tokens; every peer holds twelve
    prompts, each one prefix plus a short suffix."""
    V = _LONG_VOCAB
    prefixes = [rng.integers(0, V, int(rng.integers(3000, 7000))).astype(np.int32) for _ in range(6)]
    seqs, owners = [], []
    for p in range(P):
        for j in range(12):
            k = int(rng.integers(0, len(prefixes)))
            seqs.append(np.concatenate([prefixes[k], rng.integers(0, V, int(rng.integers(1, 400))).astype(np.int32)]))
            owners.append(p)
    return W.from_lists([s.tolist() for s in seqs], owners), prefixes


def _long_batch(rng, prefixes, nq, lo, hi):
    """nq queries of lo..hi tokens, each a stored prefix (cut to the length)
    and fresh tokens; at least 4,096 tokens per query on average."""
    qs = []
    for i in range(nq):
        k = int(rng.integers(0, len(prefixes)))
        L = int(rng.integers(lo, hi))
        body = prefixes[k][:min(L, len(prefixes[k]))]
        qs.append(np.concatenate([body, rng.integers(0, _LONG_VOCAB, max(0, L - len(body))).astype(np.int32)]))
    lens = np.array([len(q) for q in qs], dtype=np.int64)
    assert lens.sum() >= 4096 * nq
    offs = np.zeros(nq + 1, dtype=np.int64)
    offs[1:] = np.cumsum(lens)
    return W.SeqSet(np.concatenate(qs).astype(np.int32), offs, None)


def _index_order_rows(f, queries, what):
    """Reference rows: the batch routed in pieces of at most 8,192 queries,
    which are taken in index order."""
    ms, cs = [], []
    for a in range(0, len(queries), 8192):
        sub = queries.subset(np.arange(a, min(a + 8192, len(queries))))
        m, c = gpu_route(f, sub, f"{what} index-order piece at {a}")
        ms.append(m)
        cs.append(c)
    return np.concatenate(ms), np.concatenate(cs)


@pytest.mark.timeout(600)
def test_longest_first_batches_on_two_streams():
    """The forest keeps one order buffer.  Three long batches routed back to
    back without a host wait, on two streams: the second, larger than the
    first, on another stream (the buffer grows once the first route is done
    with it), the third on the first stream again (it waits for the second
    route before reusing the buffer).  Each result equals its index-order
    reference."""
    import torch
    rng = np.random.default_rng(4242)
    P = 8
    snap, prefixes = _long_forest(rng, P)
    batches = [_long_batch(rng, prefixes, n, 4096, 6000) for n in (8192 + 8, 9000, 8192 + 300)]
    f = _forest(snap, P)
    dev = device()
    ins = [to_dev(b) for b in batches]
    outs = [(torch.empty((len(b), P), dtype=torch.int32, device=dev), torch.empty(len(b), dtype=torch.int32, device=dev))
            for b in batches]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    announce("longest-first: three long batches on two streams, no host wait between them")
    for i, st in enumerate((s1, s2, s1)):
        with torch.cuda.stream(st):
            f.route(ins[i][0], ins[i][1], outs[i][0], outs[i][1], stream=st)
    torch.cuda.synchronize()
    for i, b in enumerate(batches):
        m, c = outs[i][0].cpu().numpy(), outs[i][1].cpu().numpy()
        assert_properties(m, c, b, f"two streams, batch {i}")
        m_ref, c_ref = _index_order_rows(f, b, f"two streams, batch {i}")
        assert_rows_equal(m, c, m_ref, c_ref, what=f"two streams, batch {i}")
    f.close()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("nq,lo,hi", [(8192 + 77, 2048, 10240), (65536, 4096, 4400)])
def test_longest_first_order_batches(nq, lo, hi):
    """Batches with more queries than wave slots (8,192) and at least 4,096
    tokens per query on average are taken longest first through a permutation;
    every row must still land at its own index.  The same queries routed in
    batches of at most 8,192 (index order) give the reference rows, and a
    sample is checked against the oracle.  65,536 queries is the largest batch
    the order takes (sixteen workgroups of the counting sort)."""
    rng = np.random.default_rng(41 + nq)
    P = 8
    snap, prefixes = _long_forest(rng, P)
    queries = _long_batch(rng, prefixes, nq, lo, hi)
    f = _forest(snap, P)
    m, c = gpu_route(f, queries, "longest-first batch")
    assert_properties(m, c, queries, "longest-first batch")
    m_ref, c_ref = _index_order_rows(f, queries, "longest-first batch")
    assert_rows_equal(m, c, m_ref, c_ref, what="longest-first vs index order")
    o = oracle_for(snap, P)
    idx = np.unique(np.concatenate([rng.choice(nq, 200, replace=False), np.arange(nq - 5, nq)]))
    m_or, c_or = o.route_seqset(queries, idx, nthreads())
    assert_rows_equal(m, c, m_or, c_or, idx, "longest-first batch sample")
    o.close()
    f.close()


def test_launcher_keeps_its_forest():
    """A route launcher holds its forest: dropping every other reference does
    not free the forest under it; after an explicit close the launcher
    refuses to run instead of passing a freed handle to the library."""
    import gc

    import torch
    from paper_2606_17059_amd import Forest
    w = W.make_config(1)
    P = w.num_peers
    f = Forest(P)
    f.load_seqset(w.snapshot)
    x = w.queries.subset(np.arange(64))
    qt, qo = to_dev(x)
    ml = torch.empty((len(x), P), dtype=torch.int32, device=device())
    ch = torch.empty(len(x), dtype=torch.int32, device=device())
    launch = f.route_launcher(qt, qo, ml, ch)
    del f
    gc.collect()
    announce("launcher after its forest's last other reference went")
    launch()
    torch.cuda.synchronize()
    o = oracle_for(w.snapshot, P)
    m_or, c_or = o.route(x.tokens, x.offsets, 2)
    o.close()
    assert_rows_equal(ml.cpu().numpy(), ch.cpu().numpy(), m_or, c_or, what="launcher keeps its forest")
    launch.buffers[0].close()
    with pytest.raises(RuntimeError, match="closed"):
        launch()


def test_label_width_follows_the_tokens():
    """Routes read 16-bit labels while every label token fits in [0, 65535],
    16-bit labels plus a plane of bit 16 while every token fits in
    [0, 131071], and int32 labels otherwise, with identical results: a
    small-token forest starts at 16 bits, stays there through merges that grow
    its label pool (the narrow copy grows with it) and through compaction,
    goes to 17 bits when a merge brings a token of 70,000 (the layout epoch
    advances, since routes switch kernels), keeps them through compaction and
    a growth, and goes to 32 bits when a merge brings a token of 200,000; a
    forest uploaded with tokens up to 131,071 starts at 17 bits, one with a
    negative token at 32."""
    import torch
    rng = np.random.default_rng(616)
    P = 3
    w = W.tiny_random(7, num_peers=P, vocab=8, max_seqs=12, n_queries=150)
    f = _forest(w.snapshot, P)
    o = oracle_for(w.snapshot, P)
    queries = [w.queries.seq(i).tolist() for i in range(len(w.queries))]

    def check(what, bits):
        t, off = pins._csr(queries)
        m, c = gpu_route(f, W.SeqSet(t, off, None), what)
        m_or, c_or = o.route(t, off, 2)
        assert_rows_equal(m, c, m_or, c_or, what=what)
        info = f.info()
        assert info["label_bits"] == bits and info["label_token_bytes"] == (4 if bits == 32 else 2), (what, info)

    def merge(seqs, what):
        peers = np.array([int(rng.integers(0, P)) for _ in seqs], np.int32)
        t, off = pins._csr(seqs)
        announce(f"label width: merge {what}")
        f.merge(torch.from_numpy(peers).to(device()), torch.from_numpy(t).to(device()),
                torch.from_numpy(off).to(device()))
        o.merge(peers, t, off)
        torch.cuda.synchronize()

    check("uploaded", 16)
    pool0 = f.info()["pool_tokens"]
    # long small-token sequences: the label pool outgrows its spare capacity
    merge([rng.integers(0, 8, int(rng.integers(200, 400))).tolist() for _ in range(60)], "long small tokens")
    assert f.info()["pool_tokens"] > 2 * pool0 + 4096
    queries += [s[:150] for s in pins.csr_to_list(*o.export(0))[:20]]
    check("after growth", 16)
    f.compact()
    check("after compaction", 16)
    epoch = f.info()["layout_epoch"]
    merge([[1, 2, 70000, 3], [5, 70000], [1, 2, 65536, 65535, 131071]], "tokens of 65,536 to 131,071")
    assert f.info()["layout_epoch"] > epoch
    queries += [[1, 2, 70000, 3, 9], [5, 70000], [1, 2, 65536, 65535, 131071], [1, 2, 65536, 65535, 65535],
                [1, 2, 70000 - 65536], [5, 70000 + 65536], [1, 2, 0, 65535, 131071]]
    check("after tokens of up to 17 bits", 17)
    # 17-bit labels of every alignment against the bit words: sequences of
    # 1..300 tokens mixing both halves of the range, then a growth of the pool
    merge([(rng.integers(0, 2, L) * 65536 + rng.integers(0, 5, L)).tolist() for L in range(1, 300, 7)],
          "17-bit sequences of many lengths")
    queries += [s for s in pins.csr_to_list(*o.export(1))[:30]]
    queries += [[(x ^ 65536) if i == len(s) // 2 else x for i, x in enumerate(s)]
                for s in pins.csr_to_list(*o.export(2))[:30] if s]
    check("17-bit sequences", 17)
    f.compact()
    check("17 bits after compaction", 17)
    merge([rng.integers(0, 131072, int(rng.integers(500, 1500))).tolist() for _ in range(40)], "growth at 17 bits")
    check("17 bits after growth", 17)
    epoch = f.info()["layout_epoch"]
    merge([[1, 2, 200000, 3], [9, 9]], "a token of 200,000")
    assert f.info()["layout_epoch"] > epoch
    queries += [[1, 2, 200000, 3, 9], [1, 2, 200000 - 131072]]
    check("after a wide token", 32)
    f.close()
    o.close()

    for seqs, qs, bits in (([[3, 131071, 4], [3, 1, 65536]], [[3, 131071, 4, 4], [3, 1, 65536], [3, 1, 0], [3, 2]], 17),
                           ([[3, -1, 4], [3, 1]], [[3, -1, 4, 4], [3, 1], [3, 2]], 32)):
        snap = W.from_lists(seqs, [0, 1])
        g = _forest(snap, 2)
        og = oracle_for(snap, 2)
        t, off = pins._csr(qs)
        m, c = gpu_route(g, W.SeqSet(t, off, None), f"uploaded forest, {bits}-bit labels")
        m_or, c_or = og.route(t, off, 1)
        assert_rows_equal(m, c, m_or, c_or, what=f"uploaded forest, {bits}-bit labels")
        assert g.info()["label_bits"] == bits
        g.close()
        og.close()


def _wide_block_sets(rng, n_children, P):
    """Sequences under one node with n_children distinct next tokens: a shared
    3-token head, then one of n_children distinct tokens (even numbers, so that
    odd tokens fall between two children), then a short random tail; spread
    over P peers.  Also n_children sequences that start with distinct tokens,
    so the root's block is as wide."""
    kids = np.sort(rng.choice(np.arange(0, 8 * n_children, 2), n_children, replace=False)).astype(np.int64)
    head = [900001, 900002, 900003]
    seqs, owners = [], []
    for i, t in enumerate(kids.tolist()):
        tail = rng.integers(0, 4, int(rng.integers(0, 6))).tolist()
        seqs.append(head + [t] + tail)
        owners.append(i % P)
        seqs.append([t, 5] + tail)
        owners.append((i + 1) % P)
    return seqs, owners, kids, head


def _wide_block_queries(rng, seqs, kids, head):
    """Hits, misses between, below and above the children, and the tokens at
    and around the block's separator positions (rank k * n / 64)."""
    n = len(kids)
    qs = []
    for r in sorted({(k * n) // 64 for k in range(64)} | {n - 1}):
        for d in (-1, 0, 1):
            t = int(kids[r]) + d
            qs.append(head + [t, 0, 1])
            qs.append([t, 5, 0])
    for t in (int(kids[0]) - 2, int(kids[-1]) + 2, -5, 2 ** 31 - 1):
        qs.append(head + [t])
        qs.append([t, 5])
    # every child of the first, a middle and the last separator range, and the
    # odd tokens between them: hits and misses at every vector of the sub-range
    for k in (0, 31, 63):
        lo, hi = (k * n) // 64, n if k == 63 else ((k + 1) * n) // 64
        for r in range(lo, hi):
            qs.append(head + [int(kids[r])])
            qs.append([int(kids[r]) + 1, 5])
    for i in rng.choice(len(seqs), 300, replace=False).tolist():
        s = list(seqs[i])
        qs.append(s)
        qs.append(s + [7])
        if len(s) > 4:
            qs.append(s[:-1] + [s[-1] + 1])
    return qs


@pytest.mark.timeout(600)
@pytest.mark.parametrize("n_children", [4097, 5000, 20000, 70000])
def test_child_blocks_wider_than_4096(n_children):
    """Child blocks of more than 64 x 64 children take a 64-ary search after
    the separators (one step up to 64 x 64 x 64 children, two above), in the
    route's child locate and in the merge walk's.
    Built by a host load, and again by a load of half the sequences followed
    by merges of the other half (new children, extensions through the wide
    block, duplicates), then compacted; every row against the oracle."""
    import torch
    rng = np.random.default_rng(n_children)
    P = 3
    seqs, owners, kids, head = _wide_block_sets(rng, n_children, P)
    qs = W.from_lists(_wide_block_queries(rng, seqs, kids, head))
    snap = W.from_lists(seqs, owners)
    o = oracle_for(snap, P)
    m_or, c_or = o.route(qs.tokens, qs.offsets, nthreads())
    o.close()
    f = _forest(snap, P)
    m, c = gpu_route(f, qs, f"wide block {n_children}: host load")
    assert_rows_equal(m, c, m_or, c_or, what=f"wide block {n_children} host load")
    f.close()
    # half by host load, the rest (and extensions of the loaded half) by merges
    half = np.arange(0, len(seqs), 2)
    rest = np.arange(1, len(seqs), 2)
    g = _forest(snap.subset(half), P)
    gpu_route(g, qs.subset(np.arange(4)), "wide block: first upload")
    ext = [list(seqs[i]) + [int(rng.integers(0, 4))] for i in half[::3]]
    batches = [(np.array([owners[i] for i in rest], np.int32), [seqs[i] for i in rest]),
               (np.array([owners[i] for i in half[::3]], np.int32), ext),
               (np.array([owners[i] for i in rest[:500]], np.int32), [seqs[i] for i in rest[:500]])]
    og = oracle_for(snap.subset(half), P)
    for k, (peers, bseqs) in enumerate(batches):
        t, off = pins._csr(bseqs)
        announce(f"wide block {n_children}: merge batch {k} of {len(bseqs)}")
        g.merge(torch.from_numpy(peers).to(device()), torch.from_numpy(t).to(device()),
                torch.from_numpy(off).to(device()))
        og.merge(peers, t, off)
        m, c = gpu_route(g, qs, f"wide block {n_children}: after merge {k}")
        m_or, c_or = og.route(qs.tokens, qs.offsets, nthreads())
        assert_rows_equal(m, c, m_or, c_or, what=f"wide block {n_children} merge {k}")
    # compaction rebuilds the image, separators (both levels) included
    announce(f"wide block {n_children}: compaction")
    before, after = g.compact()
    assert after <= before
    m, c = gpu_route(g, qs, f"wide block {n_children}: after compaction")
    assert_rows_equal(m, c, m_or, c_or, what=f"wide block {n_children} compacted")
    g.check()
    g.close()
    og.close()


@pytest.mark.parametrize("bits", [16, 17])
def test_narrow_labels_with_query_tokens_out_of_range(bits):
    """While labels are read as 16- or 17-bit values, a query token outside
    their range, or equal to a label token in its low 16 bits only, must still
    differ from it: in the middle of a label, the label token k is replaced by
    k with bit 16 flipped, k + 131072, k - 65536, k + 2^31 (wrapped) and -1;
    the walk must stop there, as the oracle's int32 compare does."""
    rng = np.random.default_rng(99 + bits)
    P = 2
    top = 65536 if bits == 16 else 131072
    seqs = [rng.integers(0, top, int(rng.integers(40, 300))).tolist() for _ in range(30)]
    owners = [i % P for i in range(len(seqs))]
    snap = W.from_lists(seqs, owners)
    f = _forest(snap, P)
    qs = []
    for s in seqs:
        for pos in (0, 1, len(s) // 2, len(s) - 1):
            k = s[pos]
            for bad in (k ^ 65536, k + 131072, k - 65536, (k + 2 ** 31) % 2 ** 32 - 2 ** 31, -1):
                q = list(s)
                q[pos] = int(bad)
                qs.append(q)
        qs.append(list(s))
    queries = W.from_lists(qs)
    m, c = gpu_route(f, queries, f"narrow labels ({bits} bits), wide query tokens")
    assert f.info()["label_bits"] == bits
    o = oracle_for(snap, P)
    m_or, c_or = o.route(queries.tokens, queries.offsets, nthreads())
    assert_rows_equal(m, c, m_or, c_or, what="narrow labels, wide query tokens")
    o.close()
    f.close()


@pytest.mark.parametrize("vocab", [32000, 128256, 2 ** 31 - 1])
def test_wide_first_window(vocab):
    """A forest whose root has one child with a label of 256 tokens or more
    (a long shared system prompt) routes with the 256-token first-level
    window; results must not depend on it.  Queries end or mismatch at every
    vector edge of both windows, with 16-, 17- and 32-bit labels.  Merges then
    give the root a second child and cut its first label short of 256 tokens,
    so the forest keeps the wide window without its reason; routes must still
    equal the oracle's."""
    import torch
    rng = np.random.default_rng(vocab % 1000 + 7)
    P = 5
    head = rng.integers(0, vocab, 300).tolist()
    seqs, owners = [], []
    for i in range(40):
        seqs.append(head + rng.integers(0, vocab, int(rng.integers(0, 200))).tolist())
        owners.append(i % P)
    snap = W.from_lists(seqs, owners)
    f = _forest(snap, P)
    qs = [[]]
    cuts = (1, 2, 63, 64, 65, 127, 128, 129, 191, 192, 200, 255, 256, 257, 299, 300)
    for n in cuts:
        qs.append(head[:n])
        q = list(head)
        q[n - 1] = (q[n - 1] + 1) % vocab
        qs.append(q)
    qs += [list(s) for s in seqs[:10]]
    qs += [s[:len(head) + 5] + [(s[len(head) + 5] + 1) % vocab] if len(s) > len(head) + 5 else list(s)
           for s in seqs[10:20]]
    queries = W.from_lists(qs)
    m, c = gpu_route(f, queries, f"wide first window, vocab {vocab}")
    info = f.info()
    assert info["first_window_tokens"] == 256, info
    o = oracle_for(snap, P)
    m_or, c_or = o.route(queries.tokens, queries.offsets, nthreads())
    assert_rows_equal(m, c, m_or, c_or, what="wide first window")
    # merges: a sequence with another first token, and one leaving the head at 100
    alt = [(head[0] + 1) % vocab] + rng.integers(0, vocab, 50).tolist()
    cut = head[:100] + [(head[100] + 1) % vocab] + rng.integers(0, vocab, 30).tolist()
    ins = W.from_lists([alt, cut], [1, 3])
    dev = device()
    announce(f"wide first window: merge of {len(ins)} inserts")
    f.merge(torch.from_numpy(ins.peer).to(dev), torch.from_numpy(ins.tokens).to(dev),
            torch.from_numpy(ins.offsets).to(dev))
    o.merge(ins.peer, ins.tokens, ins.offsets)
    q2 = W.from_lists(qs + [alt, cut, cut[:101], alt[:1]])
    m, c = gpu_route(f, q2, "wide first window after merges")
    assert f.info()["first_window_tokens"] == 256
    m_or, c_or = o.route(q2.tokens, q2.offsets, nthreads())
    assert_rows_equal(m, c, m_or, c_or, what="wide first window after merges")
    f.check()
    o.close()
    f.close()


def test_narrow_first_window_for_short_root_labels():
    """A root with a single child whose label is shorter than 256 tokens, or
    with several children, keeps the 128-token window."""
    rng = np.random.default_rng(5)
    head = rng.integers(0, 1000, 200).tolist()
    snap = W.from_lists([head + [1, 2], head + [3]], [0, 1])
    f = _forest(snap, 2)
    q = W.from_lists([head + [1, 2, 9]])
    m, c = gpu_route(f, q, "short root label")
    assert f.info()["first_window_tokens"] == 128
    assert m.tolist() == [[len(head) + 2, len(head)]] and c.tolist() == [0]
    f.close()
    snap = W.from_lists([[1] + head + [5] * 300, [2] + head + [5] * 300], [0, 1])
    f = _forest(snap, 2)
    q = W.from_lists([[2] + head])
    m, c = gpu_route(f, q, "two root children")
    assert f.info()["first_window_tokens"] == 128
    assert m.tolist() == [[0, len(head) + 1]] and c.tolist() == [1]
    f.close()


@pytest.mark.timeout(600)
def test_child_block_past_the_second_separator_level():
    """A block of 270,000 children: its sub-ranges of about 4,219 first tokens
    leave second-level ranges of 66 children, which take one step of the
    64-ary search; every child of two sub-ranges, the odd tokens between them
    and the block's ends, by host load and after a merge, against the
    radix-tree oracle."""
    import torch
    rng = np.random.default_rng(270000)
    n = 270000
    P = 2
    kids = np.sort(rng.choice(np.arange(0, 4 * n, 2), n, replace=False)).astype(np.int64)
    head = [77, 78]
    seqs = [head + [int(t), 9] for t in kids.tolist()]
    owners = [i % P for i in range(n)]
    snap = W.from_lists(seqs, owners)
    qs = []
    for k in (5, 63):
        lo, hi = (k * n) // 64, n if k == 63 else ((k + 1) * n) // 64
        for r in range(lo, hi):
            qs.append(head + [int(kids[r]), 9])
            qs.append(head + [int(kids[r]) + 1])
    qs += [head + [int(kids[0]) - 1], head + [int(kids[-1]) + 1], head + [int(kids[0])], head]
    queries = W.from_lists(qs)
    o = radix_for(snap, P)
    m_or, c_or = o.route(queries.tokens, queries.offsets, nthreads())
    f = _forest(snap, P)
    m, c = gpu_route(f, queries, "block of 270,000 children: host load")
    assert_rows_equal(m, c, m_or, c_or, what="270,000 children, host load")
    # a merge rebuilds the block (new children between the old ones)
    new = [head + [int(t) + 1, 4] for t in kids[::97].tolist()]
    ins = W.from_lists(new, [1] * len(new))
    announce(f"block of 270,000 children: merge of {len(ins)}")
    dev = device()
    f.merge(torch.from_numpy(ins.peer).to(dev), torch.from_numpy(ins.tokens).to(dev),
            torch.from_numpy(ins.offsets).to(dev))
    o.merge(ins.peer, ins.tokens, ins.offsets)
    q2 = W.from_lists(qs + new[:2000])
    m, c = gpu_route(f, q2, "block of 270,000 children after a merge")
    m_or, c_or = o.route(q2.tokens, q2.offsets, nthreads())
    assert_rows_equal(m, c, m_or, c_or, what="270,000 children after a merge")
    f.check()
    o.close()
    f.close()


@pytest.mark.parametrize("P", [32, 96, 160])
def test_rows_of_whole_lines_with_a_partial_mask_word(P):
    """Rows of P a multiple of 32 are stored non-temporally through a buffer
    range of the row; with P = 96 or 160 the last mask word is only partly
    used, and its lanes past the row must store nothing (the next row is
    another query's).  Every row against the oracle, also through the route
    without allocation."""
    import torch
    for sd in range(3):
        w = W.tiny_random(sd, num_peers=P, vocab=3, max_seqs=4, n_queries=131)
        f = _forest(w.snapshot, P)
        m, c = gpu_route(f, w.queries, f"rows of whole lines P={P} seed={sd}")
        o = oracle_for(w.snapshot, P)
        m_or, c_or = o.route(w.queries.tokens, w.queries.offsets, 2)
        assert_rows_equal(m, c, m_or, c_or, what=f"P={P} seed={sd}")
        qt, qo = to_dev(w.queries)
        ml = torch.full((len(w.queries), P), -7, dtype=torch.int32, device=device())
        ch = torch.full((len(w.queries),), -7, dtype=torch.int32, device=device())
        announce(f"rows of whole lines P={P} seed={sd}: route without allocation")
        f.route_noalloc(qt, qo, ml, ch)
        torch.cuda.synchronize()
        assert_rows_equal(ml.cpu().numpy(), ch.cpu().numpy(), m_or, c_or, what=f"P={P} seed={sd} noalloc")
        o.close()
        f.close()


def test_route_without_allocation_on_the_wide_first_window():
    """pr_route_noalloc on a forest that takes the 256-token first window:
    every row equals pr_route's and the oracle's."""
    import torch
    rng = np.random.default_rng(2561)
    V = 128256
    head = rng.integers(0, V, 280).tolist()
    seqs = [head + rng.integers(0, V, int(rng.integers(0, 90))).tolist() for _ in range(40)]
    snap = W.from_lists(seqs, [i % 4 for i in range(40)])
    qs = [head[:n] for n in (5, 128, 255, 256, 257, 280)]
    qs += [s[:k] + [(s[k] + 1) % V] for s in seqs[:20] for k in (100, 260) if k < len(s)]
    qs += [list(s) for s in seqs[20:]]
    queries = W.from_lists(qs)
    f = _forest(snap, 4)
    m, c = gpu_route(f, queries, "wide first window: pr_route")
    assert f.info()["first_window_tokens"] == 256
    qt, qo = to_dev(queries)
    ml = torch.full((len(queries), 4), -7, dtype=torch.int32, device=device())
    ch = torch.full((len(queries),), -7, dtype=torch.int32, device=device())
    announce("wide first window: route without allocation")
    f.route_noalloc(qt, qo, ml, ch)
    torch.cuda.synchronize()
    assert_rows_equal(ml.cpu().numpy(), ch.cpu().numpy(), m, c, what="noalloc against pr_route")
    o = oracle_for(snap, 4)
    m_or, c_or = o.route(queries.tokens, queries.offsets, 2)
    assert_rows_equal(m, c, m_or, c_or, what="wide window against the oracle")
    o.close()
    f.close()
