"""The union-forest layout built by the library's host code, checked on the CPU.

A plain-Python reader walks the flattened image exactly as the layout's
contract says (child slots sorted by first token, peer masks uniform along
edges) and must reproduce the oracle's match lengths.  Structural invariants of
the image are checked too.  No GPU is touched: the image comes from
pr_forest_host_image.
"""
import numpy as np
import pytest

import oracle
import pins
import workloads as W

pytest.importorskip("ctypes")
from paper_2606_17059_amd import router as R  # noqa: E402


def _mask_int(row):
    v = 0
    for w, x in enumerate(row.tolist()):
        v |= int(x) << (64 * w)
    return v


def walk(img, P, q):
    """Walk the image as the layout contract states: the children of node x are
    ids [ct_beg, ct_beg + ct_cnt) sorted by first token; masks are uniform
    along each edge."""
    nodes, masks, pool = img["nodes"], img["masks"], img["pool"]
    alive = (1 << P) - 1
    m = [0] * P
    d, x = 0, 0
    q = [int(t) for t in q]
    while d < len(q) and nodes[x, 4] > 0:
        beg, cnt = int(nodes[x, 3]), int(nodes[x, 4])
        toks = nodes[beg:beg + cnt, 0]
        j = int(np.searchsorted(toks, q[d]))
        if j >= cnt or int(toks[j]) != q[d]:
            break
        c = beg + j
        nm = alive & _mask_int(masks[c])
        dead = alive & ~nm
        for p in range(P):
            if (dead >> p) & 1:
                m[p] = d
        alive = nm
        if not alive:
            break
        off, ln = int(np.uint32(nodes[c, 1])), int(nodes[c, 2])
        lab = pool[off:off + ln].tolist()
        l = 0
        while l < ln and d + l < len(q) and lab[l] == q[d + l]:
            l += 1
        d += l
        if l < ln:
            break
        x = c
    for p in range(P):
        if (alive >> p) & 1:
            m[p] = d
    return m


def check_structure(img, P):
    nodes, masks, pool, ntok = img["nodes"], img["masks"], img["pool"], img["ntok"]
    n = nodes.shape[0]
    assert nodes[0, 2] == 0  # root label empty
    assert np.array_equal(ntok, nodes[:, 0])
    parents = np.zeros(n, dtype=np.int64)
    for x in range(n):
        beg, cnt = int(nodes[x, 3]), int(nodes[x, 4])
        toks = nodes[beg:beg + cnt, 0]
        assert (np.diff(toks.astype(np.int64)) > 0).all(), "child blocks must be strictly sorted"
        mx = _mask_int(masks[x])
        for c in range(beg, beg + cnt):
            parents[c] += 1
            assert nodes[c, 2] >= 1
            assert int(pool[int(np.uint32(nodes[c, 1]))]) == int(nodes[c, 0]), "tok = label's first token"
            mc = _mask_int(masks[c])
            assert mc & ~mx == 0, "a child's peers are a subset of its parent's"
        if x != 0 and cnt == 1:
            assert _mask_int(masks[beg]) != mx, "single-child chains with equal masks are compressed"
        if cnt > 64:  # separators of wide blocks
            seps = img["nsep"][beg:beg + 64]
            want = ntok[beg + (np.arange(64) * cnt) // 64]
            assert np.array_equal(seps, want), "separators of a wide child block"
        if cnt >= 64 + 64 * 64:  # second-level separators, per sub-range
            for k in range(64):
                lo, hi = (k * cnt) // 64, cnt if k == 63 else ((k + 1) * cnt) // 64
                got = img["nsep"][beg + 64 + 64 * k:beg + 128 + 64 * k]
                want = ntok[beg + lo + (np.arange(64) * (hi - lo)) // 64]
                assert np.array_equal(got, want), "second-level separators of a wide child block"
        assert mx >> P == 0
    assert parents[0] == 0 and (parents[1:] == 1).all(), "every non-root node has one parent"


def build_forest(w, snapshot=None):
    f = R.Forest(w.num_peers)
    f.load_seqset(snapshot if snapshot is not None else w.snapshot)
    return f


def _compare(w, idx=None, snapshot=None):
    f = build_forest(w, snapshot)
    img = f.host_image()
    check_structure(img, w.num_peers)
    o = oracle.Oracle(w.num_peers)
    pins.load_all(o, snapshot if snapshot is not None else w.snapshot, w.num_peers)
    qs = w.queries if idx is None else w.queries.subset(idx)
    m_or, c_or = o.route(qs.tokens, qs.offsets, 4)
    for i in range(len(qs)):
        m = walk(img, w.num_peers, qs.seq(i))
        assert m == m_or[i].tolist(), f"query {i}: image walk {m} != oracle {m_or[i].tolist()}"
    f.close()


@pytest.mark.parametrize("vocab", [2, 3, 8])
def test_tiny_random_images(vocab):
    for sd in range(10):
        w = W.tiny_random(sd, num_peers=2 + sd % 5, vocab=vocab, n_queries=40)
        _compare(w)


def test_many_peers_mask_words():
    # 130 peers -> 4 mask words (3 used); peers share sequences heavily
    w = W.tiny_random(5, num_peers=130, vocab=3, max_seqs=3, n_queries=60)
    _compare(w)


def test_wide_blocks_carry_separators():
    """Blocks of more than 64 children carry separators, and blocks of 4,160
    children or more a second level of them per sub-range."""
    rng = np.random.default_rng(11)
    for n_children in (65, 100, 513, 4097, 4159, 4160, 5000, 70000):
        first = rng.choice(np.arange(-200000, 200000), size=n_children, replace=False)
        seqs = [[int(a), int(rng.integers(0, 9))] for a in first]
        ss = W.from_lists(seqs, sorted(int(rng.integers(0, 3)) for _ in seqs))
        w = W.Workload(0, "wide", 3, 0, ss, W.from_lists([[int(first[0]), 1], [int(first[-1])], [7777777]]))
        _compare(w)


def test_config1_image():
    w = W.make_config(1)
    _compare(w, idx=np.arange(0, 2048, 8))


def test_config3_small_image_estimates_and_truth():
    w = W.make_config(3, n_queries=48, prompts_per_peer=12)
    _compare(w)
    _compare(w, snapshot=w.true_snapshot)


def test_snapshot_replace_and_duplicate_load():
    w = W.make_config(1, n_queries=64, prompts_per_peer=20)
    f = build_forest(w)
    a = f.host_image()
    # loading the same snapshot again is a no-op (a duplicated broadcast)
    lo, hi = w.snapshot.peer_range(2)
    f.load_snapshot(2, w.snapshot.tokens[w.snapshot.offsets[lo]:w.snapshot.offsets[hi]],
                    w.snapshot.offsets[lo:hi + 1] - w.snapshot.offsets[lo])
    b = f.host_image()
    for k in ("nodes", "masks", "ntok", "pool"):
        assert np.array_equal(a[k], b[k])
    # an empty snapshot (crashed peer) removes that peer everywhere
    f.load_snapshot(2, np.zeros(0, np.int32), np.zeros(1, np.int64))
    c = f.host_image()
    assert all(((int(r[0]) >> 2) & 1) == 0 for r in c["masks"])
    f.close()


def test_abi_errors_without_gpu():
    f = R.Forest(3)
    with pytest.raises(R.RouterError) as e:
        f.load_snapshot(3, np.zeros(1, np.int32), np.array([0, 1]))
    assert e.value.status == R.PR_EINVAL
    with pytest.raises(R.RouterError):
        f.load_snapshot(0, np.zeros(2, np.int32), np.array([0, 2, 1]))
    with pytest.raises(R.RouterError):
        f.load_snapshot(0, np.zeros(2, np.int32), np.array([1, 2]))
    with pytest.raises(R.RouterError):
        R.pr_forest_create(0)
    with pytest.raises(R.RouterError):
        R.pr_forest_create(R.PR_MAX_PEERS + 1)
    assert f.info()["num_peers"] == 3
    f.close()
