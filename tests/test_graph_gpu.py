"""pr_route captured into a HIP graph (through torch.cuda.CUDAGraph) for a
serving loop of small batches: the launch reads its inputs from fixed
buffers, so each replay routes whatever batch was copied there.  Every
replay, with eager routes and host waits between them, must equal the eager
route of the same batch and the CPU oracle's."""
import numpy as np
import pytest

import workloads as W
from gpu_util import announce, assert_rows_equal, device, gpu_route, nthreads, oracle_for, radix_for, to_dev

pytestmark = pytest.mark.gpu


def _capture(fn):
    """fn() captured into a graph (after a warm-up run on a side stream)."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn(side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn(torch.cuda.current_stream())
    torch.cuda.synchronize()
    return g


def test_route_replayed_from_a_graph():
    import torch
    from paper_2606_17059_amd import Forest
    w = W.make_config(1)
    P = w.num_peers
    f = Forest(P)
    f.load_seqset(w.snapshot)
    dev = device()
    rng = np.random.default_rng(515)
    b = 64
    batches = [w.queries.subset(np.sort(rng.choice(len(w.queries), b, replace=False))) for _ in range(6)]
    cap = max(int(x.offsets[-1]) for x in batches)
    qt = torch.zeros(cap, dtype=torch.int32, device=dev)
    qo = torch.zeros(b + 1, dtype=torch.int64, device=dev)
    ml = torch.empty((b, P), dtype=torch.int32, device=dev)
    ch = torch.empty(b, dtype=torch.int32, device=dev)

    def fill(x):
        qt.zero_()
        qt[:int(x.offsets[-1])].copy_(torch.from_numpy(x.tokens))
        qo.copy_(torch.from_numpy(x.offsets))

    o = oracle_for(w.snapshot, P)
    # the first route builds and uploads the forest; capture needs it built
    fill(batches[0])
    f.route(qt, qo, ml, ch)
    torch.cuda.synchronize()
    announce(f"graph: capture pr_route on {b} queries")
    g = _capture(lambda st: f.route_launcher(qt, qo, ml, ch, stream=st)())
    for i, x in enumerate(batches):
        fill(x)
        announce(f"graph: replay {i}")
        ml.fill_(-7)
        ch.fill_(-7)
        g.replay()
        torch.cuda.synchronize()
        m, c = ml.cpu().numpy().copy(), ch.cpu().numpy().copy()
        m_ref, c_ref = gpu_route(f, x, f"eager reference of replay {i}")
        assert_rows_equal(m, c, m_ref, c_ref, what=f"graph replay {i}")
        m_or, c_or = o.route(x.tokens, x.offsets, 4)
        assert_rows_equal(m, c, m_or, c_or, what=f"graph replay {i} against the oracle")
    o.close()
    f.close()


def test_select_replayed_from_a_graph():
    """pr_route_select under capture, the eligibility words in a fixed buffer
    too: each replay takes the mask that buffer holds."""
    import torch
    import oracle as O
    from paper_2606_17059_amd import Forest, eligible_words
    w = W.make_config(1)
    P = w.num_peers
    f = Forest(P)
    f.load_seqset(w.snapshot)
    dev = device()
    x = w.queries.subset(np.arange(200))
    qt, qo = to_dev(x)
    nq = len(x)
    el = torch.zeros(1, dtype=torch.int64, device=dev)
    ml = torch.empty((nq, P), dtype=torch.int32, device=dev)
    b1 = torch.empty(nq, dtype=torch.int32, device=dev)
    b2 = torch.empty(nq, dtype=torch.int32, device=dev)
    f.route(qt, qo)
    torch.cuda.synchronize()
    announce("graph: capture pr_route_select")
    g = _capture(lambda st: f.route_select(qt, qo, el, 1, True, ml, b1, b2, stream=st))
    o = O.Oracle(P)
    import pins
    pins.load_all(o, w.snapshot, P)
    rng = np.random.default_rng(77)
    for i in range(5):
        mask = (rng.random(P) < 0.5).astype(np.uint8)
        el.copy_(torch.from_numpy(eligible_words(mask)))
        b1.fill_(-7)
        b2.fill_(-7)
        announce(f"graph: select replay {i} eligible={mask.tolist()}")
        g.replay()
        torch.cuda.synchronize()
        m_or, b1_or, b2_or = o.route_select(x.tokens, x.offsets, mask, 1, True, 2)
        assert np.array_equal(ml.cpu().numpy(), m_or), i
        assert np.array_equal(b1.cpu().numpy(), b1_or), i
        assert np.array_equal(b2.cpu().numpy(), b2_or), i
    o.close()
    f.close()


@pytest.mark.timeout(600)
def test_long_batch_captured_in_index_order():
    """A batch that an eager route takes longest first is captured in index
    order (no order buffer, event or wait under capture): same rows, which
    equal the radix-tree oracle's."""
    import torch
    from test_route_gpu import _forest, _long_batch, _long_forest
    rng = np.random.default_rng(808)
    P = 8
    snap, prefixes = _long_forest(rng, P)
    x = _long_batch(rng, prefixes, 8192 + 40, 4096, 6000)
    f = _forest(snap, P)
    m_ref, c_ref = gpu_route(f, x, "eager, longest first")
    o = radix_for(snap, P)
    m_or, c_or = o.route(x.tokens, x.offsets, nthreads())
    o.close()
    assert_rows_equal(m_ref, c_ref, m_or, c_or, what="long batch, eager route against the oracle")
    qt, qo = to_dev(x)
    ml = torch.empty((len(x), P), dtype=torch.int32, device=device())
    ch = torch.empty(len(x), dtype=torch.int32, device=device())
    announce("graph: capture a long batch")
    g = _capture(lambda st: f.route_launcher(qt, qo, ml, ch, stream=st)())
    for i in range(2):
        ml.fill_(-7)
        g.replay()
        torch.cuda.synchronize()
        assert_rows_equal(ml.cpu().numpy(), ch.cpu().numpy(), m_ref, c_ref, what=f"long batch replay {i}")
    f.close()


@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")
def test_capture_refuses_a_forest_that_changed():
    """A host snapshot load leaves the device image stale; capturing a route
    before anything uploads it is refused (PR_ESTATE), and the capture stays
    valid (nothing was enqueued).  An eager route afterwards uploads and
    routes as usual."""
    import torch
    from paper_2606_17059_amd import Forest, RouterError
    w = W.make_config(1)
    P = w.num_peers
    f = Forest(P)
    f.load_seqset(w.snapshot)
    x = w.queries.subset(np.arange(50))
    qt, qo = to_dev(x)
    ml = torch.empty((len(x), P), dtype=torch.int32, device=device())
    ch = torch.empty(len(x), dtype=torch.int32, device=device())
    f.route(qt, qo, ml, ch)
    f.load_snapshot(0, np.zeros(0, np.int32), np.zeros(1, np.int64))
    torch.cuda.synchronize()
    announce("graph: capture on a changed forest (refused on the host)")
    g = torch.cuda.CUDAGraph()
    with pytest.raises(RouterError, match="graph capture"):
        with torch.cuda.graph(g):
            f.route_launcher(qt, qo, ml, ch, stream=torch.cuda.current_stream())()
    torch.cuda.synchronize()
    m, c = gpu_route(f, x, "eager route after the refused capture")
    assert (m[:, 0] == 0).all()
    f.close()


def test_layout_epoch_marks_moved_arrays():
    """Routes leave layout_epoch alone and a small merge that fits the spare
    capacity does too, so a graph captured before it replays on the merged
    forest; an upload after host loads and a compaction move the arrays and
    advance it."""
    import torch
    from paper_2606_17059_amd import Forest
    w = W.make_config(1)
    P = w.num_peers
    f = Forest(P)
    f.load_seqset(w.snapshot)
    assert f.info()["layout_epoch"] == 0  # nothing uploaded yet
    x = w.queries.subset(np.arange(100))
    qt, qo = to_dev(x)
    ml = torch.empty((len(x), P), dtype=torch.int32, device=device())
    ch = torch.empty(len(x), dtype=torch.int32, device=device())
    f.route(qt, qo, ml, ch)
    torch.cuda.synchronize()
    e1 = f.info()["layout_epoch"]
    assert e1 >= 1
    announce("graph: capture before a small merge")
    g = _capture(lambda st: f.route_launcher(qt, qo, ml, ch, stream=st)())
    assert f.info()["layout_epoch"] == e1
    # insert a few of the queries themselves into peer 2: their rows change
    ins = x.subset(np.arange(5))
    it, io = to_dev(ins)
    f.merge(torch.full((len(ins),), 2, dtype=torch.int32, device=device()), it, io)
    torch.cuda.synchronize()
    assert f.info()["layout_epoch"] == e1, "a merge within the spare capacity moved the arrays"
    ml.fill_(-7)
    g.replay()
    torch.cuda.synchronize()
    m, c = ml.cpu().numpy().copy(), ch.cpu().numpy().copy()
    m_ref, c_ref = gpu_route(f, x, "eager route after the merge")
    assert_rows_equal(m, c, m_ref, c_ref, what="replay after a merge in place")
    assert (m[:5, 2] == x.lengths()[:5]).all()
    del g
    f.compact()
    e2 = f.info()["layout_epoch"]
    assert e2 > e1
    f.load_snapshot(1, np.zeros(0, np.int32), np.zeros(1, np.int64))
    gpu_route(f, x, "route after a device load")
    assert f.info()["layout_epoch"] >= e2
    f.close()
