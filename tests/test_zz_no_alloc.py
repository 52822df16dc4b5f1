"""pr_route_noalloc, the route entry point that allocates nothing (for callers
that cannot allocate: code under HIP graph capture, tight serving loops), called
through the C ABI and compared with pr_route, the entry point it is a variant
of, and with the oracle.  Two long batches in a row, the second smaller, both
taken longest first, so that both use the library's static scratch array."""
import numpy as np
import pytest

import workloads as W
from gpu_util import announce, assert_rows_equal, device, nthreads, radix_for, to_dev

pytestmark = pytest.mark.gpu

_V = 50000


def _long_world(rng, P):
    prefixes = [rng.integers(0, _V, int(rng.integers(3000, 7000))).astype(np.int32) for _ in range(6)]
    seqs, owners = [], []
    for p in range(P):
        for _ in range(12):
            k = int(rng.integers(0, len(prefixes)))
            seqs.append(np.concatenate([prefixes[k], rng.integers(0, _V, int(rng.integers(1, 400))).astype(np.int32)]))
            owners.append(p)
    return W.from_lists([s.tolist() for s in seqs], owners), prefixes


def _long_queries(rng, prefixes, nq, lo, hi):
    qs = []
    for _ in range(nq):
        k = int(rng.integers(0, len(prefixes)))
        L = int(rng.integers(lo, hi))
        body = prefixes[k][:min(L, len(prefixes[k]))]
        qs.append(np.concatenate([body, rng.integers(0, _V, max(0, L - len(body))).astype(np.int32)]))
    lens = np.array([len(q) for q in qs], dtype=np.int64)
    offs = np.zeros(nq + 1, dtype=np.int64)
    offs[1:] = np.cumsum(lens)
    return W.SeqSet(np.concatenate(qs).astype(np.int32), offs, None)


def test_noalloc_route_matches_pr_route_and_oracle():
    import torch
    from paper_2606_17059_amd import Forest, RouterError
    from paper_2606_17059_amd import router as R
    rng = np.random.default_rng(2026)
    P = 8
    snap, prefixes = _long_world(rng, P)
    # both batches exceed the 8,192 wave slots and average over 4,096 tokens,
    # so both are walked longest first through the static scratch
    big = _long_queries(rng, prefixes, 9000, 4096, 6000)
    small = _long_queries(rng, prefixes, 8400, 4200, 5200)
    assert big.offsets[-1] >= 4096 * len(big) and small.offsets[-1] >= 4096 * len(small)
    f = Forest(P)
    f.load_seqset(snap)
    dev = device()
    r = radix_for(snap, P)
    first = True
    outs = []
    for what, qs in (("9,000 queries", big), ("8,400 queries", small)):
        qt, qo = to_dev(qs)
        nq = len(qs)
        m_ref = torch.full((nq, P), -7, dtype=torch.int32, device=dev)
        c_ref = torch.full((nq,), -7, dtype=torch.int32, device=dev)
        if first:
            # the forest is not on the device yet: the variant refuses to upload it
            with pytest.raises(RouterError) as e:
                f.route_noalloc(qt, qo, m_ref, c_ref)
            assert e.value.status == R.PR_ESTATE
            first = False
        announce(f"noalloc: pr_route of {what}")
        f.route(qt, qo, m_ref, c_ref)
        torch.cuda.synchronize()
        m_na = torch.full((nq, P), -7, dtype=torch.int32, device=dev)
        c_na = torch.full((nq,), -7, dtype=torch.int32, device=dev)
        outs.append((qs, qt, qo, m_na, c_na, m_ref, c_ref))
    # the two no-alloc calls back to back on one stream, no host wait between
    announce("noalloc: pr_route_noalloc of 9,000 then 8,400 queries")
    for qs, qt, qo, m_na, c_na, _, _ in outs:
        f.route_noalloc(qt, qo, m_na, c_na)
    torch.cuda.synchronize()
    for qs, qt, qo, m_na, c_na, m_ref, c_ref in outs:
        m1, c1 = m_na.cpu().numpy(), c_na.cpu().numpy()
        assert_rows_equal(m1, c1, m_ref.cpu().numpy(), c_ref.cpu().numpy(), what=f"noalloc vs pr_route {len(qs)}")
        m_or, c_or = r.route(qs.tokens, qs.offsets, nthreads())
        assert_rows_equal(m1, c1, m_or, c_or, what=f"noalloc vs oracle {len(qs)}")
    # a small batch (index order, no scratch) and an empty one
    qs = big.subset(np.arange(37))
    qt, qo = to_dev(qs)
    m_na = torch.empty((37, P), dtype=torch.int32, device=dev)
    c_na = torch.empty(37, dtype=torch.int32, device=dev)
    announce("noalloc: 37 queries")
    f.route_noalloc(qt, qo, m_na, c_na)
    torch.cuda.synchronize()
    m_or, c_or = r.route(qs.tokens, qs.offsets, 2)
    assert_rows_equal(m_na.cpu().numpy(), c_na.cpu().numpy(), m_or, c_or, what="noalloc 37 queries")
    # more queries than the scratch holds: refused on the host, nothing enqueued
    n_over = R.PR_NOALLOC_MAX_QUERIES + 1
    qo_over = torch.zeros(n_over + 1, dtype=torch.int64, device=dev)
    with pytest.raises(RouterError) as e:
        f.route_noalloc(qt, qo_over, torch.empty((n_over, P), dtype=torch.int32, device=dev),
                        torch.empty(n_over, dtype=torch.int32, device=dev))
    assert e.value.status == R.PR_EINVAL
    f.check()
    f.close()
    r.close()
