"""Every forest operation in one random sequence on the GPU, checked against
the CPU oracle after each step: host and device snapshot loads, merges,
touches, evictions, compaction, export, tree token counts, routing and peer
selection with random eligibility.

Half of the seeds draw first tokens from 150 values, so merges grow the root's
child block past 64 children (the width at which it needs separators) while
routing runs between them; the others use a vocabulary of 2-4 tokens, so edges
split at every depth.  5, 65, 130 and 1,024 peers run the route kernel's
one-, two-, four- and sixteen-word peer-mask forms.
"""
import numpy as np
import pytest

import pins
import workloads as W
from gpu_util import announce, assert_rows_equal, device, gpu_route
from test_compact_gpu import _compact
from test_lru_gpu import Both

pytestmark = pytest.mark.gpu


def _select_check(b, queries, rng, what):
    import torch
    from paper_2606_17059_amd import eligible_words
    P = b.P
    el = (rng.random(P) < rng.choice([0.0, 0.3, 0.9])).astype(np.uint8)
    local = int(rng.integers(-1, P))
    prefer = bool(rng.integers(0, 2))
    t, off = pins._csr(queries)
    dev = device()
    announce(f"mixed select {what}: local={local} prefer={prefer} eligible={int(el.sum())}/{P}")
    m, b1, b2 = b.f.route_select(torch.from_numpy(t).to(dev), torch.from_numpy(off).to(dev),
                                 torch.from_numpy(eligible_words(el)).to(dev), local, prefer)
    torch.cuda.synchronize()
    m_or, b1_or, b2_or = b.o.route_select(t, off, el, local, prefer, 2)
    assert np.array_equal(m.cpu().numpy(), m_or), (what, "match lengths")
    assert np.array_equal(b1.cpu().numpy(), b1_or), (what, "best")
    assert np.array_equal(b2.cpu().numpy(), b2_or), (what, "second")


def _root_width(b):
    """Children of the root: distinct first tokens over every peer's tree."""
    return len({int(t[o]) for p in range(b.P) for t, off in [b.o.export(p)] for o in off[:-1]
                if off[-1] > o})


def _device_load(b, p, seqs):
    import torch
    t, off = pins._csr(seqs)
    dev = device()
    announce(f"mixed device load peer {p}: {len(seqs)} sequences")
    b.f.load_snapshot_device(p, torch.from_numpy(t).to(dev), torch.from_numpy(off).to(dev))
    b.o.load(p, t, off)


@pytest.mark.parametrize("seed", range(8))
def test_mixed_operations(seed):
    rng = np.random.default_rng(9300 + seed)
    P = {6: 65, 7: 1024}.get(seed, 130 if seed % 3 == 2 else 5)
    wide = seed % 2 == 0
    vocab = 2 + seed % 3

    def seq(lo=1, hi=9):
        n = int(rng.integers(lo, hi))
        if n == 0:
            return []
        first = int(rng.integers(0, 150 if wide else vocab))
        return [first] + rng.integers(0, vocab, size=n - 1).tolist()

    def seqs(k, lo=1, hi=9):
        return [seq(lo, hi) for _ in range(k)]

    local = int(rng.integers(0, P))
    b = Both(P, local)
    t = 1
    b.time(t)
    for p in range(P):  # the root starts with fewer than 64 children
        if rng.random() < (0.5 if P < 64 else 0.2 if P < 1000 else 0.03):
            b.load(p, seqs(int(rng.integers(0, 5))))
    queries = seqs(40, 0, 11)
    widths = []
    for step in range(24):
        what = f"seed={seed} step={step}"
        t += int(rng.integers(0, 3))
        b.time(t)
        op = rng.choice(["merge", "merge", "touch", "evict", "load", "device_load", "compact"])
        announce(f"mixed {what}: {op}")
        if op == "merge":
            b.merge([(int(rng.integers(0, P)), s) for s in seqs(int(rng.integers(1, 40)))])
        elif op == "touch":
            b.touch([queries[i] for i in rng.integers(0, len(queries), size=6)])
        elif op == "evict":
            g, o = b.evict(int(rng.integers(1, 12)))
            assert g == o, (what, g, o)
        elif op == "load":
            b.load(int(rng.integers(0, P)), seqs(int(rng.integers(0, 8))))
        elif op == "device_load":
            _device_load(b, int(rng.integers(0, P)), seqs(int(rng.integers(0, 8))))
        else:
            _compact(b.f, what)
        if step % 4 == 3 or step == 23:
            b.check(queries, what)
            b.f.check()
        else:
            tq, oq = pins._csr(queries)
            m, c = gpu_route(b.f, W.SeqSet(tq, oq, np.zeros(len(queries), np.int32)), what)
            m_or, c_or = b.o.route(tq, oq, 2)
            assert_rows_equal(m, c, m_or, c_or, what=what)
        _select_check(b, queries, rng, what)
        widths.append(_root_width(b))
    if wide:  # the root's block was routed both narrower and wider than 64 children
        assert min(widths) <= 64 < max(widths), widths
    b.f.close()
