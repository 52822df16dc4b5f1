"""The round structure of the device batch insert, modelled in plain Python on
the flattened layout and checked against the oracle (no GPU)."""
import numpy as np
import pytest

import oracle
import pins
import workloads as W
from merge_model import FlatForest
from paper_2606_17059_amd import router as R


def _seqs(ss):
    return [ss.seq(i).tolist() for i in range(len(ss))]


@pytest.mark.parametrize("vocab", [2, 3, 8])
def test_model_merges_match_oracle(vocab):
    for sd in range(10):
        P = [1, 3, 5, 70][sd % 4]
        base = W.tiny_random(sd, num_peers=P, vocab=vocab, max_seqs=6 if P < 10 else 1, n_queries=50)
        f = R.Forest(P)
        if sd % 3:
            f.load_seqset(base.snapshot)
        model = FlatForest(f.host_image(), P)
        f.close()
        o = oracle.Oracle(P)
        if sd % 3:
            pins.load_all(o, base.snapshot, P)
        for r in range(3):
            ins = W.tiny_random(1000 * sd + r, num_peers=P, vocab=vocab, max_seqs=max(1, 20 // P),
                                n_queries=1).snapshot
            model.merge(_seqs(ins), ins.peer.tolist())
            o.merge(ins.peer, ins.tokens, ins.offsets)
            m_or, _ = o.route(base.queries.tokens, base.queries.offsets, 1)
            for i in range(len(base.queries)):
                assert model.route(base.queries.seq(i).tolist()) == m_or[i].tolist(), (vocab, sd, r, i)
        if P > 1:  # a snapshot replaced after merges: clear the peer, insert the new set
            new = W.tiny_random(77 + sd, num_peers=1, vocab=vocab, max_seqs=6, n_queries=1).snapshot
            model.clear_peer(1)
            model.merge(_seqs(new), [1] * len(new))
            o.load(1, new.tokens, new.offsets)
            m_or, _ = o.route(base.queries.tokens, base.queries.offsets, 1)
            for i in range(len(base.queries)):
                assert model.route(base.queries.seq(i).tolist()) == m_or[i].tolist(), (vocab, sd, "reload", i)
