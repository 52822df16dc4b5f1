"""The simulator's router calls on the CPU oracle (test infrastructure): the
same closed loop replayed against the oracle must give the same trace."""
import numpy as np

import oracle


class OracleBackend:
    def __init__(self, num_peers: int, local: int):
        self.o = oracle.Oracle(num_peers)
        self.local = local
        self.o.set_local(local)

    @staticmethod
    def _csr(seqs):
        t = np.concatenate([np.asarray(s, np.int32) for s in seqs]) if seqs else np.zeros(0, np.int32)
        o = np.zeros(len(seqs) + 1, np.int64)
        o[1:] = np.cumsum([len(s) for s in seqs])
        return t, o

    def set_time(self, t: int) -> None:
        self.o.set_time(t)

    def route(self, q):
        t, o = self._csr([q])
        m, b1, b2 = self.o.route_select(t, o, None, self.local, True, 1)
        return m[0], int(b1[0]), int(b2[0])

    def touch(self, q) -> None:
        t, o = self._csr([q])
        self.o.touch(t, o)

    def tree_tokens(self) -> int:
        return self.o.tree_tokens(self.local)

    def evict(self, n: int) -> int:
        return self.o.evict(n)

    def insert(self, peer: int, q) -> None:
        t, o = self._csr([q])
        self.o.merge(np.array([peer], np.int32), t, o)

    def export_local(self):
        return self.o.export(self.local)

    def load_estimate(self, peer: int, snapshot) -> None:
        t, o = snapshot
        self.o.load(peer, t, o)

    def close(self) -> None:
        self.o.close()
