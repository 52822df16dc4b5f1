"""CPU oracle for the prefix-cache-aware router -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never calls it and
shares no code with it.

Two independent oracles, sharing no code:

* ``Oracle`` (``prefix_oracle.c``) computes the plain definition of the
  paper's routing rule (System Design; Algorithm 1): for every peer p,
  m[q][p] is the longest common prefix of q with any sequence inserted into
  p's tree, and the chosen peer is the lowest id attaining the maximum, by a
  linear scan over every stored sequence.  ``route_select`` adds the push-back
  and failover selection (best and second-best eligible peer).
* ``RadixOracle`` (``radix_oracle.c``) keeps one radix tree per peer, as the
  paper does, and walks each with the query (INSERT and MATCH step by step).
  It reaches the same result far faster on large forests, so it checks every
  row of the full-size workloads.

Every function here is pinned by ``tests/test_oracle_pins.py`` and
``tests/test_radix_oracle.py`` against independent formulations (hand-worked
examples, the prefix-set definition of a trie, numpy brute force, invariants
the paper states, and each other).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "prefix_oracle.c")
_SRC_RADIX = os.path.join(_HERE, "radix_oracle.c")
LIB_PATH = os.path.join(_HERE, "liboracle.so")

_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)


def build(plant: Optional[str] = None, out: Optional[str] = None) -> str:
    """Compile the oracle with gcc.  ``plant`` names a deliberate mistake
    (PLANT_* macro) for the tests that check the pins catch it."""
    out = out or (LIB_PATH if plant is None else os.path.join(_HERE, f"liboracle_{plant.lower()}.so"))
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread", _SRC, _SRC_RADIX, "-o", out + ".tmp"]
    if plant:
        cmd.insert(1, f"-D{plant}")
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def _load(path: str) -> ctypes.CDLL:
    lib = ctypes.CDLL(path)
    lib.or_create.restype = ctypes.c_void_p
    lib.or_create.argtypes = [ctypes.c_int32]
    lib.or_destroy.restype = None
    lib.or_destroy.argtypes = [ctypes.c_void_p]
    lib.or_load.restype = ctypes.c_int
    lib.or_load.argtypes = [ctypes.c_void_p, ctypes.c_int32, _i32p, _i64p, ctypes.c_int64]
    lib.or_merge.restype = ctypes.c_int
    lib.or_merge.argtypes = [ctypes.c_void_p, _i32p, _i32p, _i64p, ctypes.c_int64]
    lib.or_route.restype = ctypes.c_int
    lib.or_route.argtypes = [ctypes.c_void_p, _i32p, _i64p, ctypes.c_int64, _i32p, _i32p, ctypes.c_int32]
    lib.or_route_select.restype = ctypes.c_int
    lib.or_route_select.argtypes = [ctypes.c_void_p, _i32p, _i64p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int32,
                                    ctypes.c_int32, _i32p, _i32p, _i32p, ctypes.c_int32]
    lib.or_export.restype = ctypes.c_int
    lib.or_export.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                              ctypes.c_int64, _i64p, _i64p]
    lib.or_set_local.restype = ctypes.c_int
    lib.or_set_local.argtypes = [ctypes.c_void_p, ctypes.c_int32]
    lib.or_set_time.restype = ctypes.c_int
    lib.or_set_time.argtypes = [ctypes.c_void_p, ctypes.c_int64]
    lib.or_touch.restype = ctypes.c_int
    lib.or_touch.argtypes = [ctypes.c_void_p, _i32p, _i64p, ctypes.c_int64]
    lib.or_evict.restype = ctypes.c_int64
    lib.or_evict.argtypes = [ctypes.c_void_p, ctypes.c_int64]
    lib.or_tree_tokens.restype = ctypes.c_int64
    lib.or_tree_tokens.argtypes = [ctypes.c_void_p, ctypes.c_int32]
    lib.or_lcp.restype = ctypes.c_int64
    lib.or_lcp.argtypes = [_i32p, ctypes.c_int64, _i32p, ctypes.c_int64]
    lib.or_prefix_match.restype = ctypes.c_int64
    lib.or_prefix_match.argtypes = [ctypes.c_void_p, ctypes.c_int32, _i32p, ctypes.c_int64]
    lib.or_set_size.restype = ctypes.c_int64
    lib.or_set_size.argtypes = [ctypes.c_void_p, ctypes.c_int32]
    lib.rx_create.restype = ctypes.c_void_p
    lib.rx_create.argtypes = [ctypes.c_int32, ctypes.c_int32]
    lib.rx_destroy.restype = None
    lib.rx_destroy.argtypes = [ctypes.c_void_p]
    lib.rx_load.restype = ctypes.c_int
    lib.rx_load.argtypes = [ctypes.c_void_p, ctypes.c_int32, _i32p, _i64p, ctypes.c_int64]
    lib.rx_merge.restype = ctypes.c_int
    lib.rx_merge.argtypes = [ctypes.c_void_p, _i32p, _i32p, _i64p, ctypes.c_int64]
    lib.rx_match.restype = ctypes.c_int64
    lib.rx_match.argtypes = [ctypes.c_void_p, ctypes.c_int32, _i32p, ctypes.c_int64]
    lib.rx_route.restype = ctypes.c_int
    lib.rx_route.argtypes = [ctypes.c_void_p, _i32p, _i64p, ctypes.c_int64, _i32p, _i32p, ctypes.c_int32]
    for name in ("rx_node_count", "rx_tree_tokens"):
        getattr(lib, name).restype = ctypes.c_int64
        getattr(lib, name).argtypes = [ctypes.c_void_p, ctypes.c_int32]
    lib.rx_check.restype = ctypes.c_int
    lib.rx_check.argtypes = [ctypes.c_void_p, ctypes.c_int32]
    return lib


_LIBS = {}


def lib(path: Optional[str] = None) -> ctypes.CDLL:
    path = path or LIB_PATH
    if path not in _LIBS:
        if not os.path.exists(path):
            if path == LIB_PATH:
                build()
            else:
                raise FileNotFoundError(path)
        _LIBS[path] = _load(path)
    return _LIBS[path]


def _p32(a: np.ndarray):
    return a.ctypes.data_as(_i32p)


def _p64(a: np.ndarray):
    return a.ctypes.data_as(_i64p)


def _csr(tokens, offsets) -> Tuple[np.ndarray, np.ndarray]:
    t = np.ascontiguousarray(tokens, dtype=np.int32)
    o = np.ascontiguousarray(offsets, dtype=np.int64)
    if t.size == 0:
        t = np.zeros(1, np.int32)  # valid pointer for empty batches
    return t, o


class Oracle:
    """Per-peer multisets S_p with load (replace), merge (insert) and route."""

    def __init__(self, num_peers: int, lib_path: Optional[str] = None):
        self._lib = lib(lib_path)
        self.num_peers = int(num_peers)
        self._h = self._lib.or_create(self.num_peers)
        if not self._h:
            raise ValueError("or_create failed")

    def close(self):
        if self._h:
            self._lib.or_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def load(self, peer: int, tokens, offsets) -> None:
        t, o = _csr(tokens, offsets)
        r = self._lib.or_load(self._h, int(peer), _p32(t), _p64(o), o.shape[0] - 1)
        if r:
            raise ValueError(f"or_load failed ({r})")

    def load_seqset(self, ss) -> None:
        """Load every peer's snapshot from a peer-major SeqSet."""
        for p in range(self.num_peers):
            lo, hi = ss.peer_range(p)
            o = ss.offsets[lo:hi + 1] - ss.offsets[lo]
            self.load(p, ss.tokens[ss.offsets[lo]:ss.offsets[hi]], o)

    def merge(self, peer_of, tokens, offsets) -> None:
        t, o = _csr(tokens, offsets)
        po = np.ascontiguousarray(peer_of, dtype=np.int32)
        if po.size == 0:
            po = np.zeros(1, np.int32)
        r = self._lib.or_merge(self._h, _p32(po), _p32(t), _p64(o), o.shape[0] - 1)
        if r:
            raise ValueError(f"or_merge failed ({r})")

    def route(self, tokens, offsets, nthreads: int = 0) -> Tuple[np.ndarray, np.ndarray]:
        t, o = _csr(tokens, offsets)
        nq = o.shape[0] - 1
        m = np.zeros((max(nq, 1), self.num_peers), dtype=np.int32)
        c = np.zeros(max(nq, 1), dtype=np.int32)
        nt = nthreads or (os.cpu_count() or 1)
        r = self._lib.or_route(self._h, _p32(t), _p64(o), nq, _p32(m), _p32(c), nt)
        if r:
            raise ValueError(f"or_route failed ({r})")
        return m[:nq], c[:nq]

    def route_select(self, tokens, offsets, eligible=None, local: int = -1, prefer_local: bool = False,
                     nthreads: int = 0) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
        """Match lengths, best and second-best eligible peer (push-back and
        failover selection; see or_route_select in prefix_oracle.c)."""
        t, o = _csr(tokens, offsets)
        nq = o.shape[0] - 1
        m = np.zeros((max(nq, 1), self.num_peers), dtype=np.int32)
        b1 = np.zeros(max(nq, 1), dtype=np.int32)
        b2 = np.zeros(max(nq, 1), dtype=np.int32)
        el = None
        if eligible is not None:
            el = np.ascontiguousarray(eligible, dtype=np.uint8)
            if el.shape != (self.num_peers,):
                raise ValueError("eligible must hold one flag per peer")
        nt = nthreads or (os.cpu_count() or 1)
        r = self._lib.or_route_select(self._h, _p32(t), _p64(o), nq, el.ctypes.data if el is not None else None,
                                      int(local), int(bool(prefer_local)), _p32(m), _p32(b1), _p32(b2), nt)
        if r:
            raise ValueError(f"or_route_select failed ({r})")
        return m[:nq], b1[:nq], b2[:nq]

    def route_seqset(self, qs, idx: Optional[Sequence[int]] = None, nthreads: int = 0):
        """Route all queries of a SeqSet, or only the sampled indices ``idx``."""
        if idx is None:
            return self.route(qs.tokens, qs.offsets, nthreads)
        sub = qs.subset(np.asarray(idx))
        return self.route(sub.tokens, sub.offsets, nthreads)

    def export(self, peer: int) -> Tuple[np.ndarray, np.ndarray]:
        """sendTrie: the members of S_p that are no proper prefix of another
        (each once, empty ones left out), in lexicographic order, as CSR."""
        ns, nt = ctypes.c_int64(0), ctypes.c_int64(0)
        r = self._lib.or_export(self._h, int(peer), None, 0, None, 0, ctypes.byref(ns), ctypes.byref(nt))
        if r:
            raise ValueError(f"or_export failed ({r})")
        t = np.zeros(max(nt.value, 1), np.int32)
        o = np.zeros(ns.value + 1, np.int64)
        r = self._lib.or_export(self._h, int(peer), t.ctypes.data, t.shape[0], o.ctypes.data, o.shape[0],
                                ctypes.byref(ns), ctypes.byref(nt))
        if r:
            raise ValueError(f"or_export failed ({r})")
        return t[:nt.value], o

    # ---- local LRU tree (Algorithm 1's EvictLRUTrie) ----
    def set_local(self, peer: int) -> None:
        """Make peer the local one: its tree keeps access times (-1: none)."""
        if self._lib.or_set_local(self._h, int(peer)):
            raise ValueError("or_set_local failed")

    def set_time(self, t: int) -> None:
        """Current time for loads, merges and touches of the local peer."""
        if self._lib.or_set_time(self._h, int(t)):
            raise ValueError("or_set_time failed (time went backwards)")

    def touch(self, tokens, offsets) -> None:
        t, o = _csr(tokens, offsets)
        if self._lib.or_touch(self._h, _p32(t), _p64(o), o.shape[0] - 1):
            raise ValueError("or_touch failed")

    def evict(self, n: int) -> int:
        r = int(self._lib.or_evict(self._h, int(n)))
        if r < 0:
            raise ValueError("or_evict failed")
        return r

    def tree_tokens(self, peer: int) -> int:
        """Distinct non-empty prefixes of peer's set (tokens its tree holds)."""
        r = int(self._lib.or_tree_tokens(self._h, int(peer)))
        if r < 0:
            raise ValueError("or_tree_tokens failed")
        return r

    def prefix_match(self, peer: int, q) -> int:
        qa = np.ascontiguousarray(q, dtype=np.int32)
        if qa.size == 0:
            return int(self._lib.or_prefix_match(self._h, int(peer), _p32(np.zeros(1, np.int32)), 0))
        return int(self._lib.or_prefix_match(self._h, int(peer), _p32(qa), qa.shape[0]))

    def set_size(self, peer: int) -> int:
        return int(self._lib.or_set_size(self._h, int(peer)))

    def lcp(self, a, b) -> int:
        a = np.ascontiguousarray(a, dtype=np.int32)
        b = np.ascontiguousarray(b, dtype=np.int32)
        pa = _p32(a if a.size else np.zeros(1, np.int32))
        pb = _p32(b if b.size else np.zeros(1, np.int32))
        return int(self._lib.or_lcp(pa, a.shape[0], pb, b.shape[0]))


class RadixOracle:
    """One radix tree per peer, as the paper keeps them (radix_oracle.c):
    load (replace), merge (insert), route (MATCH on every tree, then the
    lowest-id argmax).  ``split_block`` B > 0 keeps a node at every depth that
    is a multiple of B (the long-context workload's 16-token blocks); match
    lengths do not depend on it."""

    def __init__(self, num_peers: int, split_block: int = 0, lib_path: Optional[str] = None):
        self._lib = lib(lib_path)
        self.num_peers = int(num_peers)
        self.split_block = int(split_block)
        self._h = self._lib.rx_create(self.num_peers, self.split_block)
        if not self._h:
            raise ValueError("rx_create failed")

    def close(self):
        if self._h:
            self._lib.rx_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def load(self, peer: int, tokens, offsets) -> None:
        t, o = _csr(tokens, offsets)
        r = self._lib.rx_load(self._h, int(peer), _p32(t), _p64(o), o.shape[0] - 1)
        if r:
            raise ValueError(f"rx_load failed ({r})")

    def load_seqset(self, ss) -> None:
        """Load every peer's snapshot from a peer-major SeqSet."""
        for p in range(self.num_peers):
            lo, hi = ss.peer_range(p)
            o = ss.offsets[lo:hi + 1] - ss.offsets[lo]
            self.load(p, ss.tokens[ss.offsets[lo]:ss.offsets[hi]], o)

    def merge(self, peer_of, tokens, offsets) -> None:
        t, o = _csr(tokens, offsets)
        po = np.ascontiguousarray(peer_of, dtype=np.int32)
        if po.size == 0:
            po = np.zeros(1, np.int32)
        r = self._lib.rx_merge(self._h, _p32(po), _p32(t), _p64(o), o.shape[0] - 1)
        if r:
            raise ValueError(f"rx_merge failed ({r})")

    def route(self, tokens, offsets, nthreads: int = 0) -> Tuple[np.ndarray, np.ndarray]:
        t, o = _csr(tokens, offsets)
        nq = o.shape[0] - 1
        m = np.zeros((max(nq, 1), self.num_peers), dtype=np.int32)
        c = np.zeros(max(nq, 1), dtype=np.int32)
        nt = nthreads or (os.cpu_count() or 1)
        r = self._lib.rx_route(self._h, _p32(t), _p64(o), nq, _p32(m), _p32(c), nt)
        if r:
            raise ValueError(f"rx_route failed ({r})")
        return m[:nq], c[:nq]

    def route_seqset(self, qs, idx: Optional[Sequence[int]] = None, nthreads: int = 0):
        """Route all queries of a SeqSet, or only the sampled indices ``idx``."""
        if idx is None:
            return self.route(qs.tokens, qs.offsets, nthreads)
        sub = qs.subset(np.asarray(idx))
        return self.route(sub.tokens, sub.offsets, nthreads)

    def prefix_match(self, peer: int, q) -> int:
        qa = np.ascontiguousarray(q, dtype=np.int32)
        r = int(self._lib.rx_match(self._h, int(peer), _p32(qa if qa.size else np.zeros(1, np.int32)),
                                   qa.shape[0]))
        if r < 0:
            raise ValueError("rx_match failed")
        return r

    def node_count(self, peer: int) -> int:
        """Nodes of peer's tree, the root not counted."""
        return int(self._lib.rx_node_count(self._h, int(peer)))

    def tree_tokens(self, peer: int) -> int:
        """Sum of peer's label lengths: its distinct non-empty prefixes."""
        return int(self._lib.rx_tree_tokens(self._h, int(peer)))

    def check(self, peer: int) -> int:
        """0 if peer's tree has the structure INSERT leaves (see rx_check)."""
        return int(self._lib.rx_check(self._h, int(peer)))
