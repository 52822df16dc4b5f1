"""Seeded synthetic workloads for the prefix-cache-aware router.

The paper evaluates on MMLU few-shot prompts (a shared few-shot prefix per topic
plus a unique question, one output token, requests drawn uniformly or with an
80/20 skew; Experimental Setup).  That dataset is not used here: these
generators produce integer token sequences with the same *structure* (shared
system prefix, shared per-topic prefix, unique suffix; Zipf-skewed topic
choice) at the sizes of the five benchmark configurations.

This module holds none of the routing method's arithmetic.  It only draws
token sequences; both the CPU oracle and the device path consume its output.

Every configuration is a pure function of (config id, seed base, size
overrides).  Random streams come from ``SeedSequence([seed_base, cfg])``
spawned once, in this fixed order: prefixes, homing, cache, queries, stale,
inserts.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

SEED_BASE = 20261202
STREAM_NAMES = ("prefixes", "homing", "cache", "queries", "stale", "inserts")
MAX_STREAM_ROUNDS = 256  # rounds per distribution the streaming configuration can generate

I32 = np.int32
I64 = np.int64


# --------------------------------------------------------------------------
# containers
# --------------------------------------------------------------------------
@dataclass
class SeqSet:
    """A batch of int32 token sequences in CSR form.

    ``tokens[offsets[i]:offsets[i+1]]`` is sequence i.  ``peer`` (optional)
    gives the owning peer of each sequence; for snapshots it is non-decreasing
    (peer-major) and sequences of one peer are in insert order.
    """

    tokens: np.ndarray
    offsets: np.ndarray
    peer: Optional[np.ndarray] = None

    def __len__(self) -> int:
        return int(self.offsets.shape[0] - 1)

    def seq(self, i: int) -> np.ndarray:
        return self.tokens[self.offsets[i]:self.offsets[i + 1]]

    def lengths(self) -> np.ndarray:
        return np.diff(self.offsets)

    def peer_range(self, p: int) -> Tuple[int, int]:
        assert self.peer is not None
        lo = int(np.searchsorted(self.peer, p, side="left"))
        hi = int(np.searchsorted(self.peer, p, side="right"))
        return lo, hi

    def peer_subset(self, p: int) -> "SeqSet":
        lo, hi = self.peer_range(p)
        return self.subset(np.arange(lo, hi))

    def subset(self, idx: np.ndarray) -> "SeqSet":
        idx = np.asarray(idx, dtype=I64)
        lens = (self.offsets[idx + 1] - self.offsets[idx]).astype(I64)
        offs = np.zeros(idx.shape[0] + 1, dtype=I64)
        np.cumsum(lens, out=offs[1:])
        toks = np.empty(int(offs[-1]), dtype=I32)
        for j, i in enumerate(idx.tolist()):
            toks[offs[j]:offs[j + 1]] = self.tokens[self.offsets[i]:self.offsets[i + 1]]
        peer = None if self.peer is None else self.peer[idx].copy()
        return SeqSet(toks, offs, peer)


@dataclass
class StreamPhase:
    """One (merge, lookup) round of the streaming configuration."""

    dist: str
    round: int
    inserts: SeqSet  # .peer = target replica of each insert
    queries: SeqSet


@dataclass
class Workload:
    cfg: int
    name: str
    num_peers: int
    vocab: int
    snapshot: SeqSet  # what the router's forest holds (estimates for cfg 3)
    queries: SeqSet
    true_snapshot: Optional[SeqSet] = None  # cfg 3: the peers' exact trees
    meta: Dict = field(default_factory=dict)
    _insert_fn: Optional[object] = None
    _query_fn: Optional[object] = None

    def phases(self, dist: str) -> List[StreamPhase]:
        assert self._insert_fn is not None, "only the streaming configuration has phases"
        return [self.phase(dist, r) for r in range(self.meta["rounds"])]

    def phase(self, dist: str, rnd: int) -> StreamPhase:
        """Round rnd of the streaming configuration: its merge batch, then its
        lookup batch."""
        assert self._insert_fn is not None, "only the streaming configuration has phases"
        return StreamPhase(dist, rnd, self._insert_fn(dist, rnd), self._query_fn(dist, rnd))

    def insert_batch(self, dist: str, rnd: int) -> SeqSet:
        """The merge batch of round rnd (any rnd < MAX_STREAM_ROUNDS; rounds
        past meta["rounds"] continue the same recipe)."""
        assert self._insert_fn is not None, "only the streaming configuration has insert batches"
        return self._insert_fn(dist, rnd)

    def query_batch(self, dist: str, rnd: int) -> SeqSet:
        assert self._query_fn is not None, "only the streaming configuration has lookup batches"
        return self._query_fn(dist, rnd)


# --------------------------------------------------------------------------
# helpers
# --------------------------------------------------------------------------
def _streams(cfg: int, seed_base: int):
    ss = np.random.SeedSequence([seed_base, cfg])
    kids = ss.spawn(len(STREAM_NAMES))
    return dict(zip(STREAM_NAMES, kids))


def _rng(ss: np.random.SeedSequence) -> np.random.Generator:
    return np.random.default_rng(ss)


def _uniform_int(rng, lo: int, hi: int, n: int) -> np.ndarray:
    """n draws of U{lo..hi} (inclusive)."""
    return rng.integers(lo, hi + 1, size=n, dtype=I64)


def zipf_probs(n_items: int, s: float) -> np.ndarray:
    """Finite Zipf law: P(rank r) proportional to (r+1)^-s, r = 0..n-1."""
    w = np.power(np.arange(1, n_items + 1, dtype=np.float64), -float(s))
    return w / w.sum()


def _draw_topics(rng, n: int, n_topics: int, s: Optional[float], perm: np.ndarray) -> np.ndarray:
    """Topic ids for n requests: uniform when s is None, else Zipf(s) over
    ranks mapped to topics through the seeded permutation ``perm``."""
    if s is None:
        return rng.integers(0, n_topics, size=n, dtype=I64)
    ranks = rng.choice(n_topics, size=n, p=zipf_probs(n_topics, s))
    return perm[ranks].astype(I64)


def _assemble(heads: List[np.ndarray], head_id: np.ndarray, suffix_len: np.ndarray,
              rng, vocab: int, peer: Optional[np.ndarray] = None) -> SeqSet:
    """Sequence i = heads[head_id[i]] followed by suffix_len[i] fresh uniform tokens."""
    n = int(head_id.shape[0])
    hl = np.array([h.shape[0] for h in heads], dtype=I64)
    lens = hl[head_id] + suffix_len
    offs = np.zeros(n + 1, dtype=I64)
    np.cumsum(lens, out=offs[1:])
    toks = np.empty(int(offs[-1]), dtype=I32)
    suffix = rng.integers(0, vocab, size=int(suffix_len.sum()), dtype=I32)
    so = 0
    hid = head_id.tolist()
    sl = suffix_len.tolist()
    ol = offs.tolist()
    for i in range(n):
        h = heads[hid[i]]
        o = ol[i]
        k = h.shape[0]
        toks[o:o + k] = h
        s = sl[i]
        toks[o + k:o + k + s] = suffix[so:so + s]
        so += s
    return SeqSet(toks, offs, None if peer is None else np.asarray(peer, dtype=I32))


def _two_homes(rng, n_topics: int, P: int, perm: np.ndarray) -> List[List[int]]:
    """Each topic lives on two distinct peers: primary perm[t] mod P (balanced),
    secondary uniform over the other P-1 peers.  Returns homed topics per peer."""
    homed: List[List[int]] = [[] for _ in range(P)]
    prim = (perm % P).astype(I64)
    sec_draw = rng.integers(0, P - 1, size=n_topics, dtype=I64)
    for t in range(n_topics):
        a = int(prim[t])
        b = int(sec_draw[t])
        b = b + 1 if b >= a else b
        homed[a].append(t)
        homed[b].append(t)
    return [sorted(h) for h in homed]


def _cache_heads(rng, homed: List[List[int]], per_peer: int) -> Tuple[np.ndarray, np.ndarray]:
    """Topic of every cached prompt, peer-major, uniform over the peer's homed set."""
    P = len(homed)
    peer = np.repeat(np.arange(P, dtype=I32), per_peer)
    topic = np.empty(P * per_peer, dtype=I64)
    for p in range(P):
        h = np.asarray(homed[p], dtype=I64)
        topic[p * per_peer:(p + 1) * per_peer] = h[rng.integers(0, h.shape[0], size=per_peer)]
    return peer, topic


# --------------------------------------------------------------------------
# the five benchmark configurations (+ config 0 for tiny random tests)
# --------------------------------------------------------------------------
CONFIG_NAMES = {1: "tiny", 2: "medium", 3: "stale", 4: "long", 5: "stream"}


def make_config(cfg: int, seed_base: int = SEED_BASE, *, n_queries: Optional[int] = None,
                prompts_per_peer: Optional[int] = None, rounds: Optional[int] = None,
                phase_queries: Optional[int] = None, phase_inserts: Optional[int] = None) -> Workload:
    """Build configuration ``cfg`` (1..5).  Size overrides shrink a config for
    quick tests while keeping its recipe."""
    st = _streams(cfg, seed_base)
    if cfg == 1:
        return _cfg_tiny(st, n_queries, prompts_per_peer)
    if cfg == 2:
        return _cfg_medium(st, n_queries, prompts_per_peer)
    if cfg == 3:
        return _cfg_stale(st, n_queries, prompts_per_peer)
    if cfg == 4:
        return _cfg_long(st, n_queries, prompts_per_peer)
    if cfg == 5:
        return _cfg_stream(st, prompts_per_peer, rounds, phase_queries, phase_inserts)
    raise ValueError(f"unknown config {cfg}")


def _topic_world(st, vocab: int, sys_len: int, topic_lens: np.ndarray, n_unseen: int):
    """Draw the shared system prefix, the seen topic heads and the unseen pool.

    heads[t] = system prefix + topic t's prefix (t < T); heads[T + u] = system
    prefix + unseen topic u's prefix.  Unseen topics are drawn by the same law
    and never cached anywhere."""
    rng = _rng(st["prefixes"])
    sys_p = rng.integers(0, vocab, size=sys_len, dtype=I32)
    T = int(topic_lens.shape[0])
    heads = []
    for t in range(T):
        heads.append(np.concatenate([sys_p, rng.integers(0, vocab, size=int(topic_lens[t]), dtype=I32)]))
    unseen_lens = topic_lens[rng.integers(0, T, size=n_unseen)] if n_unseen else np.zeros(0, I64)
    for u in range(n_unseen):
        heads.append(np.concatenate([sys_p, rng.integers(0, vocab, size=int(unseen_lens[u]), dtype=I32)]))
    perm = rng.permutation(T).astype(I64)  # Zipf rank -> topic
    return sys_p, heads, perm


def _queries(rng, n: int, T: int, n_unseen: int, unseen_frac: float, zipf_s: Optional[float],
             perm: np.ndarray, heads, suffix_lo: int, suffix_hi, vocab: int, head_lens=None):
    unseen = rng.random(n) < unseen_frac if unseen_frac > 0 else np.zeros(n, dtype=bool)
    topic = _draw_topics(rng, n, T, zipf_s, perm)
    head_id = topic.copy()
    if n_unseen:
        u = rng.integers(0, n_unseen, size=n, dtype=I64)
        head_id[unseen] = T + u[unseen]
    if callable(suffix_hi):
        hi = suffix_hi(head_id)
        slen = suffix_lo + (rng.random(n) * (hi - suffix_lo + 1)).astype(I64)
    else:
        slen = _uniform_int(rng, suffix_lo, suffix_hi, n)
    qs = _assemble(heads, head_id, slen, rng, vocab)
    return qs, head_id, unseen


def _cfg_tiny(st, n_queries, per_peer) -> Workload:
    P, V, SYS, T, TL = 4, 32000, 64, 16, 256
    per_peer = 200 if per_peer is None else per_peer
    nq = 2048 if n_queries is None else n_queries
    sys_p, heads, perm = _topic_world(st, V, SYS, np.full(T, TL, I64), T)
    rng_h = _rng(st["homing"])
    homed: List[List[int]] = [[] for _ in range(P)]
    extra = rng_h.random(T) < 0.25
    other = rng_h.integers(0, P - 1, size=T)
    for t in range(T):
        a = t % P
        homed[a].append(t)
        if extra[t]:
            b = int(other[t])
            b = b + 1 if b >= a else b
            homed[b].append(t)
    homed = [sorted(h) for h in homed]
    rng_c = _rng(st["cache"])
    peer, topic = _cache_heads(rng_c, homed, per_peer)
    snap = _assemble(heads, topic, _uniform_int(rng_c, 32, 128, topic.shape[0]), rng_c, V, peer)
    rng_q = _rng(st["queries"])
    qs, head_id, unseen = _queries(rng_q, nq, T, T, 0.10, 1.0, perm, heads, 32, 128, V)
    meta = dict(sys_len=SYS, head_len=np.array([h.shape[0] for h in heads], I64), n_topics=T,
                homed=homed, cache_topic=topic, query_head=head_id, query_unseen=unseen, zipf_s=1.0)
    return Workload(1, "tiny", P, V, snap, qs, meta=meta)


def _cfg_medium(st, n_queries, per_peer) -> Workload:
    P, V, SYS, T, TL = 16, 32000, 128, 64, 1024
    per_peer = 2000 if per_peer is None else per_peer
    nq = 65536 if n_queries is None else n_queries
    sys_p, heads, perm = _topic_world(st, V, SYS, np.full(T, TL, I64), T)
    homed = _two_homes(_rng(st["homing"]), T, P, perm)
    rng_c = _rng(st["cache"])
    peer, topic = _cache_heads(rng_c, homed, per_peer)
    snap = _assemble(heads, topic, _uniform_int(rng_c, 64, 256, topic.shape[0]), rng_c, V, peer)
    qs, head_id, unseen = _queries(_rng(st["queries"]), nq, T, T, 0.05, 1.1, perm, heads, 64, 256, V)
    meta = dict(sys_len=SYS, head_len=np.array([h.shape[0] for h in heads], I64), n_topics=T,
                homed=homed, cache_topic=topic, query_head=head_id, query_unseen=unseen, zipf_s=1.1)
    return Workload(2, "medium", P, V, snap, qs, meta=meta)


def _cfg_stale(st, n_queries, per_peer) -> Workload:
    P, V, SYS, T = 64, 128256, 256, 512
    per_peer = 4000 if per_peer is None else per_peer
    nq = 262144 if n_queries is None else n_queries
    window = min(1000, per_peer)
    rng_pre = _rng(st["prefixes"])
    task_len = _uniform_int(rng_pre, 512, 2048, T)
    # the task lengths use the prefixes stream first; _topic_world continues on a fresh stream
    sys_p, heads, perm = _topic_world({"prefixes": st["prefixes"].spawn(1)[0]}, V, SYS, task_len, 0)
    homed = _two_homes(_rng(st["homing"]), T, P, perm)
    rng_c = _rng(st["cache"])
    peer, topic = _cache_heads(rng_c, homed, per_peer)
    hi_of = lambda hid: (4096 - SYS - task_len[hid]).astype(I64)
    n = topic.shape[0]
    hi = hi_of(topic)
    slen = 64 + (rng_c.random(n) * (hi - 64 + 1)).astype(I64)
    true_snap = _assemble(heads, topic, slen, rng_c, V, peer)
    # observer 0 holds its own exact tree; its replica of each other peer misses
    # a Bernoulli(0.2) subset of that peer's last `window` inserts.
    rng_s = _rng(st["stale"])
    keep = np.ones(n, dtype=bool)
    for p in range(1, P):
        lo = p * per_peer + per_peer - window
        drop = rng_s.random(window) < 0.2
        keep[lo:lo + window] = ~drop
    est_snap = true_snap.subset(np.nonzero(keep)[0])
    qs, head_id, unseen = _queries(_rng(st["queries"]), nq, T, 0, 0.0, 1.2, perm, heads, 64, hi_of, V)
    meta = dict(sys_len=SYS, head_len=np.array([h.shape[0] for h in heads], I64), n_topics=T,
                homed=homed, cache_topic=topic, query_head=head_id, query_unseen=unseen, zipf_s=1.2,
                stale_keep=keep, stale_window=window)
    return Workload(3, "stale", P, V, est_snap, qs, true_snapshot=true_snap, meta=meta)


def _cfg_long(st, n_queries, per_peer) -> Workload:
    P, V, T = 32, 128256, 256
    per_peer = 500 if per_peer is None else per_peer
    nq = 32768 if n_queries is None else n_queries
    rng_pre = _rng(st["prefixes"])
    plen = _uniform_int(rng_pre, 8192, 32768, T)
    sys_p, heads, perm = _topic_world({"prefixes": st["prefixes"].spawn(1)[0]}, V, 0, plen, 0)
    homed = _two_homes(_rng(st["homing"]), T, P, perm)
    rng_c = _rng(st["cache"])
    peer, topic = _cache_heads(rng_c, homed, per_peer)
    snap = _assemble(heads, topic, _uniform_int(rng_c, 128, 1024, topic.shape[0]), rng_c, V, peer)
    qs, head_id, unseen = _queries(_rng(st["queries"]), nq, T, 0, 0.0, 1.0, perm, heads, 128, 1024, V)
    meta = dict(sys_len=0, head_len=np.array([h.shape[0] for h in heads], I64), n_topics=T,
                homed=homed, cache_topic=topic, query_head=head_id, query_unseen=unseen, zipf_s=1.0,
                split_block=16)
    return Workload(4, "long", P, V, snap, qs, meta=meta)


def _cfg_stream(st, per_peer, rounds, phase_queries, phase_inserts) -> Workload:
    P, V, SYS, T, TL = 128, 128256, 128, 512, 1024
    per_peer = 2000 if per_peer is None else per_peer
    R = 4 if rounds is None else rounds
    NQ = 1048576 if phase_queries is None else phase_queries
    NI = 10000 if phase_inserts is None else phase_inserts
    sys_p, heads, perm = _topic_world(st, V, SYS, np.full(T, TL, I64), T)
    homed = _two_homes(_rng(st["homing"]), T, P, perm)
    rng_c = _rng(st["cache"])
    peer, topic = _cache_heads(rng_c, homed, per_peer)
    snap = _assemble(heads, topic, _uniform_int(rng_c, 64, 256, topic.shape[0]), rng_c, V, peer)
    dists = ("uniform", "zipf")
    # one child stream per (dist, round), spawned up front so any round's
    # batches can be generated on their own
    q_kids = st["queries"].spawn(2 * MAX_STREAM_ROUNDS)
    i_kids = st["inserts"].spawn(2 * MAX_STREAM_ROUNDS)

    def kid(dist: str, rnd: int) -> int:
        if not 0 <= rnd < MAX_STREAM_ROUNDS:
            raise ValueError(f"round {rnd} outside [0, {MAX_STREAM_ROUNDS})")
        return dists.index(dist) * MAX_STREAM_ROUNDS + rnd

    def inserts(dist: str, rnd: int) -> SeqSet:
        s = None if dist == "uniform" else 1.2
        rng_i = _rng(i_kids[kid(dist, rnd)])
        tgt = rng_i.integers(1, P, size=NI, dtype=I64).astype(I32)
        itopic = _draw_topics(rng_i, NI, T, s, perm)
        return _assemble(heads, itopic, _uniform_int(rng_i, 64, 256, NI), rng_i, V, tgt)

    def lookups(dist: str, rnd: int) -> SeqSet:
        s = None if dist == "uniform" else 1.2
        qs, _, _ = _queries(_rng(q_kids[kid(dist, rnd)]), NQ, T, T, 0.05, s, perm, heads, 64, 256, V)
        return qs

    # the first-round query batch stands in as `queries` for generic code paths
    meta = dict(sys_len=SYS, head_len=np.array([h.shape[0] for h in heads], I64), n_topics=T,
                homed=homed, cache_topic=topic, rounds=R, phase_queries=NQ, phase_inserts=NI)
    empty = SeqSet(np.zeros(0, I32), np.zeros(1, I64))
    return Workload(5, "stream", P, V, snap, empty, meta=meta, _insert_fn=inserts, _query_fn=lookups)


# --------------------------------------------------------------------------
# config 0: tiny random forests for exhaustive tests
# --------------------------------------------------------------------------
def tiny_random(seed: int, *, num_peers: int = 3, vocab: int = 3, max_len: int = 12,
                max_seqs: int = 12, n_queries: int = 64, with_empty: bool = True) -> Workload:
    """Small random instances over a tiny vocabulary, so that shared prefixes,
    sequences ending inside an edge, duplicates and prefixes-of-prompts all occur.
    Sequences are built by extending random earlier ones, which forces sharing."""
    rng = np.random.default_rng(np.random.SeedSequence([SEED_BASE, 0, seed]))
    pool: List[np.ndarray] = []

    def draw_seq() -> np.ndarray:
        if pool and rng.random() < 0.6:
            base = pool[int(rng.integers(0, len(pool)))]
            cut = int(rng.integers(0, base.shape[0] + 1))
            ext = int(rng.integers(0, max_len - cut + 1))
            return np.concatenate([base[:cut], rng.integers(0, vocab, size=ext, dtype=I32)]).astype(I32)
        lo = 0 if with_empty else 1
        return rng.integers(0, vocab, size=int(rng.integers(lo, max_len + 1)), dtype=I32)

    seqs, owners = [], []
    for p in range(num_peers):
        k = int(rng.integers(0, max_seqs + 1))
        for _ in range(k):
            s = draw_seq()
            pool.append(s)
            seqs.append(s)
            owners.append(p)
    snap = _from_list(seqs, owners)
    qs = []
    for _ in range(n_queries):
        if pool and rng.random() < 0.3:
            qs.append(pool[int(rng.integers(0, len(pool)))].copy())  # exact cached prompt
        else:
            qs.append(draw_seq())
    return Workload(0, f"tiny_random_{seed}", num_peers, vocab, snap, _from_list(qs, None))


def _from_list(seqs: List[np.ndarray], owners: Optional[List[int]]) -> SeqSet:
    offs = np.zeros(len(seqs) + 1, dtype=I64)
    if seqs:
        np.cumsum([s.shape[0] for s in seqs], out=offs[1:])
    toks = np.concatenate(seqs).astype(I32) if seqs and offs[-1] > 0 else np.zeros(0, I32)
    peer = None if owners is None else np.asarray(owners, dtype=I32)
    return SeqSet(toks, offs, peer)


def from_lists(seqs, owners=None) -> SeqSet:
    """CSR from a Python list of token lists."""
    return _from_list([np.asarray(s, dtype=I32) for s in seqs], owners)
