"""Pins for the CPU oracle: independent ways to know the right answer.

Each check takes a factory ``make(num_peers) -> oracle-like object`` (with
load / merge / route) and returns a list of failure strings, so the same checks
run against the real oracle and against builds with a planted mistake.

* hand-worked examples (tests/golden/hand_examples.txt, derived by hand from the
  paper's definitions: System Design, Algorithm 1, "Trie-broadcast loss");
* the prefix-set formulation of a trie: a tree over S holds exactly the
  prefixes of S's members, so m = the largest k with q[:k] among them;
* numpy brute force of max_s LCP(q, s) by padded-matrix comparison;
* numpy's argmax, which returns the first (lowest-index) maximum;
* invariants: m <= |q|; a cached prompt used as a query matches its owner in
  full; merging never lowers a match and yields the union's match; set
  semantics under permutation / duplication / repeated loads (a snapshot is a
  complete state, so applying it twice is applying it once).
"""
from __future__ import annotations

import os
import re
from dataclasses import dataclass, field
from typing import Callable, List, Sequence, Tuple

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "hand_examples.txt")


# --------------------------------------------------------------------------
# golden examples
# --------------------------------------------------------------------------
@dataclass
class Example:
    name: str
    peers: int = 0
    ops: List[Tuple] = field(default_factory=list)  # ("load", p, seqs) | ("merge", [(p, seq)]) | ("query", q, m, c)


def _toks(s: str) -> List[int]:
    s = s.strip()
    if s == "[]":
        return []
    return [int(x) for x in s.split()] if s else []


def parse_golden(path: str = GOLDEN) -> List[Example]:
    exs: List[Example] = []
    cur = None
    for raw in open(path):
        line = raw.strip()
        if not line or line.startswith("#"):
            continue
        kw, _, rest = line.partition(" ")
        if kw == "example":
            cur = Example(rest.strip())
            exs.append(cur)
        elif kw == "peers":
            cur.peers = int(rest)
        elif kw == "load":
            p, _, seqs = rest.partition("|")
            items = [x for x in seqs.split(";")] if seqs.strip() else []
            cur.ops.append(("load", int(p), [_toks(x) for x in items]))
        elif kw == "merge":
            items = []
            for it in rest.split(";"):
                p, _, s = it.partition(":")
                items.append((int(p), _toks(s)))
            cur.ops.append(("merge", items))
        elif kw == "query":
            q, _, res = rest.partition("->") if rest.strip() != "" else ("", "", "")
            if line.startswith("query ->"):
                q, res = "", line[len("query ->"):]
            ms, _, c = res.partition(";")
            cur.ops.append(("query", _toks(q), [int(x) for x in ms.split()], int(c)))
        else:
            raise ValueError(f"bad golden line: {line}")
    return exs


def _csr(seqs: Sequence[Sequence[int]]):
    offs = np.zeros(len(seqs) + 1, dtype=np.int64)
    if seqs:
        np.cumsum([len(s) for s in seqs], out=offs[1:])
    toks = np.array([t for s in seqs for t in s], dtype=np.int32)
    return toks, offs


def check_golden(make: Callable) -> List[str]:
    fails = []
    for ex in parse_golden():
        o = make(ex.peers)
        for op in ex.ops:
            if op[0] == "load":
                t, off = _csr(op[2])
                o.load(op[1], t, off)
            elif op[0] == "merge":
                t, off = _csr([s for _, s in op[1]])
                o.merge(np.array([p for p, _ in op[1]], np.int32), t, off)
            else:
                _, q, m_exp, c_exp = op
                t, off = _csr([q])
                m, c = o.route(t, off, 1)
                if list(m[0]) != m_exp or int(c[0]) != c_exp:
                    fails.append(f"{ex.name}: q={q} got m={list(m[0])} c={int(c[0])}, want m={m_exp} c={c_exp}")
    return fails


# --------------------------------------------------------------------------
# independent formulations
# --------------------------------------------------------------------------
def prefix_set_match(seqs: Sequence[np.ndarray], q: np.ndarray) -> int:
    """Largest k such that q[:k] is a prefix of some stored sequence."""
    prefixes = set()
    for s in seqs:
        s = tuple(int(x) for x in s)
        for k in range(len(s) + 1):
            prefixes.add(s[:k])
    if not prefixes:
        return 0
    qt = tuple(int(x) for x in q)
    best = 0
    for k in range(len(qt) + 1):
        if qt[:k] in prefixes:
            best = k
    return best


def numpy_lcp_match(seqs: Sequence[np.ndarray], q: np.ndarray) -> int:
    """max over s of LCP(q, s) with a padded matrix compare (no loops over tokens)."""
    if len(seqs) == 0:
        return 0
    L = max([len(s) for s in seqs] + [len(q)])
    if L == 0:
        return 0
    M = np.zeros((len(seqs), L), dtype=np.int64)
    valid = np.zeros((len(seqs), L), dtype=bool)
    for i, s in enumerate(seqs):
        M[i, :len(s)] = s
        valid[i, :len(s)] = True
    qq = np.zeros(L, dtype=np.int64)
    qv = np.zeros(L, dtype=bool)
    qq[:len(q)] = q
    qv[:len(q)] = True
    eq = (M == qq[None, :]) & valid & qv[None, :]
    # first False per row (or L if none) = LCP
    notq = ~eq
    first = np.where(notq.any(axis=1), notq.argmax(axis=1), L)
    return int(first.max())


def reference_matrix(peer_sets: List[List[np.ndarray]], queries: List[np.ndarray], fn=numpy_lcp_match):
    m = np.array([[fn(S, q) for S in peer_sets] for q in queries], dtype=np.int64)
    if m.size == 0:
        return m.reshape(len(queries), len(peer_sets)), np.zeros(len(queries), np.int64)
    return m, np.argmax(m, axis=1)


def _peer_lists(w) -> List[List[np.ndarray]]:
    out = []
    for p in range(w.num_peers):
        lo, hi = w.snapshot.peer_range(p)
        out.append([w.snapshot.seq(i) for i in range(lo, hi)])
    return out


def load_all(o, ss, num_peers):
    for p in range(num_peers):
        lo, hi = ss.peer_range(p)
        o.load(p, ss.tokens[ss.offsets[lo]:ss.offsets[hi]], ss.offsets[lo:hi + 1] - ss.offsets[lo])


def check_tiny_random(make: Callable, seeds: Sequence[int], vocabs=(2, 3, 8)) -> List[str]:
    import workloads as W
    fails = []
    for v in vocabs:
        for sd in seeds:
            w = W.tiny_random(sd, num_peers=2 + sd % 4, vocab=v, n_queries=40)
            o = make(w.num_peers)
            load_all(o, w.snapshot, w.num_peers)
            m, c = o.route(w.queries.tokens, w.queries.offsets, 2)
            sets = _peer_lists(w)
            qs = [w.queries.seq(i) for i in range(len(w.queries))]
            m_ps, c_ps = reference_matrix(sets, qs, prefix_set_match)
            m_np, c_np = reference_matrix(sets, qs, numpy_lcp_match)
            if not np.array_equal(m, m_ps) or not np.array_equal(m, m_np):
                bad = np.nonzero((m != m_ps).any(axis=1))[0][:3]
                fails.append(f"vocab={v} seed={sd}: match mismatch at queries {bad.tolist()}")
            if not np.array_equal(c, c_np):
                fails.append(f"vocab={v} seed={sd}: chosen differs from numpy argmax")
    return fails


def check_merge_semantics(make: Callable, seeds: Sequence[int]) -> List[str]:
    """Merging a batch gives exactly max(before, batch alone); permuting or
    duplicating the batch changes nothing; loading twice equals loading once."""
    import workloads as W
    fails = []
    for sd in seeds:
        base = W.tiny_random(sd, num_peers=3, vocab=3, n_queries=50)
        extra = W.tiny_random(sd + 1000, num_peers=3, vocab=3, n_queries=1)
        qt, qo = base.queries.tokens, base.queries.offsets
        P = 3
        a = make(P)
        load_all(a, base.snapshot, P)
        m0, _ = a.route(qt, qo, 1)
        ins = extra.snapshot
        a.merge(ins.peer, ins.tokens, ins.offsets)
        m1, c1 = a.route(qt, qo, 1)
        b = make(P)
        load_all(b, ins, P)
        mb, _ = b.route(qt, qo, 1)
        if (m1 < m0).any():
            fails.append(f"seed {sd}: merge lowered a match")
        if not np.array_equal(m1, np.maximum(m0, mb)):
            fails.append(f"seed {sd}: merge result != max(before, batch alone)")
        # permuted + duplicated batch, and a doubled snapshot load
        perm = np.random.default_rng(sd).permutation(len(ins))
        dup = np.concatenate([perm, perm[: len(perm) // 2]])
        sub = ins.subset(dup)
        d = make(P)
        load_all(d, base.snapshot, P)
        load_all(d, base.snapshot, P)
        d.merge(sub.peer, sub.tokens, sub.offsets)
        m2, c2 = d.route(qt, qo, 1)
        if not np.array_equal(m1, m2) or not np.array_equal(c1, c2):
            fails.append(f"seed {sd}: order/duplicate/reload changed the result")
    return fails


def check_config_invariants(make: Callable, w, idx: np.ndarray, nthreads: int = 4) -> List[str]:
    """Invariants and generator closed forms on a real configuration sample."""
    fails = []
    o = make(w.num_peers)
    load_all(o, w.snapshot, w.num_peers)
    sub = w.queries.subset(idx)
    m, c = o.route(sub.tokens, sub.offsets, nthreads)
    qlen = sub.lengths()
    if (m > qlen[:, None]).any():
        fails.append("m exceeds |q|")
    if not np.array_equal(c, np.argmax(m, axis=1)):
        fails.append("chosen != first argmax")
    # closed forms of the generator: a peer caching the query's topic matches at
    # least the whole shared head; a peer not caching it matches less than that;
    # any peer with a cached prompt matches at least the system prefix.
    meta = w.meta
    head = meta["query_head"][idx]
    hl = meta["head_len"][head]
    cached = [set() for _ in range(w.num_peers)]
    for t, p in zip(meta["cache_topic"].tolist(), w.snapshot.peer.tolist()):
        cached[p].add(t)
    for i in range(len(idx)):
        for p in range(w.num_peers):
            has = int(head[i]) in cached[p]
            if has and m[i, p] < hl[i]:
                fails.append(f"q{idx[i]} p{p}: caches the topic but m={m[i, p]} < {hl[i]}")
            if not has and m[i, p] >= hl[i]:
                fails.append(f"q{idx[i]} p{p}: lacks the topic but m={m[i, p]} >= {hl[i]}")
            if cached[p] and m[i, p] < meta["sys_len"]:
                fails.append(f"q{idx[i]} p{p}: below the system prefix")
        if len(fails) > 5:
            break
    # a cached prompt used as a query matches its owner in full
    rng = np.random.default_rng(7)
    pick = rng.choice(len(w.snapshot), size=min(32, len(w.snapshot)), replace=False)
    ps = w.snapshot.subset(pick)
    mp, _ = o.route(ps.tokens, ps.offsets, nthreads)
    own = w.snapshot.peer[pick]
    if not np.array_equal(mp[np.arange(len(pick)), own], ps.lengths()):
        fails.append("a cached prompt does not match its owner in full")
    return fails


# ---- selection with push-back and failover ----------------------------------
SELECT_GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "select_examples.txt")


def parse_select_golden(path: str = SELECT_GOLDEN):
    """[(name, P, loads {p: [seqs]}, [(eligible, local, prefer, query, best, second)])]."""
    out, cur = [], None
    sel = None
    for raw in open(path):
        line = raw.split("#", 1)[0].strip()
        if not line:
            continue
        kw, _, rest = line.partition(" ")
        if kw == "example":
            cur = [rest.strip(), 0, {}, []]
            out.append(cur)
        elif kw == "peers":
            cur[1] = int(rest)
        elif kw == "load":
            p, _, body = rest.partition("|")
            body = body.strip()
            cur[2][int(p)] = [] if not body else [_toks(x) for x in body.split(";")]
        elif kw == "select":
            bits, local, prefer = rest.split()
            sel = (np.array([int(c) for c in bits], np.uint8), int(local), bool(int(prefer)))
        elif kw == "query":
            q, _, res = rest.partition("->")
            b1, b2 = (int(x) for x in res.split())
            cur[3].append((sel[0], sel[1], sel[2], _toks(q), b1, b2))
        else:
            raise ValueError(f"bad directive {kw!r}")
    return out


def select_order(m_row: np.ndarray, eligible, local: int, prefer: bool) -> List[int]:
    """The candidate order written as a sort: key (-m, local-first flag, id),
    keeping eligible peers and the local one."""
    P = m_row.shape[0]
    ids = np.arange(P)
    loc_key = np.where(prefer & (ids == local), 0, 1)
    order = np.lexsort((ids, loc_key, -m_row.astype(np.int64)))
    keep = np.ones(P, bool) if eligible is None else np.asarray(eligible).astype(bool).copy()
    if local >= 0:
        keep[local] = True
    return [int(p) for p in order if keep[p]]


def check_select_golden(make: Callable) -> List[str]:
    fails = []
    for name, P, loads, cases in parse_select_golden():
        o = make(P)
        for p, seqs in loads.items():
            t, off = _csr(seqs)
            o.load(p, t, off)
        for el, local, prefer, q, b1, b2 in cases:
            t, off = _csr([q])
            _, g1, g2 = o.route_select(t, off, el, local, prefer, 1)
            if (int(g1[0]), int(g2[0])) != (b1, b2):
                fails.append(f"{name}: q={q} eligible={el.tolist()} local={local} prefer={prefer}: "
                             f"got ({int(g1[0])}, {int(g2[0])}) want ({b1}, {b2})")
    return fails


def check_select_random(make: Callable, seeds: Sequence[int]) -> List[str]:
    """Random eligibility, local peer and prefer flag over tiny random forests:
    the oracle's best and second equal the first two of the sorted order, and
    its match matrix equals route()'s."""
    import workloads as W
    fails = []
    for sd in seeds:
        rng = np.random.default_rng(1000 + sd)
        w = W.tiny_random(sd, num_peers=2 + sd % 5, vocab=3, n_queries=40)
        P = w.num_peers
        o = make(P)
        load_all(o, w.snapshot, P)
        m0, c0 = o.route(w.queries.tokens, w.queries.offsets, 2)
        for trial in range(6):
            el = (rng.random(P) < 0.6).astype(np.uint8)
            local = int(rng.integers(-1, P))
            prefer = bool(rng.integers(0, 2))
            m, b1, b2 = o.route_select(w.queries.tokens, w.queries.offsets, el, local, prefer, 2)
            if not np.array_equal(m, m0):
                fails.append(f"seed={sd}: route_select match matrix differs from route")
            for i in range(len(w.queries)):
                order = select_order(m0[i], el, local, prefer) + [-1, -1]
                if (int(b1[i]), int(b2[i])) != (order[0], order[1]):
                    fails.append(f"seed={sd} trial={trial} q={i}: got ({b1[i]}, {b2[i]}) want {order[:2]}")
                    break
        # everyone eligible, no local peer: best is route()'s chosen
        _, b1, _ = o.route_select(w.queries.tokens, w.queries.offsets, None, -1, False, 2)
        if not np.array_equal(b1, c0):
            fails.append(f"seed={sd}: unrestricted best differs from chosen")
    return fails


# ---- snapshot export (sendTrie) -----------------------------------------------
EXPORT_GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "export_examples.txt")


def _seqs(body: str) -> List[List[int]]:
    body = body.strip()
    return [] if not body else [_toks(x) for x in body.split(";")]


def parse_export_golden(path: str = EXPORT_GOLDEN):
    """[(name, P, [("load", p, seqs) | ("merge", [(p, seq)]) | ("export", p, seqs)])]."""
    out, cur = [], None
    for raw in open(path):
        line = raw.split("#", 1)[0].strip()
        if not line:
            continue
        kw, _, rest = line.partition(" ")
        if kw == "example":
            cur = [rest.strip(), 0, []]
            out.append(cur)
        elif kw == "peers":
            cur[1] = int(rest)
        elif kw == "load":
            p, _, body = rest.partition("|")
            cur[2].append(("load", int(p), _seqs(body)))
        elif kw == "merge":
            items = []
            for part in rest.split(";"):
                p, _, seq = part.partition(":")
                items.append((int(p), _toks(seq)))
            cur[2].append(("merge", items))
        elif kw == "export":
            p, _, body = rest.partition("->")
            cur[2].append(("export", int(p), _seqs(body)))
        else:
            raise ValueError(f"bad directive {kw!r}")
    return out


def csr_to_list(t: np.ndarray, o: np.ndarray) -> List[List[int]]:
    return [t[o[i]:o[i + 1]].tolist() for i in range(len(o) - 1)]


def maximal_members(seqs) -> List[tuple]:
    """Brute force: non-empty members that are no proper prefix of another
    member, each once, sorted."""
    S = {tuple(int(x) for x in s) for s in seqs}
    keep = [s for s in S if s and not any(len(t) > len(s) and t[:len(s)] == s for t in S)]
    return sorted(keep)


def check_export_golden(make: Callable) -> List[str]:
    fails = []
    for name, P, ops in parse_export_golden():
        o = make(P)
        for op in ops:
            if op[0] == "load":
                t, off = _csr(op[2])
                o.load(op[1], t, off)
            elif op[0] == "merge":
                t, off = _csr([s for _, s in op[1]])
                o.merge(np.array([p for p, _ in op[1]], np.int32), t, off)
            else:
                got = csr_to_list(*o.export(op[1]))
                if got != op[2]:
                    fails.append(f"{name}: export {op[1]} got {got} want {op[2]}")
    return fails


def check_export_random(make: Callable, seeds: Sequence[int]) -> List[str]:
    """Tiny random forests with merges: the export equals the brute-force
    maximal members (as a sorted list), and loading it into a fresh peer gives
    the same match for every query (the same tree)."""
    import workloads as W
    fails = []
    for sd in seeds:
        w = W.tiny_random(sd, num_peers=3, vocab=2 + sd % 3, n_queries=60)
        P = w.num_peers
        o = make(P)
        load_all(o, w.snapshot, P)
        ins = W.tiny_random(sd + 500, num_peers=P, vocab=2 + sd % 3, n_queries=1)
        o.merge(ins.snapshot.peer, ins.snapshot.tokens, ins.snapshot.offsets)
        sets = [list(x) for x in _peer_lists(w)]
        for i in range(len(ins.snapshot)):
            sets[int(ins.snapshot.peer[i])].append(ins.snapshot.seq(i))
        for p in range(P):
            t, off = o.export(p)
            got = [tuple(x) for x in csr_to_list(t, off)]
            if sorted(got) != maximal_members(sets[p]) or len(set(got)) != len(got):
                fails.append(f"seed={sd} peer={p}: export differs from the maximal members")
                continue
            o2 = make(1)
            o2.load(0, t, off)
            for i in range(len(w.queries)):
                q = w.queries.seq(i)
                if o2.prefix_match(0, q) != o.prefix_match(p, q):
                    fails.append(f"seed={sd} peer={p} q={i}: the exported set matches differently")
                    break
    return fails


# ---- local LRU tree ------------------------------------------------------------
LRU_GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "lru_examples.txt")


def parse_lru_golden(path: str = LRU_GOLDEN):
    out, cur = [], None
    for raw in open(path):
        line = raw.split("#", 1)[0].strip()
        if not line:
            continue
        kw, _, rest = line.partition(" ")
        if kw == "example":
            cur = [rest.strip(), []]
            out.append(cur)
        elif kw == "time":
            cur[1].append(("time", int(rest)))
        elif kw == "load":
            cur[1].append(("load", _seqs(rest.partition("|")[2])))
        elif kw in ("merge", "touch"):
            cur[1].append((kw, _seqs(rest)))
        elif kw == "evict":
            n, _, c = rest.partition("->")
            cur[1].append(("evict", int(n), int(c)))
        elif kw == "export":
            cur[1].append(("export", _seqs(rest.partition("->")[2])))
        elif kw == "match":
            q, _, m = rest.partition("->")
            cur[1].append(("match", _toks(q), int(m)))
        else:
            raise ValueError(f"bad directive {kw!r}")
    return out


def run_lru_ops(make: Callable, ops, check: bool = True) -> List[str]:
    """Apply golden LRU operations to an oracle-like object (local peer 0 of 2)."""
    fails = []
    o = make(2)
    o.set_local(0)
    for op in ops:
        if op[0] == "time":
            o.set_time(op[1])
        elif op[0] == "load":
            t, off = _csr(op[1])
            o.load(0, t, off)
        elif op[0] == "merge":
            t, off = _csr(op[1])
            o.merge(np.zeros(len(op[1]), np.int32), t, off)
        elif op[0] == "touch":
            t, off = _csr(op[1])
            o.touch(t, off)
        elif op[0] == "evict":
            got = o.evict(op[1])
            if got != op[2]:
                fails.append(f"evict {op[1]}: got {got} want {op[2]}")
        elif op[0] == "export":
            got = csr_to_list(*o.export(0))
            if got != op[1]:
                fails.append(f"export: got {got} want {op[1]}")
        elif op[0] == "match":
            got = o.prefix_match(0, np.array(op[1], np.int32))
            if got != op[2]:
                fails.append(f"match {op[1]}: got {got} want {op[2]}")
    return fails


def check_lru_golden(make: Callable) -> List[str]:
    fails = []
    for name, ops in parse_lru_golden():
        fails += [f"{name}: {x}" for x in run_lru_ops(make, ops)]
    return fails


class LruModel:
    """Independent formulation: a dict from every path to its access time;
    n evictions remove the first n paths in the order (time, -length, path)."""

    def __init__(self):
        self.tau = {}

    def load(self, seqs, t):
        self.tau = {}
        self.merge(seqs, t)

    def merge(self, seqs, t):
        for s in seqs:
            s = tuple(int(x) for x in s)
            for k in range(1, len(s) + 1):
                self.tau[s[:k]] = max(self.tau.get(s[:k], t), t)

    def match(self, q) -> int:
        q = tuple(int(x) for x in q)
        m = 0
        while m < len(q) and q[:m + 1] in self.tau:
            m += 1
        return m

    def touch(self, qs, t):
        for q in qs:
            q = tuple(int(x) for x in q)
            for k in range(1, self.match(q) + 1):
                self.tau[q[:k]] = max(self.tau[q[:k]], t)

    def evict(self, n) -> int:
        order = sorted(self.tau, key=lambda p: (self.tau[p], -len(p), p))[:n]
        for p in order:
            del self.tau[p]
        return len(order)

    def export(self):
        return sorted(p for p in self.tau if not any(q[:len(p)] == p and len(q) > len(p) for q in self.tau))


def check_lru_random(make: Callable, seeds: Sequence[int]) -> List[str]:
    """Random loads, merges, touches and evictions on tiny tries: the oracle's
    tree (export and matches) equals the sort-based model's after every step."""
    fails = []
    for sd in seeds:
        rng = np.random.default_rng(4000 + sd)
        vocab = 2 + sd % 3

        def seqs(k, lo=0, hi=7):
            return [rng.integers(0, vocab, size=int(rng.integers(lo, hi))).tolist() for _ in range(k)]

        o = make(2)
        o.set_local(0)
        mdl = LruModel()
        t = 0
        first = seqs(8)
        o.set_time(t)
        tt, off = _csr(first)
        o.load(0, tt, off)
        mdl.load(first, t)
        queries = seqs(12, 0, 9)
        for step in range(14):
            t += int(rng.integers(0, 2))
            o.set_time(t)
            kind = step % 3
            if kind == 0:
                batch = seqs(3)
                tt, off = _csr(batch)
                o.merge(np.zeros(len(batch), np.int32), tt, off)
                mdl.merge(batch, t)
            elif kind == 1:
                batch = [queries[i] for i in rng.integers(0, len(queries), size=4)]
                tt, off = _csr(batch)
                o.touch(tt, off)
                mdl.touch(batch, t)
            else:
                n = int(rng.integers(0, 6))
                got, want = o.evict(n), mdl.evict(n)
                if got != want:
                    fails.append(f"seed={sd} step={step}: evicted {got}, model {want}")
            exp = [tuple(x) for x in csr_to_list(*o.export(0))]
            if exp != mdl.export():
                fails.append(f"seed={sd} step={step}: tree differs from the model")
                break
            for q in queries:
                if o.prefix_match(0, np.array(q, np.int32)) != mdl.match(q):
                    fails.append(f"seed={sd} step={step}: match of {q} differs")
                    break
    return fails
