"""Closed-loop simulation of the decentralized router (Algorithm 1) on N nodes.

Every node owns one forest: its own tree (the local peer, with access times)
and its estimates of the other nodes' trees.  Requests arrive one at a time,
round robin over the nodes, and each runs to completion before the next starts
(the paper's batching-free setup, Section "Experimental Setup").  For request
r arriving at node i:

  * node i routes r: k = the peer with the longest match in i's forest
    (pr_route_select; on equal match its own tree first);
  * if k = i, i runs r; otherwise r is forwarded (a round trip of 2 * comm
    with jitter), k runs it, and i inserts r into its estimate of k
    (UpdateTrieEstimate);
  * running r at node k: serving r refreshes the prefix it reuses (pr_touch),
    then least-recently-used tokens are evicted (pr_evict_lru) until the new
    tokens fit the node's KV budget, and r is inserted into k's own tree
    (UpdateTrie);
  * every poll period each node exports its own tree (sendTrie) and every
    other node replaces its estimate with it (anti-entropy, Section
    "Trie-broadcast loss").

The cost model is synthetic: latency = base + prefill_ms_per_token * (tokens
not cached at the processing node) + the forward's round trip.  The hit of a
request is the match at the processing node's own tree ("actual") and at the
routing node's estimate of it ("expected"), as fractions of the prompt.

The routing itself is the library's; the simulator only drives it through a
backend (RouterBackend below), so that the same trace can be replayed against
another implementation of the calls.
"""
from __future__ import annotations

import argparse
import json
import time
from dataclasses import dataclass, field, asdict
from typing import Dict, List, Optional

import numpy as np


@dataclass
class SimConfig:
    nodes: int = 4
    requests: int = 4000
    topics: int = 57
    prefix_len: tuple = (380, 520)     # few-shot prefix tokens per topic, U{a..b}
    question_len: tuple = (40, 140)    # fresh question tokens per request, U{a..b}
    vocab: int = 32000
    skew: Optional[float] = None       # None: uniform topics; else Zipf exponent over topic ranks
    comm_ms: float = 2.0               # one-way communication latency
    jitter_ms: float = 0.5             # uniform jitter added to each one-way delay
    poll_ms: float = 500.0             # anti-entropy period
    kv_tokens: int = 20000             # KV-cache budget of one node, in tokens
    base_ms: float = 20.0              # fixed cost of a request
    prefill_ms_per_token: float = 0.5  # cost of every token not found in the processing node's cache
    route: bool = True                 # False: every request runs where it arrives (no-routing baseline)
    seed: int = 20261202


class RouterBackend:
    """One node's router: the calls the simulation makes, on the library."""

    def __init__(self, num_peers: int, local: int, device=None):
        import torch
        from .router import Forest
        self.dev = device if device is not None else torch.device("cuda", torch.cuda.current_device())
        self.f = Forest(num_peers)
        self.local = local
        self.f.set_local_peer(local)

    def _csr(self, seqs):
        import torch
        t = np.concatenate([np.asarray(s, np.int32) for s in seqs]) if seqs else np.zeros(0, np.int32)
        o = np.zeros(len(seqs) + 1, np.int64)
        o[1:] = np.cumsum([len(s) for s in seqs])
        return torch.from_numpy(t).to(self.dev), torch.from_numpy(o).to(self.dev)

    def set_time(self, t: int) -> None:
        self.f.set_time(t)

    def route(self, q):
        import torch
        t, o = self._csr([q])
        m, b1, b2 = self.f.route_select(t, o, None, self.local, True)
        torch.cuda.synchronize()
        return m.cpu().numpy()[0], int(b1.cpu()[0]), int(b2.cpu()[0])

    def touch(self, q) -> None:
        t, o = self._csr([q])
        self.f.touch(t, o)

    def tree_tokens(self) -> int:
        return self.f.tree_tokens(self.local)

    def evict(self, n: int) -> int:
        return self.f.evict_lru(n)

    def insert(self, peer: int, q) -> None:
        import torch
        t, o = self._csr([q])
        self.f.merge(torch.tensor([peer], dtype=torch.int32, device=self.dev), t, o)

    def export_local(self):
        return self.f.export_snapshot(self.local)

    def load_estimate(self, peer: int, snapshot) -> None:
        t, o = snapshot
        self.f.load_snapshot_device(peer, t.contiguous(), o)

    def close(self) -> None:
        self.f.close()


def make_workload(cfg: SimConfig):
    """Seeded synthetic prompts: topic prefixes plus fresh questions."""
    rng = np.random.default_rng(np.random.SeedSequence([cfg.seed, 4]))
    heads = [rng.integers(0, cfg.vocab, size=int(rng.integers(cfg.prefix_len[0], cfg.prefix_len[1] + 1)),
                          dtype=np.int32) for _ in range(cfg.topics)]
    if cfg.skew is None:
        p = np.full(cfg.topics, 1.0 / cfg.topics)
    else:
        w = 1.0 / np.power(np.arange(1, cfg.topics + 1, dtype=np.float64), cfg.skew)
        p = (w / w.sum())[rng.permutation(cfg.topics)]
    topic = rng.choice(cfg.topics, size=cfg.requests, p=p)
    qlen = rng.integers(cfg.question_len[0], cfg.question_len[1] + 1, size=cfg.requests)
    prompts = [np.concatenate([heads[t], rng.integers(0, cfg.vocab, size=int(n), dtype=np.int32)])
               for t, n in zip(topic, qlen)]
    jitter = rng.uniform(-cfg.jitter_ms, cfg.jitter_ms, size=(cfg.requests, 2))
    return prompts, topic, jitter


def simulate(cfg: SimConfig, backends: Optional[List] = None, make_backend=None) -> Dict:
    """Run the closed loop.  backends: one RouterBackend-like object per node
    (created with make_backend(num_peers, local) if not given)."""
    N = cfg.nodes
    mk = make_backend or (lambda P, local: RouterBackend(P, local))
    nodes = backends or [mk(N, i) for i in range(N)]
    prompts, topic, jitter = make_workload(cfg)
    clock = 0.0
    next_poll = cfg.poll_ms
    trace = []
    t_calls = 0.0

    def stamp():
        return int(round(clock * 1000))  # microseconds

    def run_at(k, q, hit):
        nonlocal t_calls
        nd = nodes[k]
        t0 = time.perf_counter()
        nd.set_time(stamp())
        nd.touch(q)
        need = max(0, len(q) - hit)
        have = nd.tree_tokens()
        ev = 0
        if have + need > cfg.kv_tokens:
            ev = nd.evict(have + need - cfg.kv_tokens)
        nd.insert(nd.local, q)
        t_calls += time.perf_counter() - t0
        return ev

    for j, q in enumerate(prompts):
        i = j % N
        while clock >= next_poll:  # anti-entropy rounds due before this request
            t0 = time.perf_counter()
            snaps = [nodes[a].export_local() for a in range(N)]
            for b in range(N):
                for a in range(N):
                    if a != b:
                        nodes[b].load_estimate(a, snaps[a])
            t_calls += time.perf_counter() - t0
            next_poll += cfg.poll_ms
        t0 = time.perf_counter()
        for nd in nodes:
            nd.set_time(stamp())
        m_row, best, second = nodes[i].route(q)
        t_calls += time.perf_counter() - t0
        k = best if cfg.route else i
        expected = int(m_row[k])
        delay = 0.0
        if k != i:
            delay = 2 * cfg.comm_ms + jitter[j, 0] + jitter[j, 1]
            t0 = time.perf_counter()
            actual = int(nodes[k].route(q)[0][k])  # the processing node's own tree
            t_calls += time.perf_counter() - t0
        else:
            actual = int(m_row[i])
        ev = run_at(k, q, actual)
        if k != i:
            t0 = time.perf_counter()
            nodes[i].insert(k, q)  # UpdateTrieEstimate after a successful forward
            t_calls += time.perf_counter() - t0
        lat = cfg.base_ms + cfg.prefill_ms_per_token * (len(q) - actual) + delay
        clock += lat
        trace.append({"origin": i, "target": k, "second": second, "topic": int(topic[j]), "len": len(q),
                      "expected": expected, "actual": actual, "evicted": ev, "latency_ms": lat})
    if backends is None:
        for nd in nodes:
            nd.close()
    return {"config": asdict(cfg), "trace": trace, "library_seconds": t_calls, "sim_ms": clock}


def summarize(res: Dict, window: int = 300, stride: int = 30) -> Dict:
    tr = res["trace"]
    N = res["config"]["nodes"]
    tgt = np.array([r["target"] for r in tr])
    ln = np.array([r["len"] for r in tr], np.float64)
    share = np.bincount(tgt, minlength=N) / len(tr)
    tops = np.array([r["topic"] for r in tr])
    # per-topic specialisation: the share of a topic's requests its busiest node takes, per window
    spec = []
    for t in np.unique(tops):
        idx = np.nonzero(tops == t)[0]
        if len(idx) >= window:
            for s in range(0, len(idx) - window + 1, stride):
                spec.append(np.bincount(tgt[idx[s:s + window]], minlength=N).max() / window)
    return {
        "requests": len(tr),
        "hotspot_share": float(share.max()),
        "node_share": share.tolist(),
        "forwarded": float(np.mean([r["origin"] != r["target"] for r in tr])),
        "expected_hit": float(np.sum([r["expected"] for r in tr]) / ln.sum()),
        "actual_hit": float(np.sum([r["actual"] for r in tr]) / ln.sum()),
        "mean_latency_ms": float(np.mean([r["latency_ms"] for r in tr])),
        "evicted_tokens": int(np.sum([r["evicted"] for r in tr])),
        "topic_window_top_share": float(np.mean(spec)) if spec else None,
        "library_seconds": res["library_seconds"],
        "library_us_per_request": res["library_seconds"] / len(tr) * 1e6,
    }


def main() -> int:
    ap = argparse.ArgumentParser(description="closed-loop simulation of Algorithm 1 on the library")
    ap.add_argument("--nodes", type=int, default=4)
    ap.add_argument("--requests", type=int, default=4000)
    ap.add_argument("--skew", type=float, default=None)
    ap.add_argument("--comm-ms", type=float, default=2.0)
    ap.add_argument("--poll-ms", type=float, default=500.0)
    ap.add_argument("--kv-tokens", type=int, default=20000)
    ap.add_argument("--no-route", action="store_true")
    ap.add_argument("--seed", type=int, default=20261202)
    a = ap.parse_args()
    cfg = SimConfig(nodes=a.nodes, requests=a.requests, skew=a.skew, comm_ms=a.comm_ms, poll_ms=a.poll_ms,
                    kv_tokens=a.kv_tokens, route=not a.no_route, seed=a.seed)
    out = summarize(simulate(cfg))
    out["config"] = asdict(cfg)
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
