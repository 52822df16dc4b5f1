#!/usr/bin/env python3
"""Throughput of the batched prefix-cache-aware router on one MI355X.

One step = one pr_route over a full query batch of the workload: every query's
longest-prefix match against every peer's tree plus the argmax over peers
(walk, child locate, label compare, per-peer lengths, argmax, output write).
Queries, offsets, outputs and the forest are resident in HBM before the timed
region; four device copies of the query batch rotate so that the 256 MB
last-level cache cannot serve the query stream from one step to the next (with
one copy, lines read with the default cache policy come back from it).

Prints one JSON line (rank 0 = the only rank).  Algorithmic bytes per query:
  B_q = 4*min(|q|, M_q + 1) + 4*(P + 1) + 8
(the query tokens a walk must read, including the mismatching one; the output
row plus the chosen peer; the int64 query offset).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E, AMD public specification

WORKLOADS = {
    1: "tiny: 4 peers x 200 prompts (64 sys + 16 topics x 256 + 32-128 suffix), 2,048 queries Zipf(1.0), 10% unseen",
    2: "medium: 16 peers x 2,000 prompts (128 sys + 64 topics x 1,024 + 64-256 suffix, 2 homes/topic), "
       "65,536 queries Zipf(1.1), 5% unseen",
    3: "stale: 64 peers x 4,000 prompts (256 sys + 512 tasks x 512-2,048 + suffix, <= 4,096 tokens), "
       "observer-0 estimates with Bernoulli(0.2) drops of the last 1,000 inserts, 262,144 queries Zipf(1.2)",
    4: "long: 32 peers x 500 prompts (256 prefixes x 8,192-32,768 + 128-1,024 suffix), 32,768 queries Zipf(1.0)",
    5: "stream: 128 peers x 2,000 prompts (128 sys + 512 topics x 1,024 + 64-256 suffix), 1,048,576-query lookup batch",
}


def kernel_code_sha(path: str) -> str:
    """sha256 prefix of a kernel source with comments and whitespace removed:
    it changes when the code does, not when a comment does."""
    import hashlib
    import re
    src = open(path).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    return hashlib.sha256(re.sub(r"\s+", " ", src).strip().encode()).hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per launch of the route kernel from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary, or None if it does not cover this workload
    or the kernel code changed since it was taken."""
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", "route_kernel_traffic.json")))[workload]
        sha = kernel_code_sha(os.path.join(ROOT, "paper_2606_17059_amd", "csrc", "route_kernels.h"))
    except (OSError, KeyError, ValueError):
        return None
    return rec["traffic_bytes_per_launch"] if rec.get("kernel_code_sha256_16") == sha else None


def step_kernels(nq: int, ntok: int) -> list:
    """Kernels one pr_route call launches (the library's rule: batches of more
    than 8,192 and at most 65,536 queries averaging at least 4,096 tokens are
    walked longest first, after two order launches).  kernel_ms is the time of
    the whole call, so there it includes the order launches."""
    if 8192 < nq <= 65536 and ntok >= 4096 * nq:
        return ["route_order_count_kernel", "route_order_scatter_kernel", "route_kernel<W, false>"]
    return ["route_kernel<W, false>"]


def route_kernel_name(f) -> str:
    """The plain route kernel instantiation a forest's routes run: mask words
    and label token type (16-bit while every label token fits)."""
    info = f.info()
    lt = "unsigned short" if info["label_token_bytes"] == 2 else "int"
    return f"route_kernel<{info['mask_words']}, false, {lt}>"


def log(msg: str) -> None:
    sys.stderr.write(msg + "\n")
    sys.stderr.flush()


def cpu_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, queries, target_s: float):
    """Time the CPU oracle, as it stands, on a bounded sample of the same batch."""
    import oracle
    o = oracle.Oracle(w.num_peers)
    ss = w.snapshot
    for p in range(w.num_peers):
        lo, hi = ss.peer_range(p)
        o.load(p, ss.tokens[ss.offsets[lo]:ss.offsets[hi]], ss.offsets[lo:hi + 1] - ss.offsets[lo])
    T = cpu_threads()
    rng = np.random.default_rng(12345)
    n = min(len(queries), 4 * T)
    while True:
        idx = np.sort(rng.choice(len(queries), n, replace=False))
        sub = queries.subset(idx)
        t0 = time.perf_counter()
        o.route(sub.tokens, sub.offsets, T)
        dt = time.perf_counter() - t0
        if dt >= 0.25 * target_s or n >= len(queries):
            break
        n = int(min(len(queries), max(2 * n, n * target_s / max(dt, 1e-3))))
    # the same oracle on one thread, over a sample sized to about a fifth of the target time
    n1 = max(1, min(n, int(n * 0.2 * target_s / max(dt * T, 1e-3))))
    sub1 = queries.subset(np.sort(rng.choice(len(queries), n1, replace=False)))
    t0 = time.perf_counter()
    o.route(sub1.tokens, sub1.offsets, 1)
    dt1 = time.perf_counter() - t0
    o.close()
    return {"value": n / dt, "unit": "queries/s", "cores": T, "kind": "oracle",
            "sample": f"{n} of {len(queries)} queries drawn uniformly (seed 12345), {dt:.1f} s with {T} threads",
            "one_thread": {"value": n1 / dt1, "unit": "queries/s", "sample": f"{n1} queries, {dt1:.1f} s"},
            "cpu_model": cpu_model()}


def bench_stream(args, w, dev):
    """Streaming configuration: per round, one delta-merge of the insert batch
    into the replica trees, then lookups of the round's query batch."""
    import torch
    from paper_2606_17059_amd import Forest
    P = w.num_peers
    phases_out = []
    tot_ins = tot_merge_s = tot_q = tot_route_s = tot_bytes = 0.0
    kern_all = []
    compact_out = []
    cpu = None
    # untimed warm-up on a throwaway forest: the first launch of each kernel
    # loads its code object, a one-time cost of the process, not of a merge
    wf = Forest(P)
    wf.load_seqset(w.snapshot.subset(np.arange(min(len(w.snapshot), 4 * P))))
    ph0 = w.phase("uniform", 0)
    wi = ph0.inserts.subset(np.arange(min(len(ph0.inserts), 256)))
    wf.merge(torch.from_numpy(wi.peer).to(dev), torch.from_numpy(wi.tokens).to(dev),
             torch.from_numpy(wi.offsets).to(dev))
    wq = ph0.queries.subset(np.arange(min(len(ph0.queries), 256)))
    wf.route(torch.from_numpy(wq.tokens).to(dev), torch.from_numpy(wq.offsets).to(dev))
    torch.cuda.synchronize()
    wf.close()
    del ph0, wi, wq
    for dist in ("uniform", "zipf"):
        f = Forest(P)
        f.load_seqset(w.snapshot)
        for rnd in range(w.meta["rounds"]):
            t0 = time.perf_counter()
            ph = w.phase(dist, rnd)
            gen_s = time.perf_counter() - t0
            ins, qs = ph.inserts, ph.queries
            ip = torch.from_numpy(ins.peer).to(dev)
            it = torch.from_numpy(ins.tokens).to(dev)
            io = torch.from_numpy(ins.offsets).to(dev)
            qt = torch.from_numpy(qs.tokens).to(dev)
            qo = torch.from_numpy(qs.offsets).to(dev)
            nq = len(qs)
            ml = torch.empty((nq, P), dtype=torch.int32, device=dev)
            ch = torch.empty(nq, dtype=torch.int32, device=dev)
            if rnd == 0:
                f.route(qt, qo, ml, ch)  # builds and uploads the base forest
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            t0 = time.perf_counter()
            e0.record()
            f.merge(ip, it, io)
            e1.record()
            torch.cuda.synchronize()
            merge_s = time.perf_counter() - t0
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for _ in range(args.steps)]
            for a, b in ev:
                a.record()
                f.route(qt, qo, ml, ch)
                b.record()
            torch.cuda.synchronize()
            f.check()
            km = np.array([a.elapsed_time(b) for a, b in ev])
            m = ml.cpu().numpy()
            M = m.max(axis=1).astype(np.int64)
            bq = float((4 * np.minimum(qs.lengths(), M + 1) + 4 * (P + 1) + 8).sum())
            kern_all.extend(km.tolist())
            tot_ins += len(ins)
            tot_merge_s += merge_s
            tot_q += nq * len(km)
            tot_route_s += km.sum() / 1e3
            tot_bytes += bq * len(km)
            ph_rec = {"dist": dist, "round": rnd, "inserts": len(ins), "merge_ms": merge_s * 1e3,
                      "merge_inserts_per_s": len(ins) / merge_s, "lookups": nq,
                      "route_ms": float(km.mean()), "route_gbps": bq / (km.mean() / 1e3) / 1e9,
                      "forest_nodes": f.info()["num_nodes"]}
            phases_out.append(ph_rec)
            log(f"[bench] stream {dist} round {rnd}: gen {gen_s:.1f} s; {ph_rec}")
            if cpu is None and not args.no_cpu_baseline:
                import oracle
                o = oracle.Oracle(P)
                ss = w.snapshot
                for p in range(P):
                    lo, hi = ss.peer_range(p)
                    o.load(p, ss.tokens[ss.offsets[lo]:ss.offsets[hi]], ss.offsets[lo:hi + 1] - ss.offsets[lo])
                t0 = time.perf_counter()
                o.merge(ins.peer, ins.tokens, ins.offsets)
                o_merge_s = time.perf_counter() - t0
                T = cpu_threads()
                rng = np.random.default_rng(12345)
                n = 4 * T
                while True:
                    sub = qs.subset(np.sort(rng.choice(nq, n, replace=False)))
                    t0 = time.perf_counter()
                    o.route(sub.tokens, sub.offsets, T)
                    dt = time.perf_counter() - t0
                    if dt >= 0.25 * args.cpu_seconds or n >= nq:
                        break
                    n = int(min(nq, max(2 * n, n * args.cpu_seconds / max(dt, 1e-3))))
                o.close()
                cpu = {"value": n / dt, "unit": "queries/s", "cores": T, "kind": "oracle",
                       "sample": f"{n} of {nq} lookups of the first uniform round, {dt:.1f} s with {T} threads; "
                                 f"oracle merge of that round's {len(ins)} inserts: "
                                 f"{len(ins) / o_merge_s:.0f} inserts/s (1 thread)",
                       "cpu_model": cpu_model()}
                log(f"[bench] cpu baseline: {cpu}")
            if args.compact and rnd == w.meta["rounds"] - 1:
                compact_out.append(bench_compact(f, qt, qo, ml, ch, qs, args.steps, dist, float(km.mean())))
                log(f"[bench] compact: {compact_out[-1]}")
            del qt, qo, ml, ch
        kname = route_kernel_name(f)
        f.close()
    kern = np.array(kern_all)
    achieved = tot_bytes / tot_route_s / 1e9
    return {
        "value": tot_q / tot_route_s, "ms_per_step": float(kern.mean()), "kernel_ms": float(kern.mean()),
        "achieved": achieved, "bytes_per_launch": tot_bytes / len(kern), "kernel": kname,
        "merge": {"inserts_per_s": tot_ins / tot_merge_s, "inserts": tot_ins, "seconds": tot_merge_s,
                  "note": "wall time of pr_merge calls (host-synchronous), 8 rounds x 10,000 inserts"},
        "phases": phases_out, "cpu": cpu, "compact": compact_out or None}


def bench_compact(f, qt, qo, ml, ch, qs, steps, dist, route_ms_before) -> dict:
    """Compaction after the last merge round: records and label tokens before
    and after, wall time of the (host-synchronous) call, and the lookup kernel
    time on the same batch before and after."""
    import torch
    i0 = f.info()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    before, after = f.compact()
    ms = (time.perf_counter() - t0) * 1e3
    i1 = f.info()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in ev:
        a.record()
        f.route(qt, qo, ml, ch)
        b.record()
    torch.cuda.synchronize()
    f.check()
    km = np.array([a.elapsed_time(b) for a, b in ev])
    return {"dist": dist, "nodes_before": before, "nodes_after": after, "pool_before": i0["pool_tokens"],
            "pool_after": i1["pool_tokens"], "compact_ms": ms, "nodes_per_s": before / (ms / 1e3),
            "route_ms_before": route_ms_before, "route_ms_after": float(km.mean())}


def bench_select(f, w, qt, qo, needed, K, warmup, dev) -> dict:
    """Time pr_route_select on the same batch: 75% of peers eligible (seeded),
    local peer 0 preferred on ties, best and second-best written; once with the
    match-length matrix and once with the two picks only."""
    import torch
    from paper_2606_17059_amd import eligible_words
    P = w.num_peers
    nq = len(w.queries)
    el = (np.random.default_rng(20261202).random(P) < 0.75).astype(np.uint8)
    elw = torch.from_numpy(eligible_words(el)).to(dev)
    ml = torch.empty((nq, P), dtype=torch.int32, device=dev)
    b1 = torch.empty(nq, dtype=torch.int32, device=dev)
    b2 = torch.empty(nq, dtype=torch.int32, device=dev)
    out = {"eligible_peers": int(el.sum()), "local_peer": 0, "prefer_local": True}
    for name, mlx, extra_bytes in (("with_match_len", ml, 4 * (P + 2)), ("picks_only", None, 8)):
        def call(k):
            f.route_select(qt[k % len(qt)], qo[k % len(qo)], elw, 0, True, mlx, b1, b2,
                           want_match_len=mlx is not None)
        for i in range(warmup):
            call(i)
        torch.cuda.synchronize()
        # as for pr_route: K calls back to back between one pair of events
        # (the host enqueues faster than the kernel runs), then the spread
        # with each launch between its own events
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for k in range(K):
            call(k)
        e1.record()
        torch.cuda.synchronize()
        region_ms = e0.elapsed_time(e1) / K
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
        for k in range(K):
            ev[k][0].record()
            call(k)
            ev[k][1].record()
        torch.cuda.synchronize()
        ms = np.array([a.elapsed_time(b) for a, b in ev])
        byts = float((4 * needed + extra_bytes + 8).sum())
        out[name] = {"kernel_ms": region_ms,
                     "kernel_ms_own_events": {"mean": float(ms.mean()), "median": float(np.median(ms))},
                     "queries_per_s": nq / (region_ms / 1e3),
                     "algorithmic_bytes_per_launch": byts,
                     "hbm_gbps": byts / (region_ms / 1e3) / 1e9,
                     "frac": byts / (region_ms / 1e3) / 1e9 / PEAK_HBM_GBPS}
    f.check()
    return out


def bench_latency(f, w, dev, reps: int = 200) -> dict:
    """Small batches, as a router serving requests as they arrive would send
    them: the first b queries of the batch, per call the host wall time of
    pr_route plus a stream synchronisation, and of pr_route plus the copy of
    the chosen peers into pinned host memory, and of one replay of a HIP graph
    holding the launch (medians over `reps` calls), and the GPU time per
    launch of back-to-back launches."""
    import torch
    q = w.queries
    P = w.num_peers
    out = {}
    for b in (1, 8, 64, 512, 4096, 32768):
        if b > len(q):
            break
        end = int(q.offsets[b])
        qt = torch.from_numpy(q.tokens[:end].copy()).to(dev)
        qo = torch.from_numpy(q.offsets[:b + 1].copy()).to(dev)
        ml = torch.empty((b, P), dtype=torch.int32, device=dev)
        ch = torch.empty(b, dtype=torch.int32, device=dev)
        host = torch.empty(b, dtype=torch.int32, pin_memory=True)
        launch = f.route_launcher(qt, qo, ml, ch)
        for _ in range(20):
            launch()
        torch.cuda.synchronize()
        sync_us, copy_us = np.empty(reps), np.empty(reps)
        for i in range(reps):
            t0 = time.perf_counter()
            launch()
            torch.cuda.synchronize()
            sync_us[i] = (time.perf_counter() - t0) * 1e6
        for i in range(reps):
            t0 = time.perf_counter()
            launch()
            host.copy_(ch, non_blocking=True)
            torch.cuda.synchronize()
            copy_us[i] = (time.perf_counter() - t0) * 1e6
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            launch()
        e1.record()
        torch.cuda.synchronize()
        # the same launch captured into a HIP graph and replayed
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            f.route_launcher(qt, qo, ml, ch, stream=side)()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            f.route_launcher(qt, qo, ml, ch, stream=torch.cuda.current_stream())()
        torch.cuda.synchronize()
        graph_us = np.empty(reps)
        for i in range(reps):
            t0 = time.perf_counter()
            g.replay()
            torch.cuda.synchronize()
            graph_us[i] = (time.perf_counter() - t0) * 1e6
        del g
        out[str(b)] = {"query_tokens": end, "route_sync_us": float(np.median(sync_us)),
                       "route_sync_p99_us": float(np.percentile(sync_us, 99)),
                       "route_chosen_to_host_us": float(np.median(copy_us)),
                       "graph_replay_sync_us": float(np.median(graph_us)),
                       "gpu_us_per_launch_back_to_back": e0.elapsed_time(e1) * 1e3 / reps}
        log(f"[bench] latency b={b}: {out[str(b)]}")
    f.check()
    return out


def bench_snapshot(f, w, dev, peers: int = 4) -> dict:
    """Anti-entropy on the device: export peers 0..peers-1 (sendTrie) and load
    each export back into the same peer (receive side, device input).  The
    exported set rebuilds the same tree, so routing does not change.  Both
    calls are host-synchronous; wall time per call."""
    import torch
    out = {"peers": peers, "export": [], "load": []}
    for p in range(min(peers, w.num_peers)):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        toks, offs = f.export_snapshot(p)
        t1 = time.perf_counter()
        ns, nt = offs.numel() - 1, toks.numel()
        f.load_snapshot_device(p, toks.contiguous(), offs)
        t2 = time.perf_counter()
        out["export"].append({"peer": p, "ms": (t1 - t0) * 1e3, "seqs": ns, "tokens": nt,
                              "tokens_per_s": nt / (t1 - t0)})
        out["load"].append({"peer": p, "ms": (t2 - t1) * 1e3, "seqs": ns, "tokens": nt,
                            "inserts_per_s": ns / (t2 - t1), "tokens_per_s": nt / (t2 - t1)})
    f.check()
    return out


def bench_lru(f, w, qt, qo, dev) -> dict:
    """Local tree LRU on the device: peer 0 is local; the whole query batch is
    touched at time 2 (its matched prefixes refreshed), then 1%, 5% and 20% of
    the local tree's tokens are evicted in turn.  Host-synchronous calls; wall
    time each."""
    import torch
    out = {"local_peer": 0}
    f.set_time(1)
    f.set_local_peer(0)
    toks0, _ = f.export_snapshot(0)
    f.set_time(2)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    f.touch(qt[0], qo[0])
    out["touch"] = {"queries": len(w.queries), "ms": (time.perf_counter() - t0) * 1e3}
    out["touch"]["queries_per_s"] = len(w.queries) / (out["touch"]["ms"] / 1e3)
    total = int(toks0.numel())  # tokens of the local tree's maximal paths (an upper bound of its size)
    out["evict"] = []
    for frac in (0.01, 0.05, 0.20):
        n = max(1, int(total * frac))
        t0 = time.perf_counter()
        got = f.evict_lru(n)
        ms = (time.perf_counter() - t0) * 1e3
        out["evict"].append({"requested": n, "evicted": got, "ms": ms, "tokens_per_s": got / (ms / 1e3)})
    f.check()
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=2, choices=sorted(WORKLOADS))
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU time of the oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--lru", action="store_true",
                    help="also time touching the batch in the local tree and LRU evictions")
    ap.add_argument("--snapshot", action="store_true",
                    help="also time snapshot export and device-input load of a few peers")
    ap.add_argument("--compact", action="store_true",
                    help="config 5: compact the forest after the last merge round and time it")
    ap.add_argument("--latency", action="store_true",
                    help="also time small batches (1 to 32,768 queries) per call, host wall time included")
    ap.add_argument("--no-select", action="store_true",
                    help="skip timing pr_route_select (push-back / failover selection)")
    ap.add_argument("--copies", type=int, default=4, help="device copies of the query batch to rotate")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="first copy a buffer of this size device-to-device three times (a plain copy kernel "
                         "of known size for scaling profiler byte counters)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        sys.stderr.write("bench.py: measures one GPU only; runs on several GPUs are not supported "
                         "(queries would shard across GPUs with the forest replicated)\n")
        return 2

    import torch

    import workloads as W
    from paper_2606_17059_amd import Forest

    if not torch.cuda.is_available():
        sys.stderr.write("bench.py needs a HIP device\n")
        return 1
    dev = torch.device("cuda:0")
    if args.copy_probe_mib > 0:
        a = torch.empty(args.copy_probe_mib << 18, dtype=torch.int32, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        log(f"[bench] copy probe: 3 copies of {args.copy_probe_mib} MiB")
        del a, b
    t0 = time.perf_counter()
    w = W.make_config(args.config)
    if args.config == 5:
        r = bench_stream(args, w, dev)
        out = {
            "metric": "routed queries/sec (batched LPM over all peer trees) + achieved HBM GB/s",
            "value": r["value"], "unit": "queries/s", "n_gpus": 1, "steps": args.steps, "warmup": 0,
            "ms_per_step": r["ms_per_step"], "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": "int32", "data": "synthetic",
            "config": {"workload": WORKLOADS[5], "config_index": 5, "peers": w.num_peers,
                       "queries_per_step": w.meta["phase_queries"], "parallelism": "single GPU"},
            "hbm_gbps": r["achieved"],
            "roofline": {"bound": "hbm", "achieved": r["achieved"], "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                         "frac": r["achieved"] / PEAK_HBM_GBPS, "traffic": measured_traffic("stream"),
                         "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                         "kernel": r["kernel"],
                         "kernel_ms": r["kernel_ms"], "algorithmic_bytes_per_launch": r["bytes_per_launch"]},
            "cpu_baseline": r["cpu"], "merge": r["merge"], "phases": r["phases"]}
        if r["compact"]:
            out["compact"] = r["compact"]
        print(json.dumps(out), flush=True)
        return 0
    queries = w.queries
    log(f"[bench] generated config {args.config} in {time.perf_counter() - t0:.1f} s: "
        f"{len(w.snapshot)} cached prompts, {len(queries)} queries")

    f = Forest(w.num_peers)
    f.load_seqset(w.snapshot)
    qt = [torch.from_numpy(queries.tokens).to(dev) for _ in range(max(1, args.copies))]
    qo = [torch.from_numpy(queries.offsets).to(dev) for _ in range(max(1, args.copies))]
    nq = len(queries)
    P = w.num_peers
    ml = torch.empty((nq, P), dtype=torch.int32, device=dev)
    ch = torch.empty(nq, dtype=torch.int32, device=dev)
    t0 = time.perf_counter()
    f.route(qt[0], qo[0], ml, ch)  # first route builds and uploads the forest
    torch.cuda.synchronize()
    log(f"[bench] forest build + upload + first route {time.perf_counter() - t0:.2f} s; {f.info()}")

    # buffers checked once; the timed loop only launches (host time per launch
    # well below the kernel's, so the queue never runs dry)
    launch = [f.route_launcher(qt[i], qo[i], ml, ch) for i in range(len(qt))]
    for i in range(args.warmup):
        launch[i % len(launch)]()
    torch.cuda.synchronize()

    # timed region: K launches back to back on the current stream between one
    # pair of HIP events; the host enqueues far faster than the kernel runs, so
    # the region's length over K is the kernel's average launch duration (event
    # markers between launches would add GPU time of their own)
    K = args.steps
    all0, all1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    all0.record()
    for k in range(K):
        launch[k % len(launch)]()
    all1.record()
    torch.cuda.synchronize()
    total_ms = all0.elapsed_time(all1)
    f.check()
    # after the timed region: per-launch spread, each launch between its own events
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    for k in range(K):
        ev[k][0].record()
        launch[k % len(launch)]()
        ev[k][1].record()
    torch.cuda.synchronize()
    kern_ms = np.array([a.elapsed_time(b) for a, b in ev])

    m = ml.cpu().numpy()
    M = m.max(axis=1).astype(np.int64)
    qlen = queries.lengths()
    needed = np.minimum(qlen, M + 1)
    bytes_q = 4 * needed + 4 * (P + 1) + 8
    total_bytes = float(bytes_q.sum())
    avg_kernel_s = total_ms / K / 1e3
    achieved = total_bytes / avg_kernel_s / 1e9
    value = nq * K / (total_ms / 1e3)
    log(f"[bench] timed region: {K} launches in {total_ms:.4f} ms, {total_ms / K:.4f} ms per launch; "
        f"algorithmic bytes/launch {total_bytes / 1e6:.1f} MB")
    log(f"[bench] per-launch ms (own events, after the timed region): mean {kern_ms.mean():.4f} "
        f"median {np.median(kern_ms):.4f} min {kern_ms.min():.4f} max {kern_ms.max():.4f}")

    extra = {}
    if args.config == 3:
        # the same batch routed on the peers' true trees: how often the stale
        # estimates pick the same peer, and the prefill reuse they predict vs get
        ft = Forest(P)
        ft.load_seqset(w.true_snapshot)
        mt, ct = ft.route(qt[0], qo[0])
        torch.cuda.synchronize()
        ft.close()
        mt, ct = mt.cpu().numpy(), ct.cpu().numpy()
        ce = ch.cpu().numpy()
        rows = np.arange(nq)
        tot = float(qlen.sum())
        extra["stale_report"] = {
            "route_agreement": float((ce == ct).mean()),
            "expected_hit": float(m[rows, ce].sum() / tot),
            "actual_hit": float(mt[rows, ce].sum() / tot),
            "oracle_true_hit": float(mt[rows, ct].sum() / tot)}
        log(f"[bench] stale report: {extra['stale_report']}")

    if not args.no_select:
        extra["select"] = bench_select(f, w, qt, qo, needed, K, args.warmup, dev)
        log(f"[bench] select: {extra['select']}")
    if args.latency:
        extra["latency"] = bench_latency(f, w, dev)
    if args.lru:
        # after the timed routes: touches and evictions change the forest
        extra["lru"] = bench_lru(f, w, qt, qo, dev)
        log(f"[bench] lru: {extra['lru']}")
    if args.snapshot:
        # after the timed routes: the device loads switch the forest to its device path
        extra["snapshot"] = bench_snapshot(f, w, dev)
        log(f"[bench] snapshot: {extra['snapshot']}")

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, queries, args.cpu_seconds)
        log(f"[bench] cpu baseline: {cpu}")

    out = {
        "metric": "routed queries/sec (batched LPM over all peer trees) + achieved HBM GB/s",
        "value": value,
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": total_ms / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": WORKLOADS[args.config], "config_index": args.config, "peers": P,
                   "queries_per_step": nq, "query_tokens": int(qlen.sum()), "parallelism": "single GPU"},
        "hbm_gbps": achieved,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBPS, "traffic": measured_traffic(W.CONFIG_NAMES[args.config]),
                     "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "kernel": route_kernel_name(f), "kernel_ms": total_ms / K,
                     "kernel_ms_own_events": {"mean": float(kern_ms.mean()), "median": float(np.median(kern_ms))},
                     "kernels_per_step": step_kernels(nq, int(qlen.sum())),
                     "algorithmic_bytes_per_launch": total_bytes},
        "cpu_baseline": cpu,
    }
    out.update(extra)
    print(json.dumps(out), flush=True)
    f.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
