#!/usr/bin/env python3
"""Throughput of the batched prefix-cache-aware router on one MI355X.

Default workload: the largest single-GPU one, the streaming workload (128
peers x 2,000 prompts).  One step = for each of its two topic distributions
(uniform, Zipf 1.2), the delta-merge of a fresh 10,000-insert batch into that
distribution's forest followed by a lookup batch of 1,048,576 queries on it:
every row of the hot path (walk, child locate, label compare, per-peer
lengths, argmax, output write, merge).  `value` is the lookups routed per
second of step wall time (merges included); the lookup kernel alone and the
merges are reported beside it.  `--config N` (1-4) makes a single lookup batch
of that workload the step instead; `--extra-configs` (default 2,3,4) measures
those workloads' lookup batches too, under "configs".

Inputs are resident in HBM before the timed region.  Every timed output is
compared with the radix-tree CPU oracle afterwards (bit-exact or the run
fails), and the oracle's match lengths give the algorithmic bytes per query:
  B_q = 4*min(|q|, M_q + 1) + 4*(P + 1) + 8
(the query tokens a walk must read, including the mismatching one; the output
row plus the chosen peer; the int64 query offset).  Lookup workloads rotate
four device copies of their batch so that the 256 MB last-level cache cannot
serve the query stream from one launch to the next.

Prints one JSON line (rank 0 = the only rank).
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
    """The plain route kernel instantiation a forest's routes run: mask words,
    label token type (16-bit while every label token fits 17 bits), whether
    bit 16 comes from the bit plane, and the first-level window in 64-token
    vectors."""
    info = f.info()
    lt = "int" if info["label_bits"] == 32 else "unsigned short"
    hb = "true" if info["label_bits"] == 17 else "false"
    return f"route_kernel<{info['mask_words']}, false, {lt}, {hb}, {info['first_window_tokens'] // 64}>"


def log(msg: str) -> None:
    sys.stderr.write(msg + "\n")
    sys.stderr.flush()


def cpu_threads() -> int:
    """Threads for the CPU oracle: the CPUs this process may run on, at most 16
    (one GPU's share of a host with several GPUs)."""
    return max(1, min(16, host_cpus()["affinity"]))


def host_cpus() -> dict:
    try:
        aff = len(os.sched_getaffinity(0))
    except AttributeError:
        aff = os.cpu_count() or 1
    return {"logical": os.cpu_count() or 1, "affinity": aff}


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _time_oracle(o, queries, idx, T):
    sub = queries.subset(idx)
    t0 = time.perf_counter()
    o.route(sub.tokens, sub.offsets, T)
    return time.perf_counter() - t0


def cpu_baseline(make_oracles, queries, target_s: float, what: str):
    """The CPU oracles, as they stand, timed on bounded samples of the batch the
    GPU routes: the radix-tree oracle (one tree per peer, the paper's own
    structure) on T threads and on one thread, and the linear-scan oracle on T
    threads.  ``make_oracles()`` returns (radix, linear) loaded with the forest
    the GPU routes on."""
    radix, linear = make_oracles()
    T = cpu_threads()
    rng = np.random.default_rng(12345)
    nq = len(queries)

    def grow(o, threads, budget):
        n = min(nq, 4 * threads)
        while True:
            idx = np.sort(rng.choice(nq, n, replace=False))
            dt = _time_oracle(o, queries, idx, threads)
            if dt >= 0.25 * budget or n >= nq:
                return n, dt
            n = int(min(nq, max(2 * n, n * budget / max(dt, 1e-3))))

    n, dt = grow(radix, T, 0.5 * target_s)
    n1, dt1 = grow(radix, 1, 0.15 * target_s)
    nl, dtl = grow(linear, T, 0.25 * target_s)
    radix.close()
    linear.close()
    cpus = host_cpus()
    return {"value": n / dt, "unit": "queries/s", "cores": T, "kind": "oracle",
            "oracle": "radix trees, one per peer (oracle/radix_oracle.c)",
            "sample": f"{n} of {nq} {what} drawn uniformly (seed 12345), {dt:.1f} s on {T} threads",
            "one_thread": {"value": n1 / dt1, "unit": "queries/s", "sample": f"{n1} queries, {dt1:.1f} s"},
            "linear_scan": {"value": nl / dtl, "unit": "queries/s", "threads": T,
                            "oracle": "max over stored sequences of the LCP (oracle/prefix_oracle.c)",
                            "sample": f"{nl} queries, {dtl:.1f} s"},
            "host_logical_cpus": cpus["logical"], "affinity_cpus": cpus["affinity"],
            "threads_note": "threads = the CPUs this process may use, at most 16 (one GPU's share of the host)",
            "cpu_model": cpu_model()}


def _upload(ss, dev):
    import torch
    return (torch.from_numpy(np.ascontiguousarray(ss.tokens, dtype=np.int32)).to(dev),
            torch.from_numpy(np.ascontiguousarray(ss.offsets, dtype=np.int64)).to(dev))


def _alg_bytes(queries, M, P) -> np.ndarray:
    """B_q = 4 min(|q|, M_q + 1) + 4 (P + 1) + 8 per query."""
    return 4 * np.minimum(queries.lengths(), M.astype(np.int64) + 1) + 4 * (P + 1) + 8


def cu_split_streams(dev, merge_cus_per_xcd: int):
    """Two streams over disjoint sets of compute units (hipExtStreamCreateWithCUMask):
    merges on merge_cus_per_xcd CUs of each of the 8 XCDs, lookups on the rest.
    The CU picked as the c-th of XCD j has mask bit per*j + j + 8*c (per = CUs
    per XCD): that is a CU of XCD j whether the mask numbers CUs XCD by XCD or
    round-robin over the XCDs.  Returns (lookup stream, merge stream, counts)."""
    import ctypes

    import torch
    hip = ctypes.CDLL("libamdhip64.so.7")  # torch's HIP runtime, already loaded
    n_cu = torch.cuda.get_device_properties(dev).multi_processor_count
    n_xcd = 8
    per = n_cu // n_xcd
    if per * n_xcd != n_cu or not 0 < merge_cus_per_xcd <= per // n_xcd:
        raise SystemExit(f"bench.py: cannot reserve {merge_cus_per_xcd} CUs per XCD on {n_cu} CUs")
    merge_bits = {per * j + j + n_xcd * c for j in range(n_xcd) for c in range(merge_cus_per_xcd)}
    n_words = (n_cu + 31) // 32

    def make(bits):
        words = (ctypes.c_uint32 * n_words)()
        for b in bits:
            words[b // 32] |= 1 << (b % 32)
        h = ctypes.c_void_p()
        if hip.hipExtStreamCreateWithCUMask(ctypes.byref(h), ctypes.c_uint32(n_words), words) != 0:
            raise SystemExit("bench.py: hipExtStreamCreateWithCUMask failed")
        return torch.cuda.ExternalStream(h.value, device=dev), h

    look, hl = make(set(range(n_cu)) - merge_bits)
    merge, hm = make(merge_bits)
    return look, merge, {"lookup_cus": n_cu - len(merge_bits), "merge_cus": len(merge_bits),
                         "handles": (hip, hl, hm)}


def bench_stream(args, dev) -> dict:
    """The streaming workload, 128 peers.  One step = for each topic
    distribution (uniform, Zipf 1.2), the delta-merge of a fresh batch of
    10,000 inserts into that distribution's forest, then a lookup batch of
    1,048,576 queries on it.  Each forest has its own stream and host thread;
    the two fall into step: both merges (latency-bound: small kernels and one
    readback each) run side by side, then both lookups share HBM.  A kernel
    queued on one stream while a lookup's million waves fill the chip on the
    other waits for that lookup to drain, so a merge gains nothing from
    running beside the other forest's lookup (--schedule pipelined: one host
    thread issuing merge A, lookup A, merge B, lookup B, with no wait between
    them, measures that); --schedule serial runs everything in turn on one
    stream.  Merges are also timed alone after the timed region.  Every lookup of every timed step is compared
    with the radix-tree oracle after the timed region, and the algorithmic
    bytes come from the oracle's match lengths."""
    import torch

    import oracle
    import workloads as W
    from paper_2606_17059_amd import Forest
    t_gen = time.perf_counter()
    w = W.make_config(5)
    P, R = w.num_peers, w.meta["rounds"]
    dists = ("uniform", "zipf")
    Wu, K = args.warmup, args.steps
    n_steps = Wu + K
    if n_steps + 4 > W.MAX_STREAM_ROUNDS:
        raise SystemExit(f"bench.py: at most {W.MAX_STREAM_ROUNDS} warm-up + timed steps on the streaming workload")
    # lookups: the R rounds' batches of each distribution, taken in turn by
    # the steps (fresh for the first R rounds, then again on the grown forest)
    qhost = {d: [] for d in dists}
    qdev = {d: [] for d in dists}
    for d in dists:
        for r in range(R):
            q = w.query_batch(d, r)
            qhost[d].append(q)
            qdev[d].append(_upload(q, dev))
            log(f"[bench] stream: lookup batch {d} {r}: {len(q)} queries, {q.tokens.size} tokens "
                f"({time.perf_counter() - t_gen:.1f} s)")
    ihost = {d: [w.insert_batch(d, k) for k in range(n_steps)] for d in dists}
    idev = {d: [(torch.from_numpy(b.peer).to(dev),) + _upload(b, dev) for b in ihost[d]] for d in dists}
    log(f"[bench] stream: {n_steps} insert batches per distribution generated and uploaded "
        f"({time.perf_counter() - t_gen:.1f} s)")
    nq = len(qhost[dists[0]][0])
    # outputs: one pair per timed step and distribution (checked afterwards),
    # one scratch pair for the warm-up steps
    outs = {d: [(torch.empty((nq, P), dtype=torch.int32, device=dev), torch.empty(nq, dtype=torch.int32, device=dev))
                for _ in range(K)] for d in dists}
    warm_out = (torch.empty((nq, P), dtype=torch.int32, device=dev), torch.empty(nq, dtype=torch.int32, device=dev))
    # the first launch of each kernel in a process loads its code object: a
    # one-time cost of the process, paid on a throwaway forest
    wf = Forest(P)
    wf.load_seqset(w.snapshot.subset(np.arange(4 * P)))
    wi = ihost[dists[0]][0].subset(np.arange(256))
    wf.merge(torch.from_numpy(wi.peer).to(dev), *_upload(wi, dev))
    wq = qhost[dists[0]][0].subset(np.arange(256))
    wf.route(*_upload(wq, dev))
    torch.cuda.synchronize()
    wf.close()
    forests, streams = {}, {}
    for d in dists:
        forests[d] = Forest(P)
        forests[d].load_seqset(w.snapshot)
        streams[d] = (torch.cuda.Stream(device=dev) if args.schedule != "serial" or d == dists[0]
                      else streams[dists[0]])
        forests[d].route(*qdev[d][0], *warm_out)  # builds and uploads the base forest
    torch.cuda.synchronize()
    log(f"[bench] stream: base forests uploaded ({forests[dists[0]].info()})")
    ev = {d: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
          for d in dists}
    merge_s = {d: np.zeros(n_steps) for d in dists}
    t_region = time.perf_counter()

    # lookups: each forest's own stream, or one stream both forests' lookups
    # queue on in turn (--schedule shared)
    look_s = torch.cuda.Stream(device=dev) if args.schedule == "shared" else None
    last_lookup = {d: None for d in dists}

    def run_steps(d, ks):
        f, s = forests[d], streams[d]
        ls = look_s if look_s is not None else s
        for k in ks:
            if args.schedule == "serial":
                s.synchronize()  # the previous lookup is done: the merge's wall time is its own
            if look_s is not None and last_lookup[d] is not None:
                s.wait_event(last_lookup[d])  # the merge changes records that lookup reads
            t0 = time.perf_counter()
            f.merge(*idev[d][k], stream=s)  # returns when the forest holds the batch
            merge_s[d][k] = time.perf_counter() - t0
            if look_s is not None:
                ls.wait_stream(s)
            qt, qo = qdev[d][k % R]
            if k >= Wu:
                a, b = ev[d][k - Wu]
                a.record(ls)
                f.route(qt, qo, *outs[d][k - Wu], stream=ls)
                b.record(ls)
            else:
                f.route(qt, qo, *warm_out, stream=ls)
            if look_s is not None:
                last_lookup[d] = torch.cuda.Event()
                last_lookup[d].record(ls)

    cu_split = None
    if args.schedule == "cusplit":
        # one host thread; lookups on one stream over most of the CUs, merges
        # on another over the few CUs kept from the lookups.  A forest's merge
        # waits for its previous lookup (it changes records that lookup reads)
        # and its lookup for the merge; the other forest's lookup runs meanwhile
        lstream, mstream, cu_split = cu_split_streams(dev, args.merge_cus)
        last_lookup = {d: None for d in dists}
        for k in range(n_steps):
            if k == Wu:
                torch.cuda.synchronize()
                t_region = time.perf_counter()
            for d in dists:
                f = forests[d]
                if last_lookup[d] is not None:
                    mstream.wait_event(last_lookup[d])
                t0 = time.perf_counter()
                f.merge(*idev[d][k], stream=mstream)  # returns when the forest holds the batch
                merge_s[d][k] = time.perf_counter() - t0
                done = torch.cuda.Event()
                done.record(mstream)
                lstream.wait_event(done)
                qt, qo = qdev[d][k % R]
                if k >= Wu:
                    a, b = ev[d][k - Wu]
                    a.record(lstream)
                    f.route(qt, qo, *outs[d][k - Wu], stream=lstream)
                    b.record(lstream)
                else:
                    f.route(qt, qo, *warm_out, stream=lstream)
                last_lookup[d] = torch.cuda.Event()
                last_lookup[d].record(lstream)
    elif args.schedule in ("threads", "shared"):
        # one host thread per forest (the library's calls release the
        # interpreter lock): each forest's merge, then lookup, on its own
        # stream, while the other forest's run beside them
        import threading
        barrier = threading.Barrier(len(dists) + 1)
        errors = []

        def worker(d):
            try:
                run_steps(d, range(Wu))
                torch.cuda.synchronize()
                barrier.wait()
                barrier.wait()  # the main thread has started the clock
                run_steps(d, range(Wu, n_steps))
            except BaseException as e:  # reported by the main thread
                errors.append(e)
                barrier.abort()

        threads = [threading.Thread(target=worker, args=(d,)) for d in dists]
        for t in threads:
            t.start()
        try:
            barrier.wait()
            torch.cuda.synchronize()
            t_region = time.perf_counter()
            barrier.wait()
        except threading.BrokenBarrierError:
            pass
        for t in threads:
            t.join()
        if errors:
            raise errors[0]
    else:
        for k in range(n_steps):
            if k == Wu:
                torch.cuda.synchronize()
                t_region = time.perf_counter()
            for d in dists:
                run_steps(d, [k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_region
    if cu_split is not None:
        hip, hl, hm = cu_split.pop("handles")
        hip.hipStreamDestroy(hl)
        hip.hipStreamDestroy(hm)
    for d in dists:
        forests[d].check()
    route_ms = {d: np.array([a.elapsed_time(b) for a, b in ev[d]]) for d in dists}
    log(f"[bench] stream: timed region {K} steps in {wall * 1e3:.2f} ms; route ms mean "
        f"{ {d: round(float(route_ms[d].mean()), 4) for d in dists} }; merge ms mean "
        f"{ {d: round(float(merge_s[d][Wu:].mean() * 1e3), 3) for d in dists} }")
    # the lookup kernel alone, for the roofline: K launches back to back on
    # each forest as the timed steps left it, over the last step's batch (whose
    # algorithmic bytes the oracle gives below)
    iso_ms = {}
    for d in dists:
        qt, qo = qdev[d][(n_steps - 1) % R]
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(streams[d])
        for _ in range(K):
            forests[d].route(qt, qo, *warm_out, stream=streams[d])
        b.record(streams[d])
        torch.cuda.synchronize()
        iso_ms[d] = a.elapsed_time(b) / K
    log(f"[bench] stream: lookup kernel alone, ms per launch {iso_ms}")
    # merges timed alone: further fresh batches after the last timed lookup,
    # each with the GPU otherwise idle (they change nothing the oracle checks)
    alone = {}
    for d in dists:
        ts = []
        for k in range(n_steps, n_steps + 4):
            b = w.insert_batch(d, k)
            dev_b = (torch.from_numpy(b.peer).to(dev),) + _upload(b, dev)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            forests[d].merge(*dev_b, stream=streams[d])
            ts.append(time.perf_counter() - t0)
        alone[d] = ts
    n_alone = sum(len(v) for v in alone.values()) * len(ihost[dists[0]][0])
    alone_s = sum(sum(v) for v in alone.values())
    log(f"[bench] stream: merges alone ms {({d: [round(x * 1e3, 3) for x in v] for d, v in alone.items()})}")
    kname = route_kernel_name(forests[dists[0]])
    info = {d: forests[d].info() for d in dists}
    compact = None
    if args.compact:
        compact = [bench_compact(forests[d], *qdev[d][(n_steps - 1) % R], *warm_out, None, 5, d,
                                 float(route_ms[d].mean())) for d in dists]
        log(f"[bench] compact: {compact}")
    for d in dists:
        forests[d].close()
    # every lookup of every timed step against the radix-tree oracle, which
    # takes the same merges in the same order
    T = cpu_threads()
    tot_bytes = 0.0
    rows = 0
    per_dist = {}
    for d in dists:
        o = oracle.RadixOracle(P)
        o.load_seqset(w.snapshot)
        byts = []
        for k in range(n_steps):
            b = ihost[d][k]
            o.merge(b.peer, b.tokens, b.offsets)
            if k < Wu:
                continue
            q = qhost[d][k % R]
            m_or, c_or = o.route(q.tokens, q.offsets, T)
            m = outs[d][k - Wu][0].cpu().numpy()
            c = outs[d][k - Wu][1].cpu().numpy()
            if not (np.array_equal(m, m_or) and np.array_equal(c, c_or)):
                bad = np.nonzero((m != m_or).any(axis=1) | (c != c_or))[0]
                raise SystemExit(f"bench.py: stream {d} step {k}: {bad.size} rows differ from the oracle "
                                 f"(first {bad[:5].tolist()})")
            byts.append(float(_alg_bytes(q, m_or.max(axis=1), P).sum()))
            rows += len(q)
        log(f"[bench] stream {d}: every row of {K} steps equals the oracle")
        tot_bytes += sum(byts)
        per_dist[d] = {"route_ms_mean": float(route_ms[d].mean()), "route_ms_median": float(np.median(route_ms[d])),
                       "route_ms_alone": iso_ms[d], "last_step_bytes": byts[-1],
                       "algorithmic_bytes_per_launch": float(np.mean(byts)),
                       "merge_ms_mean": float(merge_s[d][Wu:].mean() * 1e3),
                       "merge_inserts_per_s": float(len(ihost[d][0]) * K / merge_s[d][Wu:].sum()),
                       "forest_nodes_after": info[d]["num_nodes"], "forest_device_bytes": info[d]["device_bytes"]}
        o.close()
    all_ms = np.concatenate([route_ms[d] for d in dists])
    route_s = all_ms.sum() / 1e3
    n_lookups = 2 * K * nq
    iso_bytes = float(np.mean([per_dist[d]["last_step_bytes"] for d in dists]))
    iso = float(np.mean([iso_ms[d] for d in dists]))
    n_ins = sum(len(ihost[d][k]) for d in dists for k in range(Wu, n_steps))
    merge_tot = sum(merge_s[d][Wu:].sum() for d in dists)
    achieved = iso_bytes / (iso / 1e3) / 1e9
    cpu = None
    if not args.no_cpu_baseline:
        def make():
            ra = oracle.RadixOracle(P)
            ra.load_seqset(w.snapshot)
            li = oracle.Oracle(P)
            li.load_seqset(w.snapshot)
            b = ihost["uniform"][0]
            ra.merge(b.peer, b.tokens, b.offsets)
            li.merge(b.peer, b.tokens, b.offsets)
            return ra, li
        cpu = cpu_baseline(make, qhost["uniform"][0], args.cpu_seconds,
                           "lookups of the first uniform round (after its merge)")
        log(f"[bench] cpu baseline: {cpu}")
    return {
        "value": n_lookups / wall, "ms_per_step": wall * 1e3 / K,
        "queries_per_step": 2 * nq, "inserts_per_step": 2 * len(ihost[dists[0]][0]),
        "lookup": {"queries_per_s": nq / (iso / 1e3), "route_ms_alone": iso,
                   "route_ms_in_steps": float(all_ms.mean()),
                   "queries_per_s_in_steps": n_lookups / route_s,
                   "note": "alone: K launches back to back per forest after the timed region (the roofline's "
                           "kernel time); in steps: HIP events around each route call of the timed steps, "
                           "which run beside the other forest's merge and lookup"},
        "merge": {"inserts_per_s": n_ins / merge_tot, "inserts": n_ins, "seconds": float(merge_tot),
                  "note": "wall time of the timed steps' pr_merge calls (host-synchronous), "
                          + ("each after the previous lookup on the stream finished" if args.schedule == "serial"
                             else "each queued behind its forest's previous lookup, beside the other forest's"),
                  "alone": {"inserts_per_s": n_alone / alone_s, "inserts": n_alone, "seconds": alone_s,
                            "note": "four more fresh batches per distribution after the timed region, each "
                                    "merged with the GPU otherwise idle"}},
        "per_distribution": per_dist, "cu_split": cu_split,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBPS, "traffic": measured_traffic("stream"),
                     "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "kernel": kname, "kernel_ms": iso,
                     "algorithmic_bytes_per_launch": iso_bytes,
                     "bytes_from": "match lengths of the radix-tree oracle",
                     "timing": "K launches back to back per forest, each forest as the timed steps left it, over "
                               "the last timed step's lookup batch"},
        "parity": {"oracle": "radix trees, one per peer", "rows": rows, "bit_exact": True,
                   "what": "every match length and chosen peer of every timed lookup"},
        "cpu": cpu, "compact": compact, "workload_note": f"lookup batches: the {R} rounds' batches per distribution, taken in "
                                     f"turn; insert batches: fresh for every step"}


def bench_route_config(cfg: int, args, dev, headline: bool) -> dict:
    """One configuration's lookup batch: K launches back to back between one
    pair of HIP events (four rotated query copies), every row compared with
    the radix-tree oracle, whose match lengths give the algorithmic bytes."""
    import torch

    import oracle
    import workloads as W
    from paper_2606_17059_amd import Forest
    t0 = time.perf_counter()
    w = W.make_config(cfg)
    queries = w.queries
    P = w.num_peers
    nq = len(queries)
    log(f"[bench] config {cfg}: generated in {time.perf_counter() - t0:.1f} s: {len(w.snapshot)} cached prompts, "
        f"{nq} queries")
    f = Forest(P)
    f.load_seqset(w.snapshot)
    copies = max(1, args.copies)
    qt = [torch.from_numpy(queries.tokens).to(dev) for _ in range(copies)]
    qo = [torch.from_numpy(queries.offsets).to(dev) for _ in range(copies)]
    ml = torch.empty((nq, P), dtype=torch.int32, device=dev)
    ch = torch.empty(nq, dtype=torch.int32, device=dev)
    t0 = time.perf_counter()
    f.route(qt[0], qo[0], ml, ch)  # first route builds and uploads the forest
    torch.cuda.synchronize()
    log(f"[bench] config {cfg}: forest build + upload + first route {time.perf_counter() - t0:.2f} s; {f.info()}")
    launch = [f.route_launcher(qt[i], qo[i], ml, ch) for i in range(len(qt))]
    for i in range(args.warmup):
        launch[i % len(launch)]()
    torch.cuda.synchronize()
    # K launches back to back between one pair of events: the host enqueues
    # far faster than the kernel runs, so the region over K is the kernel's
    # average launch duration
    K = args.steps
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for k in range(K):
        launch[k % len(launch)]()
    e1.record()
    torch.cuda.synchronize()
    total_ms = e0.elapsed_time(e1)
    f.check()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    for k in range(K):
        ev[k][0].record()
        launch[k % len(launch)]()
        ev[k][1].record()
    torch.cuda.synchronize()
    kern_ms = np.array([a.elapsed_time(b) for a, b in ev])
    m, c = ml.cpu().numpy(), ch.cpu().numpy()
    split = int(w.meta.get("split_block", 0))
    r = oracle.RadixOracle(P, split_block=split)
    r.load_seqset(w.snapshot)
    t0 = time.perf_counter()
    m_or, c_or = r.route(queries.tokens, queries.offsets, cpu_threads())
    oracle_s = time.perf_counter() - t0
    r.close()
    if not (np.array_equal(m, m_or) and np.array_equal(c, c_or)):
        bad = np.nonzero((m != m_or).any(axis=1) | (c != c_or))[0]
        raise SystemExit(f"bench.py: config {cfg}: {bad.size} rows differ from the oracle (first {bad[:5].tolist()})")
    bytes_q = _alg_bytes(queries, m_or.max(axis=1), P)
    total_bytes = float(bytes_q.sum())
    achieved = total_bytes / (total_ms / K / 1e3) / 1e9
    log(f"[bench] config {cfg}: {K} launches in {total_ms:.4f} ms, {total_ms / K:.4f} ms per launch, "
        f"{achieved:.0f} GB/s ({achieved / PEAK_HBM_GBPS:.3f}); every row equals the oracle ({oracle_s:.1f} s)")
    out = {
        "workload": WORKLOADS[cfg], "peers": P, "queries": nq, "query_tokens": int(queries.lengths().sum()),
        "value": nq * K / (total_ms / 1e3), "unit": "queries/s", "steps": K, "warmup": args.warmup,
        "ms_per_step": total_ms / K,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBPS, "traffic": measured_traffic(W.CONFIG_NAMES[cfg]),
                     "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "kernel": route_kernel_name(f), "kernel_ms": total_ms / K,
                     "kernel_ms_own_events": {"mean": float(kern_ms.mean()), "median": float(np.median(kern_ms))},
                     "kernels_per_step": step_kernels(nq, int(queries.lengths().sum())),
                     "algorithmic_bytes_per_launch": total_bytes,
                     "bytes_from": "match lengths of the radix-tree oracle"},
        "parity": {"oracle": "radix trees, one per peer" + (f", nodes at every {split}-token block" if split else ""),
                   "rows": nq, "bit_exact": True},
    }
    if cfg == 3:
        # the same batch routed on the peers' true trees (every row checked
        # too): how often the stale estimates pick the same peer, and the
        # prefill reuse they predict vs get (Table 2's expected / actual hit)
        ft = Forest(P)
        ft.load_seqset(w.true_snapshot)
        mt, ct = ft.route(qt[0], qo[0])
        torch.cuda.synchronize()
        ft.close()
        mt, ct = mt.cpu().numpy(), ct.cpu().numpy()
        rt = oracle.RadixOracle(P)
        rt.load_seqset(w.true_snapshot)
        mt_or, ct_or = rt.route(queries.tokens, queries.offsets, cpu_threads())
        rt.close()
        if not (np.array_equal(mt, mt_or) and np.array_equal(ct, ct_or)):
            raise SystemExit("bench.py: config 3 true forest: rows differ from the oracle")
        rows = np.arange(nq)
        tot = float(queries.lengths().sum())
        out["stale_report"] = {
            "route_agreement": float((c == ct).mean()),
            "expected_hit": float(m[rows, c].sum() / tot),
            "actual_hit": float(mt[rows, c].sum() / tot),
            "oracle_true_hit": float(mt[rows, ct].sum() / tot),
            "note": "estimates: observer 0's stale replicas; truth: the peers' exact trees; hit = matched "
                    "prefill tokens / query tokens"}
        out["parity"]["rows"] = 2 * nq
        log(f"[bench] stale report: {out['stale_report']}")
    if headline or cfg == 2:
        if not args.no_select:
            out["select"] = bench_select(f, w, qt, qo, np.minimum(queries.lengths(), m_or.max(axis=1) + 1),
                                         K, args.warmup, dev)
            log(f"[bench] select: {out['select']}")
    if headline:
        if args.latency:
            out["latency"] = bench_latency(f, w, dev)
        if args.lru:
            out["lru"] = bench_lru(f, w, qt, qo, dev)
            log(f"[bench] lru: {out['lru']}")
        if args.snapshot:
            out["snapshot"] = bench_snapshot(f, w, dev)
            log(f"[bench] snapshot: {out['snapshot']}")
        if not args.no_cpu_baseline:
            def make():
                ra = oracle.RadixOracle(P, split_block=split)
                ra.load_seqset(w.snapshot)
                li = oracle.Oracle(P)
                li.load_seqset(w.snapshot)
                return ra, li
            out["cpu"] = cpu_baseline(make, queries, args.cpu_seconds, "queries")
            log(f"[bench] cpu baseline: {out['cpu']}")
    f.close()
    del qt, qo, ml, ch, launch
    torch.cuda.empty_cache()
    return out


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
    ap.add_argument("--config", type=int, default=5, choices=sorted(WORKLOADS),
                    help="headline workload (default 5, the largest: streaming merges and lookups)")
    ap.add_argument("--extra-configs", default="2,3,4",
                    help="comma-separated lookup workloads also measured and reported under 'configs' "
                         "('' for none)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU time of the oracle samples")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--lru", action="store_true",
                    help="also time touching the batch in the local tree and LRU evictions (configs 1-4)")
    ap.add_argument("--snapshot", action="store_true",
                    help="also time snapshot export and device-input load of a few peers (configs 1-4)")
    ap.add_argument("--latency", action="store_true",
                    help="also time small batches (1 to 32,768 queries) per call, host wall time included "
                         "(configs 1-4)")
    ap.add_argument("--schedule", choices=("shared", "cusplit", "threads", "pipelined", "serial"), default="threads",
                    help="config 5: shared: a host thread and merge stream per forest, both forests' lookups "
                         "queued in turn on one stream, so each merge runs beside the other forest's lookup; "
                         "cusplit: one host thread, lookups on a stream over most CUs and merges on a "
                         "stream over the CUs kept from it (--merge-cus per XCD), each forest's merge beside the "
                         "other forest's lookup; threads (default): a stream and a host thread per forest; "
                         "pipelined: two streams, one host thread issuing each forest's merge while the other's "
                         "lookup runs; serial: one stream, in turn")
    ap.add_argument("--merge-cus", type=int, default=2,
                    help="config 5 with --schedule cusplit: CUs per XCD kept for merges")
    ap.add_argument("--compact", action="store_true",
                    help="config 5: compact both forests after the timed steps and time it")
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
    t_start = time.perf_counter()
    extras = [int(x) for x in args.extra_configs.split(",") if x.strip()]
    out = {"metric": "routed queries/sec (batched LPM over all peer trees) + achieved HBM GB/s",
           "unit": "queries/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "int32",
           "data": "synthetic"}
    if args.config == 5:
        r = bench_stream(args, dev)
        out.update({
            "value": r["value"], "ms_per_step": r["ms_per_step"],
            "config": {"workload": WORKLOADS[5], "config_index": 5, "peers": 128,
                       "queries_per_step": r["queries_per_step"], "inserts_per_step": r["inserts_per_step"],
                       "step": "for each topic distribution (uniform, Zipf 1.2): merge a fresh 10,000-insert batch "
                               "into its forest, then route a 1,048,576-query lookup batch on it; "
                               + {"shared": "a host thread and a merge stream per forest; both forests' lookups "
                                            "queued in turn on one stream",
                                  "cusplit": "one host thread; lookups on a stream over {lookup_cus} CUs, merges on a "
                                             "stream over the other {merge_cus}, each forest's merge beside the "
                                             "other forest's lookup".format(**(r["cu_split"] or
                                                                               {"lookup_cus": 0, "merge_cus": 0})),
                                  "pipelined": "the two forests on two streams from one host thread, each "
                                               "forest's merge beside the other forest's lookup",
                                  "threads": "the two forests on two streams and two host threads",
                                  "serial": "all in turn on one stream"}[args.schedule],
                       "parallelism": "single GPU"},
            "hbm_gbps": r["roofline"]["achieved"], "roofline": r["roofline"], "lookup": r["lookup"],
            "merge": r["merge"], "per_distribution": r["per_distribution"], "parity": r["parity"],
            "cpu_baseline": r["cpu"], "inputs": r["workload_note"]})
        if r["compact"]:
            out["compact"] = r["compact"]
    else:
        r = bench_route_config(args.config, args, dev, headline=True)
        out.update({
            "value": r["value"], "ms_per_step": r["ms_per_step"],
            "config": {"workload": WORKLOADS[args.config], "config_index": args.config, "peers": r["peers"],
                       "queries_per_step": r["queries"], "query_tokens": r["query_tokens"],
                       "parallelism": "single GPU"},
            "hbm_gbps": r["roofline"]["achieved"], "roofline": r["roofline"], "parity": r["parity"],
            "cpu_baseline": r.get("cpu")})
        for k in ("stale_report", "select", "latency", "lru", "snapshot"):
            if k in r:
                out[k] = r[k]
    if extras:
        out["configs"] = {}
        for cfg in extras:
            if cfg == args.config or cfg == 5:
                continue
            out["configs"][str(cfg)] = bench_route_config(cfg, args, dev, headline=False)
    out["bench_seconds"] = time.perf_counter() - t_start
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
