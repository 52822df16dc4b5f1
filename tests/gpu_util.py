"""Helpers shared by the GPU parity tests (device transfer, oracle sampling)."""
from __future__ import annotations

import os
import sys

import numpy as np

import oracle
import pins


def announce(msg: str) -> None:
    """Name the case before each GPU step, flushed, so a fault points at it."""
    sys.stdout.write(f"\n[gpu-case] {msg}\n")
    sys.stdout.flush()


def device():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a HIP device")
    return torch.device("cuda:0")


def to_dev(ss):
    import torch
    dev = device()
    toks = torch.from_numpy(np.ascontiguousarray(ss.tokens, dtype=np.int32)).to(dev)
    offs = torch.from_numpy(np.ascontiguousarray(ss.offsets, dtype=np.int64)).to(dev)
    return toks, offs


def gpu_route(forest, ss, label=""):
    import torch
    announce(f"route {label}: {len(ss)} queries, {forest.num_peers} peers")
    t, o = to_dev(ss)
    m, c = forest.route(t, o)
    torch.cuda.synchronize()
    return m.cpu().numpy(), c.cpu().numpy()


def oracle_for(snapshot, num_peers):
    o = oracle.Oracle(num_peers)
    pins.load_all(o, snapshot, num_peers)
    return o


def radix_for(snapshot, num_peers, split_block=0):
    """The per-peer radix-tree oracle loaded with a snapshot: fast enough to
    check every row of the full-size workloads."""
    o = oracle.RadixOracle(num_peers, split_block=split_block)
    o.load_seqset(snapshot)
    return o


def nthreads() -> int:
    n = os.cpu_count() or 1
    return max(1, min(n, 16))


def assert_rows_equal(m_gpu, c_gpu, m_or, c_or, idx=None, what=""):
    if idx is not None:
        m_gpu, c_gpu = m_gpu[idx], c_gpu[idx]
    bad = np.nonzero((m_gpu != m_or).any(axis=1) | (c_gpu != c_or))[0]
    assert bad.size == 0, (f"{what}: {bad.size} rows differ; first {bad[:5].tolist()}: "
                           f"gpu m={m_gpu[bad[0]].tolist()} c={int(c_gpu[bad[0]])} "
                           f"oracle m={m_or[bad[0]].tolist()} c={int(c_or[bad[0]])}")


def assert_properties(m, c, ss, what=""):
    """Properties that hold at any size: bounds, argmax rule."""
    qlen = ss.lengths()
    assert (m >= 0).all(), f"{what}: negative match"
    assert (m <= qlen[:, None]).all(), f"{what}: match longer than the query"
    assert np.array_equal(c, np.argmax(m, axis=1)), f"{what}: chosen is not the lowest-id argmax"
