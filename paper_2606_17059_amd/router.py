"""Python binding of libprefix_router.so (ctypes; argument marshalling only).

Function names follow the C ABI in include/prefix_router.h.  Every routing and
merge step runs in the library's HIP kernels; this module only checks shapes,
dtypes and devices of torch tensors and passes raw pointers and the current HIP
stream.  If the library is not built, loading it raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libprefix_router.so")

PR_OK, PR_EINVAL, PR_ENOMEM, PR_EDEVICE, PR_ESTATE = 0, -1, -2, -3, -4
PR_MAX_PEERS = 1024
PR_NOALLOC_MAX_QUERIES = 65536

EXPORTED = ("pr_abi_version", "pr_last_error", "pr_forest_create", "pr_forest_destroy",
            "pr_load_snapshot", "pr_load_snapshot_device", "pr_export_snapshot", "pr_merge", "pr_route",
            "pr_route_noalloc",
            "pr_route_select", "pr_tree_tokens", "pr_forest_compact", "pr_set_local_peer", "pr_set_time", "pr_touch", "pr_evict_lru",
            "pr_forest_check",
            "pr_forest_info_get", "pr_forest_host_image")

PR_SELECT_PREFER_LOCAL = 1


class RouterError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"status {status}: {msg}")
        self.status = status


class ForestInfo(ctypes.Structure):
    _fields_ = [("num_peers", ctypes.c_int32), ("mask_words", ctypes.c_int32),
                ("num_nodes", ctypes.c_int64),
                ("pool_tokens", ctypes.c_int64), ("device_bytes", ctypes.c_int64),
                ("host_seq_tokens", ctypes.c_int64), ("layout_epoch", ctypes.c_int64),
                ("label_token_bytes", ctypes.c_int64), ("label_bits", ctypes.c_int64),
                ("merge_refusals", ctypes.c_int64), ("first_window_tokens", ctypes.c_int64)]


class ImageView(ctypes.Structure):
    _fields_ = [("mask_words", ctypes.c_int32), ("num_nodes", ctypes.c_int64),
                ("pool_tokens", ctypes.c_int64),
                ("nodes", ctypes.POINTER(ctypes.c_int32)), ("ntok", ctypes.POINTER(ctypes.c_int32)),
                ("nsep", ctypes.POINTER(ctypes.c_int32)), ("mext", ctypes.POINTER(ctypes.c_uint64)),
                ("pool", ctypes.POINTER(ctypes.c_int32))]


_lib_handle = None
_vp = ctypes.c_void_p
_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)


def lib() -> ctypes.CDLL:
    """Load the library (import torch first so that one HIP runtime serves both)."""
    global _lib_handle
    if _lib_handle is not None:
        return _lib_handle
    try:
        import torch  # noqa: F401  (binds libamdhip64 to torch's copy)
    except ImportError:
        pass
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run paper_2606_17059_amd.build.build()")
    L = ctypes.CDLL(LIB_PATH)
    L.pr_abi_version.restype = ctypes.c_int32
    L.pr_last_error.restype = ctypes.c_char_p
    L.pr_forest_create.argtypes = [ctypes.c_int32, ctypes.POINTER(_vp)]
    L.pr_forest_create.restype = ctypes.c_int32
    L.pr_forest_destroy.argtypes = [_vp]
    L.pr_forest_destroy.restype = None
    L.pr_load_snapshot.argtypes = [_vp, ctypes.c_int32, _vp, _vp, ctypes.c_int64]
    L.pr_load_snapshot.restype = ctypes.c_int32
    L.pr_load_snapshot_device.argtypes = [_vp, ctypes.c_int32, _vp, ctypes.c_int64, _vp, ctypes.c_int64, _vp]
    L.pr_load_snapshot_device.restype = ctypes.c_int32
    L.pr_export_snapshot.argtypes = [_vp, ctypes.c_int32, _vp, ctypes.c_int64, _vp, ctypes.c_int64, _i64p, _i64p,
                                     _vp]
    L.pr_export_snapshot.restype = ctypes.c_int32
    L.pr_tree_tokens.argtypes = [_vp, ctypes.c_int32, _i64p, _vp]
    L.pr_tree_tokens.restype = ctypes.c_int32
    L.pr_forest_compact.argtypes = [_vp, _i64p, _i64p, _vp]
    L.pr_forest_compact.restype = ctypes.c_int32
    L.pr_set_local_peer.argtypes = [_vp, ctypes.c_int32]
    L.pr_set_local_peer.restype = ctypes.c_int32
    L.pr_set_time.argtypes = [_vp, ctypes.c_int64]
    L.pr_set_time.restype = ctypes.c_int32
    L.pr_touch.argtypes = [_vp, _vp, ctypes.c_int64, _vp, ctypes.c_int64, _vp]
    L.pr_touch.restype = ctypes.c_int32
    L.pr_evict_lru.argtypes = [_vp, ctypes.c_int64, _i64p, _vp]
    L.pr_evict_lru.restype = ctypes.c_int32
    L.pr_merge.argtypes = [_vp, _vp, _vp, ctypes.c_int64, _vp, ctypes.c_int64, _vp]
    L.pr_merge.restype = ctypes.c_int32
    L.pr_route.argtypes = [_vp, _vp, ctypes.c_int64, _vp, ctypes.c_int64, _vp, _vp, _vp]
    L.pr_route_noalloc.restype = ctypes.c_int32
    L.pr_route_noalloc.argtypes = [_vp, _vp, ctypes.c_int64, _vp, ctypes.c_int64, _vp, _vp, _vp]
    L.pr_route.restype = ctypes.c_int32
    L.pr_route_select.argtypes = [_vp, _vp, ctypes.c_int64, _vp, ctypes.c_int64, _vp, ctypes.c_int32,
                                  ctypes.c_uint32, _vp, _vp, _vp, _vp]
    L.pr_route_select.restype = ctypes.c_int32
    L.pr_forest_check.argtypes = [_vp]
    L.pr_forest_check.restype = ctypes.c_int32
    L.pr_forest_info_get.argtypes = [_vp, ctypes.POINTER(ForestInfo)]
    L.pr_forest_info_get.restype = ctypes.c_int32
    L.pr_forest_host_image.argtypes = [_vp, ctypes.POINTER(ImageView)]
    L.pr_forest_host_image.restype = ctypes.c_int32
    if L.pr_abi_version() != 7:
        raise RuntimeError("libprefix_router ABI version mismatch")
    _lib_handle = L
    return L


def _check(status: int) -> None:
    if status != PR_OK:
        raise RouterError(status, lib().pr_last_error().decode())


def pr_last_error() -> str:
    return lib().pr_last_error().decode()


# ---- thin wrappers with the C names -----------------------------------------
def pr_forest_create(num_peers: int) -> int:
    h = _vp()
    _check(lib().pr_forest_create(int(num_peers), ctypes.byref(h)))
    return h.value


def pr_forest_destroy(f: int) -> None:
    lib().pr_forest_destroy(f)


def pr_load_snapshot(f: int, peer: int, tokens: np.ndarray, offsets: np.ndarray) -> None:
    t = np.ascontiguousarray(tokens, dtype=np.int32)
    o = np.ascontiguousarray(offsets, dtype=np.int64)
    if o.ndim != 1 or o.shape[0] < 1:
        raise ValueError("offsets must be 1-D with at least one entry")
    _check(lib().pr_load_snapshot(f, int(peer), t.ctypes.data if t.size else None, o.ctypes.data,
                                  o.shape[0] - 1))


def _dev(t, dtype, name):
    import torch
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name} must be a CUDA (HIP) torch tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _stream_ptr(stream, device) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return int(s.cuda_stream)


def pr_load_snapshot_device(f: int, peer: int, tokens, offsets, stream=None) -> None:
    import torch
    _dev(tokens, torch.int32, "tokens")
    _dev(offsets, torch.int64, "offsets")
    n = offsets.numel() - 1
    if n < 0:
        raise ValueError("offsets must have at least one entry")
    _check(lib().pr_load_snapshot_device(f, int(peer), tokens.data_ptr() or None, tokens.numel(),
                                         offsets.data_ptr(), n, _stream_ptr(stream, offsets.device)))


def pr_export_snapshot(f: int, peer: int, device=None, stream=None):
    """Export peer's tree: (tokens, offsets) as CUDA tensors (int32, int64)."""
    import torch
    dev = device if device is not None else torch.device("cuda", torch.cuda.current_device())
    ns, nt = ctypes.c_int64(0), ctypes.c_int64(0)
    st = _stream_ptr(stream, dev)
    _check(lib().pr_export_snapshot(f, int(peer), None, 0, None, 0, ctypes.byref(ns), ctypes.byref(nt), st))
    toks = torch.empty(max(nt.value, 1), dtype=torch.int32, device=dev)
    offs = torch.empty(ns.value + 1, dtype=torch.int64, device=dev)
    _check(lib().pr_export_snapshot(f, int(peer), toks.data_ptr(), toks.numel(), offs.data_ptr(), offs.numel(),
                                    ctypes.byref(ns), ctypes.byref(nt), st))
    return toks[:nt.value], offs


def pr_tree_tokens(f: int, peer: int, stream=None) -> int:
    import torch
    n = ctypes.c_int64(0)
    st = _stream_ptr(stream, torch.device("cuda", torch.cuda.current_device()))
    _check(lib().pr_tree_tokens(f, int(peer), ctypes.byref(n), st))
    return n.value


def pr_forest_compact(f: int, stream=None) -> tuple:
    """Drop unreachable and unheld node records; returns (nodes_before, nodes_after)."""
    import torch
    a, b = ctypes.c_int64(0), ctypes.c_int64(0)
    st = _stream_ptr(stream, torch.device("cuda", torch.cuda.current_device()))
    _check(lib().pr_forest_compact(f, ctypes.byref(a), ctypes.byref(b), st))
    return a.value, b.value


def pr_set_local_peer(f: int, peer: int) -> None:
    _check(lib().pr_set_local_peer(f, int(peer)))


def pr_set_time(f: int, t: int) -> None:
    _check(lib().pr_set_time(f, int(t)))


def pr_touch(f: int, q_tokens, q_offsets, stream=None) -> None:
    import torch
    _dev(q_tokens, torch.int32, "q_tokens")
    _dev(q_offsets, torch.int64, "q_offsets")
    n = q_offsets.numel() - 1
    if n < 0:
        raise ValueError("q_offsets must have at least one entry")
    _check(lib().pr_touch(f, q_tokens.data_ptr() or None, q_tokens.numel(), q_offsets.data_ptr(), n,
                          _stream_ptr(stream, q_offsets.device)))


def pr_evict_lru(f: int, max_tokens: int, stream=None) -> int:
    import torch
    ev = ctypes.c_int64(0)
    st = _stream_ptr(stream, torch.device("cuda", torch.cuda.current_device()))
    _check(lib().pr_evict_lru(f, int(max_tokens), ctypes.byref(ev), st))
    return ev.value


def pr_merge(f: int, peer_of, tokens, offsets, stream=None) -> None:
    import torch
    _dev(peer_of, torch.int32, "peer_of")
    _dev(tokens, torch.int32, "tokens")
    _dev(offsets, torch.int64, "offsets")
    n = offsets.numel() - 1
    if n < 0 or peer_of.numel() != n:
        raise ValueError("peer_of must have len(offsets) - 1 entries")
    _check(lib().pr_merge(f, peer_of.data_ptr() or None, tokens.data_ptr() or None, tokens.numel(),
                          offsets.data_ptr(), n, _stream_ptr(stream, offsets.device)))


def pr_route(f: int, q_tokens, q_offsets, match_len, chosen, num_peers: int, stream=None) -> None:
    import torch
    _dev(q_tokens, torch.int32, "q_tokens")
    _dev(q_offsets, torch.int64, "q_offsets")
    _dev(match_len, torch.int32, "match_len")
    _dev(chosen, torch.int32, "chosen")
    nq = q_offsets.numel() - 1
    if nq < 0:
        raise ValueError("q_offsets must have at least one entry")
    if match_len.numel() != nq * num_peers or chosen.numel() != nq:
        raise ValueError("match_len must hold [num_queries][num_peers] and chosen [num_queries]")
    _check(lib().pr_route(f, q_tokens.data_ptr() or None, q_tokens.numel(), q_offsets.data_ptr(), nq,
                          match_len.data_ptr() or None, chosen.data_ptr() or None,
                          _stream_ptr(stream, q_offsets.device)))


def pr_route_noalloc(f: int, q_tokens, q_offsets, match_len, chosen, num_peers: int, stream=None) -> None:
    """pr_route without allocation (at most PR_NOALLOC_MAX_QUERIES queries;
    the forest must be on the device already)."""
    import torch
    _dev(q_tokens, torch.int32, "q_tokens")
    _dev(q_offsets, torch.int64, "q_offsets")
    _dev(match_len, torch.int32, "match_len")
    _dev(chosen, torch.int32, "chosen")
    nq = q_offsets.numel() - 1
    if nq < 0:
        raise ValueError("q_offsets must have at least one entry")
    if match_len.numel() != nq * num_peers or chosen.numel() != nq:
        raise ValueError("match_len must hold [num_queries][num_peers] and chosen [num_queries]")
    _check(lib().pr_route_noalloc(f, q_tokens.data_ptr() or None, q_tokens.numel(), q_offsets.data_ptr(), nq,
                                  match_len.data_ptr() or None, chosen.data_ptr() or None,
                                  _stream_ptr(stream, q_offsets.device)))


def pr_route_select(f: int, q_tokens, q_offsets, eligible, local_peer: int, flags: int, match_len, best, second,
                    num_peers: int, stream=None) -> None:
    """eligible: CUDA uint64 tensor of ceil(num_peers / 64) words (torch.int64
    holding the bits) or None; match_len and second may be None."""
    import torch
    _dev(q_tokens, torch.int32, "q_tokens")
    _dev(q_offsets, torch.int64, "q_offsets")
    _dev(best, torch.int32, "best")
    nq = q_offsets.numel() - 1
    if nq < 0:
        raise ValueError("q_offsets must have at least one entry")
    if best.numel() != nq:
        raise ValueError("best must hold [num_queries]")
    if match_len is not None:
        _dev(match_len, torch.int32, "match_len")
        if match_len.numel() != nq * num_peers:
            raise ValueError("match_len must hold [num_queries][num_peers]")
    if second is not None:
        _dev(second, torch.int32, "second")
        if second.numel() != nq:
            raise ValueError("second must hold [num_queries]")
    if eligible is not None:
        _dev(eligible, torch.int64, "eligible")
        if eligible.numel() != (num_peers + 63) // 64:
            raise ValueError("eligible must hold ceil(num_peers / 64) words")
    _check(lib().pr_route_select(f, q_tokens.data_ptr() or None, q_tokens.numel(), q_offsets.data_ptr(), nq,
                                 eligible.data_ptr() if eligible is not None else None, int(local_peer),
                                 int(flags), match_len.data_ptr() if match_len is not None else None,
                                 best.data_ptr() or None, second.data_ptr() if second is not None else None,
                                 _stream_ptr(stream, q_offsets.device)))


def eligible_words(flags) -> np.ndarray:
    """Pack per-peer 0/1 flags into the int64 words pr_route_select reads."""
    b = np.asarray(flags).astype(bool)
    words = np.zeros((b.shape[0] + 63) // 64, dtype=np.uint64)
    for p in np.nonzero(b)[0]:
        words[p // 64] |= np.uint64(1) << np.uint64(p % 64)
    return words.view(np.int64)


def pr_forest_check(f: int) -> None:
    _check(lib().pr_forest_check(f))


def pr_forest_info_get(f: int) -> dict:
    info = ForestInfo()
    _check(lib().pr_forest_info_get(f, ctypes.byref(info)))
    return {k: getattr(info, k) for k, _ in ForestInfo._fields_}


def pr_forest_host_image(f: int) -> dict:
    """Copy of the host-side layout image (numpy arrays)."""
    v = ImageView()
    _check(lib().pr_forest_host_image(f, ctypes.byref(v)))

    def arr(ptr, n, dt):
        if n == 0:
            return np.zeros(0, dtype=dt)
        return np.ctypeslib.as_array(ptr, shape=(n,)).astype(dt, copy=True)

    W = v.mask_words
    nodes = arr(v.nodes, v.num_nodes * 8, np.int32).reshape(-1, 8)
    mask0 = nodes[:, 6].astype(np.uint32).astype(np.uint64) | (nodes[:, 7].astype(np.uint32).astype(np.uint64) << np.uint64(32))
    mext = arr(v.mext, v.num_nodes * (W - 1), np.uint64).reshape(-1, W - 1) if W > 1 \
        else np.zeros((v.num_nodes, 0), np.uint64)
    return dict(mask_words=W, nodes=nodes, ntok=arr(v.ntok, v.num_nodes, np.int32),
                nsep=arr(v.nsep, v.num_nodes, np.int32),
                masks=np.concatenate([mask0[:, None], mext], axis=1), pool=arr(v.pool, v.pool_tokens, np.int32))


# ---- convenience object ------------------------------------------------------
class Forest:
    """Owning handle of a pr_forest (one node's view of all peers' trees)."""

    def __init__(self, num_peers: int):
        self.num_peers = int(num_peers)
        self._h = pr_forest_create(self.num_peers)

    @property
    def handle(self) -> int:
        if not self._h:
            raise RuntimeError("forest is closed")
        return self._h

    def close(self) -> None:
        if getattr(self, "_h", None):
            pr_forest_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def load_snapshot(self, peer: int, tokens, offsets) -> None:
        pr_load_snapshot(self.handle, peer, tokens, offsets)

    def load_seqset(self, ss) -> None:
        """Load every peer's snapshot from a peer-major CSR batch (workloads.SeqSet)."""
        for p in range(self.num_peers):
            lo = int(np.searchsorted(ss.peer, p, side="left"))
            hi = int(np.searchsorted(ss.peer, p, side="right"))
            o = ss.offsets[lo:hi + 1] - ss.offsets[lo]
            self.load_snapshot(p, ss.tokens[ss.offsets[lo]:ss.offsets[hi]], o)

    def merge(self, peer_of, tokens, offsets, stream=None) -> None:
        pr_merge(self.handle, peer_of, tokens, offsets, stream)

    def load_snapshot_device(self, peer: int, tokens, offsets, stream=None) -> None:
        pr_load_snapshot_device(self.handle, peer, tokens, offsets, stream)

    def export_snapshot(self, peer: int, device=None, stream=None):
        return pr_export_snapshot(self.handle, peer, device, stream)

    def tree_tokens(self, peer: int, stream=None) -> int:
        return pr_tree_tokens(self.handle, peer, stream)

    def compact(self, stream=None) -> tuple:
        return pr_forest_compact(self.handle, stream)

    def set_local_peer(self, peer: int) -> None:
        pr_set_local_peer(self.handle, peer)

    def set_time(self, t: int) -> None:
        pr_set_time(self.handle, t)

    def touch(self, q_tokens, q_offsets, stream=None) -> None:
        pr_touch(self.handle, q_tokens, q_offsets, stream)

    def evict_lru(self, max_tokens: int, stream=None) -> int:
        return pr_evict_lru(self.handle, max_tokens, stream)

    def route(self, q_tokens, q_offsets, match_len=None, chosen=None, stream=None) -> Tuple:
        import torch
        nq = q_offsets.numel() - 1
        dev = q_offsets.device
        if match_len is None:
            match_len = torch.empty((nq, self.num_peers), dtype=torch.int32, device=dev)
        if chosen is None:
            chosen = torch.empty(nq, dtype=torch.int32, device=dev)
        pr_route(self.handle, q_tokens, q_offsets, match_len, chosen, self.num_peers, stream)
        return match_len, chosen

    def route_noalloc(self, q_tokens, q_offsets, match_len, chosen, stream=None) -> Tuple:
        """pr_route_noalloc into caller-allocated outputs."""
        pr_route_noalloc(self.handle, q_tokens, q_offsets, match_len, chosen, self.num_peers, stream)
        return match_len, chosen

    def route_launcher(self, q_tokens, q_offsets, match_len, chosen, stream=None):
        """Check the buffers once and return a callable that launches pr_route on
        them with no per-call checks or conversions (tight launch loops).  The
        callable keeps the tensors alive; it raises RouterError on a failed call."""
        import torch
        _dev(q_tokens, torch.int32, "q_tokens")
        _dev(q_offsets, torch.int64, "q_offsets")
        _dev(match_len, torch.int32, "match_len")
        _dev(chosen, torch.int32, "chosen")
        nq = q_offsets.numel() - 1
        if nq < 0:
            raise ValueError("q_offsets must have at least one entry")
        if match_len.numel() != nq * self.num_peers or chosen.numel() != nq:
            raise ValueError("match_len must hold [num_queries][num_peers] and chosen [num_queries]")
        fn = lib().pr_route
        args = (ctypes.c_void_p(self.handle), ctypes.c_void_p(q_tokens.data_ptr() or None),
                ctypes.c_int64(q_tokens.numel()), ctypes.c_void_p(q_offsets.data_ptr()), ctypes.c_int64(nq),
                ctypes.c_void_p(match_len.data_ptr() or None), ctypes.c_void_p(chosen.data_ptr() or None),
                ctypes.c_void_p(_stream_ptr(stream, q_offsets.device)))
        # the launcher holds the forest too, so that the forest outlives it
        keep = (self, q_tokens, q_offsets, match_len, chosen, stream)

        def launch() -> None:
            if not self._h:
                raise RuntimeError("forest is closed")
            st = fn(*args)
            if st != PR_OK:
                _check(st)

        launch.buffers = keep
        return launch

    def route_select(self, q_tokens, q_offsets, eligible=None, local_peer: int = -1, prefer_local: bool = False,
                     match_len=None, best=None, second=None, want_match_len: bool = True,
                     want_second: bool = True, stream=None) -> Tuple:
        """Best and second-best eligible peer (pr_route_select).  eligible: a
        CUDA int64 tensor of packed words (see eligible_words) or None."""
        import torch
        nq = q_offsets.numel() - 1
        dev = q_offsets.device
        if match_len is None and want_match_len:
            match_len = torch.empty((nq, self.num_peers), dtype=torch.int32, device=dev)
        if best is None:
            best = torch.empty(nq, dtype=torch.int32, device=dev)
        if second is None and want_second:
            second = torch.empty(nq, dtype=torch.int32, device=dev)
        pr_route_select(self.handle, q_tokens, q_offsets, eligible, local_peer,
                        PR_SELECT_PREFER_LOCAL if prefer_local else 0, match_len, best, second,
                        self.num_peers, stream)
        return match_len, best, second

    def check(self) -> None:
        pr_forest_check(self.handle)

    def info(self) -> dict:
        return pr_forest_info_get(self.handle)

    def host_image(self) -> dict:
        return pr_forest_host_image(self.handle)
