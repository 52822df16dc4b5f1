"""The C-ABI library loads and exports every entry point its header declares
(no GPU calls)."""
import ctypes
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "prefix_router.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(pr_[a-z_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for must in ("pr_forest_create", "pr_forest_destroy", "pr_load_snapshot", "pr_merge", "pr_route"):
        assert must in names


def test_library_exports_every_declared_symbol():
    from paper_2606_17059_amd import router as R
    L = R.lib()
    for name in declared_functions():
        assert hasattr(L, name), f"{name} not exported"
        assert isinstance(getattr(L, name), ctypes._CFuncPtr)
    assert set(declared_functions()) == set(R.EXPORTED)


def test_abi_version_and_info_layout_agree():
    """The library reports the header's PR_ABI_VERSION, and the binding's copy
    of pr_forest_info has the header's fields in the header's order."""
    from paper_2606_17059_amd import router as R
    src = open(os.path.join(ROOT, "include", "prefix_router.h")).read()
    version = int(re.search(r"#define PR_ABI_VERSION (\d+)", src).group(1))
    assert R.lib().pr_abi_version() == version
    body = re.search(r"typedef struct \{(.*?)\} pr_forest_info;", src, flags=re.S).group(1)
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    fields = re.findall(r"(int32_t|int64_t)\s+(\w+);", body)
    ctypes_of = {"int32_t": ctypes.c_int32, "int64_t": ctypes.c_int64}
    assert [(n, ctypes_of[t]) for t, n in fields] == list(R.ForestInfo._fields_)


def test_binding_refuses_missing_library(monkeypatch, tmp_path):
    from paper_2606_17059_amd import router as R
    monkeypatch.setattr(R, "_lib_handle", None)
    monkeypatch.setattr(R, "LIB_PATH", str(tmp_path / "missing.so"))
    try:
        R.lib()
        raise AssertionError("loading a missing library must raise")
    except RuntimeError as e:
        assert "not built" in str(e)


def test_route_select_argument_errors_without_gpu():
    """Host-side checks of pr_route_select run before any device work."""
    from paper_2606_17059_amd import router as R
    L = R.lib()
    f = R.pr_forest_create(3)
    try:
        for local, flags in [(3, 0), (-2, 0), (0, 2)]:
            st = L.pr_route_select(f, None, 0, None, 0, None, local, flags, None, None, None, None)
            assert st == R.PR_EINVAL, (local, flags)
        assert L.pr_route_select(f, None, 0, None, 0, None, 2, 1, None, None, None, None) == R.PR_OK
        assert L.pr_route_select(f, None, -1, None, 0, None, -1, 0, None, None, None, None) == R.PR_EINVAL
    finally:
        R.pr_forest_destroy(f)


def test_lru_argument_errors_without_gpu():
    """Host-side checks of the LRU calls run before any device work."""
    import ctypes
    from paper_2606_17059_amd import router as R
    L = R.lib()
    f = R.pr_forest_create(3)
    try:
        ev = ctypes.c_int64(-1)
        assert L.pr_evict_lru(f, 5, ctypes.byref(ev), None) == R.PR_ESTATE  # no local peer yet
        assert L.pr_touch(f, None, 0, None, 0, None) == R.PR_ESTATE
        assert L.pr_set_local_peer(f, 3) == R.PR_EINVAL
        assert L.pr_set_local_peer(f, -2) == R.PR_EINVAL
        assert L.pr_set_local_peer(f, 1) == R.PR_OK  # no device image yet: no GPU work
        assert L.pr_set_time(f, 10) == R.PR_OK
        assert L.pr_set_time(f, 9) == R.PR_EINVAL
        assert L.pr_evict_lru(f, -1, ctypes.byref(ev), None) == R.PR_EINVAL
        assert L.pr_evict_lru(f, 0, ctypes.byref(ev), None) == R.PR_OK and ev.value == 0
        assert L.pr_evict_lru(f, 1, None, None) == R.PR_EINVAL
        assert L.pr_touch(f, None, -1, None, 0, None) == R.PR_EINVAL
    finally:
        R.pr_forest_destroy(f)


def test_route_noalloc_argument_errors_without_gpu():
    """pr_route_noalloc refuses a NULL forest and more queries than its scratch
    holds before any device work (the pointers are never read)."""
    from paper_2606_17059_amd import router as R
    L = R.lib()
    f = R.pr_forest_create(3)
    try:
        dummy = ctypes.c_void_p(16)
        n_over = R.PR_NOALLOC_MAX_QUERIES + 1
        assert L.pr_route_noalloc(None, dummy, 4, dummy, 1, dummy, dummy, None) == R.PR_EINVAL
        assert L.pr_route_noalloc(f, dummy, 4, dummy, n_over, dummy, dummy, None) == R.PR_EINVAL
        assert "at most" in R.pr_last_error()
        assert L.pr_route_noalloc(f, dummy, 4, dummy, -1, dummy, dummy, None) == R.PR_EINVAL
        assert L.pr_route_noalloc(f, None, 0, None, 0, None, None, None) == R.PR_OK
        # a forest never uploaded: refused, nothing enqueued
        assert L.pr_route_noalloc(f, dummy, 4, dummy, 1, dummy, dummy, None) == R.PR_ESTATE
    finally:
        R.pr_forest_destroy(f)
