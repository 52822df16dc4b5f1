"""Build libprefix_router.so in-tree for gfx950 (hipcc cross-compiles without a GPU)."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(PKG, "_build")
LIB_PATH = os.path.join(PKG, "libprefix_router.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# packed-fp32 instruction selection stays off for every HIP object in this library
HIP_FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wall", "-Wno-unused-result"]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    noise = "is not a recognized feature for this target"
    out = "\n".join(l for l in r.stdout.splitlines() if noise not in l)
    if r.returncode != 0:
        sys.stderr.write(out + "\n")
        raise RuntimeError("build step failed: " + " ".join(cmd))
    return out


def build(verbose: bool = False, defines=(), out_path: str = LIB_PATH) -> str:
    """Compile the library.  ``defines`` (e.g. "PR_LCP_VECTORS=16") override the
    kernels' compile-time tile constants."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    host_obj = os.path.join(BUILD_DIR, "forest_host.o")
    out = _run(["g++", *HOST_FLAGS, "-I", CSRC, "-c", os.path.join(CSRC, "forest_host.cpp"), "-o", host_obj])
    dev_obj = os.path.join(BUILD_DIR, "router.o")
    out += _run([HIPCC, *HIP_FLAGS, *["-D" + d for d in defines], "-I", INCLUDE, "-I", CSRC, "-c",
                 os.path.join(CSRC, "router.hip"), "-o", dev_obj])
    tmp = out_path + ".tmp"
    out += _run([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", dev_obj, host_obj, "-o", tmp])
    os.replace(tmp, out_path)
    if verbose and out.strip():
        print(out)
    return out_path


if __name__ == "__main__":
    print(build(verbose=True))
