"""The C ABI from plain C11: tests/c/abi_check.c is compiled with gcc against
include/prefix_router.h (-pedantic, warnings as errors), linked with the built
library, and run: argument and state checks on the host, then a small forest
on the GPU (load, route, merge, selection, export) against hand-worked values."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2606_17059_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


@pytest.fixture(scope="module")
def abi_check(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("c_client") / "abi_check")
    cmd = ["gcc", "-std=c11", "-Wall", "-Wextra", "-pedantic", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-isystem", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "c", "abi_check.c"), "-o", exe,
           "-L", PKG, "-lprefix_router", "-Wl,-rpath," + PKG,
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, r.stdout
    return exe


def test_c_client_host_checks(abi_check):
    r = subprocess.run([abi_check, "host"], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                       timeout=120)
    assert r.returncode == 0, r.stdout
    assert "abi_check host: ok" in r.stdout


@pytest.mark.gpu
def test_c_client_device_checks(abi_check):
    from gpu_util import announce
    announce("C client: load, route, merge, select, export on a 3-peer forest")
    r = subprocess.run([abi_check, "device"], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                       timeout=120)
    assert r.returncode == 0, r.stdout
    assert "abi_check device: ok" in r.stdout
