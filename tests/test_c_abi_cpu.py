"""CPU checks that the boundary is plain C: include/sdnn.h compiles as strict C99, and
the plain-C caller that the GPU test runs compiles against it (no GPU is touched)."""
import os
import runpy
import shutil
import subprocess

import pytest

from conftest import ROOT

pytestmark = pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not installed")


def test_header_is_strict_c99():
    for std in ("c99", "c11"):
        r = subprocess.run(["gcc", f"-std={std}", "-Wall", "-Wextra", "-pedantic", "-Werror",
                            "-x", "c", "-fsyntax-only", os.path.join(ROOT, "include", "sdnn.h")],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr


def test_c_caller_compiles():
    if not os.path.isdir("/opt/rocm/include"):
        pytest.skip("HIP headers not installed")
    cmd = runpy.run_path(os.path.join(ROOT, "tests", "c_abi", "build_check.py"))["command"]
    r = subprocess.run(cmd(syntax_only=True), capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_c_caller_agrees_on_struct_layouts():
    """The built C caller (if present) was compiled with the struct sizes the binding
    uses: a host-only query, no device work."""
    import ctypes
    import paper_2101_07948_amd as sd
    exe = os.path.join(ROOT, "tests", "c_abi", "sdnn_c_check")
    if not os.path.exists(exe):
        pytest.skip("the C caller is built by __graft_entry__.build()")
    r = subprocess.run([exe, "-sizes"], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    assert r.stdout.split() == [str(ctypes.sizeof(sd.PlanOpts)), str(ctypes.sizeof(sd.PlanInfo))]
