"""The host code (CSR validation, Algorithm 1 and the other row orders, packing and the
packed stream's self-check, the C ABI's argument checks) built for the CPU with
AddressSanitizer and UndefinedBehaviorSanitizer, and the host-only ABI tests run against
that build in a child process that preloads the sanitizer runtime.  Any out-of-bounds
access, use after free or undefined operation in that code aborts the child."""
import os
import subprocess
import sys

import pytest

from conftest import ROOT

MODULES = ["tests/test_abi_cpu.py", "tests/test_row_orders.py", "tests/test_split_cpu.py"]

RUNNER = r'''
import sys
sys.path.insert(0, {root!r}); sys.path.insert(0, {tests!r})
import paper_2101_07948_amd as sd
sd.LIB_PATH = {lib!r}
import pytest
rc = pytest.main(["-q", "-x", "-p", "no:cacheprovider"] + {modules!r})
maps = open("/proc/self/maps").read()
assert {lib!r} in maps, "the sanitizer build was not the library the tests loaded"
assert "libasan" in maps, "the sanitizer runtime is not loaded"
print("SANITIZED_RUN_RC", int(rc))
sys.exit(int(rc))
'''


def _asan_runtime():
    r = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


def test_host_code_under_asan_and_ubsan(tmp_path):
    runtime = _asan_runtime()
    if runtime is None:
        pytest.skip("no AddressSanitizer runtime for g++ on this host")
    from paper_2101_07948_amd import build
    lib = build.build_host_sanitized(str(tmp_path / "libsdnn_host_asan.so"))
    script = tmp_path / "run.py"
    script.write_text(RUNNER.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=lib,
                                    modules=MODULES))
    env = dict(os.environ)
    env["LD_PRELOAD"] = runtime
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([sys.executable, str(script)], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=1200)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0 and "SANITIZED_RUN_RC 0" in r.stdout, tail
