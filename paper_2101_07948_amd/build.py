"""Builds libsdnn.so (the gfx950 HIP kernels + C ABI) and libsdnn_probes.so (the
measurement probes of include/sdnn_probes.h) in place with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libsdnn.so")
SOURCES = [os.path.join(HERE, "csrc", "sdnn_host.cpp"), os.path.join(HERE, "csrc", "sdnn_kernels.hip")]
PROBES_LIB = os.path.join(HERE, "libsdnn_probes.so")
PROBES_SOURCES = [os.path.join(HERE, "csrc", "sdnn_probes.hip")]

# -packed-fp32-ops: keep the compiler from forming packed FP32 instructions.
HIPCC_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-Wall",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if cand and (os.path.isabs(cand) and os.path.exists(cand) or not os.path.isabs(cand)):
            return cand
    return "hipcc"


def build(verbose: bool = False) -> str:
    # regenerate the inline-assembly inner loop (a pure function of its generator)
    sys.path.insert(0, os.path.join(HERE, "csrc"))
    try:
        import gen_spmm_asm
        gen_spmm_asm.main()
    finally:
        sys.path.pop(0)
    for lib, sources in ((LIB, SOURCES), (PROBES_LIB, PROBES_SOURCES)):
        tmp = lib + ".tmp%d" % os.getpid()
        cmd = [hipcc()] + HIPCC_FLAGS + ["-o", tmp] + sources
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            sys.stderr.write(res.stdout + res.stderr)
            raise RuntimeError(f"hipcc failed building {os.path.basename(lib)}")
        if verbose:
            sys.stderr.write(res.stderr)
        os.replace(tmp, lib)
    return LIB


HOST_SANITIZED_SOURCES = [os.path.join(HERE, "csrc", "sdnn_host.cpp"),
                          os.path.join(HERE, "csrc", "sdnn_launch_stubs.cpp")]


def build_host_sanitized(out: str) -> str:
    """The host code alone (CSR validation, row orders, packing and its self-check, the
    C ABI's argument checks) built for the CPU under AddressSanitizer and
    UndefinedBehaviorSanitizer, with the kernel launchers replaced by stubs that fail
    (sdnn_launch_stubs.cpp).  It serves the host-only entry points; load it in a process
    started with the sanitizer runtime preloaded (tests/test_host_sanitized.py)."""
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-shared", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I" + os.path.join(rocm, "include"), "-o", out]
    cmd += HOST_SANITIZED_SOURCES
    cmd += ["-L" + os.path.join(rocm, "lib"), "-lamdhip64", "-Wl,-rpath," + os.path.join(rocm, "lib")]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("g++ failed building the sanitizer build of the host code")
    return out


if __name__ == "__main__":
    if "--host-sanitized" in sys.argv:
        print(build_host_sanitized(os.path.join(HERE, "libsdnn_host_asan.so")))
    else:
        print(build(verbose=True))
