"""Compiles sdnn_c_check.c (a plain C99 caller of include/sdnn.h) against the built
libsdnn.so with gcc.  Test infrastructure, called by the repository's build step."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "sdnn_c_check.c")
EXE = os.path.join(HERE, "sdnn_c_check")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def command(out=EXE, syntax_only=False):
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
           "-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(ROCM, "include"), SRC]
    if syntax_only:
        return cmd + ["-fsyntax-only"]
    return cmd + ["-L" + os.path.join(ROOT, "paper_2101_07948_amd"), "-lsdnn",
                  "-L" + os.path.join(ROCM, "lib"), "-lamdhip64",
                  "-Wl,-rpath,$ORIGIN/../../paper_2101_07948_amd",
                  "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-o", out]


def build() -> str:
    tmp = EXE + ".tmp%d" % os.getpid()
    res = subprocess.run(command(tmp), capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("gcc failed building sdnn_c_check:\n" + res.stderr[-4000:])
    os.replace(tmp, EXE)
    return EXE


if __name__ == "__main__":
    print(build())
