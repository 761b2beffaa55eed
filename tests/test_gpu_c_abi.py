"""The C ABI driven from a plain C99 program (tests/c_abi/sdnn_c_check.c, built by the
repository's build step) in a child process: plan creation, sdnn_spmm, sdnn_spmm_split
and sdnn_spmm from a plan fixed to 128-column tiles, with a GELU epilogue, results
checked here against the CPU oracle with the parity bar (|err| <= 1.13 * (1e-5 * sum |w||b|
+ 1e-6) for GELU) and the permutation against the oracle's Algorithm 1 bit for bit."""
import os
import subprocess

import numpy as np
import pytest

import oracle
from conftest import ROOT, tol_fp32
from paper_2101_07948_amd import inputs

pytestmark = pytest.mark.gpu
EXE = os.path.join(ROOT, "tests", "c_abi", "sdnn_c_check")


@pytest.mark.parametrize("N", [130, 132])
def test_c_caller_matches_oracle(tmp_path, N):
    """N = 130 stages B in 4-byte pieces (no 128-column tiles); N = 132 allows the
    128-column tiles, whose result equals the 256-column one bit for bit."""
    assert os.path.exists(EXE), f"{EXE} is missing: run __graft_entry__.build() first"
    # a binary built against another sdnn.h would disagree with the library on struct
    # layouts: compare the sizes it was compiled with (a host-only query) first
    import ctypes
    import paper_2101_07948_amd as sd
    r = subprocess.run([EXE, "-sizes"], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    assert r.stdout.split() == [str(ctypes.sizeof(sd.PlanOpts)), str(ctypes.sizeof(sd.PlanInfo))], \
        f"{EXE} was built against another sdnn.h: run __graft_entry__.build() again"
    M, K = 70, 333
    W = inputs.pattern_uniform(M, K, 0.1, inputs.CFG_TEST, 8100, 0.05)
    B = inputs.dense_B(K, N, inputs.CFG_TEST, 8100)
    bias = inputs.bias_normal(M, inputs.CFG_TEST, 8100, 0.02)
    for name, arr in (("row_ptr.i32", W.row_ptr.astype(np.int32)),
                      ("col_idx.i32", W.col_idx.astype(np.int32)),
                      ("values.f32", W.values.astype(np.float32)),
                      ("B.f32", B.astype(np.float32)), ("bias.f32", bias.astype(np.float32))):
        arr.tofile(tmp_path / name)
    print(f"c_abi: M={M} K={K} N={N}", flush=True)
    r = subprocess.run([EXE, str(tmp_path), str(M), str(K), str(N)], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, K, B, bias, "gelu")
    tol = tol_fp32(bound, "gelu")
    for name in ("C_plain.f32", "C_split.f32", "C_narrow.f32"):
        got = np.fromfile(tmp_path / name, dtype=np.float32).reshape(M, N).astype(np.float64)
        bad = ~(np.abs(got - ref) <= tol)
        assert not bad.any(), f"{name}: {int(bad.sum())} of {bad.size} out of tolerance"
    plain = np.fromfile(tmp_path / "C_plain.f32", dtype=np.float32)
    assert np.array_equal(plain, np.fromfile(tmp_path / "C_narrow.f32", dtype=np.float32))
    assert f"tile={128 if N % 4 == 0 else 256}" in r.stdout, r.stdout
    perm = np.fromfile(tmp_path / "perm.i32", dtype=np.int32)
    assert np.array_equal(perm, oracle.reorder(W.row_ptr, W.col_idx, K))
