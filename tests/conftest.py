import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


# GELU's derivative x*phi(x) + Phi(x) peaks at 1.1289 (x = sqrt(2)): an input error e
# moves GELU by at most 1.13 e.
GELU_LIPSCHITZ = 1.13


def tol_fp32(bound, epi="none"):
    """Parity tolerance for an fp32 result against the double-precision reference:
    |err| <= 1e-5 * sum_p |w_p| |B[c_p, n]| + 1e-6, per element; after GELU the same
    bound times GELU's Lipschitz constant (the activation's own float rounding, a few ulp
    of |C|, stays far inside the 1e-6 floor for the |C| <= ~10 these workloads reach)."""
    tol = 1e-5 * bound + 1e-6
    return tol * GELU_LIPSCHITZ if epi == "gelu" else tol


def random_csr(rng, M, K, density):
    """Tiny random CSR for oracle pins (not a workload generator)."""
    mask = rng.random((M, K)) < density
    W = np.where(mask, rng.standard_normal((M, K)), 0.0).astype(np.float32)
    rows, cols = np.nonzero(mask)
    row_ptr = np.zeros(M + 1, dtype=np.int32)
    np.cumsum(mask.sum(axis=1), out=row_ptr[1:])
    return row_ptr, cols.astype(np.int32), W[rows, cols].astype(np.float32), W


def dense_to_csr(W):
    W = np.asarray(W, dtype=np.float32)
    M, K = W.shape
    mask = W != 0
    rows, cols = np.nonzero(mask)
    row_ptr = np.zeros(M + 1, dtype=np.int32)
    np.cumsum(mask.sum(axis=1), out=row_ptr[1:])
    return row_ptr, cols.astype(np.int32), W[rows, cols].astype(np.float32)


def pattern_to_csr(rows_cols, K):
    """CSR (values 1.0) from a list of column lists."""
    row_ptr = np.zeros(len(rows_cols) + 1, dtype=np.int32)
    cols = []
    for i, cs in enumerate(rows_cols):
        cs = sorted(cs)
        cols.extend(cs)
        row_ptr[i + 1] = row_ptr[i] + len(cs)
    col_idx = np.array(cols, dtype=np.int32)
    return row_ptr, col_idx, np.ones(len(cols), dtype=np.float32)


def load_reorder_examples():
    path = os.path.join(ROOT, "tests", "golden", "reorder_examples.txt")
    out = []
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        name, K, rows, perm = [x.strip() for x in line.split("|")]
        rc = [[] if r.strip() == "-" else [int(c) for c in r.split(",")] for r in rows.split(";")]
        out.append((name, int(K), rc, [int(x) for x in perm.split(",")]))
    return out


def load_normal_cdf():
    path = os.path.join(ROOT, "tests", "golden", "normal_cdf.txt")
    xs, ps = [], []
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        x, p = line.split()
        xs.append(float(x))
        ps.append(float(p))
    return np.array(xs), np.array(ps)
