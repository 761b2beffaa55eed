"""CPU-only pins of the oracle (no GPU): it must agree with what the paper and the
mathematics fix before it can judge the GPU path."""
import numpy as np
import pytest

import _pins
import oracle
from conftest import tol_fp32
from paper_2101_07948_amd import inputs


@pytest.mark.parametrize("check", _pins.ALL_CHECKS, ids=lambda c: c.__name__)
def test_oracle_pin(check):
    fails = check()
    assert not fails, "\n".join(fails)


def test_f32_baseline_within_tolerance():
    """The timed fp32 baseline stays within the parity tolerance of the double
    reference on a BERT-shaped layer (a sanity check of the tolerance's margin)."""
    w = inputs.workload("c2", N=96)
    L = w.layers[0]
    C64, bound = oracle.spmm_f64(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.K, w.B, L.bias, L.epi)
    C32 = oracle.spmm_f32(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.K, w.B, L.bias, L.epi)
    err = np.abs(C32.astype(np.float64) - C64)
    assert np.all(err <= tol_fp32(bound))
    # the margin is real: typical error is far below the bound
    assert np.median(err / tol_fp32(bound)) < 0.2


@pytest.mark.parametrize("epi", ["relu", "gelu"])
def test_f32_baseline_epilogues(epi):
    w = inputs.workload("c1")
    L = w.layers[0]
    C64, bound = oracle.spmm_f64(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.K, w.B, L.bias, epi)
    C32 = oracle.spmm_f32(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.K, w.B, L.bias, epi)
    assert np.all(np.abs(C32 - C64) <= tol_fp32(bound) * 1.13 + 1e-7)


def test_reorder_on_workload_is_permutation():
    w = inputs.workload("c1")
    W = w.layers[0].W
    perm = oracle.reorder(W.row_ptr, W.col_idx, W.K)
    assert sorted(perm.tolist()) == list(range(W.M))
    nnz = np.diff(W.row_ptr)
    assert nnz[perm[0]] == nnz.max()
