"""The non-allocating K-split call (sdnn_spmm_split_noalloc), through the C ABI, against
the allocating one (sdnn_spmm_split with a caller workspace) and the CPU oracle: two
calls in a row on the same device scratch, the second with a smaller input, each equal
bit for bit to the workspace call with the same run count (same kernels, same summation
order) and within the parity bar of the oracle."""
import ctypes

import numpy as np
import pytest

import oracle
import paper_2101_07948_amd as sd
from conftest import tol_fp32
from paper_2101_07948_amd import inputs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _call_noalloc(plan, B, C, bias, epi, splits):
    L = sd.lib()
    N = B.shape[1]
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return L.sdnn_spmm_split_noalloc(plan.handle, B.data_ptr(), C.data_ptr(), N,
                                     None if bias is None else bias.data_ptr(), sd.EPI[epi],
                                     splits, stream)


@pytest.mark.parametrize("splits", [0, 3])
def test_noalloc_matches_workspace_call(splits):
    cases = [  # (M, K, N, seed): the second call is smaller than the first
        (700, 2048, 1024, 1),
        (300, 1100, 200, 2),
    ]
    for M, K, N, seed in cases:
        print(f"noalloc: M={M} K={K} N={N} splits={splits}", flush=True)
        W = inputs.pattern_uniform(M, K, 0.1, inputs.CFG_TEST, 9000 + seed, 0.05)
        Bn = inputs.dense_B(K, N, inputs.CFG_TEST, 9000 + seed)
        bn = inputs.bias_normal(M, inputs.CFG_TEST, 9000 + seed, 0.02)
        B = torch.from_numpy(Bn).to(DEV)
        bias = torch.from_numpy(bn).to(DEV)
        with sd.Plan.from_csr(W, split_chunks=4) as plan:
            runs = plan.info["splits"]
            assert runs > 1
            C_ws = torch.full((M, N), float("nan"), device=DEV)
            ws = torch.full((plan.workspace_floats(N),), float("nan"), device=DEV)
            plan.spmm_split(B, C_ws, bias, "gelu", workspace=ws, splits=splits)
            C_na = torch.full((M, N), float("nan"), device=DEV)
            assert _call_noalloc(plan, B, C_na, bias, "gelu", splits) == 0
            torch.cuda.synchronize()
            assert torch.equal(C_na, C_ws), f"M={M} N={N}: differs from the workspace call"
        ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, K, Bn, bn, "gelu")
        err = np.abs(C_na.cpu().numpy().astype(np.float64) - ref)
        assert (err <= tol_fp32(bound, "gelu")).all(), f"M={M} N={N}: out of tolerance"


def test_noalloc_rejects_scratch_overflow():
    """A call whose partial products would exceed the fixed scratch returns SDNN_ERR_DIM
    (checked on the host before any launch)."""
    M, K, N = 4096, 1024, 8192
    W = inputs.pattern_uniform(M, K, 0.01, inputs.CFG_TEST, 9100, 0.05)
    with sd.Plan.from_csr(W, split_chunks=1) as plan:
        B = torch.zeros((K, N), device=DEV)
        C = torch.zeros((M, N), device=DEV)
        # 32 runs x 4096 x 8192 floats is far above 16 Mi floats
        assert _call_noalloc(plan, B, C, None, "none", 32) == 2
    torch.cuda.synchronize()
