"""GPU parity of the sparse 3x3 convolution (stride 1, padding 1; Sec. 3.2.3 direct
convolution as an SpMM on a virtual dense operand) against the CPU oracle's direct
definition, element by element, with the same tolerance as the SpMM:

    |C_gpu - C_ref| <= 1e-5 * sum |w| |x| + 1e-6   (GELU: x 1.13)."""
import numpy as np
import pytest

import oracle
import paper_2101_07948_amd as sd
from conftest import tol_fp32
from paper_2101_07948_amd import inputs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def tolerance(bound, ref, epi):
    return tol_fp32(bound, epi)


def gpu_conv(plan, X, bias, epi):
    Xt = torch.from_numpy(np.ascontiguousarray(X)).to(DEV)
    IC, H, W, NB = X.shape
    C = torch.full((plan.M, H, W, NB), float("nan"), device=DEV)
    bt = None if bias is None else torch.from_numpy(bias).to(DEV)
    plan.conv3x3(Xt, C, bt, epi)
    torch.cuda.synchronize()
    return C.cpu().numpy()


def check_conv(L, label="", **plan_kw):
    F = L.F
    with sd.Plan.from_csr(F, **plan_kw) as plan:
        got = gpu_conv(plan, L.X, L.bias, L.epi)
        perm = plan.perm
    ref, bound = oracle.conv3x3_f64(F.row_ptr, F.col_idx, F.values, L.X, L.bias, L.epi)
    if plan_kw.get("out_permuted"):
        ref, bound = ref[perm], bound[perm]
    err = np.abs(got.astype(np.float64) - ref)
    tol = tolerance(bound, ref, L.epi)
    bad = ~(err <= tol)
    assert not bad.any(), (f"{label}: {int(bad.sum())} of {bad.size} out of tolerance; "
                           f"worst err/tol {np.nanmax(err / tol):.3g}")
    return got


@pytest.mark.parametrize("OC,IC,H,W,NB,sparsity,epi", [
    (5, 3, 5, 7, 4, 0.5, "none"),        # one ragged tile, K = 27 (one chunk)
    (8, 4, 1, 1, 4, 0.3, "relu"),        # a single pixel: only the centre tap is in range
    (6, 2, 1, 9, 8, 0.2, "gelu"),        # one image row: every ky != 1 tap is padding
    (48, 32, 14, 14, 8, 0.9, "none"),    # paper-shaped: 14 x 14, 90 %
    (64, 64, 28, 28, 4, 0.95, "relu"),   # 28 x 28, 95 %, K = 576 over 18 chunks
    (40, 16, 7, 7, 12, 0.9, "gelu"),     # 7 x 7 images, N = 588 (ragged last tile)
])
def test_conv_parity(OC, IC, H, W, NB, sparsity, epi):
    L = inputs.conv_layer(OC, IC, H, W, NB, sparsity, layer=OC + IC + H, epi=epi)
    check_conv(L, f"OC={OC} IC={IC} {H}x{W}x{NB} s={sparsity} {epi}")


def test_conv_tall_panels_and_out_permuted():
    """96 channels over 256 column tiles: 4-row panels need two rounds of workgroups on
    256 CUs, 12-row panels one, so the call runs on the tall packing; the out_permuted
    plan writes output channels in its permutation order."""
    L = inputs.conv_layer(96, 16, 32, 32, 64, 0.9, layer=5, epi="relu")
    got = check_conv(L, "tall")
    gotp = check_conv(L, "tall permuted", out_permuted=True)
    with sd.Plan.from_csr(L.F) as plan:
        assert np.array_equal(gotp, got[plan.perm])


@pytest.mark.parametrize("OC,IC,HW", [(64, 64, 56), (128, 128, 28), (256, 256, 14)])
def test_conv_benchmark_shapes(OC, IC, HW):
    """The timed convolution shapes (16 images, 90 %): 64 x 64 on 56 x 56 runs on the
    tall packing (one round of workgroups instead of two), 128 x 128 on 28 x 28 on
    4-row panels with enough consumer waves per workgroup to fit one round."""
    L = inputs.conv_layer(OC, IC, HW, HW, 16, 0.9, layer=OC + HW)
    check_conv(L, f"{OC}x{IC} {HW}x{HW}x16")


def test_conv_chain():
    """Two convolutions chained on the GPU's own output (C of one is X of the next)."""
    L1 = inputs.conv_layer(24, 8, 10, 12, 4, 0.8, layer=31, epi="relu")
    Y = check_conv(L1, "chain 1")
    F2 = inputs.pattern_uniform(16, 24 * 9, 0.2, inputs.CFG_CONV, 32, 0.05)
    L2 = inputs.ConvLayer(F2, Y.astype(np.float32), None, "none")
    check_conv(L2, "chain 2")


def test_conv_rejects_bad_shapes():
    L = inputs.conv_layer(8, 4, 6, 6, 4, 0.5, layer=40)
    X = torch.from_numpy(L.X).to(DEV)
    with sd.Plan.from_csr(L.F) as plan:
        lib = plan._lib
        C = torch.empty((8, 6, 6, 4), device=DEV)
        # NB not a multiple of 4
        X3 = torch.zeros((4, 6, 6, 3), device=DEV)
        C3 = torch.empty((8, 6, 6, 3), device=DEV)
        assert lib.sdnn_conv3x3(plan.handle, X3.data_ptr(), C3.data_ptr(), 6, 6, 3, None, 0,
                                None) == 2
        # misaligned X
        assert lib.sdnn_conv3x3(plan.handle, X.data_ptr() + 4, C.data_ptr(), 6, 6, 4, None, 0,
                                None) == 2
        # X overlapping C
        assert lib.sdnn_conv3x3(plan.handle, C.data_ptr(), C.data_ptr(), 6, 6, 4, None, 0,
                                None) == 2
        # empty image: no-op
        assert lib.sdnn_conv3x3(plan.handle, X.data_ptr(), C.data_ptr(), 0, 6, 4, None, 0,
                                None) == 0
    # K not a multiple of 9
    W = inputs.pattern_uniform(8, 20, 0.3, inputs.CFG_TEST, 41, 0.05)
    with sd.Plan.from_csr(W) as plan:
        assert plan._lib.sdnn_conv3x3(plan.handle, X.data_ptr(), C.data_ptr(), 6, 6, 4, None,
                                      0, None) == 2
    # a plan built with in_perm
    with sd.Plan.from_csr(L.F, in_perm=np.arange(36)[::-1].copy()) as plan:
        assert plan._lib.sdnn_conv3x3(plan.handle, X.data_ptr(), C.data_ptr(), 6, 6, 4, None,
                                      0, None) == 2
