"""GPU parity of the 128-column tiles (plan option tile_cols = 128: two columns per lane,
a 64 KB staging ring, two workgroups per CU) against the CPU oracle with the parity bar,
and against the 256-column tiles bit for bit (both sum each row's entries in ascending
column order).  Covers every panel height, ragged N (N % 128 != 0) and ragged K (the
clamped staging of a partial last chunk), each epilogue, forced consumer counts, the
persistent launches (tile-major and per-tile), out_permuted plans, K-split calls, the
fallback to 256-column tiles where a call does not allow 128 (N % 4 != 0, a misaligned B),
the poll budget and tuning over both widths and over the workgroups along K."""
import os

import numpy as np
import pytest

import oracle
import paper_2101_07948_amd as sd
from conftest import tol_fp32
from paper_2101_07948_amd import inputs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"


class Env:
    """Sets environment overrides of the launch for the duration of a block."""

    def __init__(self, **kv):
        self.kv = {k: str(v) for k, v in kv.items() if v is not None}

    def __enter__(self):
        self.old = {k: os.environ.get(k) for k in self.kv}
        os.environ.update(self.kv)

    def __exit__(self, *a):
        for k, v in self.old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def run(plan, B, bias, epi, Bt=None):
    Bt = torch.from_numpy(np.ascontiguousarray(B)).to(DEV) if Bt is None else Bt
    bt = None if bias is None else torch.from_numpy(np.ascontiguousarray(bias)).to(DEV)
    C = torch.full((plan.M, B.shape[1]), float("nan"), device=DEV)
    plan.spmm(Bt, C, bt, epi)
    torch.cuda.synchronize()
    return C.cpu().numpy()


def assert_parity(W, B, bias, epi, got, label):
    ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, W.K, B, bias, epi)
    err = np.abs(got.astype(np.float64) - ref)
    tol = tol_fp32(bound, epi)
    bad = ~(err <= tol)
    assert not bad.any(), (f"{label}: {int(bad.sum())} of {bad.size} elements out of tolerance; "
                           f"worst err/tol {np.nanmax(err / tol):.3g}")


def both_widths(W, B, bias, epi, label, **plan_kw):
    """The product on 128- and on 256-column tiles: parity of the first, equality of both."""
    print(f"tiles: {label}", flush=True)
    with sd.Plan.from_csr(W, tile_cols=128, **plan_kw) as plan:
        if B.shape[1] % 4 == 0:
            assert plan.launch_shape(B.shape[1])["tile_cols"] == 128, label
        narrow = run(plan, B, bias, epi)
    with sd.Plan.from_csr(W, tile_cols=256, **plan_kw) as plan:
        assert plan.launch_shape(B.shape[1])["tile_cols"] == 256, label
        wide = run(plan, B, bias, epi)
    assert_parity(W, B, bias, epi, narrow, label)
    assert np.array_equal(narrow, wide, equal_nan=False), label
    return narrow


@pytest.mark.parametrize("rw", [4, 8, 12, 16])
@pytest.mark.parametrize("M,K,N", [(200, 300, 132), (500, 768, 1000), (96, 64, 128)])
def test_every_panel_height(rw, M, K, N):
    """K = 300 and 64: a partial last chunk and an exact one; N = 132, 1000: ragged last
    tiles (4 and 104 columns), N = 128 one full tile."""
    W = inputs.pattern_uniform(M, K, 0.1, inputs.CFG_TEST, 4100 + rw + M, 0.05)
    B = inputs.dense_B(K, N, inputs.CFG_TEST, 4200 + N)
    bias = inputs.bias_normal(M, inputs.CFG_TEST, 4300 + M, 0.02)
    both_widths(W, B, bias, "none", f"RW {rw} M {M} K {K} N {N}", panel_rows=rw)


@pytest.mark.parametrize("epi", ["relu", "gelu"])
def test_epilogues(epi):
    W = inputs.pattern_uniform(300, 500, 0.15, inputs.CFG_TEST, 4400, 0.05)
    B = inputs.dense_B(500, 516, inputs.CFG_TEST, 4401)
    bias = inputs.bias_normal(300, inputs.CFG_TEST, 4402, 0.02)
    both_widths(W, B, bias, epi, epi)


@pytest.mark.parametrize("waves", [1, 3, 10])
def test_forced_consumer_counts(waves):
    W = inputs.pattern_uniform(400, 640, 0.1, inputs.CFG_TEST, 4500 + waves, 0.05)
    B = inputs.dense_B(640, 512, inputs.CFG_TEST, 4501)
    with Env(SDNN_FORCE_WAVES=waves):
        both_widths(W, B, None, "none", f"{waves} consumer waves", panel_rows=4)


def test_w0_full_size():
    """The 768 x 3072 layer at 90 % and N = 4096 (512 items of (tile, row-block) on two
    workgroups per CU) with a bias and GELU."""
    w = inputs.workload("w0")
    L = w.layers[0]
    both_widths(L.W, w.B, L.bias, "gelu", "w0")


def test_persistent_tile_major_c5_ffn1():
    """C5's 3072 x 768 layer at 97 % and N = 16384: 128 full tiles, more items than
    workgroup slots, so the workgroups take tile-major items in turn; sampled rows
    against the oracle (all columns), all of C against the 256-column tiles."""
    w = inputs.workload("c5", N=16384, num_layers=1)
    L = w.layers[4]
    assert (L.W.M, L.W.K) == (3072, 768)
    with sd.Plan.from_csr(L.W, tile_cols=128) as plan:
        narrow = run(plan, w.B, L.bias, L.epi)
    with sd.Plan.from_csr(L.W, tile_cols=256) as plan:
        wide = run(plan, w.B, L.bias, L.epi)
    assert np.array_equal(narrow, wide)
    ref, bound = oracle.spmm_f64(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.K, w.B, L.bias, L.epi)
    rows = np.random.default_rng(4600).choice(L.W.M, 48, replace=False)
    err = np.abs(narrow[rows].astype(np.float64) - ref[rows])
    assert (err <= tol_fp32(bound[rows], L.epi)).all()


def test_persistent_per_tile_ragged():
    """More items than slots with a ragged N (N % 128 = 4): workgroups of a tile take its
    row-blocks in turn."""
    W = inputs.pattern_uniform(3072, 256, 0.05, inputs.CFG_TEST, 4700, 0.05)
    B = inputs.dense_B(256, 4100, inputs.CFG_TEST, 4701)
    both_widths(W, B, None, "none", "per-tile persistence", panel_rows=4)


def test_out_permuted():
    W = inputs.pattern_uniform(333, 400, 0.1, inputs.CFG_TEST, 4800, 0.05)
    B = inputs.dense_B(400, 260, inputs.CFG_TEST, 4801)
    bias = inputs.bias_normal(333, inputs.CFG_TEST, 4802, 0.02)
    with sd.Plan.from_csr(W, tile_cols=128, out_permuted=True) as plan:
        got = run(plan, B, bias, "relu")
        perm = plan.perm
    ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, W.K, B, bias, "relu")
    err = np.abs(got.astype(np.float64) - ref[perm])
    assert (err <= tol_fp32(bound[perm], "relu")).all()


def test_fallbacks_to_256_columns():
    """Calls that do not allow 128-column tiles run on 256-column ones: N % 4 != 0 and a B
    that is not 16-byte aligned."""
    M, K = 150, 200
    W = inputs.pattern_uniform(M, K, 0.1, inputs.CFG_TEST, 4900, 0.05)
    with sd.Plan.from_csr(W, tile_cols=128) as plan:
        assert plan.launch_shape(130)["tile_cols"] == 256
        B = inputs.dense_B(K, 130, inputs.CFG_TEST, 4901)
        assert_parity(W, B, None, "none", run(plan, B, None, "none"), "N = 130")
        B = inputs.dense_B(K, 256, inputs.CFG_TEST, 4902)
        flat = torch.empty(K * 256 + 1, device=DEV)
        Bt = flat[1:].view(K, 256)
        Bt.copy_(torch.from_numpy(B))
        assert Bt.data_ptr() % 16 != 0
        assert_parity(W, B, None, "none", run(plan, B, None, "none", Bt=Bt), "misaligned B")


@pytest.mark.parametrize("rw", [4, 16])
@pytest.mark.parametrize("splits", [2, 3, 0])
def test_k_split_calls(rw, splits):
    """sdnn_spmm_split on 128-column tiles (K = 1000: 32 chunks, the last one ragged, in
    segments of 3 chunks; N = 516: a ragged last tile): each run's partial products, the
    reduction with bias and GELU, against the oracle, and bit for bit against the
    256-column tiles at the same run boundaries."""
    M, K, N = 400, 1000, 516
    W = inputs.pattern_uniform(M, K, 0.1, inputs.CFG_TEST, 5200 + rw, 0.05)
    B = inputs.dense_B(K, N, inputs.CFG_TEST, 5201)
    bias = inputs.bias_normal(M, inputs.CFG_TEST, 5202, 0.02)
    Bt = torch.from_numpy(B).to(DEV)
    bt = torch.from_numpy(bias).to(DEV)
    out = {}
    for tw in (128, 256):
        with sd.Plan.from_csr(W, tile_cols=tw, panel_rows=rw, split_chunks=3) as plan:
            runs = plan.split_runs(N, splits)
            C = torch.full((M, N), float("nan"), device=DEV)
            plan.spmm_split(Bt, C, bt, "gelu", splits=runs)
            torch.cuda.synchronize()
            out[tw] = C.cpu().numpy()
    print(f"tiles: K-split RW {rw} splits {splits} -> {runs} runs", flush=True)
    assert_parity(W, B, bias, "gelu", out[128], f"split {runs}")
    assert np.array_equal(out[128], out[256])


def test_tune_records_split_runs():
    """On a plan with K-segments sdnn_plan_tune also times the workgroup counts along K;
    spmm_split with splits = 0 then runs the recorded count, against the oracle."""
    W = inputs.pattern_uniform(768, 3072, 0.1, inputs.CFG_TEST, 5300, 0.02)
    N = 1024
    B = inputs.dense_B(3072, N, inputs.CFG_TEST, 5301)
    Bt = torch.from_numpy(B).to(DEV)
    with sd.Plan.from_csr(W, split_chunks=4) as plan:
        plan.tune(N, Bt, torch.empty(768, N, device=DEV))
        runs = plan.split_runs(N)
        assert 1 <= runs <= plan.info["splits"]
        C = torch.full((768, N), float("nan"), device=DEV)
        plan.spmm_split(Bt, C, None, "none")
        torch.cuda.synchronize()
    print(f"tiles: tuned split runs {runs}", flush=True)
    assert_parity(W, B, None, "none", C.cpu().numpy(), f"tuned {runs} runs")


@pytest.mark.parametrize("budget", [0, 2, 64])
def test_poll_budget(budget):
    """A wave whose poll budget runs out goes on without waiting and leaves NaN: every
    output is within the bar or NaN, and all NaN at budget 0."""
    M, K, N = 300, 1000, 512
    W = inputs.pattern_uniform(M, K, 0.1, inputs.CFG_TEST, 5000, 0.05)
    B = inputs.dense_B(K, N, inputs.CFG_TEST, 5001)
    with Env(SDNN_POLL_BUDGET=budget):
        with sd.Plan.from_csr(W, tile_cols=128) as plan:
            got = run(plan, B, None, "none")
    ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, K, B, None, "none")
    err = np.abs(got.astype(np.float64) - ref)
    ok = (err <= tol_fp32(bound, "none")) | np.isnan(got)
    assert ok.all(), f"{int((~ok).sum())} finite outputs out of tolerance"
    if budget == 0:
        assert np.isnan(got).all()


def test_tune_searches_both_widths():
    """sdnn_plan_tune times both tile widths; whichever it records, later calls use it and
    agree with the oracle."""
    W = inputs.pattern_uniform(768, 768, 0.1, inputs.CFG_TEST, 5100, 0.02)
    N = 1024
    B = inputs.dense_B(768, N, inputs.CFG_TEST, 5101)
    with sd.Plan.from_csr(W) as plan:
        Bt = torch.from_numpy(B).to(DEV)
        shape = plan.tune(N, Bt, torch.empty(768, N, device=DEV))
        assert shape["tile_cols"] in (128, 256)
        assert plan.launch_shape(N) == shape
        got = run(plan, B, None, "none", Bt=Bt)
    assert_parity(W, B, None, "none", got, f"tuned {shape}")


@pytest.mark.parametrize("M,K,N,waves", [(200, 300, 132, None), (900, 768, 1000, 12),
                                         (500, 640, 516, 3)])
def test_deep_panels(M, K, N, waves):
    """32-row panels (128-column tiles only, up to 14 consumer waves): parity with bias and
    GELU, and bit for bit the 256-column result (ragged K and N, forced consumer counts)."""
    W = inputs.pattern_uniform(M, K, 0.05, inputs.CFG_TEST, 5400 + M, 0.05)
    B = inputs.dense_B(K, N, inputs.CFG_TEST, 5401)
    bias = inputs.bias_normal(M, inputs.CFG_TEST, 5402, 0.02)
    with Env(SDNN_FORCE_WAVES=waves):
        with sd.Plan.from_csr(W, panel_rows=32, tile_cols=128) as plan:
            assert plan.launch_shape(N)["panel_rows"] == 32
            deep = run(plan, B, bias, "gelu")
    with sd.Plan.from_csr(W, tile_cols=256) as plan:
        wide = run(plan, B, bias, "gelu")
    print(f"tiles: deep M {M} K {K} N {N}", flush=True)
    assert_parity(W, B, bias, "gelu", deep, "deep panels")
    assert np.array_equal(deep, wide)


@pytest.mark.parametrize("splits", [2, 3])
def test_deep_panels_k_split(splits):
    M, K, N = 700, 1000, 260
    W = inputs.pattern_uniform(M, K, 0.05, inputs.CFG_TEST, 5500, 0.05)
    B = inputs.dense_B(K, N, inputs.CFG_TEST, 5501)
    Bt = torch.from_numpy(B).to(DEV)
    out = []
    for kw in ({"panel_rows": 32, "tile_cols": 128}, {"tile_cols": 256}):
        with sd.Plan.from_csr(W, split_chunks=3, **kw) as plan:
            C = torch.full((M, N), float("nan"), device=DEV)
            plan.spmm_split(Bt, C, None, "none", splits=splits)
            torch.cuda.synchronize()
            out.append(C.cpu().numpy())
    assert_parity(W, B, None, "none", out[0], f"deep split {splits}")
    assert np.array_equal(out[0], out[1])


def test_deep_panels_need_128_column_calls():
    """A plan of 32-row panels alone rejects calls that cannot run on 128-column tiles."""
    W = inputs.pattern_uniform(64, 90, 0.1, inputs.CFG_TEST, 5600, 0.05)
    with sd.Plan.from_csr(W, panel_rows=32, tile_cols=128) as plan:
        with pytest.raises(sd.SdnnError) as ei:
            plan.spmm(torch.zeros(90, 130, device=DEV), torch.zeros(64, 130, device=DEV))
        assert ei.value.code == 2
        with pytest.raises(sd.SdnnError) as ei:
            plan.conv3x3(torch.zeros(10, 4, 4, 4, device=DEV), torch.zeros(64, 4, 4, 4, device=DEV))
        assert ei.value.code == 2
        # nor can it be tuned for such a call (no packing to time), and nothing is recorded
        before = plan.launch_shape(130)
        with pytest.raises(sd.SdnnError) as ei:
            plan.tune(130, torch.zeros(90, 130, device=DEV), torch.zeros(64, 130, device=DEV))
        assert ei.value.code == 2
        assert plan.launch_shape(130) == before


def test_default_plan_takes_deep_panels_at_97_percent():
    """C5's 97 % layers at N = 16384 run on the default plan's 32-row packing with 12
    consumer waves on 128-column tiles; at N = 8192 the 768-row layers' deep grid would
    not fill the CUs and they keep the other packings."""
    if torch.cuda.get_device_properties(0).multi_processor_count != 256:
        pytest.skip("the expected shapes are those of a 256-CU device")
    c5 = inputs.workload("c5", N=4, num_layers=1).layers
    for li in (0, 4, 5):
        with sd.Plan.from_csr(c5[li].W) as plan:
            assert plan.launch_shape(16384) == {"panel_rows": 32, "waves": 12, "tile_cols": 128}
            if c5[li].W.M == 768:
                assert plan.launch_shape(8192)["panel_rows"] != 32
    w0 = inputs.workload("w0", N=4).layers[0].W
    with sd.Plan.from_csr(w0) as plan:  # 90 %: too dense for them
        assert plan.launch_shape(16384)["panel_rows"] != 32


@pytest.mark.parametrize("kw", [{"tile_cols": 128}, {"tile_cols": 128, "panel_rows": 32}])
def test_k_split_out_permuted(kw):
    """K-split calls of out_permuted plans on 128-column tiles (4-row panels and 32-row ones):
    the partials of each run are stored in the plan's row order and the reduction finds each
    stored row's bias through the plan's permutation; C row i is output row perm[i]."""
    M, K, N = 500, 900, 388
    W = inputs.pattern_uniform(M, K, 0.06, inputs.CFG_TEST, 5700, 0.05)
    B = inputs.dense_B(K, N, inputs.CFG_TEST, 5701)
    bias = inputs.bias_normal(M, inputs.CFG_TEST, 5702, 0.02)
    with sd.Plan.from_csr(W, out_permuted=True, split_chunks=2, **kw) as plan:
        C = torch.full((M, N), float("nan"), device=DEV)
        plan.spmm_split(torch.from_numpy(B).to(DEV), C, torch.from_numpy(bias).to(DEV), "gelu",
                        splits=4)
        torch.cuda.synchronize()
        perm = plan.perm
        assert plan.split_runs(N, 4) == 4
    ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, K, B, bias, "gelu")
    err = np.abs(C.cpu().numpy().astype(np.float64) - ref[perm])
    assert (err <= tol_fp32(bound[perm], "gelu")).all()


def test_tuned_deep_shape_with_a_call_that_cannot_use_it():
    """After sdnn_plan_tune records a 32-row shape at some N, a call at that N that cannot run
    on 128-column tiles (a B that is not 16-byte aligned) falls back to the rule's 256-column
    launch and still agrees with the oracle."""
    if torch.cuda.get_device_properties(0).multi_processor_count != 256:
        pytest.skip("the deep launch is chosen for a 256-CU device")
    L = inputs.workload("c5", N=4, num_layers=1).layers[5]
    W, N = L.W, 16384
    B = inputs.dense_B(W.K, N, inputs.CFG_TEST, 5800)
    with sd.Plan.from_csr(W) as plan:
        Bt = torch.from_numpy(B).to(DEV)
        plan.tune(N, Bt, torch.empty(W.M, N, device=DEV))
        flat = torch.empty(W.K * N + 1, device=DEV)
        Bm = flat[1:].view(W.K, N)
        Bm.copy_(Bt)
        assert Bm.data_ptr() % 16 != 0
        got = run(plan, B, None, "none", Bt=Bm)
    cols = np.arange(0, N, 97)
    ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, W.K, B[:, cols], None, "none")
    err = np.abs(got[:, cols].astype(np.float64) - ref)
    assert (err <= tol_fp32(bound, "none")).all()
