"""GPU parity: the HIP path (through the C ABI) against the CPU oracle, element by
element, on seeded synthetic inputs.  Bar (fp32 vs the double reference):

    |C_gpu - C_ref| <= 1e-5 * sum_p |w_p| |B[c_p, n]| + 1e-6          (none, ReLU)
    GELU: the same bound scaled by 1.13 (GELU's Lipschitz constant)

and the row permutation must equal the oracle's Algorithm 1 bit-exactly."""
import os

import numpy as np
import pytest

import oracle
import paper_2101_07948_amd as sd
from conftest import GELU_LIPSCHITZ, dense_to_csr, pattern_to_csr, random_csr, tol_fp32
from paper_2101_07948_amd import inputs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def tolerance(bound, ref, epi):
    return tol_fp32(bound, epi)


class Forced:
    """Forces the launch shape (waves per workgroup) for a call."""

    def __init__(self, waves=None):
        self.waves = waves

    def __enter__(self):
        self.old = {k: os.environ.get(k) for k in ("SDNN_FORCE_WAVES",)}
        if self.waves:
            os.environ["SDNN_FORCE_WAVES"] = str(self.waves)

    def __exit__(self, *a):
        for k, v in self.old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def gpu_spmm(plan, B, bias, epi, stream=None):
    Bt = torch.from_numpy(np.ascontiguousarray(B)).to(DEV)
    bt = None if bias is None else torch.from_numpy(np.ascontiguousarray(bias)).to(DEV)
    C = torch.full((plan.M, B.shape[1]), float("nan"), device=DEV)
    plan.spmm(Bt, C, bt, epi, stream=stream)
    torch.cuda.synchronize()
    return C.cpu().numpy()


def check(row_ptr, col_idx, values, M, K, B, bias, epi, panel_rows=0, permute=True,
          waves=None, label=""):
    with sd.Plan(row_ptr, col_idx, values, M, K, panel_rows=panel_rows, permute=permute) as plan:
        with Forced(waves):
            got = gpu_spmm(plan, B, bias, epi)
        if permute:
            assert np.array_equal(plan.perm, oracle.reorder(row_ptr, col_idx, K)), label
    ref, bound = oracle.spmm_f64(row_ptr, col_idx, values, K, B, bias, epi)
    err = np.abs(got.astype(np.float64) - ref)
    tol = tolerance(bound, ref, epi)
    bad = ~(err <= tol)  # NaN (an element never written) counts as bad
    assert not bad.any(), (f"{label}: {int(bad.sum())} of {bad.size} elements out of tolerance; "
                           f"worst err/tol {np.nanmax(err / tol):.3g}")
    return got


@pytest.mark.parametrize("name", ["c1", "c2", "c4", "w0"])
def test_workload_parity(name):
    w = inputs.workload(name)
    L = w.layers[0]
    check(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.M, L.W.K, w.B, L.bias, L.epi, label=name)


def test_w0_full_size_all_epilogues():
    """The measured workload (768 x 3072 at 90 %, N = 4096) in the launch configuration
    the benchmark times, with each epilogue."""
    w = inputs.workload("w0")
    L = w.layers[0]
    for epi in ("relu", "gelu"):
        check(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.M, L.W.K, w.B, L.bias, epi, label=epi)


def test_c3_ffn_pair_per_layer():
    """BERT FFN pair at 94 % with lognormal row lengths; layer 2 is fed the GPU's own
    layer-1 output so each layer is checked on the same input as the oracle."""
    w = inputs.workload("c3", N=4096)
    X = w.B
    for i, L in enumerate(w.layers):
        X = check(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.M, L.W.K, X, L.bias, L.epi,
                  label=f"c3 layer {i}")


def test_c5_first_encoder_layer_chain():
    """First encoder layer of the 97 % block-correlated stack at N = 16384, chained on
    the GPU's own outputs, each layer checked against the oracle."""
    w = inputs.workload("c5", N=16384, num_layers=1)
    X = w.B
    for i, L in enumerate(w.layers):
        X = check(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.M, L.W.K, X, L.bias, L.epi,
                  label=f"c5 layer {i}")


@pytest.mark.parametrize("MK,sparsity,N", [(1024, 0.70, 128), (2048, 0.90, 512),
                                            (512, 0.80, 2048), (256, 0.95, 130)])
def test_paper_shaped_problems(MK, sparsity, N):
    """The paper's kernel problems (Sec. 4.1): square W, the unit-Gaussian survivors of a
    magnitude threshold at 70-95 % sparsity, batch widths 128-2048 (130: a ragged one)."""
    L = inputs.s_layer(MK, MK, sparsity)
    B = inputs.dense_B(MK, N, inputs.CFG_S, MK + N)
    check(L.W.row_ptr, L.W.col_idx, L.W.values, MK, MK, B, None, "none",
          label=f"S {MK} {sparsity} N={N}")


@pytest.mark.parametrize("N", [1, 2, 3, 63, 64, 65, 255, 256, 257, 1000, 3136])
def test_ragged_N(N):
    W = inputs.pattern_uniform(200, 300, 0.1, inputs.CFG_TEST, N, 0.05)
    B = inputs.dense_B(300, N, inputs.CFG_TEST, N)
    bias = inputs.bias_normal(200, inputs.CFG_TEST, N, 0.02)
    check(W.row_ptr, W.col_idx, W.values, 200, 300, B, bias, "gelu", label=f"N={N}")


@pytest.mark.parametrize("panel_rows", [4, 8, 12, 16])
@pytest.mark.parametrize("N", [640, 643])
def test_kernel_variants(panel_rows, N):
    """Every compiled variant: rows per panel, aligned and unaligned N (16-byte vs
    4-byte staging), several K-chunks with a ragged last chunk."""
    M, K = 333, 451
    W = inputs.pattern_uniform(M, K, 0.12, inputs.CFG_TEST, 100 + panel_rows, 0.05)
    B = inputs.dense_B(K, N, inputs.CFG_TEST, 100 + N)
    bias = inputs.bias_normal(M, inputs.CFG_TEST, 100, 0.02)
    check(W.row_ptr, W.col_idx, W.values, M, K, B, bias, "relu", panel_rows=panel_rows,
          label=f"RW={panel_rows} N={N}")


@pytest.mark.parametrize("waves", [1, 3, 16])
def test_waves_per_workgroup(waves):
    M, K, N = 700, 300, 512
    W = inputs.pattern_uniform(M, K, 0.1, inputs.CFG_TEST, 200 + waves, 0.05)
    B = inputs.dense_B(K, N, inputs.CFG_TEST, 200)
    check(W.row_ptr, W.col_idx, W.values, M, K, B, None, "none", waves=waves,
          label=f"waves={waves}")


def test_edge_cases():
    rng = np.random.default_rng(3)
    # density 0: C = act(bias)
    M, K, N = 37, 80, 70
    B = rng.standard_normal((K, N)).astype(np.float32)
    bias = rng.standard_normal(M).astype(np.float32)
    rp = np.zeros(M + 1, np.int32)
    for epi in ("none", "relu", "gelu"):
        got = check(rp, np.zeros(0, np.int32), np.zeros(0, np.float32), M, K, B, bias, epi,
                    label=f"density0 {epi}")
        if epi != "gelu":
            want = np.maximum(bias, 0) if epi == "relu" else bias
            assert np.array_equal(got, np.repeat(want[:, None], N, axis=1))
    # density 1 and the dense comparison kernel
    Wd = rng.standard_normal((M, K)).astype(np.float32)
    rp, ci, v = dense_to_csr(Wd)
    check(rp, ci, v, M, K, B, bias, "none", label="density1")
    # empty rows, M = 1, K = 1, K = 0, K < chunk, K = chunk + 1
    for (M, K) in ((1, 50), (50, 1), (5, 64), (9, 65), (3, 0), (130, 7)):
        rp, ci, v, _ = random_csr(rng, M, K, 0.5)
        if M > 2:
            # blank out a row
            cnt = np.diff(rp)
            cnt[1] = 0
            keep = np.repeat(np.arange(M), np.diff(rp)) != 1
            ci, v = ci[keep], v[keep]
            rp = np.concatenate([[0], np.cumsum(cnt)]).astype(np.int32)
        B = rng.standard_normal((K, 33)).astype(np.float32)
        check(rp, ci, v, M, K, B, rng.standard_normal(M).astype(np.float32), "relu",
              label=f"M={M} K={K}")


def test_large_shapes():
    """Long K (3125 chunks: the stream spans the whole ring many times over), many rows
    with few columns, and one row with every column set."""
    rng = np.random.default_rng(71)
    for (M, K, N, d) in ((24, 100000, 96, 0.02), (20000, 96, 260, 0.1), (1, 4096, 512, 1.0)):
        rp, ci, v, _ = random_csr(rng, M, K, d)
        B = rng.standard_normal((K, N)).astype(np.float32)
        check(rp, ci, v, M, K, B, rng.standard_normal(M).astype(np.float32), "none",
              label=f"M={M} K={K} N={N}")


def test_c5_full_stack_sampled_columns():
    """The whole C5 workload: 12 encoder layers x 6 products, 97 % block-correlated, at
    N = 16384 on the GPU, chained on its own outputs.  Columns are independent, so the
    oracle follows the same chain on 256 sampled columns: each layer's GPU output on
    those columns is checked against the oracle applied to the GPU's previous output."""
    w = inputs.workload("c5", N=16384)
    cols = np.sort(np.random.default_rng(72).choice(w.N, 256, replace=False))
    X = torch.from_numpy(w.B).to(DEV)
    for i, L in enumerate(w.layers):
        with sd.Plan.from_csr(L.W) as plan:
            Y = torch.empty((L.W.M, w.N), device=DEV)
            bt = None if L.bias is None else torch.from_numpy(L.bias).to(DEV)
            plan.spmm(X, Y, bt, L.epi)
            torch.cuda.synchronize()
        xs = X[:, cols].cpu().numpy()
        ref, bound = oracle.spmm_f64(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.K, xs, L.bias, L.epi)
        got = Y[:, cols].cpu().numpy().astype(np.float64)
        tol = tolerance(bound, ref, L.epi)
        assert np.all(np.abs(got - ref) <= tol), f"C5 product {i}: worst {np.max(np.abs(got - ref) / tol):.3g}"
        X = Y


def test_row_permutation_equivariance_bitexact():
    """Each row sums its entries in ascending column order whatever panel it lands in,
    so permuting W's rows permutes C's rows exactly."""
    W = inputs.pattern_uniform(300, 500, 0.1, inputs.CFG_TEST, 7, 0.05)
    B = inputs.dense_B(500, 384, inputs.CFG_TEST, 7)
    bias = inputs.bias_normal(300, inputs.CFG_TEST, 7, 0.02)
    pi = np.random.default_rng(8).permutation(300)
    Wd = W.to_dense()
    rp, ci, v = dense_to_csr(Wd[pi])
    with sd.Plan.from_csr(W) as p1, sd.Plan(rp, ci, v, 300, 500) as p2:
        C1 = gpu_spmm(p1, B, bias, "gelu")
        C2 = gpu_spmm(p2, B, bias[pi], "gelu")
    assert np.array_equal(C2, C1[pi])


def test_tall_panels_at_large_N():
    """768 rows over 32 column tiles: 4-row panels need two rounds of workgroups on 256
    CUs, 8- and 12-row ones one, and 8-row panels already hold 25.6 entries per chunk at
    10 %, so the default plan runs its 8-row packing (as sdnn_plan_launch_shape reports):
    checked against the oracle, and bit-identical to a 4-row-only plan (every row sums its
    entries in ascending column order either way)."""
    M, K, N = 768, 1024, 8192
    W = inputs.pattern_uniform(M, K, 0.1, inputs.CFG_TEST, 21, 0.05)
    B = inputs.dense_B(K, N, inputs.CFG_TEST, 21)
    bias = inputs.bias_normal(M, inputs.CFG_TEST, 21, 0.02)
    with sd.Plan.from_csr(W) as plan:
        if torch.cuda.get_device_properties(0).multi_processor_count == 256:
            assert plan.launch_shape(N)["panel_rows"] == 8
    got = check(W.row_ptr, W.col_idx, W.values, M, K, B, bias, "relu", label="tall")
    with sd.Plan.from_csr(W, panel_rows=4) as p4:
        assert p4.info["tall_panel_rows"] == 0
        short = gpu_spmm(p4, B, bias, "relu")
    assert np.array_equal(got, short)


def test_out_permuted_writes_rows_in_plan_order():
    """out_permuted only moves the store: C row i is output row perm[i], bit for bit."""
    W = inputs.pattern_uniform(300, 500, 0.1, inputs.CFG_TEST, 41, 0.05)
    B = inputs.dense_B(500, 643, inputs.CFG_TEST, 41)
    bias = inputs.bias_normal(300, inputs.CFG_TEST, 41, 0.02)
    with sd.Plan.from_csr(W) as p0, sd.Plan.from_csr(W, out_permuted=True) as p1:
        assert p1.info["out_permuted"] == 1
        assert np.array_equal(p1.perm, p0.perm)
        C0 = gpu_spmm(p0, B, bias, "gelu")
        C1 = gpu_spmm(p1, B, bias, "gelu")
        assert np.array_equal(C1, C0[p1.perm])


@pytest.mark.parametrize("N", [1024, 16384])
def test_chain_in_permuted_space(N):
    """Cross-layer compensation (Sec. 3.1.2): C5's first encoder layer chained with every
    intermediate activation left in its producer's row order; each plan takes the
    previous plan's perm as in_perm, the last one writes the original order.  Each layer
    is checked against the oracle on the un-permuted input, rows permuted as stored."""
    w = inputs.workload("c5", N=N, num_layers=1)
    X = torch.from_numpy(w.B).to(DEV)
    prev = None
    for i, L in enumerate(w.layers):
        last = i == len(w.layers) - 1
        with sd.Plan.from_csr(L.W, out_permuted=not last, in_perm=prev) as plan:
            Y = torch.full((L.W.M, N), float("nan"), device=DEV)
            bt = None if L.bias is None else torch.from_numpy(L.bias).to(DEV)
            plan.spmm(X, Y, bt, L.epi)
            torch.cuda.synchronize()
            x = X.cpu().numpy()
            x_orig = x if prev is None else np.empty_like(x)
            if prev is not None:
                x_orig[prev] = x          # B row j holds input feature prev[j]
            ref, bound = oracle.spmm_f64(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.K, x_orig,
                                         L.bias, L.epi)
            order = np.arange(L.W.M) if last else plan.perm
            got = Y.cpu().numpy().astype(np.float64)
            err = np.abs(got - ref[order])
            tol = tolerance(bound[order], ref[order], L.epi)
            assert not (~(err <= tol)).any(), f"layer {i}: worst err/tol {np.nanmax(err / tol):.3g}"
            prev = None if last else plan.perm
        X = Y


def test_balanced_order():
    """permute = 2 gives each row, longest first, to the 4-row panel with the fewest
    nonzeros so far: a permutation whose panels carry nearly equal work on the
    lognormal C3 layers, with results equal to the oracle's (and bit-identical to the
    identity order, since each row still sums its entries in ascending column order)."""
    w = inputs.workload("c3", N=4)
    for i, L in enumerate(w.layers):
        W = L.W
        B = inputs.dense_B(W.K, 1024, inputs.CFG_TEST, 51 + i)
        with sd.Plan.from_csr(W, permute="balanced") as pb, \
                sd.Plan.from_csr(W, permute=False) as p0:
            perm = pb.perm
            assert np.array_equal(np.sort(perm), np.arange(W.M))
            nnz = np.diff(W.row_ptr)[perm]
            panels = nnz[: W.M // 4 * 4].reshape(-1, 4).sum(axis=1)
            # a panel can do no better than its heaviest row plus the lightest rows
            bound = max(1.02 * panels.mean(), nnz.max() + np.sort(nnz)[:3].sum())
            assert panels.max() <= bound + 4
            got = gpu_spmm(pb, B, L.bias, L.epi)
            ident = gpu_spmm(p0, B, L.bias, L.epi)
        assert np.array_equal(got, ident)
        ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, W.K, B, L.bias, L.epi)
        assert np.all(np.abs(got - ref) <= tolerance(bound, ref, L.epi))


def test_plan_tune():
    """sdnn_plan_tune times the plan's launch shapes at one N and records the fastest;
    later calls at that N use it and give bit-identical results (each row still sums in
    ascending column order), other N keep the heuristic."""
    w = inputs.workload("c2")
    L = w.layers[0]
    with sd.Plan.from_csr(L.W) as plan:
        before = gpu_spmm(plan, w.B, L.bias, L.epi)
        shape = plan.tune(w.N)
        assert shape["panel_rows"] in (4, 8, 12) and 1 <= shape["waves"] <= 12
        assert plan.launch_shape(w.N) == shape
        after = gpu_spmm(plan, w.B, L.bias, L.epi)
        assert np.array_equal(before, after)
        B2 = inputs.dense_B(L.W.K, 300, inputs.CFG_TEST, 61)
        other = gpu_spmm(plan, B2, L.bias, L.epi)
    ref, bound = oracle.spmm_f64(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.K, w.B, L.bias, L.epi)
    assert np.all(np.abs(after - ref) <= tolerance(bound, ref, L.epi))
    ref2, bound2 = oracle.spmm_f64(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.K, B2, L.bias, L.epi)
    assert np.all(np.abs(other - ref2) <= tolerance(bound2, ref2, L.epi))


def test_permute_off_and_on_agree():
    """Every row order gives the same C bit for bit (each row sums its entries in
    ascending column order wherever its panel is), and the order the plan reports is
    the host entry point's."""
    W = inputs.pattern_grouped8(256, 512, 0.05, inputs.CFG_TEST, 9, 0.05)
    B = inputs.dense_B(512, 256, inputs.CFG_TEST, 9)
    with sd.Plan.from_csr(W, permute=False) as p0:
        assert np.array_equal(p0.perm, np.arange(256))
        C0 = gpu_spmm(p0, B, None, "none")
    for mode in ("algorithm1", "balanced", "panel_union", "minhash", "bin_greedy"):
        with sd.Plan.from_csr(W, permute=mode) as p:
            assert np.array_equal(p.perm, sd.row_order(W.row_ptr, W.col_idx, W.K, mode))
            assert np.array_equal(gpu_spmm(p, B, None, "none"), C0), mode
    ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, W.K, B)
    assert (np.abs(C0 - ref) <= 1e-5 * bound + 1e-6).all()


@pytest.mark.parametrize("budget", [0, 2, 64])
def test_spent_poll_budget_turns_results_to_nan(budget):
    """Every wait in the kernel is bounded by a poll budget, here forced tiny from the
    host: a consumer that stops waiting, or whose staged chunks a producer may have
    overwritten, writes NaN for its panel.  Every output is within the oracle's bound or
    NaN, never a finite wrong value; with no budget at all every panel is NaN."""
    M, K, N = 512, 2048, 4096
    W = inputs.pattern_uniform(M, K, 0.1, inputs.CFG_TEST, 90, 0.05)
    B = inputs.dense_B(K, N, inputs.CFG_TEST, 90)
    bias = inputs.bias_normal(M, inputs.CFG_TEST, 90, 0.02)
    old = os.environ.get("SDNN_POLL_BUDGET")
    os.environ["SDNN_POLL_BUDGET"] = str(budget)
    try:
        with sd.Plan.from_csr(W) as plan:
            got = gpu_spmm(plan, B, bias, "none")
    finally:
        if old is None:
            os.environ.pop("SDNN_POLL_BUDGET", None)
        else:
            os.environ["SDNN_POLL_BUDGET"] = old
    ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, K, B, bias, "none")
    err = np.abs(got.astype(np.float64) - ref)
    ok = (err <= tolerance(bound, ref, "none")) | np.isnan(got)
    assert ok.all(), f"{int((~ok).sum())} finite outputs out of tolerance"
    if budget == 0:
        assert np.isnan(got).all()


def test_graph_capture_replays():
    """sdnn_spmm neither allocates nor synchronises, so a call can be captured in a HIP
    graph: replayed several times, with eager work and synchronisations between the
    replays, every replay gives the eager result bit for bit."""
    M, K, N = 700, 500, 1000
    W = inputs.pattern_uniform(M, K, 0.1, inputs.CFG_TEST, 77, 0.05)
    B = torch.from_numpy(inputs.dense_B(K, N, inputs.CFG_TEST, 77)).to(DEV)
    bias = torch.from_numpy(inputs.bias_normal(M, inputs.CFG_TEST, 77, 0.02)).to(DEV)
    with sd.Plan.from_csr(W) as plan:
        C_eager = torch.empty(M, N, device=DEV)
        plan.spmm(B, C_eager, bias, "gelu")
        torch.cuda.synchronize()
        C = torch.empty(M, N, device=DEV)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):  # a first call off the default stream before capture
            plan.spmm(B, C, bias, "gelu")
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            plan.spmm(B, C, bias, "gelu")
        for rep in range(4):
            C.fill_(float("nan"))
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(C, C_eager), f"replay {rep}"
    ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, K, B.cpu().numpy(),
                                 bias.cpu().numpy(), "gelu")
    err = np.abs(C_eager.cpu().numpy().astype(np.float64) - ref)
    assert (err <= tolerance(bound, ref, "gelu")).all()


def test_streams_and_concurrency():
    W = inputs.pattern_uniform(512, 512, 0.1, inputs.CFG_TEST, 11, 0.05)
    B1 = inputs.dense_B(512, 1024, inputs.CFG_TEST, 11)
    B2 = inputs.dense_B(512, 1024, inputs.CFG_TEST, 12)
    ref1, bnd1 = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, 512, B1)
    ref2, bnd2 = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, 512, B2)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    with sd.Plan.from_csr(W) as plan:
        tB1, tB2 = torch.from_numpy(B1).to(DEV), torch.from_numpy(B2).to(DEV)
        C1 = torch.full((512, 1024), float("nan"), device=DEV)
        C2 = torch.full((512, 1024), float("nan"), device=DEV)
        torch.cuda.synchronize()
        for _ in range(3):
            plan.spmm(tB1, C1, stream=s1)
            plan.spmm(tB2, C2, stream=s2)
        torch.cuda.synchronize()
    for got, ref, bnd in ((C1, ref1, bnd1), (C2, ref2, bnd2)):
        assert np.all(np.abs(got.cpu().numpy() - ref) <= tolerance(bnd, ref, "none"))


def test_overlapping_buffers_rejected():
    W = inputs.pattern_uniform(64, 64, 0.1, inputs.CFG_TEST, 13, 0.05)
    buf = torch.zeros(64 * 64 * 2, device=DEV)
    B = buf[: 64 * 64].view(64, 64)
    C = buf[64 * 32: 64 * 96].view(64, 64)
    with sd.Plan.from_csr(W) as plan:
        with pytest.raises(sd.SdnnError) as ei:
            plan.spmm(B, C)
        assert ei.value.code == 2


@pytest.mark.parametrize("M,K,N", [(64, 64, 64), (130, 97, 75), (768, 768, 512), (100, 1001, 257),
                                   (200, 33, 129)])
def test_dense_comparison_kernel(M, K, N):
    rng = np.random.default_rng(M + K + N)
    Wd = rng.standard_normal((M, K)).astype(np.float32) * 0.05
    B = rng.standard_normal((K, N)).astype(np.float32)
    bias = rng.standard_normal(M).astype(np.float32) * 0.02
    C = torch.full((M, N), float("nan"), device=DEV)
    sd.dense_gemm(torch.from_numpy(Wd).to(DEV), torch.from_numpy(B).to(DEV), C,
                  torch.from_numpy(bias).to(DEV), "gelu")
    torch.cuda.synchronize()
    rp, ci, v = dense_to_csr(Wd)
    ref, bound = oracle.spmm_f64(rp, ci, v, K, B, bias, "gelu")
    assert np.all(np.abs(C.cpu().numpy() - ref) <= tolerance(bound, ref, "gelu"))


def test_launch_shape_follows_density_and_grid():
    """The default plan's packing and tile width per call (sdnn_plan_launch_shape) on 256
    CUs: 4-row panels when they fill the device at 10 % (W0 at N = 4096), 8-row ones when
    4-row panels need more rounds (W0 at N = 16384), 12-row ones at 97 % where shorter panels
    hold too few entries per chunk (C5's 768-row layer at N = 8192), 16-row ones where they
    need the fewest rounds of workgroups (M = K = 2048 at 95 %), all on 256-column tiles;
    128-column tiles where the 256-column launch gives its workgroups at most 4 consumer
    waves (W0 and C2 at N = 1024, C5's 768 x 3072 layer at N = 1024, with 8-row panels
    there), and 32-row panels on them at 97 % where their grid fills the CUs (C5's layers
    at N = 16384)."""
    if torch.cuda.get_device_properties(0).multi_processor_count != 256:
        pytest.skip("the expected shapes are those of a 256-CU device")
    w0 = inputs.workload("w0", N=4).layers[0].W
    c2 = inputs.workload("c2", N=4).layers[0].W
    c5 = inputs.workload("c5", N=4, num_layers=1).layers
    for W, N, want, tile in ((w0, 4096, 4, 256), (w0, 16384, 8, 256), (c5[0].W, 8192, 12, 256),
                             (c5[0].W, 16384, 32, 128), (c5[4].W, 16384, 32, 128),
                             (inputs.s_layer(2048, 2048, 0.95).W, 4096, 16, 256),
                             (w0, 1024, 4, 128), (c2, 1024, 4, 128), (c5[5].W, 1024, 8, 128)):
        with sd.Plan.from_csr(W) as plan:
            got = plan.launch_shape(N)
        assert (got["panel_rows"], got["tile_cols"]) == (want, tile), (W.M, W.K, N, got)
        assert 1 <= got["waves"] <= 12
    with sd.Plan.from_csr(w0, panel_rows=16) as plan:
        assert plan.launch_shape(4096)["panel_rows"] == 16


def test_row_bytes_limit_rejected():
    """N >= 2^29 would overflow the kernels' 32-bit row offsets: sdnn_spmm and
    sdnn_plan_tune return SDNN_ERR_DIM before touching any buffer."""
    W = inputs.pattern_uniform(16, 16, 0.2, inputs.CFG_TEST, 31, 0.05)
    buf = torch.zeros(16, device=DEV)
    with sd.Plan.from_csr(W) as plan:
        L = plan._lib
        for N in (1 << 29, (1 << 31) - 1):
            assert L.sdnn_spmm(plan._h, buf.data_ptr(), buf.data_ptr() + 4096, N, None, 0, None) == 2
            assert L.sdnn_plan_tune(plan._h, buf.data_ptr(), buf.data_ptr() + 4096, N, None,
                                    None, None) == 2
    torch.cuda.synchronize()


def _chain_end_to_end(w, cols, label):
    """Runs the workload's chain of products on the GPU at its full N, each layer fed the
    GPU's previous output, and follows the same chain on the sampled columns with the
    oracle fed its own (fp32-rounded) outputs.  Columns are independent, so the GPU's
    sampled columns must stay within the propagated bound
        E_L = tol_L + Lip_L * |W_L| (E_{L-1} + 2^-24 |ref_{L-1}|),   E_0 = 0
    where tol_L is the per-layer parity bar on the oracle's input (plus the part of
    sum |w||b| that the input difference can add), Lip_L = 1.13 after GELU and 1
    otherwise, and 2^-24 |ref| is the oracle's own rounding to fp32 between layers."""
    X = torch.from_numpy(w.B).to(DEV)
    x_ref = w.B[:, cols].astype(np.float32)
    E = np.zeros_like(x_ref, dtype=np.float64)
    ref_prev = x_ref.astype(np.float64)
    for i, L in enumerate(w.layers):
        with sd.Plan.from_csr(L.W) as plan:
            Y = torch.full((L.W.M, w.N), float("nan"), device=DEV)
            bt = None if L.bias is None else torch.from_numpy(L.bias).to(DEV)
            plan.spmm(X, Y, bt, L.epi)
            torch.cuda.synchronize()
        lip = GELU_LIPSCHITZ if L.epi == "gelu" else 1.0
        absW = np.abs(L.W.values).astype(np.float32)
        slack = E + 2.0 ** -24 * np.abs(ref_prev)     # |x_gpu - x_ref| on this layer's input
        prop, _ = oracle.spmm_f64(L.W.row_ptr, L.W.col_idx, absW, L.W.K,
                                  (slack * (1 + 1e-6)).astype(np.float32), None, "none",
                                  with_bound=False)
        ref, bound = oracle.spmm_f64(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.K, x_ref,
                                     L.bias, L.epi)
        E = tol_fp32(bound + prop, L.epi) + lip * prop
        got = Y[:, cols].cpu().numpy().astype(np.float64)
        err = np.abs(got - ref)
        assert not (~(err <= E)).any(), \
            f"{label} product {i}: worst err/bound {np.nanmax(err / E):.3g}"
        X, ref_prev, x_ref = Y, ref, ref.astype(np.float32)
    return np.nanmax(err / E)


def test_c3_pair_end_to_end_propagated_bound():
    """The C3 FFN pair (3072 x 768 with bias + GELU, then 768 x 3072 with bias) at
    N = 4096, end to end against the oracle's own chain on 128 sampled columns."""
    w = inputs.workload("c3", N=4096)
    cols = np.sort(np.random.default_rng(73).choice(w.N, 128, replace=False))
    _chain_end_to_end(w, cols, "c3")


def test_c5_encoder_layer_end_to_end_propagated_bound():
    """The first C5 encoder layer (4 projections, then the FFN pair) at N = 16384 end to
    end against the oracle's own chain on 64 sampled columns.  The worst-case bound grows
    with each product by the row sums of |W| (about 4-8 on these layers), so after six
    products it is still below |C| but past about ten it no longer says anything; the
    deeper stack is checked product by product on the GPU's own inputs
    (test_c5_full_stack_sampled_columns)."""
    w = inputs.workload("c5", N=16384, num_layers=1)
    cols = np.sort(np.random.default_rng(74).choice(w.N, 64, replace=False))
    _chain_end_to_end(w, cols, "c5")


def test_dense_comparison_kernel_full_size_and_offsets():
    """The dense comparison GEMM on the W0 shape (768 x 3072 times 3072 x 4096, the tile
    shape the benchmark times) on 64 sampled columns, and on operands that start 4 bytes
    into their allocations (the element-wise edge path)."""
    rng = np.random.default_rng(4242)
    M, K, N = 768, 3072, 4096
    Wd = (rng.standard_normal((M, K)) * 0.02).astype(np.float32)
    B = rng.standard_normal((K, N)).astype(np.float32)
    bias = (rng.standard_normal(M) * 0.02).astype(np.float32)
    C = torch.full((M, N), float("nan"), device=DEV)
    sd.dense_gemm(torch.from_numpy(Wd).to(DEV), torch.from_numpy(B).to(DEV), C,
                  torch.from_numpy(bias).to(DEV), "relu")
    torch.cuda.synchronize()
    cols = np.sort(rng.choice(N, 64, replace=False))
    rp, ci, v = dense_to_csr(Wd)
    ref, bound = oracle.spmm_f64(rp, ci, v, K, B[:, cols], bias, "relu")
    assert np.all(np.abs(C[:, cols].cpu().numpy() - ref) <= tolerance(bound, ref, "relu"))
    # operands offset by one float: not 16-byte aligned
    M, K, N = 96, 300, 128
    Wd = (rng.standard_normal((M, K)) * 0.05).astype(np.float32)
    B = rng.standard_normal((K, N)).astype(np.float32)
    wbuf = torch.zeros(M * K + 1, device=DEV)
    bbuf = torch.zeros(K * N + 1, device=DEV)
    wbuf[1:] = torch.from_numpy(Wd.ravel()).to(DEV)
    bbuf[1:] = torch.from_numpy(B.ravel()).to(DEV)
    C = torch.full((M, N), float("nan"), device=DEV)
    sd.dense_gemm(wbuf[1:].view(M, K), bbuf[1:].view(K, N), C, None, "none")
    torch.cuda.synchronize()
    rp, ci, v = dense_to_csr(Wd)
    ref, bound = oracle.spmm_f64(rp, ci, v, K, B, None, "none")
    assert np.all(np.abs(C.cpu().numpy() - ref) <= tolerance(bound, ref, "none"))


@pytest.mark.parametrize("wg_per_tile", [1, 2, 3])
@pytest.mark.parametrize("N,epi", [(1024, "gelu"), (643, "relu")])
def test_persistent_workgroups(wg_per_tile, N, epi):
    """Workgroups that take several row-blocks of their column tile in turn (the ring's
    chunk numbers running on across row-blocks): forced to 1, 2 or 3 workgroups per tile
    on a problem with 8 row-blocks, with 16-byte (N = 1024) and 4-byte (N = 643)
    staging, against the oracle and bit for bit against one row-block per workgroup
    (each row sums its entries in the same order either way)."""
    M, K = 384, 512
    W = inputs.pattern_uniform(M, K, 0.1, inputs.CFG_TEST, 300 + N, 0.05)
    B = inputs.dense_B(K, N, inputs.CFG_TEST, 300 + N)
    bias = inputs.bias_normal(M, inputs.CFG_TEST, 300, 0.02)
    with sd.Plan.from_csr(W, panel_rows=4) as plan:
        with Forced(waves=12):
            one = gpu_spmm(plan, B, bias, epi)
            old = os.environ.get("SDNN_FORCE_WG_PER_TILE")
            os.environ["SDNN_FORCE_WG_PER_TILE"] = str(wg_per_tile)
            try:
                got = gpu_spmm(plan, B, bias, epi)
            finally:
                if old is None:
                    os.environ.pop("SDNN_FORCE_WG_PER_TILE", None)
                else:
                    os.environ["SDNN_FORCE_WG_PER_TILE"] = old
    assert np.array_equal(got, one)
    ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, K, B, bias, epi)
    assert np.all(np.abs(got.astype(np.float64) - ref) <= tolerance(bound, ref, epi))


@pytest.mark.parametrize("out_permuted", [False, True])
def test_panel_grouping_bitexact(out_permuted):
    """Balanced panels and the permutation's consecutive rows give the same C bit for bit
    (each row sums its entries in ascending column order in any panel), in the original
    row order and, for out_permuted plans, in the permutation's order; the reported
    permutation is Algorithm 1's either way."""
    L = inputs.workload("c3", N=4).layers[1]
    W = L.W
    B = inputs.dense_B(W.K, 1000, inputs.CFG_TEST, 77)
    with sd.Plan.from_csr(W, grouping="order", out_permuted=out_permuted) as p1, \
            sd.Plan.from_csr(W, grouping="balanced", out_permuted=out_permuted) as p2:
        assert p1.info["grouping"] == 1 and p2.info["grouping"] == 2
        want = oracle.reorder(W.row_ptr, W.col_idx, W.K)
        assert np.array_equal(p1.perm, want) and np.array_equal(p2.perm, want)
        C1 = gpu_spmm(p1, B, L.bias, "relu")
        C2 = gpu_spmm(p2, B, L.bias, "relu")
    assert np.array_equal(C1, C2)
    ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, W.K, B, L.bias, "relu")
    order = want if out_permuted else np.arange(W.M)
    assert np.all(np.abs(C2.astype(np.float64) - ref[order]) <= tolerance(bound[order], ref[order], "relu"))


@pytest.mark.parametrize("wgs", [5, 8, 13])
def test_persistent_workgroups_tile_major(wgs):
    """Persistent workgroups taking (tile, row-block) items in tile-major order (each
    workgroup's items on changing tiles, the producers moving to the next item's tile):
    forced to 5, 8 or 13 workgroups over 4 tiles x 8 row-blocks, against the oracle and
    bit for bit against one item per workgroup."""
    M, K, N = 384, 640, 1024
    W = inputs.pattern_uniform(M, K, 0.1, inputs.CFG_TEST, 400 + wgs, 0.05)
    B = inputs.dense_B(K, N, inputs.CFG_TEST, 400 + wgs)
    bias = inputs.bias_normal(M, inputs.CFG_TEST, 400, 0.02)
    with sd.Plan.from_csr(W, panel_rows=4) as plan:
        with Forced(waves=12):
            one = gpu_spmm(plan, B, bias, "gelu")
            old = os.environ.get("SDNN_FORCE_TILE_MAJOR_WGS")
            os.environ["SDNN_FORCE_TILE_MAJOR_WGS"] = str(wgs)
            try:
                got = gpu_spmm(plan, B, bias, "gelu")
            finally:
                if old is None:
                    os.environ.pop("SDNN_FORCE_TILE_MAJOR_WGS", None)
                else:
                    os.environ["SDNN_FORCE_TILE_MAJOR_WGS"] = old
    assert np.array_equal(got, one)
    ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, K, B, bias, "gelu")
    assert np.all(np.abs(got.astype(np.float64) - ref) <= tolerance(bound, ref, "gelu"))


@pytest.mark.parametrize("unaligned", [False, True])
def test_persistent_tile_major_ragged_k(unaligned):
    """Tile-major persistent items with K = 760 (a last staging chunk of 24 rows, staged by
    the clamped path) and, unaligned, a B that starts 4 bytes into its allocation (4-byte
    staging): each item's chunks come from its own tile."""
    M, K, N = 384, 760, 1024
    W = inputs.pattern_uniform(M, K, 0.1, inputs.CFG_TEST, 500, 0.05)
    Bn = inputs.dense_B(K, N, inputs.CFG_TEST, 500)
    bias = inputs.bias_normal(M, inputs.CFG_TEST, 500, 0.02)
    buf = torch.zeros(K * N + 1, device=DEV)
    off = 1 if unaligned else 0
    buf[off:off + K * N] = torch.from_numpy(Bn.ravel()).to(DEV)
    Bt = buf[off:off + K * N].view(K, N)
    outs = []
    with sd.Plan.from_csr(W, panel_rows=4) as plan:
        for wgs in (0, 7):
            old = os.environ.get("SDNN_FORCE_TILE_MAJOR_WGS")
            if wgs:
                os.environ["SDNN_FORCE_TILE_MAJOR_WGS"] = str(wgs)
            try:
                with Forced(waves=12):
                    C = torch.full((M, N), float("nan"), device=DEV)
                    plan.spmm(Bt, C, torch.from_numpy(bias).to(DEV), "relu")
                    torch.cuda.synchronize()
                    outs.append(C.cpu().numpy())
            finally:
                if old is None:
                    os.environ.pop("SDNN_FORCE_TILE_MAJOR_WGS", None)
                else:
                    os.environ["SDNN_FORCE_TILE_MAJOR_WGS"] = old
    assert np.array_equal(outs[0], outs[1])
    ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, K, Bn, bias, "relu")
    assert np.all(np.abs(outs[1].astype(np.float64) - ref) <= tolerance(bound, ref, "relu"))
