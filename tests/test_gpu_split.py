"""GPU parity of the K-split calls (sdnn_spmm_split, sdnn_conv3x3_split) against the CPU
oracle, with the bar of the unsplit calls:

    |C_gpu - C_ref| <= 1e-5 * sum_p |w_p| |B[c_p, n]| + 1e-6   (GELU: x 1.13)

Each workgroup sums one K-segment's entries and the reduction adds the segments in
order, so the rounding differs from the unsplit call but the bound is the same."""
import numpy as np
import pytest

import oracle
import paper_2101_07948_amd as sd
from conftest import pattern_to_csr, tol_fp32
from paper_2101_07948_amd import inputs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def tolerance(bound, ref, epi):
    return tol_fp32(bound, epi)


def assert_close(got, ref, bound, epi, label):
    err = np.abs(got.astype(np.float64) - ref)
    tol = tolerance(bound, ref, epi)
    bad = ~(err <= tol)  # NaN (never written) counts as bad
    assert not bad.any(), (f"{label}: {int(bad.sum())} of {bad.size} elements out of tolerance; "
                           f"worst err/tol {np.nanmax(err / tol):.3g}")


def split_spmm(plan, B, bias, epi, workspace=None, splits=0):
    Bt = torch.from_numpy(np.ascontiguousarray(B)).to(DEV)
    bt = None if bias is None else torch.from_numpy(np.ascontiguousarray(bias)).to(DEV)
    C = torch.full((plan.M, B.shape[1]), float("nan"), device=DEV)
    if workspace is None:  # a poisoned workspace: every partial must be written
        workspace = torch.full((max(plan.workspace_floats(B.shape[1]), 1),), float("nan"),
                               device=DEV)
    plan.spmm_split(Bt, C, bt, epi, workspace=workspace, splits=splits)
    torch.cuda.synchronize()
    return C.cpu().numpy()


def check_split(W, B, bias, epi, split_chunks, label="", splits=0, **kw):
    with sd.Plan.from_csr(W, split_chunks=split_chunks, **kw) as plan:
        got = split_spmm(plan, B, bias, epi, splits=splits)
        perm, splits = plan.perm, plan.info["splits"]
    nchunks = -(-W.K // 32)
    assert splits == max(1, -(-nchunks // split_chunks)), label
    ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, W.K, B, bias, epi)
    if kw.get("out_permuted"):
        ref, bound = ref[perm], bound[perm]
    assert_close(got, ref, bound, epi, label)
    return got


def rand_B(K, N, seed):
    return np.random.default_rng([2101, 7948, seed]).standard_normal((K, N), dtype=np.float32)


@pytest.mark.parametrize("split_chunks", [1, 2, 3, 7])
@pytest.mark.parametrize("N", [1, 63, 256, 257, 1000])
def test_split_parity_ragged(split_chunks, N):
    """K = 300 (ten chunks, the last one ragged) over several tiles and a ragged tail;
    N % 4 != 0 runs the 4-byte producer and scalar partial stores."""
    W = inputs.pattern_uniform(200, 300, 0.15, inputs.CFG_TEST, 500 + split_chunks, 0.05)
    bias = np.random.default_rng([5, N]).standard_normal(200).astype(np.float32) * 0.02
    check_split(W, rand_B(300, N, N), bias, "relu", split_chunks, f"sc={split_chunks} N={N}")


@pytest.mark.parametrize("splits", [0, 1, 2, 3, 4, 6, 10, 99])
@pytest.mark.parametrize("N", [129, 512])
def test_split_runs_of_segments(splits, N):
    """Ten one-chunk segments (K = 300, the last chunk ragged) in runs of
    ceil(10 / splits): every run count, the library's choice (0) and a count above the
    segments (clamped to 10).  One run is the unsplit call, bit for bit."""
    W = inputs.pattern_uniform(200, 300, 0.15, inputs.CFG_TEST, 600, 0.05)
    bias = np.random.default_rng([6, N]).standard_normal(200).astype(np.float32) * 0.02
    B = rand_B(300, N, 600 + N)
    got = check_split(W, B, bias, "gelu", 1, f"splits={splits} N={N}", splits=splits)
    if splits == 1:
        with sd.Plan.from_csr(W) as plain:
            Bt = torch.from_numpy(B).to(DEV)
            C = torch.empty(200, N, device=DEV)
            plain.spmm(Bt, C, torch.from_numpy(bias).to(DEV), "gelu")
            torch.cuda.synchronize()
            assert np.array_equal(C.cpu().numpy(), got)


@pytest.mark.parametrize("splits", [0, 3, 4, 8, 24])
def test_split_runs_w0(splits):
    """W0 at N = 1024 on 24 segments of four chunks, in runs."""
    w = inputs.workload("w0", N=1024)
    L = w.layers[0]
    check_split(L.W, w.B, L.bias, L.epi, 4, f"w0 splits={splits}", splits=splits)


@pytest.mark.parametrize("epi", ["none", "relu", "gelu"])
@pytest.mark.parametrize("panel_rows", [0, 4, 8, 12, 16])
def test_split_epilogues_and_panel_heights(epi, panel_rows):
    w = inputs.workload("c2", N=512)
    L = w.layers[0]
    check_split(L.W, w.B, L.bias, epi, 6, f"c2 {epi} rw={panel_rows}", panel_rows=panel_rows)


def test_split_out_permuted_and_no_bias():
    w = inputs.workload("c2", N=768)
    L = w.layers[0]
    got = check_split(L.W, w.B, L.bias, "gelu", 4, "c2 permuted", out_permuted=True)
    plain = check_split(L.W, w.B, L.bias, "gelu", 4, "c2")
    with sd.Plan.from_csr(L.W) as plan:
        np.testing.assert_allclose(got, plain[plan.perm], rtol=0, atol=1e-5)
    check_split(L.W, w.B, None, "none", 4, "c2 no bias")


@pytest.mark.parametrize("name,N,split_chunks", [("w0", 1024, 24), ("w0", 4096, 48),
                                                 ("c2", 1024, 6), ("c1", 64, 2)])
def test_split_workloads(name, N, split_chunks):
    w = inputs.workload(name, N=N)
    L = w.layers[0]
    check_split(L.W, w.B, L.bias, L.epi, split_chunks, f"{name} N={N} sc={split_chunks}")


def test_split_paper_shaped_problems():
    for MK, s, N in [(2048, 0.95, 256), (1024, 0.7, 512), (256, 0.9, 1024)]:
        L = inputs.s_layer(MK, MK, s)
        check_split(L.W, rand_B(MK, N, MK + N), None, "none", 8, f"S {MK} {s} N={N}")


def test_split_matches_unsplit_and_one_segment_plan():
    """A plan whose segment covers K runs the unsplit kernel (workspace untouched); a
    split plan's plain sdnn_spmm result equals a plain plan's bit for bit (the stream's
    extra cuts only add synchronisation points)."""
    w = inputs.workload("c2", N=640)
    L = w.layers[0]
    Bt = torch.from_numpy(w.B).to(DEV)
    bt = torch.from_numpy(L.bias).to(DEV)
    with sd.Plan.from_csr(L.W) as plain, sd.Plan.from_csr(L.W, split_chunks=5) as split, \
            sd.Plan.from_csr(L.W, split_chunks=1000) as one:
        assert one.info["splits"] == 1 and one.workspace_floats(640) == 768 * 640
        C0 = torch.empty(768, 640, device=DEV)
        C1 = torch.empty(768, 640, device=DEV)
        C2 = torch.empty(768, 640, device=DEV)
        plain.spmm(Bt, C0, bt, "relu")
        split.spmm(Bt, C1, bt, "relu")
        ws = torch.full((16,), 7.0, device=DEV)
        assert one._lib.sdnn_spmm_split(one.handle, Bt.data_ptr(), C2.data_ptr(), 640,
                                        bt.data_ptr(), 1, 0, ws.data_ptr(), 16, None) == 0
        torch.cuda.synchronize()
        assert torch.equal(C0, C1) and torch.equal(C0, C2)
        assert torch.all(ws == 7.0)


def test_split_rejects_bad_workspace():
    w = inputs.workload("c1", N=64)
    L = w.layers[0]
    Bt = torch.from_numpy(w.B).to(DEV)
    C = torch.empty(256, 64, device=DEV)
    with sd.Plan.from_csr(L.W, split_chunks=2) as plan, sd.Plan.from_csr(L.W) as plain:
        lib, need = plan._lib, plan.workspace_floats(64)
        assert plan.info["splits"] == 4 and need == 4 * 256 * 64
        ws = torch.empty(need + 4, device=DEV)
        h, pb, pc = plan.handle, Bt.data_ptr(), C.data_ptr()
        assert lib.sdnn_spmm_split(h, pb, pc, 64, None, 0, 0, ws.data_ptr(), need - 1, None) == 2
        assert lib.sdnn_spmm_split(h, pb, pc, 64, None, 0, 0, ws.data_ptr() + 4, need, None) == 2
        assert lib.sdnn_spmm_split(h, pb, pc, 64, None, 0, 0, None, need, None) == 1
        assert lib.sdnn_spmm_split(h, pb, pc, 64, None, 0, 0, pc, need, None) == 2       # C
        assert lib.sdnn_spmm_split(plain.handle, pb, pc, 64, None, 0, 0, ws.data_ptr(), need,
                                   None) == 2                                          # unsplit plan
        assert lib.sdnn_spmm_split(h, pb, pc, 0, None, 0, 0, None, 0, None) == 0            # N = 0
        assert lib.sdnn_spmm_split(h, pb, pc, 64, None, 0, -1, ws.data_ptr(), need, None) == 2
        assert lib.sdnn_spmm_split(h, pb, pc, 64, None, 0, 0, ws.data_ptr(), need, None) == 0
        torch.cuda.synchronize()


def test_split_graph_capture_replays():
    """Split call and reduction captured in one HIP graph: every replay equals the eager
    result."""
    w = inputs.workload("c2", N=512)
    L = w.layers[0]
    Bt = torch.from_numpy(w.B).to(DEV)
    bt = torch.from_numpy(L.bias).to(DEV)
    with sd.Plan.from_csr(L.W, split_chunks=6) as plan:
        ws = torch.empty(plan.workspace_floats(512), device=DEV)
        eager = torch.empty(768, 512, device=DEV)
        plan.spmm_split(Bt, eager, bt, "gelu", workspace=ws)
        torch.cuda.synchronize()
        C = torch.zeros(768, 512, device=DEV)
        s = torch.cuda.Stream()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(s):
            with torch.cuda.graph(g, stream=s):
                plan.spmm_split(Bt, C, bt, "gelu", workspace=ws, stream=s)
        for _ in range(3):
            C.fill_(float("nan"))
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(C, eager)


def split_conv(plan, X, bias, epi, splits=0):
    Xt = torch.from_numpy(np.ascontiguousarray(X)).to(DEV)
    IC, H, W, NB = X.shape
    C = torch.full((plan.M, H, W, NB), float("nan"), device=DEV)
    ws = torch.full((max(plan.workspace_floats(H * W * NB), 1),), float("nan"), device=DEV)
    bt = None if bias is None else torch.from_numpy(bias).to(DEV)
    plan.conv3x3_split(Xt, C, bt, epi, workspace=ws, splits=splits)
    torch.cuda.synchronize()
    return C.cpu().numpy()


@pytest.mark.parametrize("OC,IC,H,W,NB,sparsity,epi,sc,splits", [
    (5, 3, 5, 7, 4, 0.5, "none", 1, 0),        # K = 27: one segment
    (40, 16, 7, 7, 12, 0.9, "gelu", 1, 0),     # K = 144 over five segments, ragged tile
    (40, 16, 7, 7, 12, 0.9, "gelu", 1, 2),     # runs of three and two segments
    (64, 64, 28, 28, 4, 0.95, "relu", 4, 0),   # 18 chunks in segments of 4 (last ragged)
    (128, 128, 14, 14, 16, 0.9, "none", 9, 0),
    (256, 256, 7, 7, 16, 0.9, "relu", 12, 0),
    (256, 256, 7, 7, 16, 0.9, "relu", 4, 5),   # 18 segments in runs of four
])
def test_conv_split_parity(OC, IC, H, W, NB, sparsity, epi, sc, splits):
    L = inputs.conv_layer(OC, IC, H, W, NB, sparsity, layer=OC + IC + H + 1, epi=epi)
    with sd.Plan.from_csr(L.F, split_chunks=sc) as plan:
        got = split_conv(plan, L.X, L.bias, epi, splits)
    ref, bound = oracle.conv3x3_f64(L.F.row_ptr, L.F.col_idx, L.F.values, L.X, L.bias, epi)
    assert_close(got, ref, bound, epi, f"conv {OC}x{IC} {H}x{W}x{NB} sc={sc}")


def test_split_ragged_small_patterns():
    """Rows whose entries all fall in one segment, empty rows, and a segment no row
    touches: partial sums of untouched segments must still be written (as zeros)."""
    K = 200  # seven chunks
    rows = [[0, 1, 2], [], [150, 199], [40], [0, 199], [100, 101, 102, 103], [], [33, 66, 99]]
    rp, ci, v = pattern_to_csr(rows, K)
    v = np.random.default_rng([2101, 7948, 10]).standard_normal(v.size).astype(np.float32)
    W = inputs.CSR(rp, ci, v, len(rows), K)
    B = rand_B(K, 130, 9)
    for sc in (1, 2, 3):
        check_split(W, B, None, "none", sc, f"small sc={sc}", panel_rows=4)


def test_split_random_configurations():
    """Seeded random problems over every option the split call combines: shape, density,
    segment length, runs along K (0 = the library's choice), panel height, row order,
    output order, epilogue and bias."""
    rng = np.random.default_rng([2101, 7948, 4242])
    for case in range(40):
        M = int(rng.integers(1, 300))
        K = int(rng.integers(1, 700))
        N = int(rng.integers(1, 700))
        d = float(rng.choice([0.0, 0.02, 0.1, 0.3, 0.7]))
        W = inputs.pattern_uniform(M, K, d, inputs.CFG_TEST, 7000 + case, 0.05)
        sc = int(rng.integers(1, 6))
        kw = dict(panel_rows=int(rng.choice([0, 4, 8, 12, 16])),
                  permute=int(rng.integers(0, 6)), out_permuted=bool(rng.integers(0, 2)))
        epi = str(rng.choice(["none", "relu", "gelu"]))
        bias = None if rng.random() < 0.3 else \
            (rng.standard_normal(M) * 0.05).astype(np.float32)
        splits = int(rng.choice([0, 1, 2, 3, 5, 64]))
        label = (f"case {case}: M={M} K={K} N={N} d={d} sc={sc} splits={splits} {kw} {epi} "
                 f"bias={bias is not None}")
        with sd.Plan.from_csr(W, split_chunks=sc, **kw) as plan:
            got = split_spmm(plan, rand_B(K, N, 7000 + case), bias, epi, splits=splits)
            perm = plan.perm
        ref, bound = oracle.spmm_f64(W.row_ptr, W.col_idx, W.values, K, rand_B(K, N, 7000 + case),
                                     bias, epi)
        if kw["out_permuted"]:
            ref, bound = ref[perm], bound[perm]
        assert_close(got, ref, bound, epi, label)


def test_longest_k_plain_and_split():
    """K = 2^19, the longest the stream's chunk fields allow: entries up to the last
    column, through the plain call and the K-split call (24 segments, library's choice
    and 5 runs)."""
    K, M, N = 1 << 19, 16, 64
    rng = np.random.default_rng([2101, 7948, 19])
    rows = [sorted(set(rng.choice(K, 100, replace=False).tolist()) | {K - 1, K - 33, 0})
            for _ in range(M)]
    rp, ci, _ = pattern_to_csr(rows, K)
    v = rng.standard_normal(ci.size).astype(np.float32)
    W = inputs.CSR(rp, ci, v, M, K)
    B = rand_B(K, N, 19)
    bias = rng.standard_normal(M).astype(np.float32)
    ref, bound = oracle.spmm_f64(rp, ci, v, K, B, bias, "relu")
    with sd.Plan.from_csr(W) as plain:
        Bt = torch.from_numpy(B).to(DEV)
        C = torch.full((M, N), float("nan"), device=DEV)
        plain.spmm(Bt, C, torch.from_numpy(bias).to(DEV), "relu")
        torch.cuda.synchronize()
        assert_close(C.cpu().numpy(), ref, bound, "relu", "K = 2^19 plain")
        del Bt
    for splits in (0, 5):
        got = check_split(W, B, bias, "relu", 700, f"K = 2^19 split {splits}", splits=splits)
        assert got.shape == (M, N)


def test_plan_info_matches_host_check():
    """The device plan reports the statistics and byte count the host-only check computes,
    the K-segment table and the device perm of split plans included."""
    W = inputs.workload("c2", N=4).layers[0].W
    for kw in ({}, {"split_chunks": 3}, {"split_chunks": 1, "panel_rows": 8},
               {"split_chunks": 5, "out_permuted": True}):
        host = sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, **kw)
        with sd.Plan.from_csr(W, **kw) as plan:
            dev = plan.info
        for key in ("panels", "packed_bytes", "splits", "panel_rows", "tall_panel_rows", "nnz"):
            assert dev[key] == host[key], (kw, key, dev[key], host[key])
        assert dev["rho"] == pytest.approx(host["rho"]) and dev["fill"] == pytest.approx(host["fill"])


@pytest.mark.parametrize("splits", [2, 3, 8])
def test_split_row_permutation_equivariance_bitexact(splits):
    """A row's partial sums follow its entries in column order inside each run and the
    runs are added in order, whatever panel the row lands in: permuting W's rows
    permutes the K-split call's C rows bit for bit (a fixed run count, so that both
    calls cut K at the same chunks)."""
    W = inputs.pattern_uniform(300, 500, 0.1, inputs.CFG_TEST, 17, 0.05)
    B = inputs.dense_B(500, 384, inputs.CFG_TEST, 17)
    bias = inputs.bias_normal(300, inputs.CFG_TEST, 17, 0.02)
    pi = np.random.default_rng(18).permutation(300)
    Wd = W.to_dense()
    Wp = Wd[pi]
    rp = np.concatenate([[0], np.cumsum((Wp != 0).sum(axis=1))]).astype(np.int32)
    ci = np.nonzero(Wp)[1].astype(np.int32)
    v = Wp[Wp != 0].astype(np.float32)
    W2 = inputs.CSR(rp, ci, v, 300, 500)
    with sd.Plan.from_csr(W, split_chunks=2) as p1, sd.Plan.from_csr(W2, split_chunks=2) as p2:
        C1 = split_spmm(p1, B, bias, "gelu", splits=splits)
        C2 = split_spmm(p2, B, bias[pi], "gelu", splits=splits)
    assert np.array_equal(C2, C1[pi])
