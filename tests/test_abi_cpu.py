"""CPU-only tests of the C ABI library: exports, host-side preparation stage (CSR
validation, Algorithm 1 on bitsets, packing) and error codes.  No GPU is touched:
only host-only entry points are called, plus plan_create on inputs it must reject
before any device work."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import paper_2101_07948_amd as sd
from conftest import ROOT, dense_to_csr, pattern_to_csr, load_reorder_examples
from paper_2101_07948_amd import inputs


def header_functions(header="sdnn.h"):
    text = open(os.path.join(ROOT, "include", header)).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sdnn_[a-z_]+)\s*\(", text)))


def test_library_exports_every_header_symbol():
    L = sd.lib()
    names = header_functions()
    assert "sdnn_spmm" in names and "sdnn_plan_create" in names
    for n in names:
        assert hasattr(L, n), f"libsdnn.so does not export {n}"


def test_probe_library_exports_every_header_symbol():
    path = os.path.join(ROOT, "paper_2101_07948_amd", "libsdnn_probes.so")
    L = ctypes.CDLL(path)
    names = header_functions("sdnn_probes.h")
    assert names == ["sdnn_probe_fma", "sdnn_probe_lds_read", "sdnn_probe_out_floats"]
    for n in names:
        assert hasattr(L, n), f"libsdnn_probes.so does not export {n}"
    L.sdnn_probe_out_floats.restype = ctypes.c_int64
    assert L.sdnn_probe_out_floats() == 256 * 1024


def test_status_strings():
    for code, name in sd.STATUS.items():
        assert sd.status_str(code).startswith(name)


def test_destroy_null_is_noop():
    sd.lib().sdnn_plan_destroy(None)


@pytest.mark.parametrize("name", ["c1", "c2", "c4", "w0", "c3"])
def test_library_reorder_matches_oracle_on_workloads(name):
    for L in inputs.workload(name, N=4).layers:
        got = sd.reorder_rows(L.W.row_ptr, L.W.col_idx, L.W.K)
        want = oracle.reorder(L.W.row_ptr, L.W.col_idx, L.W.K)
        assert np.array_equal(got, want)


def test_library_reorder_matches_oracle_grouped():
    W = inputs.pattern_grouped8(768, 768, 0.03, inputs.CFG_C5, 0, 0.1)
    assert np.array_equal(sd.reorder_rows(W.row_ptr, W.col_idx, W.K),
                          oracle.reorder(W.row_ptr, W.col_idx, W.K))


def test_library_reorder_worked_examples_and_random():
    for name, K, rows, want in load_reorder_examples():
        rp, ci, _ = pattern_to_csr(rows, K)
        assert sd.reorder_rows(rp, ci, K).tolist() == want, name
    rng = np.random.default_rng(11)
    for _ in range(200):
        M, K = int(rng.integers(1, 12)), int(rng.integers(1, 140))
        mask = rng.random((M, K)) < rng.choice([0.05, 0.3, 0.7])
        rows = [list(np.nonzero(mask[i])[0]) for i in range(M)]
        rp, ci, _ = pattern_to_csr(rows, K)
        assert np.array_equal(sd.reorder_rows(rp, ci, K), oracle.reorder(rp, ci, K))
    for bits in range(512):  # every 3x3 pattern
        rows = [[c for c in range(3) if bits >> (3 * r + c) & 1] for r in range(3)]
        rp, ci, _ = pattern_to_csr(rows, 3)
        assert np.array_equal(sd.reorder_rows(rp, ci, 3), oracle.reorder(rp, ci, 3))


@pytest.mark.parametrize("name", ["c1", "c2", "c4", "w0", "c3"])
@pytest.mark.parametrize("panel_rows", [4, 8, 12, 16, 32])
def test_packed_stream_self_check(name, panel_rows):
    for L in inputs.workload(name, N=4).layers:
        info = sd.plan_check_host(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.M, L.W.K,
                                  panel_rows=panel_rows, tile_cols=128 if panel_rows == 32 else 0)
        assert info["nnz"] == L.W.nnz and info["M"] == L.W.M and info["K"] == L.W.K
        assert info["panels"] == -(-L.W.M // panel_rows)
        # filler closes a panel's last group, or a group whose next entry lies a whole
        # LDS ring (4 chunks) ahead: < 4 entries each, at most nchunks/4 + 1 per panel
        nchunks = -(-L.W.K // info["k_chunk"])
        stored = round(L.W.nnz / info["fill"]) if L.W.nnz else 0
        assert info["rho"] >= 1.0
        assert L.W.nnz <= stored <= L.W.nnz + 3 * info["panels"] * (nchunks // 4 + 1)
        assert stored % 4 == 0


@pytest.mark.parametrize("name", ["c2", "w0", "c3"])
def test_default_plan_packs_five_panel_heights(name):
    """With panel_rows = 0 the plan holds 4-, 12-, 8-, 16- and 32-row packings of the same
    grouping (the 32-row one, for 128-column tiles only, is left out with tile_cols = 256);
    all pass the stream self-check, taller panels share more columns, and each packing
    equals the plan with that height alone."""
    for L in inputs.workload(name, N=4).layers:
        info = sd.plan_check_host(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.M, L.W.K)
        assert info["panel_rows"] == 4 and info["tall_panel_rows"] == 12
        assert info["mid_panel_rows"] == 8 and info["tallest_panel_rows"] == 16
        assert info["deep_panel_rows"] == 32 and info["packings"] == 5
        assert info["panels"] == -(-L.W.M // 4)
        assert (info["deep_rho"] >= info["tallest_rho"] >= info["tall_rho"] >= info["mid_rho"]
                >= info["rho"] >= 1.0)
        for f in ("fill", "tall_fill", "mid_fill", "tallest_fill", "deep_fill"):
            assert 0.0 < info[f] <= 1.0
        singles = {rw: sd.plan_check_host(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.M, L.W.K,
                                          panel_rows=rw, tile_cols=128) for rw in (4, 8, 12, 16, 32)}
        for rw, one in singles.items():
            assert one["tall_panel_rows"] == 0 and one["mid_panel_rows"] == 0
            assert one["tallest_panel_rows"] == 0 and one["deep_panel_rows"] == 0
            assert one["packings"] == 1
        assert singles[12]["rho"] == info["tall_rho"] and singles[8]["rho"] == info["mid_rho"]
        assert singles[16]["rho"] == info["tallest_rho"] and singles[32]["rho"] == info["deep_rho"]
        assert info["packed_bytes"] == sum(one["packed_bytes"] for one in singles.values())
        wide = sd.plan_check_host(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.M, L.W.K,
                                  tile_cols=256)
        assert wide["packings"] == 4 and wide["deep_panel_rows"] == 0
    with pytest.raises(sd.SdnnError) as ei:  # 32-row panels need 128-column tiles
        sd.plan_check_host(L.W.row_ptr, L.W.col_idx, L.W.values, L.W.M, L.W.K, panel_rows=32)
    assert ei.value.code == 2


def test_in_perm_relabels_columns():
    """A plan told that B's rows arrive in the order in_perm (the previous layer's
    permuted output, Sec. 3.1.2) packs W with column c renamed to its position in that
    order; the packed stream passes its self-check against the renamed CSR, and the
    statistics (panels, rho, fill) do not depend on column names."""
    W = inputs.pattern_grouped8(256, 384, 0.05, inputs.CFG_TEST, 31, 0.05)
    pi = np.random.default_rng(31).permutation(384).astype(np.int32)
    base = sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K)
    got = sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, in_perm=pi,
                             out_permuted=True)
    assert got["in_permuted"] == 1 and got["out_permuted"] == 1
    assert base["in_permuted"] == 0 and base["out_permuted"] == 0
    for k in ("panels", "rho", "tall_rho"):
        assert got[k] == base[k]


def test_algorithm1_ignores_column_names():
    """Algorithm 1's keys (overlap with the last placed row, nnz, index) are invariant
    under renaming columns, so a plan built on B's permuted row order keeps the
    permutation of the original matrix."""
    W = inputs.pattern_grouped8(200, 320, 0.06, inputs.CFG_TEST, 32, 0.05)
    pi = np.random.default_rng(32).permutation(320)
    Wd = W.to_dense()
    rp, ci, v = dense_to_csr(Wd[:, pi])        # column i of W' is column pi[i] of W
    assert np.array_equal(oracle.reorder(rp, ci, 320), oracle.reorder(W.row_ptr, W.col_idx, 320))
    assert np.array_equal(sd.reorder_rows(rp, ci, 320), sd.reorder_rows(W.row_ptr, W.col_idx, 320))


def test_bad_permutation_options_rejected():
    W = inputs.pattern_uniform(64, 96, 0.1, inputs.CFG_TEST, 33, 0.05)
    bad = np.arange(96, dtype=np.int32)
    bad[5] = 6  # duplicate
    with pytest.raises(sd.SdnnError) as e:
        sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, in_perm=bad)
    assert e.value.code == 2
    bad = np.arange(96, dtype=np.int32)
    bad[0] = 96  # out of range
    with pytest.raises(sd.SdnnError) as e:
        sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, in_perm=bad)
    assert e.value.code == 2
    with pytest.raises(ValueError):
        sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, in_perm=np.arange(95))
    o = sd.PlanOpts(0, 1, 2, 0, None)
    info = sd.PlanInfo()
    L = sd.lib()
    rc = L.sdnn_plan_check_host(W.row_ptr.ctypes.data, W.col_idx.ctypes.data,
                                W.values.ctypes.data, W.M, W.K, ctypes.byref(o),
                                ctypes.byref(info))
    assert rc == 2


def test_permutation_raises_reuse_on_grouped_columns():
    """Algorithm 1's purpose (Sec. 3.1.2): adjacent rows share columns.  On block-
    correlated rows the reuse factor rho of panels of consecutive rows must improve over
    the identity order."""
    W = inputs.pattern_grouped8(768, 768, 0.03, inputs.CFG_C5, 0, 0.1)
    on = sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, panel_rows=8,
                            grouping="order")
    off = sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, panel_rows=8,
                             permute=False, grouping="order")
    assert on["rho"] > 1.3 * off["rho"]


def test_edge_shapes_pack():
    cases = [
        ([[]], 5),                 # one empty row
        ([[0]], 1),                # 1 x 1
        ([[], [], []], 0),         # K = 0
        ([[0, 63, 64, 127, 128]], 129),  # chunk boundaries
        ([list(range(200))] * 3, 200),   # dense rows spanning chunks
    ]
    for rows, K in cases:
        rp, ci, v = pattern_to_csr(rows, K)
        info = sd.plan_check_host(rp, ci, v, len(rows), K)
        assert info["nnz"] == len(ci)
    # M = 0
    info = sd.plan_check_host(np.zeros(1, np.int32), np.zeros(0, np.int32),
                              np.zeros(0, np.float32), 0, 7)
    assert info["panels"] == 0


def _expect(code, fn):
    with pytest.raises(sd.SdnnError) as ei:
        fn()
    assert ei.value.code == code, str(ei.value)


@pytest.mark.parametrize("entry", ["check", "create", "reorder"])
def test_bad_csr_rejected(entry):
    def run(rp, ci, v, M, K):
        if entry == "check":
            return sd.plan_check_host(rp, ci, v, M, K)
        if entry == "create":
            return sd.Plan(rp, ci, v, M, K)
        return sd.reorder_rows(rp, ci, K) if len(rp) == M + 1 else None

    v3 = np.ones(3, np.float32)
    _expect(3, lambda: run(np.array([1, 2, 3], np.int32), np.array([0, 1, 2], np.int32), v3, 2, 4))  # row_ptr[0] != 0
    _expect(3, lambda: run(np.array([0, 2, 1], np.int32), np.array([0, 1], np.int32), v3, 2, 4))  # non-monotone
    _expect(3, lambda: run(np.array([0, 2, 3], np.int32), np.array([0, 1, 4], np.int32), v3, 2, 4))  # col >= K
    _expect(3, lambda: run(np.array([0, 2, 3], np.int32), np.array([0, -1, 2], np.int32), v3, 2, 4))  # col < 0
    _expect(3, lambda: run(np.array([0, 2, 3], np.int32), np.array([1, 0, 2], np.int32), v3, 2, 4))  # unsorted
    _expect(3, lambda: run(np.array([0, 2, 3], np.int32), np.array([1, 1, 2], np.int32), v3, 2, 4))  # duplicate


def test_bad_dims_and_nulls():
    L = sd.lib()
    rp = np.array([0, 1], np.int32)
    ci = np.array([0], np.int32)
    v = np.ones(1, np.float32)
    P = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    perm = np.zeros(1, np.int32)
    assert L.sdnn_reorder_rows(P(rp), P(ci), -1, 4, P(perm)) == 2
    assert L.sdnn_reorder_rows(None, P(ci), 1, 4, P(perm)) == 1
    assert L.sdnn_reorder_rows(P(rp), None, 1, 4, P(perm)) == 1
    assert L.sdnn_reorder_rows(P(rp), P(ci), 1, 4, None) == 1
    info = sd.PlanInfo()
    assert L.sdnn_plan_check_host(P(rp), P(ci), None, 1, 4, None, ctypes.byref(info)) == 1
    bad = sd.PlanOpts(5, 1)
    assert L.sdnn_plan_check_host(P(rp), P(ci), P(v), 1, 4, ctypes.byref(bad), None) == 2
    bad = sd.PlanOpts(8, 6)
    assert L.sdnn_plan_check_host(P(rp), P(ci), P(v), 1, 4, ctypes.byref(bad), None) == 2
    assert L.sdnn_plan_create(P(rp), P(ci), P(v), 1, 4, None, None) == 1
    assert L.sdnn_plan_get_perm(None, P(perm)) == 1
    assert L.sdnn_plan_info(None, ctypes.byref(info)) == 1
    assert L.sdnn_spmm(None, None, None, 4, None, 0, None) == 1
    assert L.sdnn_dense_gemm(None, None, None, -1, 4, 4, None, 0, None) == 2
    assert L.sdnn_dense_gemm(None, None, None, 0, 4, 4, None, 0, None) == 0  # M = 0: no-op


def test_generated_kernel_header_in_sync():
    """The K-loop assembly header is generated; the committed copy must match."""
    import importlib.util
    path = os.path.join(ROOT, "paper_2101_07948_amd", "csrc", "gen_spmm_asm.py")
    spec = importlib.util.spec_from_file_location("gen_spmm_asm", path)
    gen = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(gen)
    assert gen.main(check=True) == 0, "spmm_asm_gen.h is stale: run the package build"


@pytest.mark.parametrize("grouping", ["order", "balanced"])
@pytest.mark.parametrize("out_permuted", [False, True])
def test_panel_grouping_self_check(grouping, out_permuted):
    """The panels may group rows differently from the reported permutation (consecutive
    rows of it, or balanced panels): the host self-check re-walks every packing, checks
    that each panel row is stored to its original row (or, for out_permuted plans, to its
    position in perm), and the reported permutation stays Algorithm 1's."""
    L = inputs.workload("c3", N=4).layers[0]
    W = L.W
    info = sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, grouping=grouping,
                              out_permuted=out_permuted)
    assert info["grouping"] == (1 if grouping == "order" else 2)


def test_panel_grouping_default_is_balanced():
    """The library's grouping is the balanced one on every workload layer (consecutive
    rows of the permutation only when asked for); the reported permutation stays
    Algorithm 1's either way, and the balanced panels' heaviest never exceeds the
    permutation's own."""
    for name, li, kw in (("c3", 0, {}), ("c3", 1, {}), ("w0", 0, {}),
                         ("c5", 0, {"num_layers": 1}), ("c5", 4, {"num_layers": 1})):
        W = inputs.workload(name, N=4, **kw).layers[li].W
        info = sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K)
        assert info["grouping"] == 2, (name, li)
        info1 = sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, grouping="order")
        assert info1["grouping"] == 1, (name, li)
        nnz = np.diff(W.row_ptr)
        perm = sd.reorder_rows(W.row_ptr, W.col_idx, W.K)
        heavy_order = nnz[perm][: W.M // 4 * 4].reshape(-1, 4).sum(1).max()
        bal = sd.row_order(W.row_ptr, W.col_idx, W.K, "balanced")
        heavy_bal = nnz[bal][: W.M // 4 * 4].reshape(-1, 4).sum(1).max()
        assert heavy_bal <= heavy_order


def test_bad_grouping_rejected():
    W = inputs.pattern_uniform(16, 16, 0.2, inputs.CFG_TEST, 1, 0.05)
    for g in (-1, 3):
        with pytest.raises(sd.SdnnError) as ei:
            sd.plan_check_host(W.row_ptr, W.col_idx, W.values, 16, 16, grouping=g)
        assert ei.value.code == 2


def test_tile_cols_option():
    """tile_cols: 0 (default) and 128 hold the stream a second time, re-encoded for the
    128-column tiles (the host self-check decodes every address word of both and compares
    the fields); 256 holds one stream; other values are rejected."""
    W = inputs.workload("c3", N=4).layers[1].W
    sizes = {}
    for t in (0, 128, 256):
        info = sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, tile_cols=t)
        assert info["tile_cols"] == t
        sizes[t] = info["packed_bytes"]
    assert sizes[0] == sizes[128] > sizes[256]
    for bad in (-1, 64, 192, 512):
        with pytest.raises(sd.SdnnError) as ei:
            sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, tile_cols=bad)
        assert ei.value.code == 2
