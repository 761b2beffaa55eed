"""CPU tests of K-segmented packing (plan option split_chunks), through the host-only
self-check: the packer's stream, re-walked, must hold every entry once, with no group
spanning two K-segments, the sync bit on each segment's first group and a segment table
that names each segment's first group.  No GPU is touched."""
import numpy as np
import pytest

import paper_2101_07948_amd as sd
from conftest import pattern_to_csr
from paper_2101_07948_amd import inputs


@pytest.mark.parametrize("name", ["w0", "c2", "c3", "c5"])
@pytest.mark.parametrize("split_chunks", [1, 3, 8, 1000])
def test_split_packing_self_check(name, split_chunks):
    W = inputs.workload(name, N=4).layers[0].W
    for rows in (0, 4, 12):
        info = sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, panel_rows=rows,
                                  split_chunks=split_chunks)
        nchunks = -(-W.K // info["k_chunk"])
        assert info["splits"] == max(1, -(-nchunks // split_chunks))
        plain = sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, panel_rows=rows)
        assert plain["splits"] == 0
        # segments only cut groups: never fewer stored entries, same reuse
        assert info["fill"] <= plain["fill"] + 1e-12
        assert info["rho"] == plain["rho"]
        if split_chunks >= nchunks:
            assert info["fill"] == plain["fill"]


def test_split_packing_ragged_and_edge_shapes():
    rng = np.random.default_rng([2101, 7948, 77])
    for M, K, d in [(1, 1, 1.0), (5, 33, 0.5), (13, 129, 0.3), (37, 1000, 0.05), (70, 96, 0.0),
                    (9, 2049, 0.02)]:
        mask = rng.random((M, K)) < d
        rp, ci, v = pattern_to_csr([np.flatnonzero(mask[i]).tolist() for i in range(M)], K)
        for sc in (1, 2, 5):
            info = sd.plan_check_host(rp, ci, v, M, K, split_chunks=sc, panel_rows=4)
            assert info["splits"] >= 1


def test_split_option_rejects_negative():
    W = inputs.workload("c2", N=4).layers[0].W
    with pytest.raises(sd.SdnnError) as e:
        sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, split_chunks=-1)
    assert e.value.code == 2


def test_split_entry_points_check_plan_before_gpu():
    """A NULL plan is reported before any device work (no GPU is needed for that)."""
    L = sd.lib()
    assert L.sdnn_spmm_split(None, None, None, 4, None, 0, 0, None, 0, None) == 1
    assert L.sdnn_conv3x3_split(None, None, None, 2, 2, 4, None, 0, 0, None, 0, None) == 1


def test_longest_k_packs_and_one_more_chunk_is_rejected():
    """K = 2^19 (16384 chunks, the stream's chunk fields full) packs, entries in the last
    chunk included, also in K-segments; one more row of B is SDNN_ERR_DIM."""
    K = 1 << 19
    rows = [[0, 5, K - 1], [K // 2, K - 33, K - 32], [], [7, 31, 32, 1000, 400000]]
    rp, ci, v = pattern_to_csr(rows, K)
    for sc in (0, 1, 700):
        info = sd.plan_check_host(rp, ci, v, len(rows), K, panel_rows=4, split_chunks=sc)
        assert info["splits"] == (0 if sc == 0 else -(-16384 // sc))
    with pytest.raises(sd.SdnnError) as e:
        sd.plan_check_host(rp, ci, v, len(rows), K + 1, panel_rows=4)
    assert e.value.code == 2
