"""Seeded generators: determinism and the structure each workload promises."""
import numpy as np

from paper_2101_07948_amd import inputs


def test_same_seed_same_bytes():
    a = inputs.workload("c2", N=32)
    b = inputs.workload("c2", N=32)
    assert a.layers[0].W.digest() == b.layers[0].W.digest()
    assert np.array_equal(a.B, b.B)
    assert np.array_equal(a.layers[0].bias, b.layers[0].bias)


def test_exact_nnz_and_csr_form():
    for name, d in (("c1", 0.1), ("c2", 0.1), ("c4", 0.2)):
        W = inputs.workload(name, N=8).layers[0].W
        assert W.nnz == int(np.rint(d * W.M * W.K))
        assert W.row_ptr[0] == 0 and np.all(np.diff(W.row_ptr) >= 0)
        for i in range(W.M):
            c = W.col_idx[W.row_ptr[i]:W.row_ptr[i + 1]]
            assert np.all(np.diff(c) > 0) and (c.size == 0 or (c[0] >= 0 and c[-1] < W.K))


def test_lognormal_rows_skewed_and_exact_total():
    w = inputs.workload("c3", N=8)
    for L in w.layers:
        cnt = np.diff(L.W.row_ptr)
        assert L.W.nnz == int(np.rint(0.06 * L.W.M * L.W.K))
        assert cnt.max() > 2 * cnt.mean() or cnt.std() > 0.3 * cnt.mean()


def test_grouped8_rows_use_whole_groups():
    W = inputs.pattern_grouped8(64, 768, 0.03, inputs.CFG_C5, 0, 0.1)
    groups = inputs.rng_for(inputs.CFG_C5, 0, inputs.T_PATTERN).permutation(768).reshape(-1, 8)
    gid = np.empty(768, np.int64)
    gid[groups.reshape(-1)] = np.repeat(np.arange(96), 8)
    for i in range(W.M):
        c = W.col_idx[W.row_ptr[i]:W.row_ptr[i + 1]]
        g, n = np.unique(gid[c], return_counts=True)
        assert (n < 8).sum() <= 1  # all groups full except possibly one
        assert len(g) == -(-len(c) // 8)


def test_gauss_threshold_keeps_largest():
    W = inputs.pattern_gauss_threshold(32, 48, 0.9, inputs.CFG_S, 0)
    assert W.nnz == int(np.rint(0.1 * 32 * 48))
    dense = inputs.rng_for(inputs.CFG_S, 0, inputs.T_PATTERN).standard_normal((32, 48))
    thr = np.sort(np.abs(dense).ravel())[-W.nnz]
    assert np.all(np.abs(W.values) >= np.float32(thr) * (1 - 1e-6))


def test_paper_shaped_layers():
    """s_layer: exact nonzero counts at every grade and a distinct seed per grade (the
    threshold itself is pinned by test_gauss_threshold_keeps_largest)."""
    seen = set()
    for sp in inputs.S_SPARSITIES:
        L = inputs.s_layer(256, 512, sp)
        assert L.W.nnz == inputs.exact_nnz(256, 512, 1.0 - sp)
        assert L.bias is None and L.epi == "none"
        seen.add(L.W.values[:8].tobytes())
    assert len(seen) == len(inputs.S_SPARSITIES)
