"""CPU tests of the library's alternative row orders (plan option permute = 2 to 5;
Sec. 3.1.2 notes that reorderings other than Algorithm 1 performed comparably), by
their defining properties, through the host-only entry point sdnn_row_order.  No GPU
is touched.  Algorithm 1 itself (permute = 1) is pinned against the oracle elsewhere."""
import numpy as np
import pytest

import oracle
import paper_2101_07948_amd as sd
from conftest import pattern_to_csr
from paper_2101_07948_amd import inputs


class Csr:
    def __init__(self, rows, K):
        self.row_ptr, self.col_idx, self.values = pattern_to_csr(rows, K)
        self.M, self.K = len(rows), K


def random_csr(M, K, density, seed):
    rng = np.random.default_rng([2101, 7948, seed])
    mask = rng.random((M, K)) < density
    return Csr([np.flatnonzero(mask[i]).tolist() for i in range(M)], K)


def row_sets(row_ptr, col_idx):
    return [set(col_idx[row_ptr[i]:row_ptr[i + 1]].tolist()) for i in range(len(row_ptr) - 1)]


def assert_panel_union_picks(row_ptr, col_idx, perm, upto=None):
    """Each pick attains the largest key (overlap with the union of the panel's rows so
    far, nonzeros, -index) over the rows not yet placed; a panel's first pick has
    overlap 0 with the empty union, so it is the row with the most nonzeros."""
    sets = row_sets(row_ptr, col_idx)
    M = len(sets)
    remaining = set(range(M))
    union = set()
    for i in range(M if upto is None else min(upto, M)):
        if i % 4 == 0:
            union = set()
        key = lambda x: (len(sets[x] & union), len(sets[x]), -x)
        best = max(remaining, key=key)
        assert perm[i] == best, f"position {i}: picked {perm[i]}, best is {best}"
        remaining.discard(best)
        union |= sets[best]


@pytest.mark.parametrize("mode", ["identity", "algorithm1", "balanced", "panel_union", "minhash",
                                  "bin_greedy"])
def test_orders_are_permutations(mode):
    for M, K, d, seed in [(1, 1, 1.0, 1), (3, 5, 0.0, 2), (7, 9, 0.4, 3), (61, 47, 0.15, 4),
                          (130, 300, 0.05, 5)]:
        W = random_csr(M, K, d, seed)
        perm = sd.row_order(W.row_ptr, W.col_idx, K, mode)
        assert np.array_equal(np.sort(perm), np.arange(M))
    W = random_csr(0, 4, 0.5, 6)
    assert sd.row_order(W.row_ptr, W.col_idx, 4, mode).shape == (0,)


def test_identity_and_algorithm1_entry_points_agree():
    W = random_csr(90, 70, 0.1, 7)
    assert np.array_equal(sd.row_order(W.row_ptr, W.col_idx, 70, "identity"), np.arange(90))
    assert np.array_equal(sd.row_order(W.row_ptr, W.col_idx, 70, "algorithm1"),
                          sd.reorder_rows(W.row_ptr, W.col_idx, 70))


def test_panel_union_worked_example():
    """Rows {0,1}, {0,1,2,3}, {2,3,9}, {0,1,7}, {9} (K = 10).  Panel-union: row 1 heads
    (most nonzeros); rows 0, 2, 3 each overlap the union {0,1,2,3} in 2 and rows 2 and
    3 have 3 nonzeros, so row 2 (lower index); the union is now {0,1,2,3,9}: rows 0
    and 3 overlap it in 2, row 4 in 1, and row 3 has more nonzeros; then row 0; row 4
    heads the next panel: [1, 2, 3, 0, 4].  Algorithm 1 compares with the previous
    row only and takes row 4 third ({2,3,9} shares 9 with it, nothing with rows 0
    and 3): [1, 2, 4, 3, 0]."""
    rows = [[0, 1], [0, 1, 2, 3], [2, 3, 9], [0, 1, 7], [9]]
    rp = np.cumsum([0] + [len(r) for r in rows]).astype(np.int32)
    ci = np.array([c for r in rows for c in r], dtype=np.int32)
    assert sd.row_order(rp, ci, 10, "panel_union").tolist() == [1, 2, 3, 0, 4]
    assert sd.row_order(rp, ci, 10, "algorithm1").tolist() == [1, 2, 4, 3, 0]


def test_panel_union_brute_force_small():
    for seed, (M, K, d) in enumerate([(5, 6, 0.5), (9, 12, 0.3), (17, 40, 0.2), (33, 64, 0.1),
                                      (64, 128, 0.05), (40, 10, 0.5)]):
        W = random_csr(M, K, d, 100 + seed)
        perm = sd.row_order(W.row_ptr, W.col_idx, K, "panel_union")
        assert_panel_union_picks(W.row_ptr, W.col_idx, perm)


def test_panel_union_on_grouped_layer():
    """The first 96 picks on a C5-shaped 768 x 768 layer (97 %, 8-column groups)."""
    W = inputs.pattern_grouped8(768, 768, 0.03, inputs.CFG_C5, 0, 0.1)
    perm = sd.row_order(W.row_ptr, W.col_idx, W.K, "panel_union")
    assert np.array_equal(np.sort(perm), np.arange(W.M))
    assert_panel_union_picks(W.row_ptr, W.col_idx, perm, upto=96)


def test_panel_union_raises_panel_reuse():
    """The order is aimed at the reuse factor rho of 4-row panels: on block-correlated
    rows it is at least Algorithm 1's and well above the identity order's."""
    W = inputs.pattern_grouped8(768, 768, 0.03, inputs.CFG_C5, 0, 0.1)
    rho = {m: sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, panel_rows=4,
                                 permute=m, grouping="order")["rho"]
           for m in ("identity", "algorithm1", "panel_union")}
    assert rho["panel_union"] >= rho["algorithm1"] > 1.3 * rho["identity"]


def test_balanced_order_replays_longest_first():
    """permute = 2: rows by nonzero count (descending, ties by index) each go to the
    4-row panel with the fewest nonzeros so far among those with room (ties: lower
    panel); position 4 p + r is panel p's r-th row."""
    for M, K, d, seed in [(13, 30, 0.3, 8), (64, 64, 0.1, 9), (101, 50, 0.2, 10)]:
        W = random_csr(M, K, d, seed)
        nnz = np.diff(W.row_ptr)
        P = (M + 3) // 4
        cap = [4] * (P - 1) + [M - 4 * (P - 1)]
        load, members = [0] * P, [[] for _ in range(P)]
        for r in sorted(range(M), key=lambda x: (-nnz[x], x)):
            p = min((q for q in range(P) if len(members[q]) < cap[q]), key=lambda q: (load[q], q))
            members[p].append(r)
            load[p] += int(nnz[r])
        want = [r for m in members for r in m]
        assert sd.row_order(W.row_ptr, W.col_idx, K, "balanced").tolist() == want


def test_balanced_order_evens_panel_work():
    """On the lognormal C3 layers no panel carries more than the mean (+2 %) or its
    heaviest row plus the three lightest rows, whichever is larger."""
    for L in inputs.workload("c3", N=4).layers:
        W = L.W
        perm = sd.row_order(W.row_ptr, W.col_idx, W.K, "balanced")
        nnz = np.diff(W.row_ptr)[perm]
        panels = nnz[: W.M // 4 * 4].reshape(-1, 4).sum(axis=1)
        bound = max(1.02 * panels.mean(), nnz.max() + np.sort(nnz)[:3].sum())
        assert panels.max() <= bound + 4


def test_row_order_rejects_bad_arguments():
    W = random_csr(8, 8, 0.5, 11)
    for mode in (-1, 6):
        with pytest.raises(sd.SdnnError) as e:
            sd.row_order(W.row_ptr, W.col_idx, 8, mode)
        assert e.value.code == 2
    bad = W.col_idx.copy()
    if bad.size >= 2:
        bad[1] = 99  # out of range
        with pytest.raises(sd.SdnnError) as e:
            sd.row_order(W.row_ptr, bad, 8, "panel_union")
        assert e.value.code == 3
    with pytest.raises(sd.SdnnError) as e:
        sd.plan_check_host(W.row_ptr, W.col_idx, W.values, 8, 8, permute=6)
    assert e.value.code == 2


def fmix32(h):
    """MurmurHash3's 32-bit finalizer, written from its published definition."""
    h ^= h >> 16
    h = (h * 0x85EBCA6B) & 0xFFFFFFFF
    h ^= h >> 13
    h = (h * 0xC2B2AE35) & 0xFFFFFFFF
    h ^= h >> 16
    return h


def test_minhash_order_replays_its_definition():
    """permute = 4: rows sorted by (min over columns of fmix32(c ^ seed_t), t = 0..3), then
    nonzeros descending, then index; rows with equal column sets end up consecutive."""
    seeds = (0x9E3779B9, 0x7F4A7C15, 0x94D049BB, 0xBF58476D)
    for M, K, d, seed in [(40, 30, 0.2, 12), (120, 200, 0.05, 13)]:
        W = random_csr(M, K, d, seed)
        sets = row_sets(W.row_ptr, W.col_idx)
        sig = [tuple(min((fmix32(c ^ t) for c in cs), default=0xFFFFFFFF) for t in seeds)
               for cs in sets]
        want = sorted(range(M), key=lambda r: (sig[r], -len(sets[r]), r))
        assert sd.row_order(W.row_ptr, W.col_idx, K, "minhash").tolist() == want
    rows = [[1, 5, 9], [2, 3], [1, 5, 9], [7], [2, 3], [1, 5, 9], [4, 8]]
    rp, ci, _ = pattern_to_csr(rows, 10)
    perm = sd.row_order(rp, ci, 10, "minhash").tolist()
    for group in ([0, 2, 5], [1, 4]):
        where = sorted(perm.index(r) for r in group)
        assert where == list(range(where[0], where[0] + len(group)))


def test_bin_greedy_order_is_algorithm1_within_bins():
    """permute = 5: bins floor(log2(nnz + 1)), densest first, each ordered by the oracle's
    Algorithm 1 on the bin's rows alone."""
    for M, K, d, seed in [(50, 60, 0.15, 14), (97, 128, 0.3, 15)]:
        W = random_csr(M, K, d, seed)
        nnz = np.diff(W.row_ptr)
        bins = np.floor(np.log2(nnz + 1)).astype(int)
        want = []
        for b in sorted(set(bins.tolist()), reverse=True):
            rows = np.flatnonzero(bins == b)
            sub = [W.col_idx[W.row_ptr[r]:W.row_ptr[r + 1]].tolist() for r in rows]
            rp, ci, _ = pattern_to_csr(sub, K)
            want += rows[oracle.reorder(rp, ci, K)].tolist()
        assert sd.row_order(W.row_ptr, W.col_idx, K, "bin_greedy").tolist() == want


@pytest.mark.parametrize("mode", ["balanced", "panel_union", "minhash", "bin_greedy"])
def test_orders_pack_and_self_check(mode):
    for name in ("c2", "c4"):
        W = inputs.workload(name, N=4).layers[0].W
        info = sd.plan_check_host(W.row_ptr, W.col_idx, W.values, W.M, W.K, permute=mode)
        assert info["rho"] >= 1.0 and 0 < info["fill"] <= 1.0
