"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Each check takes an oracle library handle (``lib=None`` means the real oracle) and
returns a list of failure messages (empty = pass), so the same checks both gate the
real oracle and are shown to reject planted mistakes (tests/test_oracle_mutants.py).
None of them re-uses the oracle's own code or formula: they compare against NumPy
float64 dense products, closed forms, tabulated normal-CDF values, invariants and
exhaustive/brute-force searches.
"""

import numpy as np
from scipy.special import ndtr

import oracle
from conftest import (dense_to_csr, load_normal_cdf, load_reorder_examples, pattern_to_csr,
                      random_csr)


def _act_np(x, epi):
    if epi == "relu":
        return np.maximum(x, 0.0)
    if epi == "gelu":
        return x * ndtr(x)  # Phi from scipy's normal CDF: a library routine, not erf
    return x


def check_bruteforce(lib=None):
    """Sparse product vs NumPy float64 dense W @ B on tiny non-square shapes."""
    fails = []
    rng = np.random.default_rng(1234)
    for trial in range(60):
        M, K, N = (int(x) for x in rng.integers(1, 17, size=3))
        d = [0.1, 0.5, 0.9][trial % 3]
        epi = ["none", "relu", "gelu"][(trial // 3) % 3]
        row_ptr, col_idx, vals, W = random_csr(rng, M, K, d)
        B = rng.standard_normal((K, N)).astype(np.float32)
        bias = rng.standard_normal(M).astype(np.float32) if trial % 2 else None
        C, bound = oracle.spmm_f64(row_ptr, col_idx, vals, K, B, bias, epi, lib=lib)
        ref = W.astype(np.float64) @ B.astype(np.float64)
        if bias is not None:
            ref = ref + bias.astype(np.float64)[:, None]
        ref = _act_np(ref, epi)
        ref_bound = np.abs(W.astype(np.float64)) @ np.abs(B.astype(np.float64))
        scale = ref_bound + np.abs(ref) + 1.0
        if not np.all(np.abs(C - ref) <= 1e-12 * scale):
            fails.append(f"bruteforce value mismatch M={M} K={K} N={N} d={d} epi={epi}")
        if not np.all(np.abs(bound - ref_bound) <= 1e-12 * (ref_bound + 1.0)):
            fails.append(f"bruteforce bound mismatch M={M} K={K} N={N}")
    return fails


def check_special_cases(lib=None):
    """Density 0 -> act(bias); identity W -> act(B + bias); one 1.0 per row -> gather;
    density 1 -> dense product."""
    fails = []
    rng = np.random.default_rng(99)
    M, K, N = 7, 9, 5
    B = rng.standard_normal((K, N)).astype(np.float32)
    bias = rng.standard_normal(M).astype(np.float32)
    for epi in ("none", "relu", "gelu"):
        # density 0
        row_ptr = np.zeros(M + 1, np.int32)
        C, bound = oracle.spmm_f64(row_ptr, np.zeros(0, np.int32), np.zeros(0, np.float32), K, B,
                                   bias, epi, lib=lib)
        want = _act_np(np.repeat(bias.astype(np.float64)[:, None], N, axis=1), epi)
        if not np.allclose(C, want, rtol=1e-15, atol=1e-15 if epi == "gelu" else 0.0) \
                or np.any(bound != 0):
            fails.append(f"density 0 != act(bias) ({epi})")
        # identity (M = K)
        I = np.eye(K, dtype=np.float32)
        rp, ci, v = dense_to_csr(I)
        biasK = rng.standard_normal(K).astype(np.float32)
        C, _ = oracle.spmm_f64(rp, ci, v, K, B, biasK, epi, lib=lib)
        want = _act_np(B.astype(np.float64) + biasK.astype(np.float64)[:, None], epi)
        # erf's form of Phi cancels for negative x: allow 1e-15 absolute there
        if not np.allclose(C, want, rtol=1e-15, atol=1e-15 if epi == "gelu" else 0.0):
            fails.append(f"identity W != act(B + bias) ({epi})")
    # gather: row i has a single 1.0 at column sigma(i)
    sigma = rng.integers(0, K, size=M)
    G = np.zeros((M, K), np.float32)
    G[np.arange(M), sigma] = 1.0
    rp, ci, v = dense_to_csr(G)
    C, _ = oracle.spmm_f64(rp, ci, v, K, B, None, "none", lib=lib)
    if not np.array_equal(C, B[sigma].astype(np.float64)):
        fails.append("single-one rows do not gather B rows")
    # density 1
    Wd = rng.standard_normal((M, K)).astype(np.float32)
    Wd[Wd == 0] = 1.0
    rp, ci, v = dense_to_csr(Wd)
    C, _ = oracle.spmm_f64(rp, ci, v, K, B, bias, "none", lib=lib)
    ref = Wd.astype(np.float64) @ B.astype(np.float64) + bias.astype(np.float64)[:, None]
    if not np.allclose(C, ref, rtol=1e-13, atol=1e-13):
        fails.append("density 1 != dense product")
    return fails


def check_gelu_table(lib=None):
    """GELU epilogue equals x * Phi(x) at tabulated normal-CDF points; ReLU = max(x, 0)."""
    fails = []
    xs, phis = load_normal_cdf()
    rp, ci, v = dense_to_csr(np.ones((1, 1), np.float32))
    for x, phi in zip(xs, phis):
        B = np.array([[x]], np.float32)
        C, _ = oracle.spmm_f64(rp, ci, v, 1, B, None, "gelu", lib=lib)
        if abs(C[0, 0] - x * phi) > 2e-10 * max(1.0, abs(x)):
            fails.append(f"gelu({x}) = {C[0, 0]!r}, table gives {x * phi!r}")
        C, _ = oracle.spmm_f64(rp, ci, v, 1, B, None, "relu", lib=lib)
        if C[0, 0] != max(x, 0.0):
            fails.append(f"relu({x}) = {C[0, 0]!r}")
    return fails


def check_invariants(lib=None):
    """Row-permutation equivariance (bit-exact) and exact linearity under scaling by 2."""
    fails = []
    rng = np.random.default_rng(7)
    for trial in range(10):
        M, K, N = 23, 31, 13
        row_ptr, col_idx, vals, W = random_csr(rng, M, K, 0.2)
        B = rng.standard_normal((K, N)).astype(np.float32)
        bias = rng.standard_normal(M).astype(np.float32)
        epi = ["none", "relu", "gelu"][trial % 3]
        C, _ = oracle.spmm_f64(row_ptr, col_idx, vals, K, B, bias, epi, lib=lib)
        pi = rng.permutation(M)
        rp, ci, v = dense_to_csr(W[pi])
        Cp, _ = oracle.spmm_f64(rp, ci, v, K, B, bias[pi], epi, lib=lib)
        if not np.array_equal(Cp, C[pi]):
            fails.append("row permutation is not bit-exactly equivariant")
        C1, _ = oracle.spmm_f64(row_ptr, col_idx, vals, K, B, None, "none", lib=lib)
        C2, _ = oracle.spmm_f64(row_ptr, col_idx, vals, K, 2 * B, None, "none", lib=lib)
        if not np.array_equal(C2, 2 * C1):
            fails.append("scaling B by 2 does not scale C by 2 exactly")
    return fails


def check_bias_linearity(lib=None):
    """With no activation the bias enters linearly and per output row:
    C(b) - C(0) = b broadcast along N, and C(b1 + b2) - C(0) = (C(b1) - C(0)) + (C(b2) - C(0)),
    both to double rounding."""
    fails = []
    rng = np.random.default_rng(17)
    for trial in range(6):
        M, K, N = 19, 27, 11
        row_ptr, col_idx, vals, _ = random_csr(rng, M, K, 0.3)
        B = rng.standard_normal((K, N)).astype(np.float32)
        b1 = rng.standard_normal(M).astype(np.float32)
        b2 = rng.standard_normal(M).astype(np.float32)
        C0, _ = oracle.spmm_f64(row_ptr, col_idx, vals, K, B, None, "none", lib=lib)
        C1, _ = oracle.spmm_f64(row_ptr, col_idx, vals, K, B, b1, "none", lib=lib)
        C2, _ = oracle.spmm_f64(row_ptr, col_idx, vals, K, B, b2, "none", lib=lib)
        C12, _ = oracle.spmm_f64(row_ptr, col_idx, vals, K, B, b1 + b2, "none", lib=lib)
        scale = np.abs(C0) + np.abs(b1)[:, None] + np.abs(b2)[:, None] + 1.0
        if not np.all(np.abs((C1 - C0) - b1.astype(np.float64)[:, None]) <= 1e-13 * scale):
            fails.append("C(b) - C(0) != b (bias not added once per row)")
        want = (C1 - C0) + (C2 - C0)
        got = C12 - C0
        # b1 + b2 is formed in float32 above: compare against that rounded sum
        exact = (b1 + b2).astype(np.float64)[:, None]
        if not np.all(np.abs(got - exact) <= 1e-13 * scale) or \
                not np.all(np.abs(want - (b1.astype(np.float64) + b2.astype(np.float64))[:, None])
                           <= 1e-13 * scale):
            fails.append("bias is not linear")
    return fails


def check_gelu_odd_part(lib=None):
    """GELU(x) - GELU(-x) = x * (Phi(x) + Phi(-x)) = x: an identity of the exact erf form
    that holds at every x, checked on a grid through a one-entry product (w = 1)."""
    fails = []
    rp, ci, v = dense_to_csr(np.ones((1, 1), np.float32))
    xs = np.linspace(-6.0, 6.0, 97).astype(np.float32)
    for x in xs:
        Cp, _ = oracle.spmm_f64(rp, ci, v, 1, np.array([[x]], np.float32), None, "gelu", lib=lib)
        Cm, _ = oracle.spmm_f64(rp, ci, v, 1, np.array([[-x]], np.float32), None, "gelu", lib=lib)
        if abs((Cp[0, 0] - Cm[0, 0]) - float(x)) > 1e-14 * max(1.0, abs(float(x))):
            fails.append(f"GELU({x}) - GELU({-x}) = {Cp[0, 0] - Cm[0, 0]!r}, not {float(x)!r}")
            break
    return fails


def _reorder_properties(row_ptr, col_idx, K, perm):
    """Tie-break-free properties of Algorithm 1: bijection, first = a densest row,
    every later pick attains the maximum overlap with its predecessor."""
    M = len(row_ptr) - 1
    sets = [set(col_idx[row_ptr[i]:row_ptr[i + 1]].tolist()) for i in range(M)]
    if sorted(perm.tolist()) != list(range(M)):
        return "not a bijection"
    if M and len(sets[perm[0]]) != max(len(s) for s in sets):
        return "first row is not a densest row"
    remaining = set(range(M)) - {int(perm[0])}
    for i in range(1, M):
        prev = sets[perm[i - 1]]
        best = max(len(prev & sets[x]) for x in remaining)
        if len(prev & sets[perm[i]]) != best:
            return f"pick {i} does not maximise overlap"
        remaining.discard(int(perm[i]))
    return None


def check_reorder(lib=None):
    """Worked examples (exact permutation, pins the tie-break), and the tie-break-free
    properties exhaustively over all 3x3 and random 5x6 binary patterns."""
    fails = []
    for name, K, rows, want in load_reorder_examples():
        rp, ci, _ = pattern_to_csr(rows, K)
        got = oracle.reorder(rp, ci, K, lib=lib).tolist()
        if got != want:
            fails.append(f"reorder {name}: got {got}, want {want}")
    for bits in range(512):
        rows = [[c for c in range(3) if bits >> (3 * r + c) & 1] for r in range(3)]
        rp, ci, _ = pattern_to_csr(rows, 3)
        msg = _reorder_properties(rp, ci, 3, oracle.reorder(rp, ci, 3, lib=lib))
        if msg:
            fails.append(f"reorder 3x3 pattern {bits}: {msg}")
            break
    rng = np.random.default_rng(5)
    for _ in range(300):
        M, K = 5, 6
        mask = rng.random((M, K)) < rng.choice([0.2, 0.4, 0.6])
        rows = [list(np.nonzero(mask[i])[0]) for i in range(M)]
        rp, ci, _ = pattern_to_csr(rows, K)
        perm = oracle.reorder(rp, ci, K, lib=lib)
        msg = _reorder_properties(rp, ci, K, perm)
        if msg:
            fails.append(f"reorder random 5x6: {msg}")
            break
        # full tie-break check by brute force over the key (overlap, nnz, -index)
        sets = [set(r) for r in rows]
        want = [max(range(M), key=lambda x: (len(sets[x]), -x))]
        rem = set(range(M)) - {want[0]}
        while rem:
            prev = sets[want[-1]]
            nxt = max(rem, key=lambda x: (len(prev & sets[x]), len(sets[x]), -x))
            want.append(nxt)
            rem.discard(nxt)
        if perm.tolist() != want:
            fails.append(f"reorder random 5x6 tie-break: got {perm.tolist()}, want {want}")
            break
    # identity cases: diagonal, empty, full
    for W in (np.eye(6), np.zeros((6, 6)), np.ones((6, 6))):
        rows = [list(np.nonzero(W[i])[0]) for i in range(6)]
        rp, ci, _ = pattern_to_csr(rows, 6)
        if oracle.reorder(rp, ci, 6, lib=lib).tolist() != list(range(6)):
            fails.append("reorder of a diagonal/empty/full pattern is not the identity")
    return fails


def _conv_filters(rng, OC, IC, density):
    """Random sparse 3x3 filters as (CSR over columns i*9 + ky*3 + kx, dense OC x IC x 3 x 3)."""
    F = rng.standard_normal((OC, IC, 3, 3)).astype(np.float32)
    F[rng.random(F.shape) >= density] = 0.0
    rp, ci, v = dense_to_csr(F.reshape(OC, IC * 9))
    return rp, ci, v, F


def _conv_numpy(F, X):
    """Zero-padded 3x3 convolution by slicing a padded copy (NumPy float64)."""
    IC, H, W, NB = X.shape
    Xp = np.pad(X.astype(np.float64), ((0, 0), (1, 1), (1, 1), (0, 0)))
    out = np.zeros((F.shape[0], H, W, NB))
    for ky in range(3):
        for kx in range(3):
            win = Xp[:, ky:ky + H, kx:kx + W, :]            # X[i][y+ky-1][x+kx-1][b]
            out += np.einsum("oi,iyxb->oyxb", F[:, :, ky, kx].astype(np.float64), win)
    return out


def check_conv(lib=None):
    """Sparse 3x3 convolution (stride 1, padding 1) against: a padded-slice NumPy
    convolution on random tiny shapes (values and the |w||x| bound); all-ones filters on
    an all-ones input (4, 6 or 9 taps in range, times IC); a centre-tap-only filter,
    which is the pointwise product W_c @ X (the SpMM reference, bit for bit); and a
    one-hot input, which places the filter taps mirrored around the hot pixel."""
    fails = []
    rng = np.random.default_rng(2024)
    for trial in range(40):
        OC, IC = (int(v) for v in rng.integers(1, 6, size=2))
        H, W = (int(v) for v in rng.integers(1, 7, size=2))
        NB = int(rng.integers(1, 5))
        epi = ["none", "relu", "gelu"][trial % 3]
        rp, ci, v, F = _conv_filters(rng, OC, IC, [0.1, 0.5, 1.0][trial % 3])
        X = rng.standard_normal((IC, H, W, NB)).astype(np.float32)
        bias = rng.standard_normal(OC).astype(np.float32) if trial % 2 else None
        C, bound = oracle.conv3x3_f64(rp, ci, v, X, bias, epi, lib=lib)
        ref = _conv_numpy(F, X)
        if bias is not None:
            ref = ref + bias.astype(np.float64)[:, None, None, None]
        ref = _act_np(ref, epi)
        ref_bound = _conv_numpy(np.abs(F), np.abs(X))
        if not np.all(np.abs(C - ref) <= 1e-12 * (ref_bound + np.abs(ref) + 1.0)):
            fails.append(f"conv value mismatch OC={OC} IC={IC} H={H} W={W} NB={NB} {epi}")
        if not np.all(np.abs(bound - ref_bound) <= 1e-12 * (ref_bound + 1.0)):
            fails.append(f"conv bound mismatch OC={OC} IC={IC} H={H} W={W}")
    # all-ones: every in-range tap contributes 1 per input channel
    for H, W, IC in ((1, 1, 2), (2, 5, 3), (4, 4, 1), (6, 3, 2)):
        rp, ci, v = dense_to_csr(np.ones((2, IC * 9), np.float32))
        C, _ = oracle.conv3x3_f64(rp, ci, v, np.ones((IC, H, W, 2), np.float32), lib=lib)
        ny = np.array([min(H - 1, y + 1) - max(0, y - 1) + 1 for y in range(H)])
        nx = np.array([min(W - 1, x + 1) - max(0, x - 1) + 1 for x in range(W)])
        want = IC * ny[:, None] * nx[None, :]
        if not all(np.array_equal(C[o, :, :, b], want) for o in range(2) for b in range(2)):
            fails.append(f"all-ones conv != in-range tap count x IC (H={H} W={W})")
    # centre tap only: a pointwise product
    OC, IC, H, W, NB = 4, 3, 5, 4, 3
    Wc = rng.standard_normal((OC, IC)).astype(np.float32)
    F = np.zeros((OC, IC, 3, 3), np.float32)
    F[:, :, 1, 1] = Wc
    rp, ci, v = dense_to_csr(F.reshape(OC, IC * 9))
    X = rng.standard_normal((IC, H, W, NB)).astype(np.float32)
    C, _ = oracle.conv3x3_f64(rp, ci, v, X, lib=lib)
    rp1, ci1, v1 = dense_to_csr(Wc)
    P, _ = oracle.spmm_f64(rp1, ci1, v1, IC, X.reshape(IC, -1))
    if not np.array_equal(C.reshape(OC, -1), P):
        fails.append("centre-tap conv != pointwise product")
    # one-hot input at (i0, y0, x0, b0): C[o][y][x][b0] = F[o][i0][y0 - y + 1][x0 - x + 1]
    OC, IC, H, W, NB = 3, 2, 5, 6, 2
    rp, ci, v, F = _conv_filters(rng, OC, IC, 1.0)
    i0, y0, x0, b0 = 1, 2, 3, 1
    X = np.zeros((IC, H, W, NB), np.float32)
    X[i0, y0, x0, b0] = 1.0
    C, _ = oracle.conv3x3_f64(rp, ci, v, X, lib=lib)
    want = np.zeros((OC, H, W, NB))
    for y in range(y0 - 1, y0 + 2):
        for x in range(x0 - 1, x0 + 2):
            want[:, y, x, b0] = F[:, i0, y0 - y + 1, x0 - x + 1]
    if not np.array_equal(C, want):
        fails.append("one-hot conv does not place the mirrored filter taps")
    return fails


ALL_CHECKS = [check_bruteforce, check_special_cases, check_gelu_table, check_gelu_odd_part,
              check_invariants, check_bias_linearity, check_reorder, check_conv]


def run_all(lib=None):
    fails = []
    for chk in ALL_CHECKS:
        fails.extend(chk(lib))
    return fails
