"""Seeded synthetic inputs for the sparse-weight x dense-activation product.

This module holds input generation only -- none of the operator's arithmetic -- and is
shared by the tests, the smoke check and the benchmark on both sides (GPU library and
CPU oracle).  Every array is drawn from ``numpy.random.default_rng([210107948, cfg,
layer, tensor])`` with tensor 0 = sparsity pattern, 1 = weight values, 2 = dense
activations B, 3 = bias.

Patterns follow the paper's synthetic suites (Sec. 4.1: unstructured sparsity, a fixed
fraction of zeros) and the layer shapes of BERT-base and MobileNet-V1 1x1 convolutions
that the paper's end-to-end models use (Sec. 4.3):

* ``uniform``      -- exactly ``round(d*M*K)`` nonzeros placed uniformly at random
                      (a Gaussian matrix thresholded at its exact magnitude quantile has
                      this support distribution).
* ``lognormal``    -- per-row nonzero counts proportional to exp(N(0, sigma^2)), rounded
                      by largest remainder to the exact total, columns uniform per row.
* ``grouped8``     -- columns partitioned at random into groups of 8; each row takes
                      whole groups (the last one partial), so rows share column blocks.
* ``gauss_threshold`` -- the paper's own recipe: unit-Gaussian matrix, smallest
                      magnitudes set to zero; the survivors keep their Gaussian values.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import Optional

import numpy as np

SEED = 210107948

# workload ids used in the seed
CFG_W0, CFG_C1, CFG_C2, CFG_C3, CFG_C4, CFG_C5, CFG_S, CFG_TEST = 0, 1, 2, 3, 4, 5, 6, 7
CFG_CONV = 8
T_PATTERN, T_VALUES, T_B, T_BIAS = 0, 1, 2, 3


def rng_for(cfg: int, layer: int, tensor: int) -> np.random.Generator:
    return np.random.default_rng([SEED, cfg, layer, tensor])


@dataclasses.dataclass
class CSR:
    """Host CSR matrix (int32 indexes, float32 values)."""
    row_ptr: np.ndarray
    col_idx: np.ndarray
    values: np.ndarray
    M: int
    K: int

    @property
    def nnz(self) -> int:
        return int(self.row_ptr[-1])

    def to_dense(self) -> np.ndarray:
        W = np.zeros((self.M, self.K), dtype=np.float32)
        rows = np.repeat(np.arange(self.M), np.diff(self.row_ptr))
        W[rows, self.col_idx] = self.values
        return W

    def digest(self) -> str:
        h = hashlib.sha256()
        for a in (self.row_ptr, self.col_idx, self.values):
            h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()


def exact_nnz(M: int, K: int, density: float) -> int:
    """round(d*M*K), round half to even."""
    return int(np.rint(density * M * K))


def _csr_from_rows(M: int, K: int, rows: np.ndarray, cols: np.ndarray, values: np.ndarray) -> CSR:
    order = np.lexsort((cols, rows))
    rows, cols, values = rows[order], cols[order], values[order]
    counts = np.bincount(rows, minlength=M)
    row_ptr = np.zeros(M + 1, dtype=np.int32)
    np.cumsum(counts, out=row_ptr[1:])
    return CSR(row_ptr, cols.astype(np.int32), values.astype(np.float32), M, K)


def _largest_remainder(weights: np.ndarray, total: int, cap: int) -> np.ndarray:
    """Integer counts proportional to ``weights`` summing to ``total``, each <= cap."""
    weights = np.asarray(weights, dtype=np.float64)
    counts = np.zeros(weights.shape[0], dtype=np.int64)
    remaining_total = total
    active = np.ones(weights.shape[0], dtype=bool)
    while remaining_total > 0 and active.any():
        w = np.where(active, weights, 0.0)
        raw = w / w.sum() * remaining_total
        base = np.floor(raw).astype(np.int64)
        rem = remaining_total - int(base.sum())
        if rem > 0:
            frac = raw - base
            frac[~active] = -1.0
            top = np.argsort(-frac, kind="stable")[:rem]
            base[top] += 1
        new = np.minimum(counts + base, cap)
        added = int((new - counts).sum())
        counts = new
        remaining_total -= added
        active = counts < cap
        if added == 0:
            break
    return counts


def values_normal(cfg: int, layer: int, n: int, std: float) -> np.ndarray:
    return rng_for(cfg, layer, T_VALUES).normal(0.0, std, n).astype(np.float32)


def pattern_uniform(M: int, K: int, density: float, cfg: int, layer: int, std: float) -> CSR:
    nnz = exact_nnz(M, K, density)
    rng = rng_for(cfg, layer, T_PATTERN)
    pos = np.sort(rng.choice(M * K, size=nnz, replace=False)) if nnz else np.zeros(0, np.int64)
    rows, cols = pos // K, pos % K
    vals = values_normal(cfg, layer, nnz, std)
    return _csr_from_rows(M, K, rows, cols, vals)


def pattern_lognormal(M: int, K: int, density: float, sigma: float, cfg: int, layer: int,
                      std: float) -> CSR:
    nnz = exact_nnz(M, K, density)
    rng = rng_for(cfg, layer, T_PATTERN)
    raw = np.exp(rng.normal(0.0, sigma, M))
    counts = _largest_remainder(raw, nnz, K)
    rows, cols = [], []
    for i in range(M):
        c = counts[i]
        if c:
            rows.append(np.full(c, i, dtype=np.int64))
            cols.append(rng.choice(K, size=c, replace=False))
    rows = np.concatenate(rows) if rows else np.zeros(0, np.int64)
    cols = np.concatenate(cols) if cols else np.zeros(0, np.int64)
    order = np.lexsort((cols, rows))
    vals = values_normal(cfg, layer, int(counts.sum()), std)
    return _csr_from_rows(M, K, rows[order], cols[order], vals)


def pattern_grouped8(M: int, K: int, density: float, cfg: int, layer: int, std: float) -> CSR:
    assert K % 8 == 0
    nnz = exact_nnz(M, K, density)
    rng = rng_for(cfg, layer, T_PATTERN)
    groups = rng.permutation(K).reshape(K // 8, 8)
    counts = _largest_remainder(np.ones(M), nnz, K)
    rows, cols = [], []
    for i in range(M):
        c = int(counts[i])
        if not c:
            continue
        ng = -(-c // 8)
        pick = rng.choice(K // 8, size=ng, replace=False)
        full = groups[pick[:-1]].reshape(-1)
        last_n = c - 8 * (ng - 1)
        last = rng.choice(groups[pick[-1]], size=last_n, replace=False)
        cc = np.concatenate([full, last])
        rows.append(np.full(c, i, dtype=np.int64))
        cols.append(cc)
    rows = np.concatenate(rows) if rows else np.zeros(0, np.int64)
    cols = np.concatenate(cols) if cols else np.zeros(0, np.int64)
    order = np.lexsort((cols, rows))
    vals = values_normal(cfg, layer, int(counts.sum()), std)
    return _csr_from_rows(M, K, rows[order], cols[order], vals)


def pattern_gauss_threshold(M: int, K: int, sparsity: float, cfg: int, layer: int) -> CSR:
    """Unit-Gaussian matrix with its smallest-magnitude entries zeroed (Sec. 4.1)."""
    nnz = exact_nnz(M, K, 1.0 - sparsity)
    dense = rng_for(cfg, layer, T_PATTERN).standard_normal((M, K))
    flat = np.abs(dense).reshape(-1)
    keep = np.sort(np.argpartition(-flat, nnz - 1)[:nnz]) if nnz else np.zeros(0, np.int64)
    rows, cols = keep // K, keep % K
    return _csr_from_rows(M, K, rows, cols, dense.reshape(-1)[keep].astype(np.float32))


def dense_B(K: int, N: int, cfg: int, layer: int, relu_clamp: bool = False) -> np.ndarray:
    B = rng_for(cfg, layer, T_B).standard_normal((K, N), dtype=np.float32)
    if relu_clamp:
        np.maximum(B, 0.0, out=B)
    return B


def bias_normal(M: int, cfg: int, layer: int, std: float) -> np.ndarray:
    if std == 0.0:
        return np.zeros(M, dtype=np.float32)
    return rng_for(cfg, layer, T_BIAS).normal(0.0, std, M).astype(np.float32)


@dataclasses.dataclass
class Layer:
    """One sparse linear layer: W (CSR), its bias and epilogue name."""
    W: CSR
    bias: Optional[np.ndarray]
    epi: str


@dataclasses.dataclass
class Workload:
    name: str
    layers: list  # list[Layer], applied in order (chained when more than one)
    B: np.ndarray  # input activations of the first layer, K0 x N
    N: int


def workload(name: str, N: Optional[int] = None, num_layers: Optional[int] = None) -> Workload:
    """The named synthetic workloads.

    w0  W 768x3072, 90% uniform, W~N(0,.02), B~N(0,1) K x N (default N=4096), bias N(0,.02)
    c1  W 256x256, 90% uniform, W~N(0,.05), B 256x64, zero bias, no activation
    c2  W 768x768, 90% uniform, W~N(0,.02), B 768x1024, bias N(0,.02)
    c3  W1 3072x768 (bias+GELU) then W2 768x3072 (bias), 94%, lognormal(0.5) rows, N=4096
    c4  W 512x512, 80% uniform, W~N(0,.05), B=max(N(0,1),0) 512x3136, bias N(0,.02), ReLU
    c5  12 x [4 x 768x768, 3072x768 (GELU), 768x3072], 97%, 8-column groups, N=16384
    """
    if name == "w0":
        M, K, N = 768, 3072, N or 4096
        W = pattern_uniform(M, K, 0.10, CFG_W0, 0, 0.02)
        return Workload(name, [Layer(W, bias_normal(M, CFG_W0, 0, 0.02), "none")],
                        dense_B(K, N, CFG_W0, 0), N)
    if name == "c1":
        M, K, N = 256, 256, N or 64
        W = pattern_uniform(M, K, 0.10, CFG_C1, 0, 0.05)
        return Workload(name, [Layer(W, bias_normal(M, CFG_C1, 0, 0.0), "none")],
                        dense_B(K, N, CFG_C1, 0), N)
    if name == "c2":
        M, K, N = 768, 768, N or 1024
        W = pattern_uniform(M, K, 0.10, CFG_C2, 0, 0.02)
        return Workload(name, [Layer(W, bias_normal(M, CFG_C2, 0, 0.02), "none")],
                        dense_B(K, N, CFG_C2, 0), N)
    if name == "c3":
        N = N or 4096
        W1 = pattern_lognormal(3072, 768, 0.06, 0.5, CFG_C3, 0, 0.02)
        W2 = pattern_lognormal(768, 3072, 0.06, 0.5, CFG_C3, 1, 0.02)
        return Workload(name, [Layer(W1, bias_normal(3072, CFG_C3, 0, 0.02), "gelu"),
                               Layer(W2, bias_normal(768, CFG_C3, 1, 0.02), "none")],
                        dense_B(768, N, CFG_C3, 0), N)
    if name == "c4":
        M, K, N = 512, 512, N or 3136
        W = pattern_uniform(M, K, 0.20, CFG_C4, 0, 0.05)
        return Workload(name, [Layer(W, bias_normal(M, CFG_C4, 0, 0.02), "relu")],
                        dense_B(K, N, CFG_C4, 0, relu_clamp=True), N)
    if name == "c5":
        N = N or 16384
        L = 12 if num_layers is None else num_layers
        d = 0.03
        layers = []
        shapes = [(768, 768)] * 4 + [(3072, 768), (768, 3072)]
        for l in range(L):
            for j, (M, K) in enumerate(shapes):
                idx = 6 * l + j
                std = 1.0 / np.sqrt(d * K)
                W = pattern_grouped8(M, K, d, CFG_C5, idx, std)
                layers.append(Layer(W, bias_normal(M, CFG_C5, idx, 0.02),
                                    "gelu" if j == 4 else "none"))
        return Workload(name, layers, dense_B(768, N, CFG_C5, 0), N)
    raise KeyError(name)


S_SPARSITIES = (0.70, 0.80, 0.90, 0.95)


def s_layer(M: int, K: int, sparsity: float) -> Layer:
    """A paper-shaped kernel problem (Sec. 4.1: M, K from 256 to 2048, 70-95 % sparse):
    the unit-Gaussian survivors of a magnitude threshold, no bias, no activation."""
    grade = S_SPARSITIES.index(sparsity) if sparsity in S_SPARSITIES else 9
    layer = (M // 256) * 1000 + (K // 256) * 10 + grade
    return Layer(pattern_gauss_threshold(M, K, sparsity, CFG_S, layer), None, "none")


@dataclasses.dataclass
class ConvLayer:
    """A sparse 3x3 convolution (stride 1, padding 1): filters as an OC x (IC*9) CSR whose
    column is i*9 + ky*3 + kx, input X of shape (IC, H, W, NB), bias, epilogue."""
    F: CSR
    X: np.ndarray
    bias: Optional[np.ndarray]
    epi: str

    @property
    def shape(self):
        IC, H, W, NB = self.X.shape
        return self.F.M, IC, H, W, NB


def conv_layer(OC: int, IC: int, H: int, W: int, NB: int, sparsity: float, layer: int = 0,
               epi: str = "none", cfg: int = CFG_CONV) -> ConvLayer:
    """The paper's convolution benchmark problems (Sec. 4.1): 3x3 filters, padding 1,
    random sparsity generated like the SpMM suite (a uniformly random support of exactly
    round(d * OC * IC * 9) taps, d = 1 - sparsity), values N(0, 0.05); input N(0, 1) in
    channel, row, column, image order; bias N(0, 0.02)."""
    F = pattern_uniform(OC, IC * 9, 1.0 - sparsity, cfg, layer, 0.05)
    X = rng_for(cfg, layer, T_B).standard_normal((IC, H, W, NB), dtype=np.float32)
    return ConvLayer(F, X, bias_normal(OC, cfg, layer, 0.02), epi)
