"""CPU oracle for SparseDNN's sparse-weight x dense-activation product (arXiv 2101.07948).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the CPU-baseline leg of
the benchmark import this package; the product library never does, and the two share
no code.  The arithmetic lives in ``oracle.c`` (plain C, double precision for the
reference); this module only loads it and marshals numpy arrays.

Functions (each cites the passage of the paper it follows):

* :func:`spmm_f64` -- the operator's plain definition (Sec. 2.2, Sec. 3.2.2) with the
  fused element-wise epilogue of Sec. 3.1: ``C = act(W @ B + bias)``, summed in double
  in ascending column order per row.  Also returns ``sum |w| |b|`` per element.
* :func:`spmm_f32` -- the same loops with a float accumulator (timed CPU baseline).
* :func:`reorder` -- Algorithm 1 of Sec. 3.1.2 (greedy weight-row permutation) with
  the tie-break reading (overlap desc, nonzero count desc, row index asc).
* :func:`conv3x3_f64` -- the sparse 3x3 convolution of Sec. 3.2.3 (stride 1, zero
  padding 1, the paper's benchmark setting of Sec. 4.1) by its definition, in double;
  filters as an OC x (IC*9) CSR (column ``i*9 + ky*3 + kx``), activations IC x H x W x NB.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_SO = os.path.join(_HERE, "liboracle.so")

EPI = {"none": 0, "relu": 1, "gelu": 2, 0: 0, 1: 1, 2: 2}

_lib_handle = None


def build(force: bool = True) -> str:
    """Compile oracle.c with gcc into liboracle.so (plain -O3, OpenMP over rows)."""
    if force or not os.path.exists(_SO):
        tmp = _SO + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O3", "-fopenmp", "-fPIC", "-shared", "-Wall", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _SO)
    return _SO


def load(path: str) -> ctypes.CDLL:
    """Load an oracle shared library and declare its signatures."""
    lib = ctypes.CDLL(path)
    i32, p = ctypes.c_int32, ctypes.c_void_p
    lib.oracle_spmm_f64.argtypes = [i32, i32, i32, p, p, p, p, p, i32, p, p]
    lib.oracle_spmm_f64.restype = ctypes.c_int
    lib.oracle_spmm_f32.argtypes = [i32, i32, i32, p, p, p, p, p, i32, p]
    lib.oracle_spmm_f32.restype = ctypes.c_int
    lib.oracle_reorder.argtypes = [i32, i32, p, p, p]
    lib.oracle_reorder.restype = ctypes.c_int
    lib.oracle_conv3x3_f64.argtypes = [i32, i32, i32, i32, i32, p, p, p, p, p, i32, p, p]
    lib.oracle_conv3x3_f64.restype = ctypes.c_int
    lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_num_threads.restype = None
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    return lib


def _lib(lib=None):
    global _lib_handle
    if lib is not None:
        return lib
    if _lib_handle is None:
        if not os.path.exists(_SO):
            build(force=False)
        _lib_handle = load(_SO)
    return _lib_handle


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _csr(row_ptr, col_idx, values):
    row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int32)
    col_idx = np.ascontiguousarray(col_idx, dtype=np.int32)
    values = None if values is None else np.ascontiguousarray(values, dtype=np.float32)
    return row_ptr, col_idx, values


def spmm_f64(row_ptr, col_idx, values, K, B, bias=None, epi="none", with_bound=True, lib=None):
    """Reference ``act(W @ B + bias)`` in double.  Returns ``(C, bound)`` as float64
    arrays of shape (M, N); ``bound`` is ``sum_p |w_p| |B[c_p, n]|`` (None if not asked)."""
    row_ptr, col_idx, values = _csr(row_ptr, col_idx, values)
    B = np.ascontiguousarray(B, dtype=np.float32)
    M = row_ptr.shape[0] - 1
    N = B.shape[1]
    assert B.shape[0] == K
    bias = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    C = np.empty((M, N), dtype=np.float64)
    bound = np.empty((M, N), dtype=np.float64) if with_bound else None
    _lib(lib).oracle_spmm_f64(M, K, N, _ptr(row_ptr), _ptr(col_idx), _ptr(values), _ptr(B),
                           _ptr(bias), EPI[epi], _ptr(C), _ptr(bound))
    return C, bound


def spmm_f32(row_ptr, col_idx, values, K, B, bias=None, epi="none", out=None, lib=None):
    """CPU baseline ``act(W @ B + bias)`` with a float accumulator (OpenMP over rows)."""
    row_ptr, col_idx, values = _csr(row_ptr, col_idx, values)
    B = np.ascontiguousarray(B, dtype=np.float32)
    M = row_ptr.shape[0] - 1
    N = B.shape[1]
    bias = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    C = out if out is not None else np.empty((M, N), dtype=np.float32)
    _lib(lib).oracle_spmm_f32(M, K, N, _ptr(row_ptr), _ptr(col_idx), _ptr(values), _ptr(B),
                           _ptr(bias), EPI[epi], _ptr(C))
    return C


def conv3x3_f64(row_ptr, col_idx, values, X, bias=None, epi="none", with_bound=True, lib=None):
    """Reference sparse 3x3 convolution (stride 1, zero padding 1) in double.  ``X`` is
    (IC, H, W, NB); the filters are an OC x (IC*9) CSR.  Returns ``(C, bound)`` of shape
    (OC, H, W, NB); ``bound`` is ``sum |w| |x|`` over the taps (None if not asked)."""
    row_ptr, col_idx, values = _csr(row_ptr, col_idx, values)
    X = np.ascontiguousarray(X, dtype=np.float32)
    IC, H, W, NB = (int(d) for d in X.shape)
    OC = row_ptr.shape[0] - 1
    assert col_idx.size == 0 or int(col_idx.max()) < IC * 9
    bias = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    C = np.empty((OC, H, W, NB), dtype=np.float64)
    bound = np.empty((OC, H, W, NB), dtype=np.float64) if with_bound else None
    _lib(lib).oracle_conv3x3_f64(OC, IC, H, W, NB, _ptr(row_ptr), _ptr(col_idx), _ptr(values),
                                 _ptr(X), _ptr(bias), EPI[epi], _ptr(C), _ptr(bound))
    return C, bound


def reorder(row_ptr, col_idx, K, lib=None):
    """Algorithm 1: ``perm[i]`` is the original row placed at position i."""
    row_ptr, col_idx, _ = _csr(row_ptr, col_idx, None)
    M = row_ptr.shape[0] - 1
    perm = np.empty(M, dtype=np.int32)
    rc = _lib(lib).oracle_reorder(M, K, _ptr(row_ptr), _ptr(col_idx), _ptr(perm))
    if rc != 0:
        raise MemoryError("oracle_reorder failed")
    return perm


def num_threads() -> int:
    return int(_lib().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """OpenMP threads of later oracle calls (timing only)."""
    _lib().oracle_set_num_threads(int(n))

