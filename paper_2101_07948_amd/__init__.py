"""MI355X (gfx950) sparse-weight x dense-activation product of SparseDNN (arXiv 2101.07948).

Thin ctypes binding over ``libsdnn.so`` (C ABI in ``include/sdnn.h``).  Every step of
the operator runs in the library: this module only checks shapes and dtypes, passes
raw pointers and the current HIP stream, and turns status codes into exceptions.
PyTorch supplies device memory and streams.  There is no fallback path: if the
library is missing, every call raises.

    plan = Plan(row_ptr, col_idx, values, M, K)    # preparation (Sec. 2.1, 3.1.2, 3.2.2)
    plan.spmm(B, C, bias, "gelu")                   # execution: C = gelu(W @ B + bias)
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsdnn.so")

EPI = {"none": 0, "relu": 1, "gelu": 2}
STATUS = {0: "SDNN_OK", 1: "SDNN_ERR_NULL", 2: "SDNN_ERR_DIM", 3: "SDNN_ERR_CSR",
          4: "SDNN_ERR_ALLOC", 5: "SDNN_ERR_HIP", 6: "SDNN_ERR_DEVICE", 7: "SDNN_ERR_INTERNAL"}


class SdnnError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {STATUS.get(code, code)}")


class PlanOpts(ctypes.Structure):
    _fields_ = [("panel_rows", ctypes.c_int32), ("permute", ctypes.c_int32),
                ("out_permuted", ctypes.c_int32), ("split_chunks", ctypes.c_int32),
                ("in_perm", ctypes.c_void_p), ("grouping", ctypes.c_int32),
                ("tile_cols", ctypes.c_int32)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int32), ("K", ctypes.c_int32), ("nnz", ctypes.c_int64),
                ("panels", ctypes.c_int64), ("packed_bytes", ctypes.c_int64),
                ("rho", ctypes.c_double), ("fill", ctypes.c_double),
                ("panel_rows", ctypes.c_int32), ("k_chunk", ctypes.c_int32),
                ("tall_panel_rows", ctypes.c_int32), ("splits", ctypes.c_int32),
                ("tall_rho", ctypes.c_double), ("tall_fill", ctypes.c_double),
                ("out_permuted", ctypes.c_int32), ("in_permuted", ctypes.c_int32),
                ("mid_panel_rows", ctypes.c_int32), ("packings", ctypes.c_int32),
                ("mid_rho", ctypes.c_double), ("mid_fill", ctypes.c_double),
                ("grouping", ctypes.c_int32), ("tile_cols", ctypes.c_int32),
                ("tallest_panel_rows", ctypes.c_int32), ("reserved2", ctypes.c_int32),
                ("tallest_rho", ctypes.c_double), ("tallest_fill", ctypes.c_double),
                ("deep_panel_rows", ctypes.c_int32), ("reserved3", ctypes.c_int32),
                ("deep_rho", ctypes.c_double), ("deep_fill", ctypes.c_double)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


_lib_handle = None


def lib() -> ctypes.CDLL:
    """The loaded libsdnn.so; raises if it has not been built."""
    global _lib_handle
    if _lib_handle is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2101_07948_amd.build` (no fallback path exists)")
        L = ctypes.CDLL(LIB_PATH)
        p, i32 = ctypes.c_void_p, ctypes.c_int32
        L.sdnn_status_str.argtypes = [ctypes.c_int]
        L.sdnn_status_str.restype = ctypes.c_char_p
        L.sdnn_reorder_rows.argtypes = [p, p, i32, i32, p]
        L.sdnn_row_order.argtypes = [p, p, i32, i32, i32, p]
        L.sdnn_plan_check_host.argtypes = [p, p, p, i32, i32, ctypes.POINTER(PlanOpts),
                                           ctypes.POINTER(PlanInfo)]
        L.sdnn_plan_create.argtypes = [p, p, p, i32, i32, ctypes.POINTER(PlanOpts),
                                       ctypes.POINTER(p)]
        L.sdnn_plan_get_perm.argtypes = [p, p]
        L.sdnn_plan_info.argtypes = [p, ctypes.POINTER(PlanInfo)]
        L.sdnn_spmm.argtypes = [p, p, p, i32, p, ctypes.c_int, p]
        L.sdnn_plan_destroy.argtypes = [p]
        L.sdnn_plan_destroy.restype = None
        L.sdnn_dense_gemm.argtypes = [p, p, p, i32, i32, i32, p, ctypes.c_int, p]
        L.sdnn_conv3x3.argtypes = [p, p, p, i32, i32, i32, p, ctypes.c_int, p]
        L.sdnn_plan_tune.argtypes = [p, p, p, i32, p, p, p]
        L.sdnn_plan_launch_shape.argtypes = [p, i32, p, p]
        L.sdnn_plan_launch_tile.argtypes = [p, i32, p]
        L.sdnn_plan_split_runs.argtypes = [p, i32, i32, p]
        i64 = ctypes.c_int64
        L.sdnn_spmm_split.argtypes = [p, p, p, i32, p, ctypes.c_int, i32, p, i64, p]
        L.sdnn_spmm_split_noalloc.argtypes = [p, p, p, i32, p, ctypes.c_int, i32, p]
        L.sdnn_conv3x3_split.argtypes = [p, p, p, i32, i32, i32, p, ctypes.c_int, i32, p, i64, p]
        for fn in ("sdnn_reorder_rows", "sdnn_row_order", "sdnn_plan_check_host", "sdnn_plan_create",
                   "sdnn_plan_get_perm", "sdnn_plan_info", "sdnn_spmm", "sdnn_dense_gemm",
                   "sdnn_conv3x3", "sdnn_plan_tune", "sdnn_spmm_split", "sdnn_conv3x3_split",
                   "sdnn_plan_launch_shape", "sdnn_spmm_split_noalloc", "sdnn_plan_launch_tile",
                   "sdnn_plan_split_runs"):
            getattr(L, fn).restype = ctypes.c_int
        _lib_handle = L
    return _lib_handle


def _check(code: int, where: str):
    if code != 0:
        raise SdnnError(code, where)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _np_ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


ORDERS = {"identity": 0, "algorithm1": 1, "balanced": 2, "panel_union": 3, "minhash": 4,
          "bin_greedy": 5}


def _order_mode(permute) -> int:
    """Plan option `permute` from a name in ORDERS, a bool (Algorithm 1 or identity)
    or its number."""
    if isinstance(permute, str):
        return ORDERS[permute]
    return (1 if permute else 0) if isinstance(permute, bool) else int(permute)


GROUPINGS = {"auto": 0, "order": 1, "balanced": 2}


def _opts(K: int, panel_rows: int, permute: bool, out_permuted: bool = False, in_perm=None,
          split_chunks: int = 0, grouping="auto", tile_cols: int = 0):
    """PlanOpts plus the in_perm array it points to (kept alive by the caller)."""
    keep = None if in_perm is None else _i32(in_perm)
    if keep is not None and keep.shape != (int(K),):
        raise ValueError(f"in_perm must hold K = {K} entries, got shape {keep.shape}")
    mode = _order_mode(permute)
    g = GROUPINGS[grouping] if isinstance(grouping, str) else int(grouping)
    o = PlanOpts(int(panel_rows), mode, 1 if out_permuted else 0, int(split_chunks),
                 None if keep is None else keep.ctypes.data, g, int(tile_cols))
    return o, keep


def reorder_rows(row_ptr, col_idx, K: int) -> np.ndarray:
    """Algorithm 1 (Sec. 3.1.2) computed by the library on the host."""
    row_ptr, col_idx = _i32(row_ptr), _i32(col_idx)
    M = row_ptr.shape[0] - 1
    perm = np.empty(M, dtype=np.int32)
    _check(lib().sdnn_reorder_rows(_np_ptr(row_ptr), _np_ptr(col_idx), M, K, _np_ptr(perm)),
           "sdnn_reorder_rows")
    return perm


def row_order(row_ptr, col_idx, K: int, permute="algorithm1") -> np.ndarray:
    """The row order of plan option `permute` (a name in ORDERS or its number),
    computed by the library on the host: perm[i] is the original row at position i."""
    row_ptr, col_idx = _i32(row_ptr), _i32(col_idx)
    M = row_ptr.shape[0] - 1
    perm = np.empty(M, dtype=np.int32)
    _check(lib().sdnn_row_order(_np_ptr(row_ptr), _np_ptr(col_idx), M, K,
                                _order_mode(permute), _np_ptr(perm)), "sdnn_row_order")
    return perm


def plan_check_host(row_ptr, col_idx, values, M: int, K: int, panel_rows: int = 0,
                    permute: bool = True, out_permuted: bool = False, in_perm=None,
                    split_chunks: int = 0, grouping="auto", tile_cols: int = 0) -> dict:
    """Host-only self-check of the preparation stage; returns the plan statistics."""
    row_ptr, col_idx, values = _i32(row_ptr), _i32(col_idx), _f32(values)
    info = PlanInfo()
    o, _keep = _opts(K, panel_rows, permute, out_permuted, in_perm, split_chunks, grouping,
                     tile_cols)
    _check(lib().sdnn_plan_check_host(_np_ptr(row_ptr), _np_ptr(col_idx), _np_ptr(values), M, K,
                                      ctypes.byref(o), ctypes.byref(info)),
           "sdnn_plan_check_host")
    return info.as_dict()


_torch = None


def _torch_mod():
    global _torch
    if _torch is None:
        import torch
        _torch = torch
    return _torch


def _stream_handle(stream) -> int:
    """The raw hipStream_t of `stream` (default: the current stream) as an integer.  The
    current stream is read through torch's raw-handle accessor, which skips building a
    Stream object (a few microseconds per call, as much as a small kernel takes)."""
    if stream is None:
        torch = _torch_mod()
        return torch._C._cuda_getCurrentRawStream(torch.cuda.current_device())
    return stream.cuda_stream


def _dev_ptr(t, name: str, shape, allow_none=False):
    """Device address of a contiguous float32 GPU tensor of the given shape (checked on a
    fast path; the slow path only builds the error message)."""
    if t is None:
        if allow_none:
            return None
        raise ValueError(f"{name} is required")
    torch = _torch_mod()
    try:
        if t.is_cuda and t.dtype is torch.float32 and t.shape == shape and t.is_contiguous():
            return t.data_ptr()
    except AttributeError:
        pass
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name} must be a CUDA/HIP torch tensor")
    if t.dtype != torch.float32:
        raise TypeError(f"{name} must be float32")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    raise ValueError(f"{name} must be contiguous (row-major)")


class Plan:
    """Preparation-stage result for one sparse weight matrix W (M x K, CSR on the host).

    The plan owns device memory on the device that is current when it is created.
    """

    def __init__(self, row_ptr, col_idx, values, M: int, K: int, panel_rows: int = 0,
                 permute: bool = True, out_permuted: bool = False, in_perm=None,
                 split_chunks: int = 0, grouping="auto", tile_cols: int = 0):
        """out_permuted: write C in the plan's permuted row order (C[i] = output row
        perm[i]); in_perm: the order of B's rows (B[i] = input feature in_perm[i]),
        e.g. the previous layer's perm when that layer used out_permuted; split_chunks:
        K-segments of that many staging chunks for spmm_split / conv3x3_split;
        grouping: "auto", "order" (panels are consecutive rows of perm) or "balanced";
        tile_cols: 0 (the library picks 256 or 128 columns per workgroup tile per call),
        256 or 128."""
        row_ptr, col_idx, values = _i32(row_ptr), _i32(col_idx), _f32(values)
        self.M, self.K = int(M), int(K)
        h = ctypes.c_void_p()
        o, _keep = _opts(self.K, panel_rows, permute, out_permuted, in_perm, split_chunks,
                         grouping, tile_cols)
        # torch first: its HIP runtime is then the one the process (and libsdnn) uses; a
        # plan created before torch's first load would leave torch without a GPU
        _torch_mod()
        self._lib = lib()
        _check(self._lib.sdnn_plan_create(_np_ptr(row_ptr), _np_ptr(col_idx), _np_ptr(values),
                                          self.M, self.K, ctypes.byref(o), ctypes.byref(h)),
               "sdnn_plan_create")
        self._h = h

    @classmethod
    def from_csr(cls, W, **kw):
        return cls(W.row_ptr, W.col_idx, W.values, W.M, W.K, **kw)

    @property
    def handle(self):
        if self._h is None:
            raise RuntimeError("plan is closed")
        return self._h

    @property
    def perm(self) -> np.ndarray:
        out = np.empty(self.M, dtype=np.int32)
        _check(self._lib.sdnn_plan_get_perm(self.handle, _np_ptr(out)), "sdnn_plan_get_perm")
        return out

    @property
    def info(self) -> dict:
        info = PlanInfo()
        _check(self._lib.sdnn_plan_info(self.handle, ctypes.byref(info)), "sdnn_plan_info")
        return info.as_dict()

    def launch_shape(self, N: int) -> dict:
        """The panel height, consumer waves per workgroup and tile width spmm uses at N
        columns (the tile width for 16-byte aligned B and C with N % 4 == 0)."""
        rw, waves, tile = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        _check(self._lib.sdnn_plan_launch_shape(self.handle, int(N), ctypes.byref(rw),
                                                ctypes.byref(waves)), "sdnn_plan_launch_shape")
        _check(self._lib.sdnn_plan_launch_tile(self.handle, int(N), ctypes.byref(tile)),
               "sdnn_plan_launch_tile")
        return {"panel_rows": rw.value, "waves": waves.value, "tile_cols": tile.value}

    def tune(self, N: int, B=None, C=None, stream=None) -> dict:
        """Times the plan's launch shapes at this N (on B / C, allocated here when not
        given) and records the fastest for later spmm calls with the same N; for plans with
        K-segments also the fastest workgroup count along K of spmm_split (split_runs)."""
        import torch
        if B is None:
            B = torch.randn(self.K, N, device="cuda")
        if C is None:
            C = torch.empty(self.M, N, device="cuda")
        pb = _dev_ptr(B, "B", (self.K, N))
        pc = _dev_ptr(C, "C", (self.M, N))
        rw, waves = ctypes.c_int32(), ctypes.c_int32()
        _check(self._lib.sdnn_plan_tune(self.handle, pb, pc, int(N), _stream_handle(stream),
                                        ctypes.byref(rw), ctypes.byref(waves)), "sdnn_plan_tune")
        tile = ctypes.c_int32()
        _check(self._lib.sdnn_plan_launch_tile(self.handle, int(N), ctypes.byref(tile)),
               "sdnn_plan_launch_tile")
        return {"panel_rows": rw.value, "waves": waves.value, "tile_cols": tile.value}

    def split_runs(self, N: int, splits: int = 0) -> int:
        """Workgroups along K that spmm_split runs at N for `splits` (0: the library's
        choice, the tuned count if tune recorded one)."""
        runs = ctypes.c_int32()
        _check(self._lib.sdnn_plan_split_runs(self.handle, int(N), int(splits), ctypes.byref(runs)),
               "sdnn_plan_split_runs")
        return runs.value

    def conv3x3(self, X, C, bias=None, epi: str = "none", stream=None):
        """Sparse 3x3 convolution (stride 1, padding 1) on the GPU: the plan holds the
        filters as an OC x (IC*9) CSR (column i*9 + ky*3 + kx); X is (IC, H, W, NB) and C
        is (OC, H, W, NB), both contiguous fp32 on the device; NB % 4 == 0."""
        if X.dim() != 4 or C.dim() != 4:
            raise ValueError("X and C must be 4-d (channels, H, W, images)")
        IC, H, W, NB = (int(d) for d in X.shape)
        if IC * 9 != self.K:
            raise ValueError(f"X has {IC} channels; the plan's K = {self.K} needs {self.K // 9}")
        px = _dev_ptr(X, "X", (IC, H, W, NB))
        pc = _dev_ptr(C, "C", (self.M, H, W, NB))
        pbias = _dev_ptr(bias, "bias", (self.M,), allow_none=True)
        _check(self._lib.sdnn_conv3x3(self.handle, px, pc, H, W, NB, pbias, EPI[epi],
                                      _stream_handle(stream)), "sdnn_conv3x3")
        return C

    def workspace_floats(self, N: int) -> int:
        """Floats of the workspace a K-split call at N columns needs (nseg * M * N, nseg =
        info["splits"], the plan's K-segments)."""
        return int(self.info["splits"]) * self.M * int(N)

    def _workspace(self, ws, N: int, stream):
        """(pointer, floats) of the caller's workspace, or of one allocated here from torch's
        caching allocator; such a block is tied to `stream` so that it is not handed out
        again before the call's kernels on that stream have run."""
        import torch
        if ws is None:
            need = self.workspace_floats(N) if int(self.info["splits"]) > 1 else 0
            ws = torch.empty(max(need, 1), device="cuda")
            if stream is not None:
                ws.record_stream(stream)
        if not isinstance(ws, torch.Tensor) or ws.device.type != "cuda" or \
                ws.dtype != torch.float32 or not ws.is_contiguous():
            raise TypeError("workspace must be a contiguous float32 CUDA/HIP tensor")
        return ctypes.c_void_p(ws.data_ptr()), int(ws.numel())

    def spmm_split(self, B, C, bias=None, epi: str = "none", workspace=None, splits: int = 0,
                   stream=None):
        """spmm with runs of a tile's K-segments in separate workgroups (plans created
        with split_chunks > 0); splits: workgroups along K (0: the library's choice);
        workspace: a float32 device tensor of at least workspace_floats(N) elements
        (allocated here when None)."""
        N = int(B.shape[1]) if B is not None and B.dim() == 2 else int(C.shape[1])
        pb = _dev_ptr(B, "B", (self.K, N))
        pc = _dev_ptr(C, "C", (self.M, N))
        pbias = _dev_ptr(bias, "bias", (self.M,), allow_none=True)
        pw, nw = self._workspace(workspace, N, stream)
        _check(self._lib.sdnn_spmm_split(self.handle, pb, pc, N, pbias, EPI[epi], int(splits),
                                         pw, nw, _stream_handle(stream)), "sdnn_spmm_split")
        return C

    def spmm_split_noalloc(self, B, C, bias=None, epi: str = "none", splits: int = 0, stream=None):
        """spmm_split with the partial products in the library's fixed per-device scratch
        (sdnn_spmm_split_noalloc): no workspace, no allocation."""
        N = int(B.shape[1]) if B is not None and B.dim() == 2 else int(C.shape[1])
        pb = _dev_ptr(B, "B", (self.K, N))
        pc = _dev_ptr(C, "C", (self.M, N))
        pbias = _dev_ptr(bias, "bias", (self.M,), allow_none=True)
        _check(self._lib.sdnn_spmm_split_noalloc(self.handle, pb, pc, N, pbias, EPI[epi],
                                                 int(splits), _stream_handle(stream)),
               "sdnn_spmm_split_noalloc")
        return C

    def conv3x3_split(self, X, C, bias=None, epi: str = "none", workspace=None, splits: int = 0,
                      stream=None):
        """conv3x3 with K-segments in separate workgroups (see spmm_split)."""
        if X.dim() != 4 or C.dim() != 4:
            raise ValueError("X and C must be 4-d (channels, H, W, images)")
        IC, H, W, NB = (int(d) for d in X.shape)
        if IC * 9 != self.K:
            raise ValueError(f"X has {IC} channels; the plan's K = {self.K} needs {self.K // 9}")
        px = _dev_ptr(X, "X", (IC, H, W, NB))
        pc = _dev_ptr(C, "C", (self.M, H, W, NB))
        pbias = _dev_ptr(bias, "bias", (self.M,), allow_none=True)
        pw, nw = self._workspace(workspace, H * W * NB, stream)
        _check(self._lib.sdnn_conv3x3_split(self.handle, px, pc, H, W, NB, pbias, EPI[epi],
                                            int(splits), pw, nw, _stream_handle(stream)),
               "sdnn_conv3x3_split")
        return C

    def spmm(self, B, C, bias=None, epi: str = "none", stream=None):
        """C = act(W @ B + bias) on the GPU, enqueued on `stream` (default: current)."""
        N = int(B.shape[1]) if B is not None and B.dim() == 2 else int(C.shape[1])
        pb = _dev_ptr(B, "B", (self.K, N))
        pc = _dev_ptr(C, "C", (self.M, N))
        pbias = _dev_ptr(bias, "bias", (self.M,), allow_none=True)
        code = self._lib.sdnn_spmm(self._h, pb, pc, N, pbias, EPI[epi], _stream_handle(stream))
        if code:
            self.handle  # a closed plan raises here
            raise SdnnError(code, "sdnn_spmm")
        return C

    def close(self):
        if getattr(self, "_h", None) is not None:
            self._lib.sdnn_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()


def dense_gemm(W, B, C, bias=None, epi: str = "none", stream=None):
    """Dense FP32 comparison GEMM: C = act(W @ B + bias) (a measurement aid)."""
    M, K = int(W.shape[0]), int(W.shape[1])
    N = int(B.shape[1])
    pw = _dev_ptr(W, "W", (M, K))
    pb = _dev_ptr(B, "B", (K, N))
    pc = _dev_ptr(C, "C", (M, N))
    pbias = _dev_ptr(bias, "bias", (M,), allow_none=True)
    _check(lib().sdnn_dense_gemm(pw, pb, pc, M, K, N, pbias, EPI[epi], _stream_handle(stream)),
           "sdnn_dense_gemm")
    return C


def status_str(code: int) -> str:
    return lib().sdnn_status_str(code).decode()
