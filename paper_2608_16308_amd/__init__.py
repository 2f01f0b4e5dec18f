"""MI355X (gfx950) dual-view blocked SpMSpV -- Python binding.

Thin marshalling over the C ABI of ``libdbspmspv.so`` (``include/dbspmspv.h``):
every step of the computation runs in the library's HIP kernels (or, for the
offline conversion, its C++ builder).  PyTorch supplies device memory and the
current stream only.

    hm = HostMatrix.from_csr(m, n, row_ptr, col_idx, vals)   # CPU-only conversion
    A = Matrix.upload(hm)                                     # or Matrix.from_csr(...)
    ctx = Context(A)
    y_idx, y_val = ctx.spmspv(A, x_idx, x_val)                # torch CUDA tensors
    y16 = ctx.spmspv_dense(A, a16)                            # decode layer
    level, parent = ctx.bfs(A, source)
"""
from __future__ import annotations

import ctypes

import numpy as np

from . import _lib
from ._lib import (BLOCK_TYPE_NAMES, DBS_F16, DBS_F32, DBS_OR_AND, DBS_PATH_AUTO, DBS_PATH_PULL,
                   DBS_PATH_PUSH, DBS_PATTERN, DBS_PLUS_TIMES, DbsError, check)

__all__ = ["HostMatrix", "Matrix", "Context", "BasicMatrix", "DbsError", "default_opts", "storage_model",
           "DBS_F32", "DBS_F16", "DBS_PATTERN", "PATHS"]

PATHS = {"auto": DBS_PATH_AUTO, "push": DBS_PATH_PUSH, "pull": DBS_PATH_PULL}
PATH_NAMES = {DBS_PATH_PUSH: "push", DBS_PATH_PULL: "pull"}


def lib():
    return _lib.load()


def default_opts(**overrides) -> _lib.BuildOpts:
    o = _lib.BuildOpts()
    lib().dbs_build_opts_default(ctypes.byref(o))
    for k, v in overrides.items():
        setattr(o, k, v)
    return o


def storage_model(rows: int, cols: int, nnz: int, value_bytes: int):
    a, b = ctypes.c_int64(), ctypes.c_int64()
    check(lib().dbs_storage_model(rows, cols, nnz, value_bytes, ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


def _dtype_code(vals):
    if vals is None:
        return DBS_PATTERN, None
    v = np.ascontiguousarray(vals)
    if v.dtype == np.float32:
        return DBS_F32, v
    if v.dtype == np.float16:
        return DBS_F16, v
    raise TypeError(f"unsupported value dtype {v.dtype}")


def _info_dict(info: _lib.MatrixInfo) -> dict:
    d = {f: getattr(info, f) for f, _ in info._fields_ if f != "blocks_by_type"}
    d["blocks_by_type"] = {BLOCK_TYPE_NAMES[t]: int(info.blocks_by_type[t]) for t in range(5)}
    return d


class HostMatrix:
    """The DB format in host memory (offline conversion; no GPU needed)."""

    def __init__(self, handle):
        self._h = ctypes.c_void_p(handle)

    @classmethod
    def from_csr(cls, m, n, row_ptr, col_idx, vals=None, opts: _lib.BuildOpts | None = None):
        row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int64)
        col_idx = np.ascontiguousarray(col_idx, dtype=np.int32)
        code, v = _dtype_code(vals)
        out = ctypes.c_void_p()
        check(lib().dbs_host_build_csr(int(m), int(n), int(row_ptr[-1]), row_ptr.ctypes.data,
                                       col_idx.ctypes.data, None if v is None else v.ctypes.data,
                                       code, ctypes.byref(opts) if opts is not None else None,
                                       ctypes.byref(out)))
        return cls(out.value)

    def info(self) -> dict:
        info = _lib.MatrixInfo()
        check(lib().dbs_host_info(self._h, ctypes.byref(info)))
        return _info_dict(info)

    def arrays(self) -> dict:
        """Copies of the host arrays (see the layout in include/dbspmspv.h)."""
        info = self.info()
        a = _lib.HostArrays()
        check(lib().dbs_host_arrays_get(self._h, ctypes.byref(a)))

        def cp(ptr, count, dt):
            if count == 0:
                return np.zeros(0, dtype=dt)
            return np.ctypeslib.as_array(ptr, shape=(count,)).astype(dt, copy=True)

        nblk, nbr, nbc = info["nblk"], info["nbr"], info["nbc"]
        return {
            "rb_ptr": cp(a.rb_ptr, nbr + 1, np.int32),
            "cb_col": cp(a.cb_col, nblk, np.int32),
            "cb_ptr": cp(a.cb_ptr, nbc + 1, np.int32),
            "csc_row": cp(a.csc_row, nblk, np.int32),
            "csc2csr": cp(a.csc2csr, nblk, np.int32),
            "desc": cp(a.desc, nblk, np.uint64),
            "payload": cp(a.payload, a.payload_bytes, np.uint8),
            "seg": cp(a.seg, a.nseg, np.uint64),
        }

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            lib().dbs_host_destroy(h)
            self._h = None


class Matrix:
    """The DB format resident on the current GPU."""

    def __init__(self, handle):
        self._h = ctypes.c_void_p(handle)

    @classmethod
    def upload(cls, hm: HostMatrix):
        out = ctypes.c_void_p()
        check(lib().dbs_matrix_upload(hm._h, ctypes.byref(out)))
        return cls(out.value)

    @classmethod
    def from_csr(cls, m, n, row_ptr, col_idx, vals=None, opts=None):
        return cls.upload(HostMatrix.from_csr(m, n, row_ptr, col_idx, vals, opts))

    @classmethod
    def from_dense(cls, w, opts=None, stream=None):
        """GPU-side conversion of a dense 2-D torch tensor on the device
        (float32 or float16, unit column stride): entries are stored iff
        nonzero.  Runs on `stream` (a torch stream; default: the current one)
        and returns when done."""
        import torch
        if w.dim() != 2 or not w.is_cuda or w.stride(1) != 1:
            raise ValueError("from_dense takes a 2-D device tensor with unit column stride")
        if w.dtype == torch.float32:
            code = DBS_F32
        elif w.dtype == torch.float16:
            code = DBS_F16
        else:
            raise ValueError(f"from_dense takes float32 or float16, not {w.dtype}")
        st = torch.cuda.current_stream(w.device) if stream is None else stream
        out = ctypes.c_void_p()
        m, n = w.shape
        check(lib().dbs_matrix_build_dense(m, n, ctypes.c_void_p(w.data_ptr()), w.stride(0) if m > 0 else n, code,
                                           ctypes.byref(opts) if opts is not None else None,
                                           ctypes.c_void_p(st.cuda_stream), ctypes.byref(out)))
        return cls(out.value)

    def info(self) -> dict:
        info = _lib.MatrixInfo()
        check(lib().dbs_matrix_info_get(self._h, ctypes.byref(info)))
        return _info_dict(info)

    def download(self) -> dict:
        """Host copies of the device arrays (for inspection and tests)."""
        lay = _lib.MatrixLayout()
        check(lib().dbs_matrix_layout_get(self._h, ctypes.byref(lay)))
        arr = {
            "sl_col": np.empty(lay.nslots, np.int32), "sl_desc": np.empty(lay.nslots, np.uint64),
            "seg_rs": np.empty(lay.nseg, np.uint32), "cb_ptr": np.empty(lay.nbc + 1, np.int32),
            "csc_row": np.empty(lay.nblk, np.int32), "csc_desc": np.empty(lay.nblk, np.uint64),
            "hv_col": np.empty(lay.nheavy, np.int32), "hv_desc": np.empty(lay.nheavy, np.uint64),
            "hv_cstart": np.empty(lay.nchunk + 1, np.int32), "hv_crow": np.empty(lay.nchunk, np.int32),
            "payload": np.empty(lay.payload_bytes, np.uint8),
        }
        ptrs = _lib.MatrixArrays(**{k: (v.ctypes.data_as(ctypes.c_void_p) if v.size else None)
                                    for k, v in arr.items()})
        check(lib().dbs_matrix_download(self._h, ctypes.byref(ptrs)))
        return arr

    @property
    def shape(self):
        i = self.info()
        return i["m"], i["n"]

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            lib().dbs_matrix_destroy(h)
            self._h = None


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


class BasicMatrix:
    """Plain CSR + CSC copies of an fp32 matrix on the current GPU for the
    basic push and pull of Alg. 1 (comparison baselines only)."""

    def __init__(self, m, n, row_ptr, col_idx, vals):
        rp = np.ascontiguousarray(row_ptr, dtype=np.int64)
        ci = np.ascontiguousarray(col_idx, dtype=np.int32)
        va = np.ascontiguousarray(vals, dtype=np.float32)
        out = ctypes.c_void_p()
        check(lib().dbs_basic_build(int(m), int(n), int(rp[-1]), rp.ctypes.data, ci.ctypes.data,
                                    va.ctypes.data, ctypes.byref(out)))
        self._h = out
        self.m, self.n = int(m), int(n)

    def spmspv(self, path, x_idx, x_val, y, stream=None):
        """Dense fp32 y[m] = A x by "push" or "pull" (torch CUDA tensors)."""
        import torch
        s = (stream or torch.cuda.current_stream()).cuda_stream
        k = 0 if x_idx is None else int(x_idx.numel())
        check(lib().dbs_basic_spmspv(self._h, PATHS[path], k, _ptr(x_idx), _ptr(x_val), _ptr(y),
                                     ctypes.c_void_p(s)))
        return y

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            lib().dbs_basic_destroy(h)
            self._h = None


class Context:
    """Per-stream workspace; runs SpMSpV, dense-activation SpMSpV and BFS."""

    def __init__(self, sizing: Matrix, stream=None):
        import torch
        self._torch = torch
        if stream is None:
            stream = torch.cuda.current_stream()
        self.stream = stream
        out = ctypes.c_void_p()
        check(lib().dbs_ctx_create(sizing._h, ctypes.c_void_p(stream.cuda_stream), ctypes.byref(out)))
        self._h = out
        self.m, self.n = sizing.shape

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            lib().dbs_ctx_destroy(h)
            self._h = None

    # -- measurement hooks
    def enable_timing(self, on: bool = True):
        check(lib().dbs_ctx_enable_timing(self._h, 1 if on else 0))

    def read_timing(self) -> dict:
        t = _lib.Timing()
        check(lib().dbs_ctx_read_timing(self._h, ctypes.byref(t)))
        return {name: (t.ms[k], int(t.launches[k])) for k, name in enumerate(_lib.DBS_K_NAMES)}

    # -- y = A x
    def spmspv_raw(self, A: Matrix, x_idx, x_val, y_idx, y_val, y_nnz, semiring=DBS_PLUS_TIMES,
                   mask=None, complement=False, path="auto", th3=0.0, stats=False):
        """All arguments are preallocated torch CUDA tensors (or None)."""
        st = _lib.CallStats() if stats else None
        k = 0 if x_idx is None else int(x_idx.numel())
        check(lib().dbs_spmspv(self._h, A._h, semiring, k, _ptr(x_idx), _ptr(x_val), _ptr(mask),
                               1 if complement else 0, PATHS[path], float(th3), _ptr(y_idx),
                               _ptr(y_val), _ptr(y_nnz), ctypes.byref(st) if st is not None else None))
        return _stats_dict(st) if st is not None else None

    def spmspv(self, A: Matrix, x_idx, x_val=None, semiring="plus_times", mask=None,
               complement=False, path="auto", th3=0.0, stats=False):
        """Returns (y_idx, y_val or None[, stats]) as CUDA tensors trimmed to nnz(y)."""
        torch = self._torch
        m, _ = A.shape
        info_dtype = A.info()["dtype"]
        sr = DBS_OR_AND if semiring in ("or_and", DBS_OR_AND) else DBS_PLUS_TIMES
        dev = x_idx.device
        y_idx = torch.empty(max(m, 1), dtype=torch.int32, device=dev)
        y_val = None
        if sr == DBS_PLUS_TIMES:
            y_val = torch.empty(max(m, 1), dtype=torch.float16 if info_dtype == DBS_F16 else torch.float32,
                                device=dev)
        y_nnz = torch.zeros(1, dtype=torch.int32, device=dev)
        st = self.spmspv_raw(A, x_idx, x_val, y_idx, y_val, y_nnz, sr, mask, complement, path, th3, stats)
        cnt = int(y_nnz.item())
        out = (y_idx[:cnt], None if y_val is None else y_val[:cnt])
        return (*out, st) if stats else out

    def spmspv_dense(self, A: Matrix, x, path="auto", th3=0.0, y=None, y32=None, stats=False):
        """Dense activation (active iff nonzero); returns y (and y32 if given)."""
        torch = self._torch
        m, _ = A.shape
        if y is None:
            y = torch.empty(max(m, 1), dtype=x.dtype, device=x.device)
        st = _lib.CallStats() if stats else None
        check(lib().dbs_spmspv_dense(self._h, A._h, _ptr(x), PATHS[path], float(th3), _ptr(y), _ptr(y32),
                                     ctypes.byref(st) if st is not None else None))
        return (y[:m], _stats_dict(st)) if stats else y[:m]

    def spmm_dense(self, A: Matrix, X, Y=None, Y32=None, stats=False):
        """Batched dense activations X [nb, n] (active iff nonzero); returns Y [nb, m]."""
        torch = self._torch
        m, n = A.shape
        nb = int(X.shape[0])
        if Y is None:
            Y = torch.empty((nb, max(m, 1)), dtype=X.dtype, device=X.device)
        st = _lib.CallStats() if stats else None
        check(lib().dbs_spmm_dense(self._h, A._h, nb, _ptr(X), _ptr(Y), _ptr(Y32),
                                   ctypes.byref(st) if st is not None else None))
        return (Y, _stats_dict(st)) if stats else Y

    def bfs(self, A: Matrix, source: int, policy="auto", th3=0.0, level=None, parent=None, stats=False):
        torch = self._torch
        m, n = A.shape
        dev = torch.device("cuda", torch.cuda.current_device())
        if level is None:
            level = torch.empty(max(n, 1), dtype=torch.int32, device=dev)
        if parent is None:
            parent = torch.empty(max(n, 1), dtype=torch.int32, device=dev)
        st = _lib.BfsStats() if stats else None
        check(lib().dbs_bfs(self._h, A._h, int(source), _ptr(level), _ptr(parent), PATHS[policy],
                            float(th3), ctypes.byref(st) if st is not None else None))
        if stats:
            L = st.levels
            s = {"levels": L, "reached": st.reached,
                 "path": [PATH_NAMES.get(st.path[i], "?") for i in range(min(L, 64))],
                 "frontier": [int(st.frontier[i]) for i in range(min(L, 64))]}
            return level[:n], parent[:n], s
        return level[:n], parent[:n]


def _stats_dict(st: _lib.CallStats) -> dict:
    return {"path": PATH_NAMES.get(st.path, "?"), "n_nzblk": st.n_nzblk, "n_blk": st.n_blk,
            "y_nnz": st.y_nnz, "tasks": st.tasks, "error_flags": st.error_flags}
