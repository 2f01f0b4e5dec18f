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
           "spmspv_noalloc",
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
        info = _lib.MatrixInfo()
        check(lib().dbs_matrix_info_get(self._h, ctypes.byref(info)))
        self.m, self.n, self.dtype = int(info.m), int(info.n), int(info.dtype)

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
        return self.m, self.n

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            lib().dbs_matrix_destroy(h)
            self._h = None


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


# ---------------------------------------------------------------------------
# Argument checks.  The C ABI takes raw device pointers and trusts the sizes
# and element types it is given, so every tensor is checked here before its
# address is passed on: its device, contiguity, element type and length.  A
# failed check raises DbsError(DBS_ERR_ARG) and nothing is launched.
# ---------------------------------------------------------------------------
def _arg_error(msg):
    return DbsError(_lib.DBS_ERR_ARG, msg)


def _value_dtype(torch, code):
    return {DBS_F32: torch.float32, DBS_F16: torch.float16}.get(code)


def _check_tensor(t, name, dtypes, min_numel, device, ndim=None):
    """One tensor argument: on `device`, contiguous, of one of `dtypes`, with
    at least `min_numel` elements (and `ndim` dimensions if given)."""
    if t is None:
        raise _arg_error(f"{name} is required")
    if t.device != device:
        raise _arg_error(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise _arg_error(f"{name} must be contiguous")
    if t.dtype not in dtypes:
        raise _arg_error(f"{name} has dtype {t.dtype}, expected {' or '.join(str(d) for d in dtypes)}")
    if ndim is not None and t.dim() != ndim:
        raise _arg_error(f"{name} must have {ndim} dimension(s), not {t.dim()}")
    if t.numel() < min_numel:
        raise _arg_error(f"{name} holds {t.numel()} elements, needs at least {min_numel}")


def _mask_dtypes(torch):
    return tuple(d for d in (torch.int32, getattr(torch, "uint32", None)) if d is not None)


def validate_spmspv(torch, m, n, dtype, semiring, device, x_idx, x_val, mask, y_idx, y_val, y_nnz):
    """Checks the tensors of one dbs_spmspv call (see Context.spmspv_raw)."""
    if semiring == DBS_PLUS_TIMES and dtype == DBS_PATTERN:
        raise _arg_error("a pattern matrix takes only the OR-AND semiring")
    k = 0
    if x_idx is not None:
        _check_tensor(x_idx, "x_idx", (torch.int32,), 0, device, ndim=1)
        k = x_idx.numel()
    if semiring == DBS_PLUS_TIMES:
        if k:
            _check_tensor(x_val, "x_val", (_value_dtype(torch, dtype),), k, device, ndim=1)
            if x_val.numel() != k:
                raise _arg_error(f"x_val holds {x_val.numel()} values for {k} indices")
        _check_tensor(y_val, "y_val", (_value_dtype(torch, dtype),), m, device)
    if mask is not None:
        _check_tensor(mask, "mask", _mask_dtypes(torch), (m + 31) // 32, device)
    _check_tensor(y_idx, "y_idx", (torch.int32,), m, device)
    _check_tensor(y_nnz, "y_nnz", (torch.int32,), 1, device)
    return k


def validate_dense(torch, m, n, dtype, device, x, y, y32):
    """Checks the tensors of one dbs_spmspv_dense call."""
    vdt = _value_dtype(torch, dtype)
    if vdt is None:
        raise _arg_error("a dense activation needs an fp32 or fp16 matrix")
    _check_tensor(x, "x", (vdt,), n, device)
    _check_tensor(y, "y", (vdt,), m, device)
    if y32 is not None:
        _check_tensor(y32, "y32", (torch.float32,), m, device)


def validate_spmm(torch, m, n, dtype, device, X, Y, Y32):
    """Checks the tensors of one dbs_spmm_dense call: X is [nb, n] and Y (and
    Y32) [nb, m], row-major."""
    vdt = _value_dtype(torch, dtype)
    if vdt is None:
        raise _arg_error("a dense activation needs an fp32 or fp16 matrix")
    _check_tensor(X, "X", (vdt,), 0, device, ndim=2)
    nb = int(X.shape[0])
    if not 1 <= nb <= _lib.DBS_MAX_BATCH:
        raise _arg_error(f"batch of {nb} activations, supported 1..{_lib.DBS_MAX_BATCH}")
    if int(X.shape[1]) != n:
        raise _arg_error(f"X has {X.shape[1]} columns, the matrix {n}")
    for t, name, dt in ((Y, "Y", vdt), (Y32, "Y32", torch.float32)):
        if t is None and name == "Y32":
            continue
        _check_tensor(t, name, (dt,), nb * m, device, ndim=2)
        if m and (int(t.shape[0]) != nb or int(t.shape[1]) != m):
            raise _arg_error(f"{name} has shape {tuple(t.shape)}, expected ({nb}, {m})")
    return nb


def validate_bfs(torch, m, n, device, source, level, parent):
    """Checks the tensors of one dbs_bfs call."""
    if m != n:
        raise _arg_error("BFS needs a square matrix")
    if not 0 <= int(source) < n:
        raise _arg_error(f"source {source} outside [0, {n})")
    _check_tensor(level, "level", (torch.int32,), n, device)
    _check_tensor(parent, "parent", (torch.int32,), n, device)


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
        dev = y.device if y is not None else torch.device("cuda", torch.cuda.current_device())
        if dev.type != "cuda":
            raise _arg_error("y must be a device tensor")
        k = 0
        if x_idx is not None:
            _check_tensor(x_idx, "x_idx", (torch.int32,), 0, dev, ndim=1)
            k = int(x_idx.numel())
            _check_tensor(x_val, "x_val", (torch.float32,), k, dev, ndim=1)
        _check_tensor(y, "y", (torch.float32,), self.m, dev)
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
        self.device = torch.device("cuda", torch.cuda.current_device())

    def _check_matrix(self, A):
        if A.m > self.m or A.n > self.n:
            raise _arg_error(f"matrix {A.m}x{A.n} exceeds the context's sizing {self.m}x{self.n}")

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            lib().dbs_ctx_destroy(h)
            self._h = None

    def set_single_launch(self, on: bool = True):
        """Short index lists (<= 2048) as one kernel launch (default off)."""
        check(lib().dbs_ctx_set_single_launch(self._h, 1 if on else 0))

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
        """All arguments are preallocated torch CUDA tensors on the context's
        device (or None): x_idx int32 [k], x_val [k] in A's value type (None
        for OR-AND), mask int32/uint32 of at least ceil(m/32) words, y_idx
        int32 and y_val (A's value type; None for OR-AND) of at least m
        entries, y_nnz int32 [1]."""
        self._check_matrix(A)
        k = validate_spmspv(self._torch, A.m, A.n, A.dtype, semiring, self.device, x_idx, x_val, mask,
                            y_idx, y_val, y_nnz)
        st = _lib.CallStats() if stats else None
        check(lib().dbs_spmspv(self._h, A._h, semiring, k, _ptr(x_idx), _ptr(x_val), _ptr(mask),
                               1 if complement else 0, PATHS[path], float(th3), _ptr(y_idx),
                               _ptr(y_val), _ptr(y_nnz), ctypes.byref(st) if st is not None else None))
        return _stats_dict(st) if st is not None else None

    def spmspv(self, A: Matrix, x_idx, x_val=None, semiring="plus_times", mask=None,
               complement=False, path="auto", th3=0.0, stats=False):
        """Returns (y_idx, y_val or None[, stats]) as CUDA tensors trimmed to nnz(y)."""
        torch = self._torch
        m = A.m
        sr = DBS_OR_AND if semiring in ("or_and", DBS_OR_AND) else DBS_PLUS_TIMES
        dev = self.device
        y_idx = torch.empty(max(m, 1), dtype=torch.int32, device=dev)
        y_val = None
        if sr == DBS_PLUS_TIMES:
            y_val = torch.empty(max(m, 1), dtype=torch.float16 if A.dtype == DBS_F16 else torch.float32,
                                device=dev)
        y_nnz = torch.zeros(1, dtype=torch.int32, device=dev)
        st = self.spmspv_raw(A, x_idx, x_val, y_idx, y_val, y_nnz, sr, mask, complement, path, th3, stats)
        cnt = int(y_nnz.item())
        out = (y_idx[:cnt], None if y_val is None else y_val[:cnt])
        return (*out, st) if stats else out

    def spmspv_dense(self, A: Matrix, x, path="auto", th3=0.0, y=None, y32=None, stats=False):
        """Dense activation (active iff nonzero); returns y (and y32 if given)."""
        torch = self._torch
        self._check_matrix(A)
        m = A.m
        if y is None and x is not None:
            y = torch.empty(max(m, 1), dtype=x.dtype, device=x.device)
        validate_dense(torch, m, A.n, A.dtype, self.device, x, y, y32)
        st = _lib.CallStats() if stats else None
        check(lib().dbs_spmspv_dense(self._h, A._h, _ptr(x), PATHS[path], float(th3), _ptr(y), _ptr(y32),
                                     ctypes.byref(st) if st is not None else None))
        return (y[:m], _stats_dict(st)) if stats else y[:m]

    def spmm_dense(self, A: Matrix, X, Y=None, Y32=None, stats=False):
        """Batched dense activations X [nb, n] (active iff nonzero); returns Y [nb, m]."""
        torch = self._torch
        self._check_matrix(A)
        m, n = A.shape
        if Y is None and X is not None and X.dim() == 2:
            Y = torch.empty((int(X.shape[0]), max(m, 1)), dtype=X.dtype, device=X.device)
        nb = validate_spmm(torch, m, n, A.dtype, self.device, X, Y, Y32)
        st = _lib.CallStats() if stats else None
        check(lib().dbs_spmm_dense(self._h, A._h, nb, _ptr(X), _ptr(Y), _ptr(Y32),
                                   ctypes.byref(st) if st is not None else None))
        return (Y, _stats_dict(st)) if stats else Y

    def bfs(self, A: Matrix, source: int, policy="auto", th3=0.0, level=None, parent=None, stats=False):
        torch = self._torch
        self._check_matrix(A)
        m, n = A.shape
        dev = self.device
        if level is None:
            level = torch.empty(max(n, 1), dtype=torch.int32, device=dev)
        if parent is None:
            parent = torch.empty(max(n, 1), dtype=torch.int32, device=dev)
        validate_bfs(torch, m, n, dev, source, level, parent)
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


def spmspv_noalloc(A: Matrix, x_idx, x_val=None, semiring="plus_times", mask=None, complement=False,
                   path="auto", th3=0.0, y_idx=None, y_val=None, y_nnz=None, stream=None):
    """y = A x through dbs_spmspv_noalloc: no context, no device allocation
    in the library (its scratch is a static device array; calls on one GPU
    must not overlap).  Outputs may be preallocated (y_idx int32 and y_val of
    at least m entries, y_nnz int32 [1]); returns (y_idx, y_val or None)
    trimmed to nnz(y), which reads y_nnz back (a synchronization)."""
    import torch
    dev = torch.device("cuda", torch.cuda.current_device())
    m = A.m
    sr = DBS_OR_AND if semiring in ("or_and", DBS_OR_AND) else DBS_PLUS_TIMES
    if y_idx is None:
        y_idx = torch.empty(max(m, 1), dtype=torch.int32, device=dev)
    if y_val is None and sr == DBS_PLUS_TIMES:
        y_val = torch.empty(max(m, 1), dtype=torch.float16 if A.dtype == DBS_F16 else torch.float32, device=dev)
    if y_nnz is None:
        y_nnz = torch.zeros(1, dtype=torch.int32, device=dev)
    if sr == DBS_OR_AND:
        y_val = None
    k = validate_spmspv(torch, A.m, A.n, A.dtype, sr, dev, x_idx, x_val, mask, y_idx, y_val, y_nnz)
    st = (stream or torch.cuda.current_stream()).cuda_stream
    check(lib().dbs_spmspv_noalloc(A._h, sr, k, _ptr(x_idx), _ptr(x_val), _ptr(mask), 1 if complement else 0,
                                   PATHS[path], float(th3), _ptr(y_idx), _ptr(y_val), _ptr(y_nnz),
                                   ctypes.c_void_p(st)))
    cnt = int(y_nnz.item())
    return y_idx[:cnt], None if y_val is None else y_val[:cnt]


def _stats_dict(st: _lib.CallStats) -> dict:
    return {"path": PATH_NAMES.get(st.path, "?"), "n_nzblk": st.n_nzblk, "n_blk": st.n_blk,
            "y_nnz": st.y_nnz, "tasks": st.tasks, "error_flags": st.error_flags}
