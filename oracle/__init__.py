"""Plain CPU oracle for DB-SpMSpV: TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The GPU library never loads it, and it
imports nothing from the GPU package: the two sides only share the seeded
input generators in ``workloads``.

What it computes (DB-SpMSpV paper):

* ``OracleMatrix.spmspv``  -- y = A x, A and x sparse, plus-times semiring,
  following the push form of Alg. 1 (Sec. 2.1) as a sequential column gather
  into a dense fp64 accumulator.  The y pattern is structural (every row with a
  stored A[i][j] at a listed j, minus rows excluded by the output mask), sorted
  ascending; also returns S_i = sum |A[i][j] x_j| for the tolerance.
* ``OracleMatrix.spmspv_bool`` -- the same pattern under the Boolean OR-AND
  semiring (values ignored), as used per level by DB-BFS (Sec. 4.2).
* ``OracleMatrix.bfs`` -- level-synchronous BFS (Sec. 4.2, Alg. 5
  semantics): edge u -> v iff A[v][u] is stored; parent[v] is the smallest id
  among level L(v)-1 vertices with an edge to v; unreachable -> -1.
* ``decode_linear`` -- DB-Decoding (Sec. 4.3): y = W a for a dense fp16
  activation a whose entries are active iff nonzero; fp64 sum, then the fp16
  result by round-to-nearest-even.

Readings where the paper is silent (structural pattern, mask bit order,
minimum-id parent, edge direction) are those listed in the design notes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(dtype=np.int64, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(dtype=np.float64, flags="C_CONTIGUOUS")
_u8p = np.ctypeslib.ndpointer(dtype=np.uint8, flags="C_CONTIGUOUS")
_u32p = np.ctypeslib.ndpointer(dtype=np.uint32, flags="C_CONTIGUOUS")


def build(src: str = _SRC, out: str = _LIB) -> str:
    """Compile the oracle with plain gcc (-O2, no fast-math)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-o", out + ".tmp", src]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def _nullable(ptr_type):
    """ndpointer that also accepts None (passed as NULL)."""
    class _P(ptr_type):  # type: ignore[misc, valid-type]
        @classmethod
        def from_param(cls, obj):
            if obj is None:
                return None
            return super().from_param(obj)
    return _P


def load(path: str = _LIB) -> ctypes.CDLL:
    if not os.path.exists(path):
        build(out=path)
    lib = ctypes.CDLL(path)
    lib.oracle_csc_from_csr.restype = ctypes.c_int
    lib.oracle_csc_from_csr.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                        _i64p, _i32p, _nullable(_f64p), _i64p, _i32p,
                                        _nullable(_f64p)]
    lib.oracle_spmspv.restype = ctypes.c_int64
    lib.oracle_spmspv.argtypes = [ctypes.c_int32, ctypes.c_int32, _i64p, _i32p, _f64p,
                                  ctypes.c_int32, _i32p, _f64p, _nullable(_u32p), ctypes.c_int,
                                  _f64p, _f64p, _u8p, _i32p, _i32p, _f64p, _f64p]
    lib.oracle_spmspv_bool.restype = ctypes.c_int64
    lib.oracle_spmspv_bool.argtypes = [ctypes.c_int32, ctypes.c_int32, _i64p, _i32p,
                                       ctypes.c_int32, _i32p, _nullable(_u32p), ctypes.c_int,
                                       _u8p, _i32p]
    lib.oracle_bfs.restype = ctypes.c_int32
    lib.oracle_bfs.argtypes = [ctypes.c_int32, _i64p, _i32p, ctypes.c_int32, _i32p, _i32p,
                               _i32p, _i32p]
    lib.oracle_time_spmspv.restype = ctypes.c_double
    lib.oracle_time_spmspv.argtypes = [ctypes.c_int32, ctypes.c_int32, _i64p, _i32p, _f64p,
                                       ctypes.c_int32, _i64p, _i32p, _f64p, ctypes.c_int32,
                                       _f64p, _f64p, _u8p, _i32p, _i32p, _f64p, _f64p]
    lib.oracle_time_bfs.restype = ctypes.c_double
    lib.oracle_time_bfs.argtypes = [ctypes.c_int32, _i64p, _i32p, ctypes.c_int32, _i32p,
                                    _i32p, _i32p, _i32p, _i32p]
    return lib


_lib_cache: dict[str, ctypes.CDLL] = {}


def _get_lib(path: str | None) -> ctypes.CDLL:
    path = path or _LIB
    if path not in _lib_cache:
        _lib_cache[path] = load(path)
    return _lib_cache[path]


def _check_x(n: int, x_idx: np.ndarray) -> np.ndarray:
    x_idx = np.ascontiguousarray(x_idx, dtype=np.int32)
    if x_idx.size:
        if x_idx.min() < 0 or x_idx.max() >= n:
            raise ValueError("x index out of range")
        if np.unique(x_idx).size != x_idx.size:
            raise ValueError("duplicate x index")
    return x_idx


def _check_mask(m: int, mask):
    if mask is None:
        return None
    mask = np.ascontiguousarray(mask, dtype=np.uint32)
    if mask.size < (m + 31) // 32:
        raise ValueError("mask too short")
    return mask


class OracleMatrix:
    """A held in the oracle's own CSC (counting sort of the input CSR).

    ``vals`` may be None for a pattern-only matrix; fp16/fp32 values are
    widened to fp64, which is exact.
    """

    def __init__(self, m, n, row_ptr, col_idx, vals=None, lib_path: str | None = None):
        self.lib = _get_lib(lib_path)
        self.m, self.n = int(m), int(n)
        row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int64)
        col_idx = np.ascontiguousarray(col_idx, dtype=np.int32)
        nnz = int(row_ptr[-1])
        self.nnz = nnz
        v64 = None if vals is None else np.ascontiguousarray(vals, dtype=np.float64)
        self.col_ptr = np.zeros(self.n + 1, dtype=np.int64)
        self.row_idx = np.zeros(max(nnz, 1), dtype=np.int32)
        self.cvals = None if v64 is None else np.zeros(max(nnz, 1), dtype=np.float64)
        rc = self.lib.oracle_csc_from_csr(self.m, self.n, nnz, row_ptr, col_idx, v64,
                                          self.col_ptr, self.row_idx, self.cvals)
        if rc != 0:
            raise ValueError(f"oracle_csc_from_csr failed ({rc})")
        mm = max(self.m, 1)
        self._acc = np.zeros(mm, dtype=np.float64)
        self._sabs = np.zeros(mm, dtype=np.float64)
        self._seen = np.zeros(mm, dtype=np.uint8)
        self._touched = np.zeros(mm, dtype=np.int32)

    def col_nnz(self, x_idx) -> np.ndarray:
        x_idx = np.asarray(x_idx, dtype=np.int64)
        return self.col_ptr[x_idx + 1] - self.col_ptr[x_idx]

    def spmspv(self, x_idx, x_val, mask=None, complement=False):
        """Returns (y_idx int32 ascending, y_val fp64, S fp64)."""
        if self.cvals is None:
            raise ValueError("pattern matrix: use spmspv_bool")
        x_idx = _check_x(self.n, x_idx)
        x_val = np.ascontiguousarray(x_val, dtype=np.float64)
        assert x_val.shape == x_idx.shape
        mask = _check_mask(self.m, mask)
        mm = max(self.m, 1)
        y_idx = np.zeros(mm, dtype=np.int32)
        y_val = np.zeros(mm, dtype=np.float64)
        y_abs = np.zeros(mm, dtype=np.float64)
        cnt = self.lib.oracle_spmspv(self.m, self.n, self.col_ptr, self.row_idx, self.cvals,
                                     int(x_idx.size), x_idx, x_val, mask, int(bool(complement)),
                                     self._acc, self._sabs, self._seen, self._touched,
                                     y_idx, y_val, y_abs)
        if cnt < 0:
            raise ValueError("oracle_spmspv failed")
        return y_idx[:cnt].copy(), y_val[:cnt].copy(), y_abs[:cnt].copy()

    def spmspv_bool(self, x_idx, mask=None, complement=False):
        """Returns y_idx (int32, ascending) under OR-AND."""
        x_idx = _check_x(self.n, x_idx)
        mask = _check_mask(self.m, mask)
        y_idx = np.zeros(max(self.m, 1), dtype=np.int32)
        cnt = self.lib.oracle_spmspv_bool(self.m, self.n, self.col_ptr, self.row_idx,
                                          int(x_idx.size), x_idx, mask, int(bool(complement)),
                                          self._seen, y_idx)
        if cnt < 0:
            raise ValueError("oracle_spmspv_bool failed")
        return y_idx[:cnt].copy()

    def bfs(self, source: int):
        """Returns (level int32[n], parent int32[n], number of nonempty levels)."""
        if self.m != self.n:
            raise ValueError("BFS needs a square matrix")
        nn = max(self.n, 1)
        level = np.zeros(nn, dtype=np.int32)
        parent = np.zeros(nn, dtype=np.int32)
        f = np.zeros(nn, dtype=np.int32)
        g = np.zeros(nn, dtype=np.int32)
        nl = self.lib.oracle_bfs(self.n, self.col_ptr, self.row_idx, int(source), level, parent, f, g)
        if nl < 0:
            raise ValueError("bad BFS source")
        return level[: self.n], parent[: self.n], int(nl)

    # ---- timing helpers for the CPU baseline (single thread) ----
    def time_spmspv(self, xs, reps: int) -> float:
        """Seconds for `reps` passes over the list of (x_idx, x_val) pairs."""
        offs = np.zeros(len(xs) + 1, dtype=np.int64)
        for i, (xi, _) in enumerate(xs):
            offs[i + 1] = offs[i] + len(xi)
        idx = np.ascontiguousarray(np.concatenate([_check_x(self.n, xi) for xi, _ in xs]), dtype=np.int32)
        val = np.ascontiguousarray(np.concatenate([np.asarray(xv, dtype=np.float64) for _, xv in xs]))
        mm = max(self.m, 1)
        y_idx = np.zeros(mm, dtype=np.int32)
        y_val = np.zeros(mm, dtype=np.float64)
        y_abs = np.zeros(mm, dtype=np.float64)
        return float(self.lib.oracle_time_spmspv(self.m, self.n, self.col_ptr, self.row_idx, self.cvals,
                                                 len(xs), offs, idx, val, int(reps),
                                                 self._acc, self._sabs, self._seen, self._touched,
                                                 y_idx, y_val, y_abs))

    def time_bfs(self, sources) -> float:
        src = np.ascontiguousarray(sources, dtype=np.int32)
        nn = max(self.n, 1)
        bufs = [np.zeros(nn, dtype=np.int32) for _ in range(4)]
        return float(self.lib.oracle_time_bfs(self.n, self.col_ptr, self.row_idx, int(src.size), src, *bufs))


def decode_linear(W: OracleMatrix, a_f16: np.ndarray):
    """DB-Decoding reference: y = W a, a dense fp16 activation.

    Entries of ``a`` are active iff nonzero (+0 and -0 inactive).  Returns
    (y64 dense fp64 [m], S dense fp64 [m], y16 = fp16 RNE of y64).
    """
    a = np.asarray(a_f16, dtype=np.float16)
    assert a.shape == (W.n,)
    idx = np.nonzero(a != 0)[0].astype(np.int32)
    y_idx, y_val, y_abs = W.spmspv(idx, a[idx].astype(np.float64))
    y64 = np.zeros(W.m, dtype=np.float64)
    S = np.zeros(W.m, dtype=np.float64)
    y64[y_idx] = y_val
    S[y_idx] = y_abs
    return y64, S, y64.astype(np.float16)


def within_tol(y_gpu, y_ref, S, rel: float = 1e-5) -> np.ndarray:
    """Element-wise acceptance of computed values against the oracle's.

    The method reaches the plain sum of products, but accumulates it in a
    different order and precision than the oracle's fp64 sum, so a value is
    accepted iff |y_gpu - y_ref| <= rel * S, S = sum_j |a_ij x_j| of its row:
    the rounding error of any summation order is bounded by that sum.  Hence

    * S == 0 demands an exact match (a row whose every product is zero);
    * the bound applies only to a finite reference: an infinite one (an
      infinite input) demands the same infinity;
    * a NaN result is accepted only where the reference is NaN too (a NaN
      input value reaches every row it multiplies), and a NaN reference
      demands a NaN result;
    * equal values are accepted (infinities of one sign);
    * the three arrays must have one shape; the result has that shape.
    """
    g = np.asarray(y_gpu, dtype=np.float64)
    r = np.asarray(y_ref, dtype=np.float64)
    s = np.asarray(S, dtype=np.float64)
    if g.shape != r.shape or g.shape != s.shape:
        raise ValueError(f"within_tol: shapes differ {g.shape} {r.shape} {s.shape}")
    with np.errstate(invalid="ignore"):
        close = np.isfinite(r) & (np.abs(g - r) <= rel * s)
        same = g == r
    both_nan = np.isnan(g) & np.isnan(r)
    return close | same | both_nan
