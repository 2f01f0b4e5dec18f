"""ctypes declarations of the C ABI in ``include/dbspmspv.h``.

Argument marshalling only.  The shared library is required: importing the
package without a built ``libdbspmspv.so`` raises, there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdbspmspv.so")

DBS_OK, DBS_ERR_ARG, DBS_ERR_ALLOC, DBS_ERR_DEVICE, DBS_ERR_UNSUPPORTED, DBS_ERR_STATE = range(6)
DBS_F32, DBS_F16, DBS_PATTERN = 0, 1, 2
DBS_PLUS_TIMES, DBS_OR_AND = 0, 1
DBS_PATH_AUTO, DBS_PATH_PUSH, DBS_PATH_PULL = 0, 1, 2
DBS_BLK_COO, DBS_BLK_DENSE, DBS_BLK_FCSR, DBS_BLK_FCSC, DBS_BLK_CSR = range(5)
BLOCK_TYPE_NAMES = ["coo", "dense", "fcsr", "fcsc", "csr"]
DBS_K_NAMES = ["scatter", "scan", "main", "finalize", "bfs_update", "other", "fused"]
DBS_BFS_MAX_LEVEL_STATS = 64
DBS_MAX_BATCH = 8

EXPORTED = [
    "dbs_build_opts_default", "dbs_host_build_csr", "dbs_host_info", "dbs_host_arrays_get",
    "dbs_host_destroy", "dbs_storage_model", "dbs_matrix_upload", "dbs_matrix_build_csr",
    "dbs_matrix_info_get", "dbs_matrix_destroy", "dbs_ctx_create", "dbs_ctx_set_stream",
    "dbs_ctx_destroy", "dbs_spmspv", "dbs_spmspv_dense", "dbs_spmm_dense", "dbs_bfs", "dbs_ctx_enable_timing",
    "dbs_ctx_read_timing", "dbs_last_error", "dbs_version", "dbs_basic_build", "dbs_basic_destroy",
    "dbs_basic_spmspv", "dbs_matrix_build_dense", "dbs_matrix_layout_get", "dbs_matrix_download",
    "dbs_spmspv_noalloc", "dbs_ctx_set_single_launch",
]
DBS_NOALLOC_MAX_DIM = 1 << 20


class BuildOpts(ctypes.Structure):
    _fields_ = [("th0", ctypes.c_int32), ("th1", ctypes.c_int32), ("th2", ctypes.c_float),
                ("seg_close", ctypes.c_int32), ("force_type", ctypes.c_int32),
                ("inline_small", ctypes.c_int32)]


class MatrixInfo(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int32), ("n", ctypes.c_int32), ("nnz", ctypes.c_int64),
                ("dtype", ctypes.c_int32), ("nbr", ctypes.c_int32), ("nbc", ctypes.c_int32),
                ("nblk", ctypes.c_int64), ("nseg", ctypes.c_int64),
                ("blocks_by_type", ctypes.c_int64 * 5), ("payload_bytes", ctypes.c_int64),
                ("db_bytes", ctypes.c_int64), ("csr_bytes", ctypes.c_int64),
                ("csr_csc_bytes", ctypes.c_int64)]


class HostArrays(ctypes.Structure):
    _fields_ = [("rb_ptr", ctypes.POINTER(ctypes.c_int32)), ("cb_col", ctypes.POINTER(ctypes.c_int32)),
                ("cb_ptr", ctypes.POINTER(ctypes.c_int32)), ("csc_row", ctypes.POINTER(ctypes.c_int32)),
                ("csc2csr", ctypes.POINTER(ctypes.c_int32)), ("desc", ctypes.POINTER(ctypes.c_uint64)),
                ("payload", ctypes.POINTER(ctypes.c_uint8)), ("payload_bytes", ctypes.c_int64),
                ("seg", ctypes.POINTER(ctypes.c_uint64)), ("nseg", ctypes.c_int64)]


class MatrixLayout(ctypes.Structure):
    _fields_ = [("nslots", ctypes.c_int64), ("nseg", ctypes.c_int64), ("nblk", ctypes.c_int64),
                ("nbc", ctypes.c_int32), ("reserved", ctypes.c_int32), ("nheavy", ctypes.c_int64),
                ("nchunk", ctypes.c_int64), ("payload_bytes", ctypes.c_int64)]


class MatrixArrays(ctypes.Structure):
    _fields_ = [("sl_col", ctypes.c_void_p), ("sl_desc", ctypes.c_void_p), ("seg_rs", ctypes.c_void_p),
                ("cb_ptr", ctypes.c_void_p), ("csc_row", ctypes.c_void_p), ("csc_desc", ctypes.c_void_p),
                ("hv_col", ctypes.c_void_p), ("hv_desc", ctypes.c_void_p), ("hv_cstart", ctypes.c_void_p),
                ("hv_crow", ctypes.c_void_p), ("payload", ctypes.c_void_p)]


class CallStats(ctypes.Structure):
    _fields_ = [("path", ctypes.c_int32), ("n_nzblk", ctypes.c_int32), ("n_blk", ctypes.c_int32),
                ("y_nnz", ctypes.c_int32), ("tasks", ctypes.c_int64), ("error_flags", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class BfsStats(ctypes.Structure):
    _fields_ = [("levels", ctypes.c_int32), ("reached", ctypes.c_int32),
                ("path", ctypes.c_int32 * DBS_BFS_MAX_LEVEL_STATS),
                ("frontier", ctypes.c_int32 * DBS_BFS_MAX_LEVEL_STATS)]


class Timing(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double * 7), ("launches", ctypes.c_int64 * 7)]


class DbsError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"dbs status {status}: {msg}")
        self.status = status


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run __graft_entry__.build() (no CPU fallback exists)")
    # torch ships its own HIP runtime (same soname as the system one).  Load it
    # first so that this library binds to it: device pointers and streams
    # from torch must belong to the runtime the library calls, and a second
    # runtime in the process would hide the GPU from torch.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    vp, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    P = ctypes.POINTER
    sig = {
        "dbs_build_opts_default": (None, [P(BuildOpts)]),
        "dbs_host_build_csr": (ctypes.c_int, [i32, i32, i64, vp, vp, vp, ctypes.c_int, P(BuildOpts), P(vp)]),
        "dbs_host_info": (ctypes.c_int, [vp, P(MatrixInfo)]),
        "dbs_host_arrays_get": (ctypes.c_int, [vp, P(HostArrays)]),
        "dbs_host_destroy": (None, [vp]),
        "dbs_storage_model": (ctypes.c_int, [i64, i64, i64, i32, P(i64), P(i64)]),
        "dbs_matrix_upload": (ctypes.c_int, [vp, P(vp)]),
        "dbs_matrix_build_csr": (ctypes.c_int, [i32, i32, i64, vp, vp, vp, ctypes.c_int, P(BuildOpts), P(vp)]),
        "dbs_matrix_info_get": (ctypes.c_int, [vp, P(MatrixInfo)]),
        "dbs_matrix_build_dense": (ctypes.c_int, [i32, i32, vp, i64, ctypes.c_int, P(BuildOpts), vp, P(vp)]),
        "dbs_matrix_layout_get": (ctypes.c_int, [vp, P(MatrixLayout)]),
        "dbs_matrix_download": (ctypes.c_int, [vp, P(MatrixArrays)]),
        "dbs_matrix_destroy": (None, [vp]),
        "dbs_ctx_create": (ctypes.c_int, [vp, vp, P(vp)]),
        "dbs_ctx_set_stream": (ctypes.c_int, [vp, vp]),
        "dbs_ctx_destroy": (None, [vp]),
        "dbs_spmspv": (ctypes.c_int, [vp, vp, ctypes.c_int, i32, vp, vp, vp, ctypes.c_int, ctypes.c_int,
                                      f32, vp, vp, vp, P(CallStats)]),
        "dbs_spmspv_noalloc": (ctypes.c_int, [vp, ctypes.c_int, i32, vp, vp, vp, ctypes.c_int, ctypes.c_int, f32,
                                              vp, vp, vp, vp]),
        "dbs_spmspv_dense": (ctypes.c_int, [vp, vp, vp, ctypes.c_int, f32, vp, vp, P(CallStats)]),
        "dbs_spmm_dense": (ctypes.c_int, [vp, vp, i32, vp, vp, vp, P(CallStats)]),
        "dbs_bfs": (ctypes.c_int, [vp, vp, i32, vp, vp, ctypes.c_int, f32, P(BfsStats)]),
        "dbs_ctx_enable_timing": (ctypes.c_int, [vp, ctypes.c_int]),
        "dbs_ctx_set_single_launch": (ctypes.c_int, [vp, ctypes.c_int]),
        "dbs_ctx_read_timing": (ctypes.c_int, [vp, P(Timing)]),
        "dbs_basic_build": (ctypes.c_int, [i32, i32, i64, vp, vp, vp, P(vp)]),
        "dbs_basic_destroy": (None, [vp]),
        "dbs_basic_spmspv": (ctypes.c_int, [vp, ctypes.c_int, i32, vp, vp, vp, vp]),
        "dbs_last_error": (ctypes.c_char_p, []),
        "dbs_version": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def check(status: int) -> None:
    if status != DBS_OK:
        msg = load().dbs_last_error().decode(errors="replace")
        raise DbsError(status, msg)
