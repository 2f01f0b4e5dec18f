"""The binding's argument checks (CPU only).

The C ABI trusts the element types and lengths of the device buffers it is
given, so the Python binding checks every tensor before passing its address:
device, contiguity, element type and length.  These tests call the checks
directly with CPU tensors (the expected device passed as "cpu"), one
rejection at a time, and check that a well-formed set passes.
"""
import pytest
import torch

import paper_2608_16308_amd as dbs
from paper_2608_16308_amd import DBS_F16, DBS_F32, DBS_OR_AND, DBS_PATTERN, DBS_PLUS_TIMES, DbsError
from paper_2608_16308_amd._lib import DBS_ERR_ARG

CPU = torch.device("cpu")
M, N = 100, 70  # mask: 4 words


def spmspv_args(**over):
    a = dict(x_idx=torch.tensor([1, 5, 9], dtype=torch.int32), x_val=torch.ones(3, dtype=torch.float32),
             mask=torch.zeros(4, dtype=torch.int32), y_idx=torch.empty(M, dtype=torch.int32),
             y_val=torch.empty(M, dtype=torch.float32), y_nnz=torch.zeros(1, dtype=torch.int32))
    a.update(over)
    return a


def call_spmspv(dtype=DBS_F32, semiring=DBS_PLUS_TIMES, device=CPU, **over):
    return dbs.validate_spmspv(torch, M, N, dtype, semiring, device, **spmspv_args(**over))


def rejects(fn, *args, **kw):
    with pytest.raises(DbsError) as e:
        fn(*args, **kw)
    assert e.value.status == DBS_ERR_ARG
    return str(e.value)


def test_spmspv_well_formed_passes():
    assert call_spmspv() == 3
    assert call_spmspv(mask=None) == 3
    assert call_spmspv(mask=torch.zeros(4, dtype=torch.uint32)) == 3
    assert call_spmspv(dtype=DBS_F16, x_val=torch.ones(3, dtype=torch.float16),
                       y_val=torch.empty(M, dtype=torch.float16)) == 3
    # OR-AND: values are ignored and may be absent
    assert call_spmspv(semiring=DBS_OR_AND, x_val=None, y_val=None) == 3
    assert call_spmspv(dtype=DBS_PATTERN, semiring=DBS_OR_AND, x_val=None, y_val=None) == 3
    # an empty x needs no values
    assert call_spmspv(x_idx=torch.zeros(0, dtype=torch.int32), x_val=None) == 0


@pytest.mark.parametrize("case", [
    "idx_int64", "idx_2d", "idx_noncontig", "val_f64", "val_f16_for_f32", "val_short", "val_long",
    "val_missing", "mask_short", "mask_int64", "mask_f32", "yidx_short", "yidx_int64", "yval_short",
    "yval_dtype", "ynnz_empty", "ynnz_int64", "device", "pattern_plus_times",
])
def test_spmspv_rejections(case):
    bad = {
        "idx_int64": dict(x_idx=torch.tensor([1, 5, 9])),
        "idx_2d": dict(x_idx=torch.tensor([[1, 5, 9]], dtype=torch.int32)),
        "idx_noncontig": dict(x_idx=torch.arange(6, dtype=torch.int32)[::2]),
        "val_f64": dict(x_val=torch.ones(3, dtype=torch.float64)),
        "val_f16_for_f32": dict(x_val=torch.ones(3, dtype=torch.float16)),
        "val_short": dict(x_val=torch.ones(2, dtype=torch.float32)),
        "val_long": dict(x_val=torch.ones(4, dtype=torch.float32)),
        "val_missing": dict(x_val=None),
        "mask_short": dict(mask=torch.zeros(3, dtype=torch.int32)),
        "mask_int64": dict(mask=torch.zeros(4, dtype=torch.int64)),
        "mask_f32": dict(mask=torch.zeros(4, dtype=torch.float32)),
        "yidx_short": dict(y_idx=torch.empty(M - 1, dtype=torch.int32)),
        "yidx_int64": dict(y_idx=torch.empty(M, dtype=torch.int64)),
        "yval_short": dict(y_val=torch.empty(M - 1, dtype=torch.float32)),
        "yval_dtype": dict(y_val=torch.empty(M, dtype=torch.float16)),
        "ynnz_empty": dict(y_nnz=torch.zeros(0, dtype=torch.int32)),
        "ynnz_int64": dict(y_nnz=torch.zeros(1, dtype=torch.int64)),
    }
    if case == "device":
        rejects(call_spmspv, device=torch.device("meta"))
    elif case == "pattern_plus_times":
        rejects(call_spmspv, dtype=DBS_PATTERN)
    else:
        rejects(call_spmspv, **bad[case])


def test_dense_activation_checks():
    x, y, y32 = torch.zeros(N, dtype=torch.float16), torch.empty(M, dtype=torch.float16), torch.empty(M)
    dbs.validate_dense(torch, M, N, DBS_F16, CPU, x, y, y32)
    dbs.validate_dense(torch, M, N, DBS_F16, CPU, x, y, None)
    rejects(dbs.validate_dense, torch, M, N, DBS_F16, CPU, x[:-1], y, y32)            # short x
    rejects(dbs.validate_dense, torch, M, N, DBS_F16, CPU, x.float(), y, y32)         # x dtype
    rejects(dbs.validate_dense, torch, M, N, DBS_F16, CPU, x, y[:-1], y32)            # short y
    rejects(dbs.validate_dense, torch, M, N, DBS_F16, CPU, x, y.float(), y32)         # y dtype
    rejects(dbs.validate_dense, torch, M, N, DBS_F16, CPU, x, y, y32.half())          # y32 dtype
    rejects(dbs.validate_dense, torch, M, N, DBS_F16, CPU, torch.zeros(2 * N, dtype=torch.float16)[::2], y, y32)
    rejects(dbs.validate_dense, torch, M, N, DBS_PATTERN, CPU, x, y, y32)             # pattern matrix


def test_batched_activation_checks():
    X, Y, Y32 = torch.zeros(3, N), torch.empty(3, M), torch.empty(3, M)
    assert dbs.validate_spmm(torch, M, N, DBS_F32, CPU, X, Y, Y32) == 3
    assert dbs.validate_spmm(torch, M, N, DBS_F32, CPU, X, Y, None) == 3
    rejects(dbs.validate_spmm, torch, M, N, DBS_F32, CPU, torch.zeros(9, N), torch.empty(9, M), None)  # nb > 8
    rejects(dbs.validate_spmm, torch, M, N, DBS_F32, CPU, torch.zeros(0, N), torch.empty(0, M), None)  # nb = 0
    rejects(dbs.validate_spmm, torch, M, N, DBS_F32, CPU, torch.zeros(3, N + 1), Y, None)   # wrong n
    rejects(dbs.validate_spmm, torch, M, N, DBS_F32, CPU, torch.zeros(3 * N), Y, None)      # 1-D X
    rejects(dbs.validate_spmm, torch, M, N, DBS_F32, CPU, X, torch.empty(3, M + 1), None)   # row stride
    rejects(dbs.validate_spmm, torch, M, N, DBS_F32, CPU, X, torch.empty(2, M), None)       # too few rows
    rejects(dbs.validate_spmm, torch, M, N, DBS_F32, CPU, X, Y.half(), None)                # Y dtype
    rejects(dbs.validate_spmm, torch, M, N, DBS_F32, CPU, X, Y, Y32.t().contiguous().t())   # Y32 strided
    rejects(dbs.validate_spmm, torch, M, N, DBS_F16, CPU, X, Y, None)                       # X dtype vs A


def test_bfs_checks():
    lv, pa = torch.empty(N, dtype=torch.int32), torch.empty(N, dtype=torch.int32)
    dbs.validate_bfs(torch, N, N, CPU, 0, lv, pa)
    dbs.validate_bfs(torch, N, N, CPU, N - 1, lv, pa)
    rejects(dbs.validate_bfs, torch, M, N, CPU, 0, lv, pa)                         # not square
    rejects(dbs.validate_bfs, torch, N, N, CPU, N, lv, pa)                         # source out of range
    rejects(dbs.validate_bfs, torch, N, N, CPU, -1, lv, pa)
    rejects(dbs.validate_bfs, torch, N, N, CPU, 0, lv[:-1], pa)                    # short level
    rejects(dbs.validate_bfs, torch, N, N, CPU, 0, lv, pa.long())                  # parent int64
