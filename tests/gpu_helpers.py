"""Shared helpers of the GPU parity tests (HIP path vs the CPU oracle)."""
from __future__ import annotations

import sys

import numpy as np

import oracle
import paper_2608_16308_amd as dbs
import workloads as wl

REL_TOL = 1e-5  # |y_gpu - y_ref| <= 1e-5 * sum_j |a_ij x_j| per row


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def torch_mod():
    import torch
    return torch


def to_dev(arr, dtype=None):
    torch = torch_mod()
    t = torch.from_numpy(np.ascontiguousarray(arr))
    if dtype is not None:
        t = t.to(dtype)
    return t.to("cuda:0")


def gpu_matrix(a: wl.CSR, opts=None):
    return dbs.Matrix.from_csr(a.m, a.n, a.row_ptr, a.col_idx, a.vals, opts)


def oracle_matrix(a: wl.CSR):
    return oracle.OracleMatrix(a.m, a.n, a.row_ptr, a.col_idx, a.vals)


def mask_words(bits: np.ndarray) -> np.ndarray:
    m = bits.size
    w = np.zeros((m + 31) // 32, dtype=np.uint32)
    idx = np.nonzero(bits)[0]
    np.bitwise_or.at(w, idx // 32, (np.uint32(1) << (idx % 32).astype(np.uint32)))
    return w


def f16_ulp_dist(a16: np.ndarray, b16: np.ndarray) -> np.ndarray:
    def key(x):
        u = x.view(np.uint16).astype(np.int64)
        mag = u & 0x7FFF
        return np.where(u & 0x8000, -mag, mag)
    return np.abs(key(a16) - key(b16))


def check_f16(g16: np.ndarray, ref64: np.ndarray, label: str):
    """fp16 outputs: NaN exactly where the fp64 reference is NaN, elsewhere
    within one fp16 ulp of its round-to-nearest-even."""
    r16 = np.asarray(ref64, dtype=np.float64).astype(np.float16)
    gn, rn = np.isnan(g16), np.isnan(r16)
    assert np.array_equal(gn, rn), f"{label}: NaN positions differ ({gn.sum()} vs {rn.sum()})"
    d = f16_ulp_dist(g16[~gn], r16[~rn])
    assert d.max(initial=0) <= 1, f"{label}: fp16 y off by {d.max()} ulp"


def check_spmspv(ctx, A, om, a: wl.CSR, x_idx, x_val, path="auto", mask=None, complement=False,
                 semiring="plus_times", expect_path=None, label="", th3=0.0):
    """Runs one SpMSpV on the GPU and checks it against the oracle."""
    torch = torch_mod()
    xi = to_dev(np.asarray(x_idx, dtype=np.int32))
    xv = None
    if semiring == "plus_times":
        vdt = np.float16 if a.vals is not None and a.vals.dtype == np.float16 else np.float32
        xv = to_dev(np.asarray(x_val, dtype=vdt))
    md = None if mask is None else to_dev(mask)
    y_idx, y_val, st = ctx.spmspv(A, xi, xv, semiring=semiring, mask=md, complement=complement,
                                  path=path, th3=th3, stats=True)
    torch.cuda.synchronize()
    gi = y_idx.cpu().numpy()
    if semiring == "plus_times":
        ri, rv, rs = om.spmspv(x_idx, np.asarray(x_val, dtype=np.float64), mask=mask, complement=complement)
    else:
        ri = om.spmspv_bool(x_idx, mask=mask, complement=complement)
    assert np.array_equal(gi, ri), f"{label}: y pattern differs ({gi.size} vs {ri.size})"
    if semiring == "plus_times":
        gv = y_val.cpu().numpy()
        if gv.dtype == np.float16:
            check_f16(gv, rv, label)
        else:
            ok = oracle.within_tol(gv, rv, rs, REL_TOL)
            if not ok.all():
                bad = np.nonzero(~ok)[0][:5]
                raise AssertionError(f"{label}: {np.sum(~ok)} values off; e.g. rows {ri[bad]} "
                                     f"gpu {gv[bad]} ref {rv[bad]} S {rs[bad]}")
    assert st["y_nnz"] == ri.size
    assert st["error_flags"] == 0
    if expect_path is not None:
        assert st["path"] == expect_path, (label, st)
    return st


def check_decode_dense(ctx, A, om, a16, path, label):
    """One dense-activation call (decode layer) against the oracle: the fp16
    output within one ulp of the fp64 sum's rounding (NaN where it is NaN),
    the fp32 sums within the tolerance."""
    torch = torch_mod()
    x = to_dev(a16)
    y32 = torch.empty(om.m, dtype=torch.float32, device="cuda:0")
    y, st = ctx.spmspv_dense(A, x, path=path, y32=y32, stats=True)
    torch.cuda.synchronize()
    y64, S, _ = oracle.decode_linear(om, a16)
    check_f16(y.cpu().numpy(), y64, label)
    ok = oracle.within_tol(y32.cpu().numpy(), y64, S, REL_TOL)
    assert ok.all(), f"{label}: {np.sum(~ok)} fp32 sums out of tolerance"
    return st
