"""GPU parity of the basic push / pull baselines (Alg. 1) against the oracle.

Both baselines return a dense fp32 y and accumulate in fp32 (pull: one
running sum per lane, then a 16-lane tree; push: fp32 atomics in arbitrary
order), so the bound is the fp32 summation bound rather than the blocked
method's 1e-5: |y - y_ref| <= (L_i + 2) * 2^-24 * S_i with L_i the number of
products of row i and S_i = sum |a_ij x_j| (never tighter than 1e-5 * S_i).
"""
from __future__ import annotations

import numpy as np
import pytest

from gpu_helpers import log, oracle_matrix, to_dev, torch_mod
import paper_2608_16308_amd as dbs
import workloads as wl

pytestmark = pytest.mark.gpu


def _check(a: wl.CSR, x_idx, x_val, label):
    torch = torch_mod()
    B = dbs.BasicMatrix(a.m, a.n, a.row_ptr, a.col_idx, a.vals)
    om = oracle_matrix(a)
    ri, rv, rs = om.spmspv(x_idx, np.asarray(x_val, dtype=np.float64))
    yref = np.zeros(a.m)
    S = np.zeros(a.m)
    yref[ri] = rv
    S[ri] = rs
    act = np.zeros(a.n, dtype=bool)
    act[np.asarray(x_idx, dtype=np.int64)] = True
    rows = np.repeat(np.arange(a.m), np.diff(a.row_ptr))
    L = np.bincount(rows[act[a.col_idx]], minlength=a.m)
    tol = np.maximum(1e-5, (L + 2) * 2.0 ** -24) * S
    xi = to_dev(np.asarray(x_idx, dtype=np.int32))
    xv = to_dev(np.asarray(x_val, dtype=np.float32))
    for path in ("pull", "push"):
        log(f"[basic] {label} path={path} m={a.m} n={a.n} nnz={a.nnz} k={len(x_idx)}")
        y = torch.full((max(a.m, 1),), float("nan"), dtype=torch.float32, device="cuda:0")
        for rep in range(2):  # the second call checks that the scratch was left clean
            B.spmspv(path, xi, xv, y)
            torch.cuda.synchronize()
            g = y.cpu().numpy()[:a.m].astype(np.float64)
            err = np.abs(g - yref)
            bad = np.nonzero(err > tol)[0]
            assert bad.size == 0, f"{label} {path} rep {rep}: row {bad[0]} gpu {g[bad[0]]} ref {yref[bad[0]]}"
            assert np.all(g[S == 0] == 0.0), f"{label} {path}: nonzero y on a row without products"


@pytest.mark.parametrize("case", ["tiny", "ragged", "wide", "crafted", "rmat14"])
def test_basic_push_pull_match_oracle(case):
    if case == "tiny":
        a = wl.tiny()
        xi, xv = wl.sparse_x(a.n, 0.01, "uniform", key=(30, 0))
    elif case == "ragged":
        a = wl.random_csr(1000, 777, 0.02, key=(30, 1))
        xi, xv = wl.sparse_x(a.n, 0.1, "uniform", key=(30, 1))
    elif case == "wide":
        a = wl.random_csr(37, 5000, 0.2, key=(30, 2))
        xi, xv = wl.sparse_x(a.n, 0.3, "clustered", key=(30, 2))
    elif case == "crafted":
        a = wl.crafted(np.float32)
        xi = np.arange(0, a.n, 3, dtype=np.int32)
        xv = np.linspace(-1, 1, xi.size).astype(np.float32)
    else:
        a = wl.rmat(14)
        xi, xv = wl.sparse_x(a.n, 0.05, "uniform", key=(30, 4))
    _check(a, xi, xv, case)


def test_basic_empty_x_and_zero_values():
    a = wl.random_csr(300, 200, 0.05, key=(30, 5))
    _check(a, np.zeros(0, dtype=np.int32), np.zeros(0, dtype=np.float32), "empty x")
    xi = np.array([0, 17, 199], dtype=np.int32)
    _check(a, xi, np.zeros(3, dtype=np.float32), "zero values")
