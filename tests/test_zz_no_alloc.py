"""dbs_spmspv_noalloc against dbs_spmspv, through the C ABI.

The no-allocation entry point runs the same kernels on a static device array
instead of a context's buffers.  On the same inputs its y pattern must equal
the context entry point's bit for bit, and both must meet the oracle's bar
(pattern exact, values within 1e-5 * sum |a_ij x_j|, NaN where the oracle has
NaN).  Calls come in pairs, the second with a smaller input, so that what a
call leaves in the shared array is exercised; a matrix above the array's
limit is refused before anything is launched.
"""
import numpy as np
import pytest

import oracle
import paper_2608_16308_amd as dbs
import workloads as wl
from gpu_helpers import REL_TOL, check_f16, gpu_matrix, log, mask_words, oracle_matrix, to_dev, torch_mod
from paper_2608_16308_amd._lib import DBS_ERR_UNSUPPORTED, DBS_NOALLOC_MAX_DIM

pytestmark = pytest.mark.gpu

PATHS = ["auto", "push", "pull"]


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def both_entry_points(torch, ctx, A, om, a, xi, xv, path, semiring="plus_times", mask=None, complement=False,
                      label=""):
    xid = to_dev(np.asarray(xi, dtype=np.int32))
    xvd = None
    if semiring == "plus_times":
        xvd = to_dev(np.asarray(xv, dtype=np.float16 if A.dtype == dbs.DBS_F16 else np.float32))
    md = None if mask is None else to_dev(mask)
    ci, cv = ctx.spmspv(A, xid, xvd, semiring=semiring, mask=md, complement=complement, path=path)
    ni, nv = dbs.spmspv_noalloc(A, xid, xvd, semiring=semiring, mask=md, complement=complement, path=path)
    torch.cuda.synchronize()
    ci, ni = ci.cpu().numpy(), ni.cpu().numpy()
    assert np.array_equal(ni, ci), f"{label}: pattern differs from dbs_spmspv ({ni.size} vs {ci.size})"
    if semiring == "plus_times":
        ri, rv, rs = om.spmspv(xi, np.asarray(xv, dtype=np.float64), mask=mask, complement=complement)
        assert np.array_equal(ni, ri), f"{label}: pattern differs from the oracle"
        for name, v in (("noalloc", nv), ("ctx", cv)):
            g = v.cpu().numpy()
            if g.dtype == np.float16:
                check_f16(g, rv, f"{label} {name}")
            else:
                ok = oracle.within_tol(g, rv, rs, REL_TOL)
                assert ok.all(), f"{label} {name}: {np.sum(~ok)} values out of tolerance"
    else:
        ri = om.spmspv_bool(xi, mask=mask, complement=complement)
        assert np.array_equal(ni, ri), f"{label}: pattern differs from the oracle"
    return ni.size


def test_noalloc_rmat16_large_then_small(torch):
    a = wl.rmat(16)
    A, om = gpu_matrix(a), oracle_matrix(a)
    ctx = dbs.Context(A)
    big = wl.sparse_x(a.n, 0.3, "uniform", key=(80,), lo=-1.0, hi=1.0)     # wide blocker route
    small = wl.sparse_x(a.n, 0.001, "clustered", key=(81,), lo=-1.0, hi=1.0)  # one-workgroup route
    assert big[0].size > 2048 and small[0].size <= 2048
    for p in PATHS:
        for name, (xi, xv) in (("large", big), ("small", small)):
            label = f"noalloc rmat16 {name} k={xi.size} path={p}"
            log(label)
            both_entry_points(torch, ctx, A, om, a, xi, xv, p, label=label)


def test_noalloc_smaller_matrix_after_larger(torch):
    """A large fp32 call, then calls on a small ragged fp16 matrix with every
    block format: plus-times, a complemented mask, OR-AND."""
    big = wl.random_csr(5000, 30000, 0.003, key=(82, 0))
    Ab, ob = gpu_matrix(big), oracle_matrix(big)
    cb = dbs.Context(Ab)
    xb = wl.sparse_x(big.n, 0.2, "uniform", key=(83,), lo=-1.0, hi=1.0)
    small = wl.crafted(np.float16, key=84)
    As, osm = gpu_matrix(small), oracle_matrix(small)
    cs = dbs.Context(As)
    rng = wl.rng_for(wl.W_RAND, 85, 0)
    xi = np.sort(rng.choice(small.n, 60, replace=False)).astype(np.int32)
    xv = wl._nonzero_normal(wl.rng_for(wl.W_RAND, 86, 0), 1.0, xi.size, dtype=np.float16)
    mw = mask_words(rng.random(small.m) < 0.5)
    for p in PATHS:
        log(f"noalloc large fp32 k={xb[0].size} path={p}")
        both_entry_points(torch, cb, Ab, ob, big, xb[0], xb[1], p, label=f"large fp32 {p}")
        log(f"noalloc small fp16 path={p}")
        both_entry_points(torch, cs, As, osm, small, xi, xv, p, label=f"small fp16 {p}")
        both_entry_points(torch, cs, As, osm, small, xi, xv, p, mask=mw, complement=True,
                          label=f"small fp16 masked {p}")
        both_entry_points(torch, cs, As, osm, small, xi, None, p, semiring="or_and", label=f"small or-and {p}")


def test_noalloc_maximum_size(torch):
    """R-MAT 20 (n = 2^20, the array's limit) at 1% and 0.01%, uniform."""
    a = wl.rmat(20)
    assert a.n == DBS_NOALLOC_MAX_DIM
    A, om = gpu_matrix(a), oracle_matrix(a)
    ctx = dbs.Context(A)
    for d, key in ((0.01, 87), (0.0001, 88)):
        xi, xv = wl.sparse_x(a.n, d, "uniform", key=(key,))
        for p in ("auto", "pull"):
            label = f"noalloc rmat20 d={d} path={p}"
            log(label)
            both_entry_points(torch, ctx, A, om, a, xi, xv, p, label=label)


def test_noalloc_refuses_above_limit(torch):
    a = wl.random_csr(1, DBS_NOALLOC_MAX_DIM + 1, 1e-5, key=(89, 0))
    A = gpu_matrix(a)
    xi = to_dev(np.array([0, 5], dtype=np.int32))
    xv = to_dev(np.ones(2, dtype=np.float32))
    log("noalloc above the limit")
    with pytest.raises(dbs.DbsError) as e:
        dbs.spmspv_noalloc(A, xi, xv)
    assert e.value.status == DBS_ERR_UNSUPPORTED
    # the array is untouched: a valid call afterwards still matches
    small = wl.random_csr(300, 400, 0.05, key=(89, 1))
    As, osm = gpu_matrix(small), oracle_matrix(small)
    both_entry_points(torch, dbs.Context(As), As, osm, small, np.array([3, 77, 390], np.int32),
                      np.array([0.5, -1.0, 2.0], np.float32), "auto", label="after refusal")
