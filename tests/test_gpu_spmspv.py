"""GPU parity of dbs_spmspv (plus-times and OR-AND, push / pull / auto, output
masks, every block format) against the CPU oracle, through the C ABI."""
import numpy as np
import pytest

import oracle
import paper_2608_16308_amd as dbs
import workloads as wl
from gpu_helpers import REL_TOL, check_spmspv, gpu_matrix, log, mask_words, oracle_matrix, to_dev, torch_mod

pytestmark = pytest.mark.gpu

PATHS = ["auto", "push", "pull"]


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def x_kinds(n, key):
    """Vector supports that drive every microkernel choice: isolated entries
    (sparse vector blocks), whole vector blocks (dense), random 30%, one entry,
    everything."""
    rng = wl.rng_for(wl.W_RAND, 31, key)
    out = {}
    out["sparse"] = np.sort(rng.choice(n, max(1, n // 40), replace=False))
    nvb = (n + 15) // 16
    blocks = rng.choice(nvb, max(1, nvb // 3), replace=False)
    full = np.concatenate([np.arange(b * 16, min(n, b * 16 + 16)) for b in blocks])
    out["blocks"] = np.sort(full)
    out["rand30"] = np.sort(rng.choice(n, max(1, int(0.3 * n)), replace=False))
    out["one"] = np.array([n - 1])
    out["all"] = np.arange(n)
    vals = {k: wl._nonzero_uniform(wl.rng_for(wl.W_RAND, 32, key, i), -1.0, 1.0, v.size)
            for i, (k, v) in enumerate(out.items())}
    return {k: (out[k].astype(np.int32), vals[k]) for k in out}


def test_tiny_config(torch):
    a = wl.tiny()
    x_idx, x_val = wl.sparse_x(a.n, 0.01, "uniform", key=(1,), lo=-1.0, hi=1.0)
    assert x_idx.size == 41
    A, om = gpu_matrix(a), oracle_matrix(a)
    ctx = dbs.Context(A)
    for p in PATHS:
        log(f"tiny 4096x4096 k=41 path={p}")
        st = check_spmspv(ctx, A, om, a, x_idx, x_val, path=p, label=f"tiny/{p}")
        if p == "auto":
            assert st["path"] == "pull"  # s_b ~ 0.14 >= th3


@pytest.mark.parametrize("dtype", ["f32", "f16"])
def test_crafted_all_formats(torch, dtype):
    npdt = np.float32 if dtype == "f32" else np.float16
    a = wl.crafted(npdt, key=11)
    A, om = gpu_matrix(a), oracle_matrix(a)
    info = A.info()
    assert all(v > 0 for v in info["blocks_by_type"].values())
    ctx = dbs.Context(A)
    rng = wl.rng_for(wl.W_RAND, 33, 0)
    bits = rng.random(a.m) < 0.6
    mw = mask_words(bits)
    for kind, (xi, xv) in x_kinds(a.n, 1).items():
        xv = xv.astype(npdt)
        for p in PATHS:
            for mask, comp in ((None, False), (mw, False), (mw, True)):
                label = f"crafted {dtype} x={kind} path={p} mask={'none' if mask is None else ('comp' if comp else 'on')}"
                log(label)
                check_spmspv(ctx, A, om, a, xi, xv.astype(np.float64), path=p, mask=mask, complement=comp,
                             label=label)


@pytest.mark.parametrize("force,inline", [(0, 1), (0, 0), (1, 1), (2, 1), (3, 1), (4, 1)])
def test_forced_single_format(torch, force, inline):
    a = wl.crafted(np.float32, key=12)
    A = gpu_matrix(a, dbs.default_opts(force_type=force, inline_small=inline))
    om = oracle_matrix(a)
    ctx = dbs.Context(A)
    for kind, (xi, xv) in x_kinds(a.n, 2).items():
        for p in ("push", "pull"):
            label = f"force_type={force} inline={inline} x={kind} path={p}"
            log(label)
            check_spmspv(ctx, A, om, a, xi, xv, path=p, label=label)


def test_or_and_and_path_equivalence(torch):
    for key, dt in ((13, None), (14, np.float32)):
        a = wl.crafted(dt, key=key)
        A, om = gpu_matrix(a), oracle_matrix(a)
        ctx = dbs.Context(A)
        rng = wl.rng_for(wl.W_RAND, 34, key)
        mw = mask_words(rng.random(a.m) < 0.5)
        for kind, (xi, _) in x_kinds(a.n, 3).items():
            outs = []
            for p in PATHS:
                for mask, comp in ((None, False), (mw, True)):
                    label = f"or_and key={key} x={kind} path={p} comp={comp}"
                    log(label)
                    check_spmspv(ctx, A, om, a, xi, None, path=p, mask=mask, complement=comp,
                                 semiring="or_and", label=label)
            del outs


@pytest.mark.parametrize("shape,density", [((77, 131), 0.08), ((300, 45), 0.5), ((1, 1), 1.0),
                                           ((1, 200), 0.3), ((200, 1), 0.3), ((513, 257), 0.02),
                                           ((64, 64), 0.0)])
def test_random_shapes(torch, shape, density):
    m, n = shape
    a = wl.random_csr(m, n, density, key=(35, m, n))
    A, om = gpu_matrix(a), oracle_matrix(a)
    ctx = dbs.Context(A)
    for kind, (xi, xv) in x_kinds(n, 4).items():
        for p in PATHS:
            label = f"random {m}x{n} d={density} x={kind} path={p}"
            log(label)
            check_spmspv(ctx, A, om, a, xi, xv, path=p, label=label)


def test_empty_x_and_threshold(torch):
    a = wl.random_csr(400, 400, 0.05, key=(36, 0))
    A, om = gpu_matrix(a), oracle_matrix(a)
    ctx = dbs.Context(A)
    log("empty x")
    st = check_spmspv(ctx, A, om, a, np.zeros(0, np.int32), np.zeros(0, np.float32), label="empty x")
    assert st["y_nnz"] == 0 and st["n_nzblk"] == 0
    # N_blk = 25, one active block: with the paper's th3 = 0.01 (also the
    # default) push needs N_nzblk < 0.25 (never); th3 = 0.05 gives
    # N_nzblk < 1.25.
    xi = np.array([5, 6], dtype=np.int32)
    xv = np.array([0.5, -2.0], dtype=np.float32)
    log("threshold paper value")
    check_spmspv(ctx, A, om, a, xi, xv, expect_path="pull", label="th 0.01", th3=0.01)
    log("threshold default")
    check_spmspv(ctx, A, om, a, xi, xv, expect_path="pull", label="th default")
    log("threshold 0.05")
    st = check_spmspv(ctx, A, om, a, xi, xv, expect_path="push", label="th 0.05", th3=0.05)
    assert st["n_nzblk"] == 1 and st["n_blk"] == 25
    # exact boundary: 2 active blocks, th3 = 0.08 -> 2 < 2.0 is false -> pull
    xi2 = np.array([5, 200], dtype=np.int32)
    check_spmspv(ctx, A, om, a, xi2, xv, expect_path="pull", label="th boundary", th3=0.08)
    check_spmspv(ctx, A, om, a, xi2, xv, expect_path="push", label="th above boundary", th3=0.0801)


def test_context_reuse_across_matrices(torch):
    """One context, a large then a smaller matrix, many calls: the scratch it
    resets after every call must leave no trace."""
    big = wl.random_csr(700, 650, 0.03, key=(37, 0))
    small = wl.crafted(np.float32, key=15)
    Ab, As = gpu_matrix(big), gpu_matrix(small)
    ob, os_ = oracle_matrix(big), oracle_matrix(small)
    ctx = dbs.Context(Ab)
    for it in range(6):
        for a, A, om in ((big, Ab, ob), (small, As, os_)):
            xs = x_kinds(a.n, 100 + it)
            kind = list(xs)[it % len(xs)]
            xi, xv = xs[kind]
            p = PATHS[it % 3]
            label = f"reuse it={it} {a.m}x{a.n} x={kind} path={p}"
            log(label)
            check_spmspv(ctx, A, om, a, xi, xv, path=p, label=label)


def test_error_flags(torch):
    a = wl.random_csr(100, 100, 0.1, key=(38, 0))
    A = gpu_matrix(a)
    ctx = dbs.Context(A)
    log("duplicate index flag")
    xi = to_dev(np.array([3, 7, 3], dtype=np.int32))
    xv = to_dev(np.array([1.0, 2.0, 3.0], dtype=np.float32))
    _, _, st = ctx.spmspv(A, xi, xv, stats=True)
    assert st["error_flags"] & 2
    log("out-of-range index flag")
    xi = to_dev(np.array([3, 100, -1], dtype=np.int32))
    _, _, st = ctx.spmspv(A, xi, xv, stats=True)
    assert st["error_flags"] & 1
    log("clean call after errors")
    om = oracle_matrix(a)
    check_spmspv(ctx, A, om, a, np.array([1, 2], np.int32), np.array([1.0, 1.0], np.float32), label="after errors")
    # host-side argument errors
    with pytest.raises(dbs.DbsError):
        ctx.spmspv(A, to_dev(np.arange(101, dtype=np.int32)), to_dev(np.ones(101, np.float32)))
    pat = wl.random_csr(50, 50, 0.1, key=(38, 1), dtype=None)
    Ap = gpu_matrix(pat)
    with pytest.raises(dbs.DbsError):
        ctx.spmspv(Ap, to_dev(np.array([1], np.int32)), to_dev(np.ones(1, np.float32)))


def test_spread_rule(torch):
    """The default selector's spread rule: push when x has under two indices
    per nonzero vector block and N_nzblk < 0.12 N_blk; otherwise, and for an
    explicit th3, the paper's rule."""
    a = wl.random_csr(2000, 3200, 0.01, key=(39, 0))  # N_blk = 200
    A, om = gpu_matrix(a), oracle_matrix(a)
    ctx = dbs.Context(A)
    rng = wl.rng_for(wl.W_RAND, 40, 0)
    blocks = np.sort(rng.choice(200, 40, replace=False))
    spread10 = (blocks[:10] * 16 + 3).astype(np.int32)             # s_b = 0.05, one index per block
    spread30 = (blocks[:30] * 16 + 7).astype(np.int32)             # s_b = 0.15
    clustered10 = np.concatenate([np.arange(b * 16, b * 16 + 16) for b in blocks[:10]]).astype(np.int32)
    pairs10 = np.concatenate([[b * 16 + 1, b * 16 + 9] for b in blocks[:10]]).astype(np.int32)  # two per block
    cases = [(spread10, 0.0, "push"), (spread10, 0.01, "pull"), (spread30, 0.0, "pull"),
             (clustered10, 0.0, "pull"), (pairs10, 0.0, "pull")]
    for xi, th3, want in cases:
        xv = wl._nonzero_uniform(wl.rng_for(wl.W_RAND, 41, xi.size), -1.0, 1.0, xi.size)
        label = f"spread rule k={xi.size} th3={th3} -> {want}"
        log(label)
        check_spmspv(ctx, A, om, a, xi, xv, expect_path=want, label=label, th3=th3)


@pytest.mark.parametrize("kind", ["uniform", "clustered"])
def test_small_x_route_boundary(torch, kind):
    """Up to 2048 indices take the one-workgroup blocker and scan, more take
    the grid-wide pair: both sides of the boundary, every path, against the
    oracle; the same x with one repeated entry (2049 indices, the wide route)
    gives the same y and statistics, with the duplicate flagged."""
    a = wl.random_csr(3000, 40000, 0.002, key=(41, 0))
    A, om = gpu_matrix(a), oracle_matrix(a)
    ctx = dbs.Context(A)
    rng = wl.rng_for(wl.W_RAND, 42, 0 if kind == "uniform" else 1)
    if kind == "uniform":
        idx = np.sort(rng.choice(a.n, 2049, replace=False))
    else:
        starts = np.sort(rng.choice(a.n // 64 - 1, 33, replace=False)) * 64
        idx = np.unique(np.concatenate([np.arange(s, s + 64) for s in starts]))[:2049]
    idx = idx.astype(np.int32)
    vals = wl._nonzero_uniform(wl.rng_for(wl.W_RAND, 43, 0), -1.0, 1.0, idx.size)
    stats = {}
    for k in (1, 2, 17, 2047, 2048, 2049):
        for p in PATHS:
            label = f"{kind} k={k} path={p}"
            log(label)
            stats[(k, p)] = check_spmspv(ctx, A, om, a, idx[:k], vals[:k], path=p, label=label)
    # 2048 distinct entries plus a repeat of the first: the wide route
    xi = np.concatenate([idx[:2048], idx[:1]])
    xv = np.concatenate([vals[:2048], vals[:1]])
    for p in PATHS:
        log(f"{kind} duplicate k=2049 path={p}")
        y_idx, y_val, st = ctx.spmspv(A, to_dev(xi), to_dev(xv), path=p, stats=True)
        torch.cuda.synchronize()
        ref = stats[(2048, p)]
        assert st["error_flags"] & 2
        assert st["n_nzblk"] == ref["n_nzblk"] and st["y_nnz"] == ref["y_nnz"] and st["path"] == ref["path"]
        ri, rv, rs = om.spmspv(idx[:2048], vals[:2048].astype(np.float64))
        assert np.array_equal(y_idx.cpu().numpy(), ri)
        assert oracle.within_tol(y_val.cpu().numpy(), rv, rs, REL_TOL).all()


def test_single_scan_tile_counts(torch):
    """More than 2048 indices on a matrix of at most 1024 vector blocks: the
    grid-wide blocker and a scan of one tile, which keeps its counts itself.
    Distinct indices against the oracle on every path; a repeated index and
    an out-of-range index are flagged, and leave y as without them."""
    a = wl.random_csr(1500, 12000, 0.004, key=(44, 0))   # N_blk = 750
    A, om = gpu_matrix(a), oracle_matrix(a)
    ctx = dbs.Context(A)
    rng = wl.rng_for(wl.W_RAND, 45, 0)
    idx = np.sort(rng.choice(a.n, 3000, replace=False)).astype(np.int32)
    vals = wl._nonzero_uniform(wl.rng_for(wl.W_RAND, 46, 0), -1.0, 1.0, idx.size)
    ref = {}
    for p in PATHS:
        label = f"one scan tile k=3000 path={p}"
        log(label)
        ref[p] = check_spmspv(ctx, A, om, a, idx, vals, path=p, label=label)
        assert ref[p]["n_nzblk"] == np.unique(idx >> 4).size
    ri, rv, rs = om.spmspv(idx, vals.astype(np.float64))
    for what, xi, xv, flag in (("repeat", np.concatenate([idx, idx[5:6]]), np.concatenate([vals, vals[5:6]]), 2),
                               ("out of range", np.concatenate([idx, [a.n]]).astype(np.int32),
                                np.concatenate([vals, [1.0]]).astype(np.float32), 1)):
        for p in PATHS:
            log(f"one scan tile {what} path={p}")
            y_idx, y_val, st = ctx.spmspv(A, to_dev(xi.astype(np.int32)), to_dev(xv.astype(np.float32)), path=p,
                                          stats=True)
            torch.cuda.synchronize()
            assert st["error_flags"] & flag, (what, p, st)
            assert st["n_nzblk"] == ref[p]["n_nzblk"] and st["path"] == ref[p]["path"]
            assert np.array_equal(y_idx.cpu().numpy(), ri)
            assert oracle.within_tol(y_val.cpu().numpy(), rv, rs, REL_TOL).all()
    log("one scan tile clean call after the flagged ones")
    check_spmspv(ctx, A, om, a, idx, vals, label="one scan tile after errors")


def coo_column_matrix(key: int) -> wl.CSR:
    """Block columns 0..3 of a 4096 x 256 matrix filled with stored COO blocks
    (2..31 entries each, in random cells), the other block columns sparse:
    a push over x in those columns stages more than 256 COO entries per wave
    iteration, so push takes the blocks' matching entries only."""
    rng = wl.rng_for(wl.W_RAND, 40, key)
    rows, cols = [], []
    for R in range(256):
        for J in range(4):
            cnt = int(rng.integers(2, 32))
            cells = rng.choice(256, size=cnt, replace=False)
            rows.append(R * 16 + cells // 16)
            cols.append(J * 16 + cells % 16)
        # a few single entries elsewhere
        for J in rng.choice(np.arange(4, 16), size=2, replace=False):
            c = int(rng.integers(0, 256))
            rows.append(np.array([R * 16 + c // 16]))
            cols.append(np.array([int(J) * 16 + c % 16]))
    r, c = np.concatenate(rows), np.concatenate(cols)
    vals = wl._nonzero_uniform(wl.rng_for(wl.W_RAND, 40, key, 1), -1.0, 1.0, r.size)
    return wl.csr_from_coo(4096, 256, r, c, vals)


def test_push_coo_matching_entries(torch):
    a = coo_column_matrix(1)
    A, om = gpu_matrix(a), oracle_matrix(a)
    ctx = dbs.Context(A)
    rng = wl.rng_for(wl.W_RAND, 41, 0)
    mw = mask_words(rng.random(a.m) < 0.5)
    cases = {
        # one column per vector block (sparse masks: matching entries only)
        "one_col": np.array([3, 21, 40, 60, 100, 200], dtype=np.int32),
        # some vector blocks whole (every column: the whole records)
        "mixed": np.concatenate([np.arange(16, 32), np.array([5, 50, 130])]).astype(np.int32),
        # a column that no COO block of its vector block uses is still fine
        "two_cols": np.array([0, 15, 33, 47], dtype=np.int32),
    }
    for name, xi in cases.items():
        xi = np.sort(xi)
        xv = wl._nonzero_uniform(wl.rng_for(wl.W_RAND, 41, len(xi)), -1.0, 1.0, xi.size)
        for mask, comp in ((None, False), (mw, False), (mw, True)):
            label = f"coo columns x={name} push mask={'none' if mask is None else ('comp' if comp else 'on')}"
            log(label)
            check_spmspv(ctx, A, om, a, xi, xv.astype(np.float64), path="push", mask=mask, complement=comp,
                         label=label)
        check_spmspv(ctx, A, om, a, xi, xv.astype(np.float64), path="auto", label=f"coo columns x={name} auto")
