"""GPU-side conversion (dbs_matrix_build_dense) against the host builder.

Bit-exact: every device array of the converted matrix (slots, segment words,
block-CSC view, non-COO list and chunks, payload) and its info equal those
of dbs_matrix_build_csr over the CSR of the same matrix's nonzero entries,
for ragged shapes, every block format (classified and forced), inline and
stored COO, other thresholds, padded leading dimensions and special values.
Then SpMSpV and a decode layer on converted matrices match the oracle.
"""
import numpy as np
import pytest

import oracle
import paper_2608_16308_amd as dbs
import workloads as wl
from gpu_helpers import REL_TOL, check_spmspv, f16_ulp_dist, log, oracle_matrix, to_dev, torch_mod

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def dense_of(a: wl.CSR, dtype):
    d = np.zeros((a.m, a.n), dtype=dtype)
    rows = np.repeat(np.arange(a.m), np.diff(a.row_ptr))
    d[rows, a.col_idx] = a.vals.astype(dtype)
    return d


def csr_of(d: np.ndarray) -> wl.CSR:
    """The stored entries of a dense matrix: nonzero values (NaN included,
    -0 excluded), columns ascending."""
    m, n = d.shape
    rows, cols = np.nonzero(d != 0)
    row_ptr = np.zeros(m + 1, dtype=np.int64)
    np.add.at(row_ptr, rows + 1, 1)
    row_ptr = np.cumsum(row_ptr)
    return wl.CSR(m, n, row_ptr, cols.astype(np.int32), np.ascontiguousarray(d[rows, cols]))


def convert_and_compare(torch, d: np.ndarray, label, opts=None, ld_pad=0):
    m, n = d.shape
    if ld_pad:
        wide = np.zeros((m, n + ld_pad), dtype=d.dtype)
        wide[:, :n] = d
        wide[:, n:] = 7  # never read
        w = torch.from_numpy(wide).to("cuda:0")[:, :n]
    else:
        w = torch.from_numpy(np.ascontiguousarray(d)).to("cuda:0")
    log(f"convert {label}: {m}x{n} {d.dtype} ld_pad={ld_pad}")
    Ag = dbs.Matrix.from_dense(w, opts=opts)
    a = csr_of(d)
    Ah = dbs.Matrix.from_csr(a.m, a.n, a.row_ptr, a.col_idx, a.vals, opts=opts)
    ig, ih = Ag.info(), Ah.info()
    assert ig == ih, f"{label}: info differs\n{ig}\n{ih}"
    ga, ha = Ag.download(), Ah.download()
    for k in ha:
        assert ga[k].shape == ha[k].shape, f"{label}: {k} shape {ga[k].shape} vs {ha[k].shape}"
        if not np.array_equal(ga[k], ha[k]):
            bad = np.nonzero(ga[k] != ha[k])[0][:5]
            raise AssertionError(f"{label}: {k} differs at {bad}: gpu {ga[k][bad]} host {ha[k][bad]}")
    return Ag, a, ig


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_convert_crafted_all_formats(torch, dtype):
    a = wl.crafted(dtype, key=21)
    _, _, info = convert_and_compare(torch, dense_of(a, dtype), f"crafted {np.dtype(dtype).name}")
    assert all(info["blocks_by_type"][t] > 0 for t in info["blocks_by_type"]), info["blocks_by_type"]


@pytest.mark.parametrize("shape,density,key", [((300, 640), 0.5, 1), ((1000, 1030), 0.03, 2), ((77, 131), 0.3, 3),
                                               ((1, 1), 1.0, 4), ((17, 1), 0.5, 5), ((1, 33), 0.5, 6),
                                               ((64, 64), 0.0, 7)])
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_convert_random_shapes(torch, shape, density, key, dtype):
    m, n = shape
    a = wl.random_csr(m, n, density, key=(70, key), dtype=dtype)
    convert_and_compare(torch, dense_of(a, dtype), f"random {m}x{n} d={density}")


@pytest.mark.parametrize("opt", ["force0", "force1", "force2", "force3", "force4", "noinline", "th", "seg1",
                                 "seg16"])
def test_convert_options(torch, opt):
    a = wl.crafted(np.float32, key=22)
    d = dense_of(a, np.float32)
    if opt.startswith("force"):
        opts = dbs.default_opts(force_type=int(opt[-1]))
    elif opt == "noinline":
        opts = dbs.default_opts(inline_small=0)
    elif opt == "th":
        opts = dbs.default_opts(th0=9, th1=200, th2=1.5)
    else:
        opts = dbs.default_opts(seg_close=int(opt[3:]))
    convert_and_compare(torch, d, f"crafted opts {opt}", opts=opts)


def test_convert_padded_ld_and_special_values(torch):
    rng = wl.rng_for(wl.W_RAND, 71, 0)
    d = rng.uniform(-1, 1, (50, 70)).astype(np.float32)
    d[rng.random(d.shape) < 0.6] = 0.0
    d[3, 5] = -0.0          # zero: not stored
    d[10, 20] = np.nan      # stored
    d[40:48, 32:48] = 0.0   # an empty tile
    convert_and_compare(torch, d, "padded ld, -0 and NaN", ld_pad=9)
    h = d.astype(np.float16)
    convert_and_compare(torch, h, "padded ld fp16", ld_pad=3)


def test_convert_empty_shapes(torch):
    for shape in ((0, 5), (5, 0), (0, 0)):
        d = np.zeros(shape, dtype=np.float32)
        A = dbs.Matrix.from_dense(torch.zeros(shape, dtype=torch.float32, device="cuda:0"))
        info = A.info()
        assert info["nblk"] == 0 and info["nnz"] == 0, (shape, info)
        assert d.size == 0


def test_convert_rejects_bad_input(torch):
    with pytest.raises(ValueError):
        dbs.Matrix.from_dense(torch.zeros((4, 4), dtype=torch.float64, device="cuda:0"))
    with pytest.raises(dbs.DbsError):
        dbs.Matrix.from_dense(torch.zeros((4, 4), dtype=torch.float32, device="cuda:0"),
                              opts=dbs.default_opts(seg_close=0))


def test_converted_matrix_spmspv_and_decode(torch):
    # SpMSpV on a converted fp32 matrix, every path
    a0 = wl.random_csr(700, 900, 0.05, key=(72, 0))
    d = dense_of(a0, np.float32)
    A, a, _ = convert_and_compare(torch, d, "spmspv matrix")
    om = oracle_matrix(a)
    ctx = dbs.Context(A)
    for frac in (0.01, 0.2):
        xi, xv = wl.sparse_x(a.n, frac, "uniform", key=(73, int(frac * 100)))
        for p in ("auto", "push", "pull"):
            label = f"converted spmspv x={frac} path={p}"
            log(label)
            check_spmspv(ctx, A, om, a, xi, xv, path=p, label=label)
    # a decode layer converted from its dense fp16 weights
    w = wl.decode_layer(320, 640, keep=0.5)
    dw = dense_of(w, np.float16)
    Aw, aw, info = convert_and_compare(torch, dw, "decode layer")
    assert info["blocks_by_type"]["coo"] == 0
    omw = oracle_matrix(aw)
    ctxw = dbs.Context(Aw)
    a16 = wl.decode_activation(640, key=3)
    for p in ("auto", "pull", "push"):
        log(f"converted decode path={p}")
        y32 = torch.empty(320, dtype=torch.float32, device="cuda:0")
        y, _ = ctxw.spmspv_dense(Aw, to_dev(a16), path=p, y32=y32, stats=True)
        torch.cuda.synchronize()
        y64, S, y16 = oracle.decode_linear(omw, a16)
        assert f16_ulp_dist(y.cpu().numpy(), y16).max() <= 1
        assert oracle.within_tol(y32.cpu().numpy(), y64, S, REL_TOL).all()


def test_converted_matrix_bfs(torch):
    # BFS on a device-converted matrix (no row-occupancy bitmap: no row
    # starts as reached) and on the host build of the same matrix (rows
    # without entries start as reached): both equal the oracle
    a0 = wl.random_csr(3000, 3000, 0.0015, key=(74, 0))
    d = dense_of(a0, np.float32)
    d[100:400, :] = 0.0  # block rows without entries and partly empty ones
    d[1000:1016:3, :] = 0.0
    Ag, a, _ = convert_and_compare(torch, d, "bfs matrix")
    Ah = dbs.Matrix.from_csr(a.m, a.n, a.row_ptr, a.col_idx, a.vals)
    om = oracle_matrix(a)
    rows_empty = np.nonzero(np.diff(a.row_ptr) == 0)[0]
    rng = wl.rng_for(wl.W_RAND, 74, 1)
    sources = [int(rows_empty[0]), int(rows_empty[-1])] + [int(s) for s in rng.choice(a.n, 4, replace=False)]
    for name, A in (("converted", Ag), ("host", Ah)):
        ctx = dbs.Context(A)
        for s in sources:
            el, ep, nl = om.bfs(s)
            for policy in ("auto", "push", "pull"):
                log(f"{name} bfs source={s} policy={policy}")
                level, parent, st = ctx.bfs(A, s, policy=policy, stats=True)
                torch.cuda.synchronize()
                assert np.array_equal(level.cpu().numpy(), el), (name, s, policy)
                assert np.array_equal(parent.cpu().numpy(), ep), (name, s, policy)
                assert st["levels"] == nl
