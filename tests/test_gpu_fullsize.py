"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times (one context, automatic path plus forced push / pull):

* R-MAT scale 20, fp32: the eight x of the density sweep, every output
  element checked against the oracle;
* R-MAT scale 22 pattern BFS from 16 giant-component sources: level[] and
  parent[] bit-exact, plus reuse of one context across calls;
* relabelled 126^3 mesh with 5% random entries, BFS-ball x at 0.1%-10%;
* fp16 decode layers 11008x4096 and 4096x14336 with 10%-dense activations;
* a FEM-like natural-order matrix (27-point stencil, 3 unknowns per node:
  72% patched-CSR blocks) with uniform and clustered x, OR-AND, BFS, and
  every block forced into each format;
* a mid-size R-MAT (scale 17) where the look-back scans span several tiles.
"""
import numpy as np
import pytest

import oracle
import paper_2608_16308_amd as dbs
import workloads as wl
from gpu_helpers import REL_TOL, check_spmspv, f16_ulp_dist, gpu_matrix, log, oracle_matrix, to_dev, torch_mod

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def bfs_exact(ctx, A, om, s, policy, label):
    torch = torch_mod()
    level, parent, st = ctx.bfs(A, int(s), policy=policy, stats=True)
    torch.cuda.synchronize()
    el, ep, nl = om.bfs(int(s))
    gl, gp = level.cpu().numpy(), parent.cpu().numpy()
    assert np.array_equal(gl, el), f"{label}: level mismatch at {np.nonzero(gl != el)[0][:5]}"
    assert np.array_equal(gp, ep), f"{label}: parent mismatch at {np.nonzero(gp != ep)[0][:5]}"
    assert st["levels"] == nl
    return st


# ------------------------------------------------------------------ mid size
@pytest.fixture(scope="module")
def rmat17(torch):
    log("generating R-MAT 17")
    a = wl.rmat(17)
    return a, gpu_matrix(a), oracle_matrix(a)


def test_rmat17_spmspv_multitile(rmat17):
    a, A, om = rmat17
    ctx = dbs.Context(A)
    for rep in range(2):
        for di, d in enumerate([1e-3, 1e-2, 1e-1, 0.5]):
            for kind in ("uniform", "clustered"):
                xi, xv = wl.sparse_x(a.n, d, kind, key=(50, di, rep))
                for p in ("auto", "push", "pull"):
                    label = f"rmat17 rep={rep} d={d} {kind} path={p}"
                    log(label)
                    check_spmspv(ctx, A, om, a, xi, xv, path=p, label=label)


def test_rmat17_bfs_repeated(rmat17):
    a, _, _ = rmat17
    p = wl.CSR(a.m, a.n, a.row_ptr, a.col_idx, None)
    A, om = gpu_matrix(p), oracle_matrix(p)
    ctx = dbs.Context(A)
    srcs = wl.bfs_sources(p, 4, key=5)
    for rep in range(2):
        for s in srcs:
            for pol in ("auto", "push", "pull"):
                label = f"rmat17 bfs rep={rep} src={s} policy={pol}"
                log(label)
                bfs_exact(ctx, A, om, s, pol, label)


# ------------------------------------------------------------------ R-MAT 20 sweep
@pytest.fixture(scope="module")
def rmat20(torch):
    log("generating R-MAT 20")
    a = wl.rmat(20)
    log("building DB + oracle CSC")
    return a, gpu_matrix(a), oracle_matrix(a)


@pytest.mark.parametrize("di", [0, 1, 2, 3])
def test_rmat20_density_sweep(rmat20, di):
    a, A, om = rmat20
    ctx = dbs.Context(A)
    d = [1e-4, 1e-3, 1e-2, 1e-1][di]
    for ki, kind in enumerate(("uniform", "clustered")):
        xi, xv = wl.sparse_x(a.n, d, kind, key=(20, di, ki))  # the benchmark's vectors
        for p in ("auto", "push", "pull"):
            label = f"rmat20 d={d} {kind} path={p}"
            log(label)
            check_spmspv(ctx, A, om, a, xi, xv, path=p, label=label)


def test_rmat20_or_and(rmat20):
    a, A, om = rmat20
    ctx = dbs.Context(A)
    rng = wl.rng_for(wl.W_RAND, 51, 0)
    bits = rng.random(a.m) < 0.5
    from gpu_helpers import mask_words
    mw = mask_words(bits)
    for d in (1e-4, 1e-2):
        xi, _ = wl.sparse_x(a.n, d, "uniform", key=(51, int(d * 1e4)))
        for p in ("push", "pull"):
            label = f"rmat20 or_and masked d={d} path={p}"
            log(label)
            check_spmspv(ctx, A, om, a, xi, None, path=p, mask=mw, complement=True, semiring="or_and", label=label)
    # masks that exclude whole 16-row blocks (85% of them) and half of the
    # rows of the others: the pull's segment loop skips the segments and
    # tasks whose block row has no admitted row; uncomplemented too
    blk = np.repeat(rng.random((a.m + 15) // 16) < 0.85, 16)[:a.m]
    bits2 = blk | (rng.random(a.m) < 0.5)
    mw2 = mask_words(bits2)
    for d in (1e-2, 0.3):
        xi, _ = wl.sparse_x(a.n, d, "uniform", key=(52, int(d * 1e4)))
        for p in ("auto", "push", "pull"):
            label = f"rmat20 or_and block-row mask d={d} path={p}"
            log(label)
            check_spmspv(ctx, A, om, a, xi, None, path=p, mask=mw2, complement=True, semiring="or_and", label=label)
        label = f"rmat20 or_and block-row mask (kept rows) d={d}"
        log(label)
        check_spmspv(ctx, A, om, a, xi, None, path="pull", mask=mask_words(~bits2), semiring="or_and", label=label)


# ------------------------------------------------------------------ R-MAT 22 BFS
@pytest.fixture(scope="module")
def rmat22(torch):
    log("generating R-MAT 22 (pattern)")
    g = wl.rmat(22, values=False)
    srcs = wl.bfs_sources(g, 16, key=0)  # the benchmark's sources
    log("building DB + oracle CSC")
    G = gpu_matrix(g)
    return g, G, oracle_matrix(g), srcs, dbs.Context(G)


@pytest.mark.parametrize("si", list(range(16)))
def test_rmat22_bfs_16_sources(rmat22, si):
    g, G, og, srcs, ctx = rmat22
    s = int(srcs[si])
    st = bfs_exact(ctx, G, og, s, "auto", f"rmat22 bfs src={s} auto")
    log(f"  levels={st['levels']} reached={st['reached']} paths={st['path']}")
    assert st["reached"] > g.n // 4  # giant component


def test_rmat22_bfs_forced_paths(rmat22):
    g, G, og, srcs, ctx = rmat22
    for pol in ("push", "pull"):
        s = int(srcs[3])
        label = f"rmat22 bfs src={s} policy={pol}"
        log(label)
        bfs_exact(ctx, G, og, s, pol, label)


# ------------------------------------------------------------------ mesh
def test_mesh_ball_x(torch):
    log("generating 126^3 mesh")
    a = wl.mesh()
    A, om = gpu_matrix(a), oracle_matrix(a)
    ctx = dbs.Context(A)
    S = wl.symmetric_pattern(a)
    for d in (1e-3, 1e-2, 1e-1):
        xi, xv = wl.ball_x(a, d, key=int(d * 1e4), S=S)
        for p in ("auto", "push", "pull"):
            label = f"mesh d={d} k={xi.size} path={p}"
            log(label)
            check_spmspv(ctx, A, om, a, xi, xv, path=p, label=label)


# ------------------------------------------------------------------ decode
@pytest.mark.parametrize("shape", [(11008, 4096), (4096, 14336)])
def test_decode_layers(torch, shape):
    out_f, in_f = shape
    log(f"generating decode layer {out_f}x{in_f}")
    w = wl.decode_layer(out_f, in_f)
    A, om = gpu_matrix(w), oracle_matrix(w)
    info = A.info()
    log(f"  blocks {info['blocks_by_type']}")
    ctx = dbs.Context(A)
    for key in range(3):
        a16 = wl.decode_activation(in_f, key=key)
        for p in ("auto", "push", "pull"):
            label = f"decode {out_f}x{in_f} act={key} path={p}"
            log(label)
            y32 = torch.empty(out_f, dtype=torch.float32, device="cuda:0")
            y, st = ctx.spmspv_dense(A, to_dev(a16), path=p, y32=y32, stats=True)
            torch.cuda.synchronize()
            y64, S, y16 = oracle.decode_linear(om, a16)
            d = f16_ulp_dist(y.cpu().numpy(), y16)
            assert d.max() <= 1, f"{label}: {d.max()} ulp"
            assert oracle.within_tol(y32.cpu().numpy(), y64, S, REL_TOL).all(), label
            if p == "auto":
                assert st["path"] == "pull"


# ------------------------------------------------------------------ FEM-like
@pytest.fixture(scope="module")
def fem(torch):
    log("generating FEM 24^3 x 3")
    a = wl.fem(24, 3)
    return a, gpu_matrix(a), oracle_matrix(a)


def test_fem_spmspv(fem):
    a, A, om = fem
    info = A.info()
    assert info["blocks_by_type"]["csr"] > info["blocks_by_type"]["coo"] > 0
    ctx = dbs.Context(A)
    for di, d in enumerate([1e-3, 1e-2, 1e-1, 0.5]):
        for kind in ("uniform", "clustered"):
            xi, xv = wl.sparse_x(a.n, d, kind, key=(60, di), lo=-1.0, hi=1.0)
            for p in ("auto", "push", "pull"):
                label = f"fem d={d} {kind} path={p}"
                log(label)
                check_spmspv(ctx, A, om, a, xi, xv, path=p, label=label)
                if d == 1e-2:
                    check_spmspv(ctx, A, om, a, xi, None, path=p, semiring="or_and", label=label + " or_and")


@pytest.mark.parametrize("force", [0, 1, 2, 3, 4])
def test_fem_forced_formats(fem, force):
    a, _, om = fem
    A = gpu_matrix(a, dbs.default_opts(force_type=force))
    ctx = dbs.Context(A)
    for di, d in enumerate([1e-2, 0.2]):
        xi, xv = wl.sparse_x(a.n, d, "uniform", key=(61, di), lo=-1.0, hi=1.0)
        for p in ("push", "pull"):
            label = f"fem force={force} d={d} path={p}"
            log(label)
            check_spmspv(ctx, A, om, a, xi, xv, path=p, label=label)


def test_fem_bfs(fem):
    a, _, _ = fem
    g = wl.CSR(a.m, a.n, a.row_ptr, a.col_idx, None)
    G, og = gpu_matrix(g), oracle_matrix(g)
    ctx = dbs.Context(G)
    rng = wl.rng_for(wl.W_RAND, 62, 0)
    for s in rng.choice(a.n, 3, replace=False):
        for policy in ("auto", "push", "pull"):
            log(f"fem bfs source={s} policy={policy}")
            bfs_exact(ctx, G, og, s, policy, f"fem bfs {s} {policy}")
