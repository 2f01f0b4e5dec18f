"""GPU parity of the structural edge cases of y = A x (Sec. 2.1) against the oracle.

The y pattern is structural: a listed x index is active whatever its value,
and a row reached by a stored entry stays in y even when its sum is 0.  The
densified x marks absent entries with all-ones bits, so an input whose bits
equal that marker must still count as present.  Every case below is run on
push, pull and the automatic choice, in fp32 and fp16, on both blocker routes
(at most 2048 indices: one workgroup; more: the grid-wide pair) and on both
sides of the pull's compaction threshold (N_nzblk / N_blk = 0.4):

* x entries of value +0.0 and -0.0 (their rows must appear in y, with 0);
* x entries whose bits equal the absent-entry marker (0xFFFFFFFF in fp32,
  0xFFFF in fp16, both NaN): their rows must appear, NaN where the oracle has
  NaN;
* rows whose products cancel exactly, inside one 16x16 block and across
  blocks of one block row;
* explicit zeros stored in A (from the CSR), in every block format, and rows
  whose every stored entry is an explicit zero;
* the Boolean OR-AND pattern of the same inputs.
"""
import numpy as np
import pytest

import oracle
import paper_2608_16308_amd as dbs
import workloads as wl
from gpu_helpers import (REL_TOL, check_decode_dense, check_spmspv, gpu_matrix, log, oracle_matrix,
                         torch_mod)

pytestmark = pytest.mark.gpu

PATHS = ["auto", "push", "pull"]
M, N = 3000, 40000            # 2500 vector blocks
CANCEL0, NCANCEL = 2000, 64   # rows 2000..2063: two cancelling entries each
ZROW0, NZROW = 2064, 16       # rows 2064..2079: only explicit zeros
COMPACT_BELOW = 0.4
F32_MARKER, F16_MARKER = 0xFFFFFFFF, 0xFFFF


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def edge_matrix(dtype):
    """Crafted blocks of every format (block rows 0-7, block columns 0-12), a
    sprinkle of COO entries elsewhere, the cancelling rows and the zero-only
    rows; ~4% of the stored values are explicit +0.0 or -0.0."""
    key = 0 if dtype == np.float32 else 1
    c = wl.crafted(dtype, key=20 + key)
    rows = [np.repeat(np.arange(c.m), np.diff(c.row_ptr))]
    cols = [c.col_idx.astype(np.int64)]
    vals = [c.vals]
    rng = wl.rng_for(wl.W_RAND, 70, key)
    # COO sprinkle: block rows 0-7 right of the crafted columns, and every
    # other row outside the special ranges
    r1 = rng.integers(0, c.m, 4000)
    c1 = rng.integers(208, N, 4000)
    r2 = rng.integers(c.m, M, 150000)
    r2 = r2[(r2 < CANCEL0) | (r2 >= ZROW0 + NZROW)]
    c2 = rng.integers(0, N, r2.size)
    rr = np.concatenate([r1, r2])
    cc = np.concatenate([c1, c2])
    keyv, first = np.unique(rr * N + cc, return_index=True)
    rr, cc = rr[first], cc[first]
    rows.append(rr)
    cols.append(cc)
    vals.append(wl._nonzero_uniform(wl.rng_for(wl.W_RAND, 71, key), -1.0, 1.0, rr.size, dtype=dtype))
    # cancelling rows: entries w and -w at two columns whose x values are
    # equal; rows CANCEL0.. +31 inside one block, the rest across blocks
    # (in-block pairs in vector blocks 100-699, cross-block pairs in 700-1099
    # and 1700-2099: every listed column is distinct)
    blocks = np.concatenate([rng.choice(np.arange(100, 700), 32, replace=False),
                             rng.choice(np.arange(700, 1100), NCANCEL - 32, replace=False)])
    pairs = []
    for t in range(NCANCEL):
        a, b = rng.choice(16, 2, replace=False)
        c1_ = int(blocks[t]) * 16 + int(a)
        c2_ = (int(blocks[t]) * 16 + int(b)) if t < 32 else (int(blocks[t]) + 1000) * 16 + int(b)
        pairs.append((c1_, c2_))
    w = wl._nonzero_uniform(wl.rng_for(wl.W_RAND, 72, key), 0.25, 2.0, NCANCEL, dtype=dtype)
    for t, (p1, p2) in enumerate(pairs):
        rows.append(np.array([CANCEL0 + t, CANCEL0 + t]))
        cols.append(np.array([p1, p2]))
        vals.append(np.array([w[t], -w[t]], dtype=dtype))
    # rows whose stored entries are all explicit zeros, in columns every x
    # set lists (those of the cancelling pairs)
    pc = np.array([p for pr in pairs for p in pr])
    for t in range(NZROW):
        zc = rng.choice(pc, 3, replace=False)
        rows.append(np.full(3, ZROW0 + t))
        cols.append(zc)
        vals.append(np.array([0.0, -0.0, 0.0], dtype=dtype))
    R = np.concatenate(rows)
    C = np.concatenate(cols)
    V = np.concatenate(vals).astype(dtype)
    # explicit zeros among the ordinary entries (crafted blocks included)
    zr = wl.rng_for(wl.W_RAND, 73, key).random(V.size)
    ordinary = (R < CANCEL0) | (R >= ZROW0 + NZROW)
    V[ordinary & (zr < 0.025)] = dtype(0.0)
    V[ordinary & (zr >= 0.025) & (zr < 0.04)] = dtype(-0.0)
    a = wl.csr_from_coo(M, N, R, C, V)
    return a, pairs


def x_sets(pairs, dtype):
    """Index lists on both blocker routes and both sides of the compaction
    threshold, each with the cancelling pairs listed, +-0 values and three
    marker-valued entries."""
    rng = wl.rng_for(wl.W_RAND, 74, 0)
    pc = np.array([p for pr in pairs for p in pr], dtype=np.int64)
    starts = rng.choice(N // 64 - 2, 47, replace=False) * 64
    base = {
        # (indices, k <= 2048 route?, compacted pull?)
        "uniform-200": (rng.choice(N, 200, replace=False), True, True),
        "uniform-1800": (rng.choice(N, 1800, replace=False), True, False),
        "clustered-3000": (np.concatenate([np.arange(s, s + 64) for s in starts])[:3000], False, True),
        "uniform-3000": (rng.choice(N, 3000, replace=False), False, False),
    }
    out = {}
    for name, (idx, small, compact) in base.items():
        idx = np.setdiff1d(idx, pc)
        k0 = idx.size
        idx = np.concatenate([idx, pc]).astype(np.int32)
        vr = wl.rng_for(wl.W_RAND, 75, k0)
        val = wl._nonzero_uniform(vr, -1.0, 1.0, idx.size, dtype=dtype)
        # each cancelling pair shares one value
        val[k0::2] = val[k0 + 1::2]
        sel = vr.permutation(k0)
        val[sel[: k0 // 20]] = dtype(0.0)
        val[sel[k0 // 20: k0 // 10]] = dtype(-0.0)
        marker = sel[k0 // 10: k0 // 10 + 3]
        if dtype == np.float32:
            val.view(np.uint32)[marker] = F32_MARKER
        else:
            val.view(np.uint16)[marker] = F16_MARKER
        perm = vr.permutation(idx.size)  # any order is allowed
        assert (idx.size <= 2048) == small, (name, idx.size)
        out[name] = (idx[perm], val[perm], compact)
    return out


@pytest.fixture(scope="module", params=["f32", "f16"])
def setup(request, torch):
    dtype = np.float32 if request.param == "f32" else np.float16
    a, pairs = edge_matrix(dtype)
    A, om = gpu_matrix(a), oracle_matrix(a)
    info = A.info()
    assert all(v > 0 for v in info["blocks_by_type"].values()), info["blocks_by_type"]
    return request.param, dtype, a, A, om, dbs.Context(A), x_sets(pairs, dtype)


@pytest.mark.parametrize("xname", ["uniform-200", "uniform-1800", "clustered-3000", "uniform-3000"])
def test_structural_values(setup, xname):
    tag, dtype, a, A, om, ctx, xs = setup
    xi, xv, compact = xs[xname]
    # what the oracle says these inputs reach: cancelled rows, rows of only
    # zero products, NaN rows -- the case must exercise all three
    ri, rv, rs = om.spmspv(xi, xv.astype(np.float64))
    cancel = np.isin(ri, np.arange(CANCEL0, CANCEL0 + NCANCEL))
    assert cancel.sum() == NCANCEL and np.all(rv[cancel] == 0.0) and np.all(rs[cancel] > 0)
    assert np.sum((rs == 0) & (rv == 0)) > 0, "no row of only zero products"
    zrow = np.isin(ri, np.arange(ZROW0, ZROW0 + NZROW))
    assert zrow.sum() == NZROW and np.all(rv[zrow] == 0.0) and np.all(rs[zrow] == 0.0)
    assert np.isnan(rv).sum() > 0, "no NaN row"
    for p in PATHS:
        label = f"edge {tag} x={xname} k={xi.size} path={p}"
        log(label)
        st = check_spmspv(ctx, A, om, a, xi, xv, path=p, label=label)
        sb = st["n_nzblk"] / st["n_blk"]
        assert (sb < COMPACT_BELOW) == compact, (label, sb)
        log(f"  s_b = {sb:.3f}, path {st['path']}, y_nnz {st['y_nnz']}")
    for p in PATHS:
        label = f"edge {tag} x={xname} OR-AND path={p}"
        log(label)
        check_spmspv(ctx, A, om, a, xi, None, path=p, semiring="or_and", label=label)


def test_structural_values_masked(setup):
    """The same values under a complemented output mask that keeps half the
    cancelling and zero-only rows."""
    tag, dtype, a, A, om, ctx, xs = setup
    from gpu_helpers import mask_words
    bits = wl.rng_for(wl.W_RAND, 76, 0).random(M) < 0.5
    mw = mask_words(bits)
    for xname in ("uniform-200", "uniform-3000"):
        xi, xv, _ = xs[xname]
        for p in PATHS:
            label = f"edge {tag} x={xname} complemented mask path={p}"
            log(label)
            check_spmspv(ctx, A, om, a, xi, xv, path=p, mask=mw, complement=True, label=label)


def test_decode_marker_and_signed_zero(torch):
    """Dense activations: +-0 are inactive, NaN entries (the marker bits and
    other NaN payloads) are active and reach their rows."""
    w = wl.decode_layer(512, 1024)
    A, om = gpu_matrix(w), oracle_matrix(w)
    ctx = dbs.Context(A)
    a16 = wl.decode_activation(1024, key=3)
    bits = a16.view(np.uint16)
    nz = np.nonzero(bits & 0x7FFF)[0]
    z = np.nonzero((bits & 0x7FFF) == 0)[0]
    bits[z[:40]] = 0x8000                       # -0: inactive
    bits[nz[:2]] = F16_MARKER                   # the marker pattern
    bits[nz[2]] = 0x7E01                        # another quiet NaN
    bits[nz[3]] = 0xFC01                        # a signalling-pattern NaN, negative
    for p in PATHS:
        label = f"decode marker/NaN/-0 path={p}"
        log(label)
        check_decode_dense(ctx, A, om, a16, p, label)
