"""GPU parity of the pull path on both sides of its compaction threshold.

Below N_nzblk / N_blk = 0.4 the pull kernel leaves the COO segments to the
compacted pass (active slots listed per wave region, then processed 256 per
round with per-run LDS sums); above it the segment loop takes them.  The cases
here pin both against the oracle: several regions per matrix and regions with
no segment, rounds that span more block rows than the per-round run capacity
(short rows), output masks, OR-AND, and one context reused across matrices of
different sizes.
"""
import numpy as np
import pytest

import paper_2608_16308_amd as dbs
import workloads as wl
from gpu_helpers import check_spmspv, gpu_matrix, log, mask_words, oracle_matrix, torch_mod

pytestmark = pytest.mark.gpu

COMPACT_BELOW = 0.4


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def _x_on_blocks(n, frac, key, clustered=False):
    """x whose active vector blocks are a given fraction of all of them."""
    rng = wl.rng_for(wl.W_RAND, 61, key)
    nvb = (n + 15) // 16
    want = max(1, int(frac * nvb))
    if clustered:
        start = int(rng.integers(0, max(1, nvb - want)))
        blocks = np.arange(start, start + want)
    else:
        blocks = np.sort(rng.choice(nvb, want, replace=False))
    # one or two entries per active vector block
    cols = []
    for b in blocks:
        c0 = b * 16 + int(rng.integers(0, 16))
        cols.append(min(c0, n - 1))
        if rng.random() < 0.5:
            cols.append(min(b * 16 + int(rng.integers(0, 16)), n - 1))
    xi = np.unique(np.array(cols, dtype=np.int64)).astype(np.int32)
    xv = wl._nonzero_uniform(wl.rng_for(wl.W_RAND, 62, key), -1.0, 1.0, xi.size)
    return xi, xv


@pytest.mark.parametrize("frac,clustered", [(0.06, False), (0.2, False), (0.39, False), (0.45, False),
                                            (0.9, False), (0.2, True)])
def test_pull_both_sides_of_threshold_rmat(torch, frac, clustered):
    a = wl.rmat(14)
    A, om = gpu_matrix(a), oracle_matrix(a)
    ctx = dbs.Context(A)
    xi, xv = _x_on_blocks(a.n, frac, (1, int(frac * 100), clustered))
    label = f"rmat14 pull active-fraction~{frac} clustered={clustered} k={xi.size}"
    log(label)
    st = check_spmspv(ctx, A, om, a, xi, xv, path="pull", label=label)
    sb = st["n_nzblk"] / st["n_blk"]
    log(f"  s_b = {sb:.3f} ({'compacted' if sb < COMPACT_BELOW else 'segment loop'})")
    # the cases straddle the threshold as intended
    if frac < COMPACT_BELOW - 0.02:
        assert sb < COMPACT_BELOW
    if frac > COMPACT_BELOW + 0.02:
        assert sb >= COMPACT_BELOW


def test_compacted_short_rows_span_many_runs(torch):
    """One entry per row: every block row holds a handful of one-entry blocks,
    so a round of 256 active slots spans far more than 32 block rows."""
    m, n = 40000, 4096
    rng = wl.rng_for(wl.W_RAND, 63, 0)
    cols = rng.integers(0, n, m).astype(np.int32)
    row_ptr = np.arange(m + 1, dtype=np.int64)
    vals = wl._nonzero_uniform(wl.rng_for(wl.W_RAND, 64, 0), -1.0, 1.0, m).astype(np.float32)
    a = wl.CSR(m, n, row_ptr, cols, vals)
    A, om = gpu_matrix(a), oracle_matrix(a)
    ctx = dbs.Context(A)
    for frac in (0.1, 0.3):
        xi, xv = _x_on_blocks(n, frac, (2, int(frac * 100)))
        label = f"short rows {m}x{n} frac={frac}"
        log(label)
        st = check_spmspv(ctx, A, om, a, xi, xv, path="pull", label=label)
        assert st["n_nzblk"] / st["n_blk"] < COMPACT_BELOW


@pytest.mark.parametrize("complement", [False, True])
def test_compacted_with_output_mask_and_or_and(torch, complement):
    a = wl.random_csr(3000, 2400, 0.01, key=(65, 0))
    A, om = gpu_matrix(a), oracle_matrix(a)
    ctx = dbs.Context(A)
    rng = wl.rng_for(wl.W_RAND, 66, int(complement))
    bits = rng.random(a.m) < 0.3
    # whole block rows masked out too
    bits[160:480] = False
    mask = mask_words(bits)
    xi, xv = _x_on_blocks(a.n, 0.15, (3, int(complement)))
    for sr in ("plus_times", "or_and"):
        label = f"masked compacted pull comp={complement} {sr}"
        log(label)
        st = check_spmspv(ctx, A, om, a, xi, xv if sr == "plus_times" else None, path="pull", mask=mask,
                          complement=complement, semiring=sr, label=label)
        assert st["n_nzblk"] / st["n_blk"] < COMPACT_BELOW


def test_compacted_context_reuse_and_repeat(torch):
    """A context sized by a large matrix serves a small one and back; calls
    repeat, so a region list left from an earlier call must not leak."""
    big = wl.rmat(13)
    small = wl.random_csr(500, 700, 0.04, key=(67, 0))
    Ab, As = gpu_matrix(big), gpu_matrix(small)
    ob, os_ = oracle_matrix(big), oracle_matrix(small)
    ctx = dbs.Context(Ab)
    for it in range(3):
        for a, A, om, frac in ((big, Ab, ob, 0.1 + 0.1 * it), (small, As, os_, 0.25)):
            xi, xv = _x_on_blocks(a.n, frac, (4, it, a.m))
            label = f"reuse it={it} {a.m}x{a.n} frac={frac:.1f}"
            log(label)
            check_spmspv(ctx, A, om, a, xi, xv, path="pull", label=label)
