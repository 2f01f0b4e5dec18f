"""Seeded synthetic inputs shaped like the DB-SpMSpV paper's workloads.

Shared by the tests, the benchmark and the oracle's timing leg; holds none of
the SpMSpV/BFS arithmetic.  The paper evaluates on SuiteSparse matrices, a
collection of symmetric graphs and Wanda-pruned LLM layers (Sec. 5.1), none
of which is available here; these generators stand in for them:

* ``tiny``       4096x4096, exactly 8 distinct uniform columns per row,
                 values U(-1,1); x: 1% unique uniform indices, values U(-1,1).
* ``rmat``       R-MAT (a,b,c,d = .57,.19,.19,.05), edge factor 16,
                 symmetrised, self-loops dropped, de-duplicated; fp32 U(0,1)
                 values or pattern only.  Power-law graphs / BFS.
* ``sparse_x``   x of a given density, uniform unique indices or
                 64-aligned runs of 64 ("clustered").
* ``mesh``       126^3 7-point stencil (non-periodic) plus 5% uniform random
                 entries, one random relabelling of rows and columns;
                 N(0,1) values.  Structured-grid / FEM class.
* ``ball_x``     x made of BFS balls around random seeds on the symmetrised
                 pattern (last level truncated by seeded choice).
* ``decode_layer`` fp16 [out, in] weight with Bernoulli(0.5) keep mask,
                 N(0, 1/in) values; activation with exactly 10% nonzeros,
                 70% of them inside 10% of the 64-wide blocks, |N(0,1)| values.
* ``crafted``    small matrices whose 16x16 blocks hit every block format and
                 every classifier boundary, with ragged (non-multiple-of-16)
                 edges.

Seeds: base seed 42 (the paper's fixed seed, Sec. 5.2) with one child stream
per (workload, array) via numpy's SeedSequence.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass

import numpy as np

BASE_SEED = 42
_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
_LIB = os.path.join(_HERE, "libworkloads.so")


def build() -> str:
    cmd = ["gcc", "-O3", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-o", _LIB + ".tmp", _SRC]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


_lib = None


def _get_lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        i64p = np.ctypeslib.ndpointer(dtype=np.int64, flags="C_CONTIGUOUS")
        i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")
        lib.wl_rmat_csr.restype = ctypes.c_int64
        lib.wl_rmat_csr.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_double, ctypes.c_double,
                                    ctypes.c_double, ctypes.c_uint64, i64p, i32p]
        lib.wl_components.restype = None
        lib.wl_components.argtypes = [ctypes.c_int32, i64p, i32p, i32p]
        _lib = lib
    return _lib


def rng_for(*key: int) -> np.random.Generator:
    """Child stream of the base seed for a (workload, array) key."""
    return np.random.default_rng(np.random.SeedSequence(BASE_SEED, spawn_key=tuple(key)))


def seed64_for(*key: int) -> int:
    return int(np.random.SeedSequence(BASE_SEED, spawn_key=tuple(key)).generate_state(1, np.uint64)[0])


# workload ids used in the seed keys
W_TINY, W_RMAT, W_MESH, W_DECODE, W_CRAFT, W_RAND, W_FEM = 1, 2, 3, 5, 7, 9, 11


@dataclass
class CSR:
    m: int
    n: int
    row_ptr: np.ndarray  # int64 [m+1]
    col_idx: np.ndarray  # int32 [nnz], ascending within each row
    vals: np.ndarray | None  # float32 / float16 [nnz] or None (pattern)

    @property
    def nnz(self) -> int:
        return int(self.row_ptr[-1])

    def dense(self) -> np.ndarray:
        d = np.zeros((self.m, self.n), dtype=np.float64)
        rows = np.repeat(np.arange(self.m), np.diff(self.row_ptr))
        d[rows, self.col_idx] = 1.0 if self.vals is None else self.vals.astype(np.float64)
        return d


def _nonzero_uniform(rng, lo, hi, size, dtype=np.float32):
    v = rng.uniform(lo, hi, size).astype(dtype)
    bad = v == 0
    while bad.any():
        v[bad] = rng.uniform(lo, hi, int(bad.sum())).astype(dtype)
        bad = v == 0
    return v


def _nonzero_normal(rng, scale, size, dtype=np.float32, absval=False):
    v = (rng.standard_normal(size) * scale).astype(dtype)
    if absval:
        v = np.abs(v)
    bad = v == 0
    while bad.any():
        w = (rng.standard_normal(int(bad.sum())) * scale).astype(dtype)
        v[bad] = np.abs(w) if absval else w
        bad = v == 0
    return v


def csr_from_coo(m, n, rows, cols, vals=None) -> CSR:
    """CSR with ascending columns from unique (row, col) pairs."""
    rows = np.asarray(rows, dtype=np.int64)
    cols = np.asarray(cols, dtype=np.int64)
    key = rows * n + cols
    order = np.argsort(key, kind="stable")
    key = key[order]
    if key.size and np.any(key[1:] == key[:-1]):
        raise ValueError("duplicate entries")
    r = rows[order]
    row_ptr = np.zeros(m + 1, dtype=np.int64)
    row_ptr[1:] = np.cumsum(np.bincount(r, minlength=m))
    v = None if vals is None else np.asarray(vals)[order]
    return CSR(m, n, row_ptr, cols[order].astype(np.int32), v)


# ----------------------------------------------------------------------------
# tiny: 4096 x 4096, 8 distinct uniform columns per row, U(-1,1)
# ----------------------------------------------------------------------------
def tiny(m: int = 4096, n: int = 4096, per_row: int = 8) -> CSR:
    rng = rng_for(W_TINY, 0)
    cols = np.empty((m, per_row), dtype=np.int64)
    for i in range(m):
        cols[i] = np.sort(rng.choice(n, per_row, replace=False))
    rows = np.repeat(np.arange(m), per_row)
    vals = _nonzero_uniform(rng_for(W_TINY, 1), -1.0, 1.0, m * per_row)
    row_ptr = np.arange(0, m * per_row + 1, per_row, dtype=np.int64)
    del rows
    return CSR(m, n, row_ptr, cols.reshape(-1).astype(np.int32), vals)


# ----------------------------------------------------------------------------
# sparse x
# ----------------------------------------------------------------------------
def sparse_x(n: int, density: float, kind: str = "uniform", key: tuple = (0,),
             lo: float = 0.0, hi: float = 1.0, k: int | None = None):
    """(idx int32 sorted-unique, val float32) with k = round(density * n).

    ``uniform``: k unique uniform indices.  ``clustered``: ceil(k/64) runs of
    64 consecutive indices at distinct 64-aligned starts; the last run is
    truncated so that exactly k indices remain.
    """
    if k is None:
        k = int(round(density * n))
    k = max(0, min(k, n))
    rng = rng_for(W_RAND, *key, 0)
    if kind == "uniform":
        idx = np.sort(rng.choice(n, k, replace=False)) if k else np.zeros(0, np.int64)
    elif kind == "clustered":
        runs = (k + 63) // 64
        nslots = n // 64
        if runs > nslots:
            raise ValueError("too many runs")
        starts = rng.choice(nslots, runs, replace=False) * 64
        idx = (starts[:, None] + np.arange(64)[None, :]).reshape(-1)[:k]
        idx = np.sort(idx)
    else:
        raise ValueError(kind)
    vals = _nonzero_uniform(rng_for(W_RAND, *key, 1), lo, hi, k) if k else np.zeros(0, np.float32)
    return idx.astype(np.int32), vals.astype(np.float32)


# ----------------------------------------------------------------------------
# R-MAT
# ----------------------------------------------------------------------------
def rmat(scale: int, edge_factor: int = 16, values: bool = True,
         abcd=(0.57, 0.19, 0.19, 0.05)) -> CSR:
    lib = _get_lib()
    n = 1 << scale
    row_ptr = np.zeros(n + 1, dtype=np.int64)
    col = np.zeros(2 * edge_factor * n, dtype=np.int32)
    nnz = lib.wl_rmat_csr(scale, edge_factor, abcd[0], abcd[1], abcd[2],
                          seed64_for(W_RMAT, scale, 0), row_ptr, col)
    if nnz < 0:
        raise MemoryError("wl_rmat_csr")
    col = col[:nnz].copy()
    vals = None
    if values:
        rng = rng_for(W_RMAT, scale, 1)
        vals = rng.random(nnz, dtype=np.float32)
        bad = vals == 0
        while bad.any():
            vals[bad] = rng.random(int(bad.sum()), dtype=np.float32)
            bad = vals == 0
    return CSR(n, n, row_ptr, col, vals)


def components(a: CSR) -> np.ndarray:
    comp = np.zeros(a.m, dtype=np.int32)
    _get_lib().wl_components(a.m, a.row_ptr, a.col_idx, comp)
    return comp


def bfs_sources(a: CSR, count: int = 16, key: int = 0) -> np.ndarray:
    """`count` distinct sources drawn uniformly from the largest component."""
    comp = components(a)
    labels, sizes = np.unique(comp, return_counts=True)
    giant = labels[np.argmax(sizes)]
    verts = np.nonzero(comp == giant)[0]
    rng = rng_for(W_RMAT, 99, key)
    return np.sort(rng.choice(verts, min(count, verts.size), replace=False)).astype(np.int32)


# ----------------------------------------------------------------------------
# relabelled 3-D 7-point mesh plus 5% random entries
# ----------------------------------------------------------------------------
def mesh(side: int = 126, extra_frac: float = 0.05) -> CSR:
    N = side ** 3
    v = np.arange(N, dtype=np.int64)
    x, rem = np.divmod(v, side * side)
    y, z = np.divmod(rem, side)
    rows = [v]
    cols = [v]
    for dim, coord, stride in ((0, x, side * side), (1, y, side), (2, z, 1)):
        for d in (-1, 1):
            ok = (coord + d >= 0) & (coord + d < side)
            rows.append(v[ok])
            cols.append(v[ok] + d * stride)
    r = np.concatenate(rows)
    c = np.concatenate(cols)
    n_stencil = r.size
    n_extra = int(round(extra_frac * n_stencil))
    rng = rng_for(W_MESH, 0)
    er = rng.integers(0, N, n_extra)
    ec = rng.integers(0, N, n_extra)
    key = np.unique(np.concatenate([r * N + c, er * N + ec]))
    r, c = np.divmod(key, N)
    perm = rng_for(W_MESH, 1).permutation(N)
    a = csr_from_coo(N, N, perm[r], perm[c])
    a.vals = _nonzero_normal(rng_for(W_MESH, 2), 1.0, a.nnz)
    return a


def fem(side: int = 56, dof: int = 3) -> CSR:
    """FEM-like matrix in natural order: a side^3 grid with `dof` unknowns per
    node and a 27-point stencil coupling every unknown of a node with every
    unknown of its (up to 26) neighbours and itself.  Rows and columns are
    node-major, dof-minor (no relabelling), so 16x16 blocks near the diagonal
    are dense-ish, the regime of the paper's FEM matrices.  Values N(0,1)."""
    N = side ** 3
    v = np.arange(N, dtype=np.int64)
    x, rem = np.divmod(v, side * side)
    y, z = np.divmod(rem, side)
    nbs = []
    for dx in (-1, 0, 1):           # lexicographic offsets: ascending neighbour ids
        for dy in (-1, 0, 1):
            for dz in (-1, 0, 1):
                ok = ((x + dx >= 0) & (x + dx < side) & (y + dy >= 0) & (y + dy < side)
                      & (z + dz >= 0) & (z + dz < side))
                nbs.append(np.where(ok, v + dx * side * side + dy * side + dz, -1))
    nb = np.stack(nbs, axis=1)                       # [N, 27], -1 = outside
    cnt = (nb >= 0).sum(axis=1)                      # neighbours per node (incl. itself)
    row_len = np.repeat(cnt * dof, dof)              # every unknown of a node: same columns
    row_ptr = np.zeros(N * dof + 1, dtype=np.int64)
    np.cumsum(row_len, out=row_ptr[1:])
    nbv = nb[nb >= 0]                                # flattened valid neighbours, node-major
    node_cols = (nbv[:, None] * dof + np.arange(dof)[None, :]).reshape(-1)
    node_ptr = np.zeros(N + 1, dtype=np.int64)
    np.cumsum(cnt * dof, out=node_ptr[1:])
    # each of the dof rows of node v repeats node_cols[node_ptr[v]:node_ptr[v+1]]
    rep_start = np.repeat(node_ptr[:-1], dof)
    lens = np.repeat(cnt * dof, dof)
    idx = np.repeat(rep_start - row_ptr[:-1], lens) + np.arange(int(row_ptr[-1]), dtype=np.int64)
    col = node_cols[idx].astype(np.int32)
    vals = _nonzero_normal(rng_for(W_FEM, side, dof), 1.0, col.size)
    return CSR(N * dof, N * dof, row_ptr, col, vals)


def symmetric_pattern(a: CSR):
    import scipy.sparse as sp
    A = sp.csr_matrix((np.ones(a.nnz, dtype=np.int8), a.col_idx, a.row_ptr), shape=(a.m, a.n))
    S = ((A + A.T) > 0).tocsr()
    return S


def ball_x(a: CSR, density: float, key: int = 0, S=None):
    """x from BFS balls grown on the symmetrised pattern around
    ceil(k/1024) random seeds; the last level is truncated by seeded choice."""
    n = a.n
    k = int(round(density * n))
    if S is None:
        S = symmetric_pattern(a)
    rng = rng_for(W_MESH, 10, key)
    nseeds = max(1, (k + 1023) // 1024)
    seeds = rng.choice(n, nseeds, replace=False)
    inball = np.zeros(n, dtype=bool)
    inball[seeds] = True
    count = nseeds
    frontier = seeds
    while count < k and frontier.size:
        nb = np.unique(S[frontier].indices)
        nb = nb[~inball[nb]]
        if count + nb.size >= k:
            nb = rng.choice(nb, k - count, replace=False)
        inball[nb] = True
        count += nb.size
        frontier = nb
    idx = np.nonzero(inball)[0].astype(np.int32)
    vals = _nonzero_uniform(rng_for(W_MESH, 11, key), -1.0, 1.0, idx.size)
    return idx, vals


# ----------------------------------------------------------------------------
# sparse decode linear layer
# ----------------------------------------------------------------------------
def decode_layer(out_f: int, in_f: int, keep: float = 0.5) -> CSR:
    rng = rng_for(W_DECODE, out_f, in_f, 0)
    mask = rng.random((out_f, in_f), dtype=np.float32) < keep
    row_ptr = np.zeros(out_f + 1, dtype=np.int64)
    row_ptr[1:] = np.cumsum(mask.sum(axis=1))
    cols = np.nonzero(mask)[1].astype(np.int32)
    vals = _nonzero_normal(rng_for(W_DECODE, out_f, in_f, 1), 1.0 / math.sqrt(in_f), cols.size,
                           dtype=np.float16)
    return CSR(out_f, in_f, row_ptr, cols, vals)


def decode_activation(in_f: int, density: float = 0.1, hot_block_frac: float = 0.1,
                      hot_share: float = 0.7, key: int = 0) -> np.ndarray:
    """Dense fp16 activation, exactly round(density*in) nonzeros, round(hot_share)
    of them in round(hot_block_frac) of the 64-wide blocks."""
    rng = rng_for(W_DECODE, in_f, 7, key)
    k = int(round(density * in_f))
    nblk = in_f // 64
    nhot = max(1, int(round(hot_block_frac * nblk)))
    hot_blocks = rng.choice(nblk, nhot, replace=False)
    hot_pos = (hot_blocks[:, None] * 64 + np.arange(64)[None, :]).reshape(-1)
    is_hot = np.zeros(in_f, dtype=bool)
    is_hot[hot_pos] = True
    cold_pos = np.nonzero(~is_hot)[0]
    k_hot = min(int(round(hot_share * k)), hot_pos.size)
    sel = np.concatenate([rng.choice(hot_pos, k_hot, replace=False),
                          rng.choice(cold_pos, k - k_hot, replace=False)])
    a = np.zeros(in_f, dtype=np.float16)
    a[sel] = _nonzero_normal(rng_for(W_DECODE, in_f, 8, key), 1.0, k, dtype=np.float16, absval=True)
    return a


# ----------------------------------------------------------------------------
# random small matrices and crafted block structures (tests)
# ----------------------------------------------------------------------------
def random_csr(m: int, n: int, density: float, key: tuple, dtype=np.float32, lo=-1.0, hi=1.0) -> CSR:
    rng = rng_for(W_RAND, *key, 100)
    mask = rng.random((m, n)) < density
    rows, cols = np.nonzero(mask)
    if dtype is None:
        vals = None
    elif dtype == np.float16:
        vals = _nonzero_normal(rng_for(W_RAND, *key, 101), 1.0, rows.size, dtype=np.float16)
    else:
        vals = _nonzero_uniform(rng_for(W_RAND, *key, 101), lo, hi, rows.size, dtype=dtype)
    return csr_from_coo(m, n, rows, cols, vals)


def crafted(dtype=np.float32, key: int = 0) -> CSR:
    """A 120 x 200 matrix (ragged: neither is a multiple of 16) whose 16x16
    blocks cover every block-format rule and boundary:

    nnz 1, 31 (< 32), 32 (= 32), 128 (= 128), 129 (> 128), 256 (full);
    two full columns (column skew), two full rows (row skew), a scattered
    64-entry block, a diagonal block, a checkerboard, and blocks that straddle
    the ragged right and bottom edges.
    """
    m, n = 120, 200
    rng = rng_for(W_CRAFT, key, 0)
    ent = set()

    def blk(bi, bj, cells):
        for r, c in cells:
            i, j = bi * 16 + r, bj * 16 + c
            if i < m and j < n:
                ent.add((i, j))

    def rand_cells(cnt):
        pos = rng.choice(256, cnt, replace=False)
        return [(int(p) // 16, int(p) % 16) for p in pos]

    blk(0, 0, [(3, 5)])                                          # 1 nnz
    blk(0, 1, rand_cells(31))                                    # 31
    blk(0, 2, rand_cells(32))                                    # 32
    blk(0, 3, rand_cells(128))                                   # 128
    blk(0, 4, rand_cells(129))                                   # 129
    blk(0, 5, [(r, c) for r in range(16) for c in range(16)])    # full
    blk(1, 0, [(r, c) for r in range(16) for c in (2, 9)])       # two full columns
    blk(1, 1, [(r, c) for r in (4, 11) for c in range(16)])      # two full rows
    blk(1, 2, rand_cells(64))                                    # scattered 64
    blk(1, 3, [(r, r) for r in range(16)])                       # diagonal
    blk(1, 4, [(r, c) for r in range(16) for c in range(16) if (r + c) % 2 == 0])  # 128 checker
    blk(2, 2, [(r, c) for r in range(16) for c in (0, 1, 2)] + [(0, 5)])  # 3 full cols + 1
    blk(2, 3, [(r, c) for r in (0, 1, 2) for c in range(16)] + [(5, 0)])  # 3 full rows + 1
    blk(2, 6, rand_cells(40))
    blk(3, 7, rand_cells(200))                                   # dense
    blk(3, 12, [(r, c) for r in range(16) for c in range(8)])    # straddles right edge (n=200)
    blk(7, 0, [(r, c) for r in range(8) for c in range(16)])     # straddles bottom edge (m=120)
    blk(7, 12, [(r, c) for r in range(16) for c in range(16)])   # corner: 8x8 valid
    blk(4, 5, [(r, c) for r in range(16) for c in range(16) if c < 2 or r == 7])  # mixed skew
    blk(5, 8, rand_cells(33))
    blk(6, 9, rand_cells(100))
    for _ in range(300):                                         # sprinkle of COO noise
        ent.add((int(rng.integers(0, m)), int(rng.integers(0, n))))
    rows, cols = zip(*sorted(ent))
    rows = np.array(rows)
    cols = np.array(cols)
    if dtype is None:
        vals = None
    elif dtype == np.float16:
        vals = _nonzero_normal(rng_for(W_CRAFT, key, 1), 1.0, rows.size, dtype=np.float16)
    else:
        vals = _nonzero_uniform(rng_for(W_CRAFT, key, 1), -1.0, 1.0, rows.size, dtype=dtype)
    return csr_from_coo(m, n, rows, cols, vals)
