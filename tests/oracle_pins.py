"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each ``check_*`` takes the path of an oracle shared library and raises
AssertionError on a mismatch.  ``test_oracle_pins.py`` runs them on the real
oracle; ``test_oracle_mutants.py`` runs them on copies of the oracle with a
planted mistake and requires every mistake to be caught.

The pins are independent of the oracle's own code:

* SpMSpV values: a dense fp64 matrix-vector product (numpy matmul) on tiny
  random inputs of every shape class; special cases with closed forms
  (identity, permutation, unit vector, full vector = SpMV via scipy,
  linearity over disjoint supports).
* y pattern and OR-AND: a dense Boolean pattern product (integer matmul).
* S_i: the dense product |A| |x|.
* Output masks: the unmasked result filtered by the bitmap, bit (i & 31) of
  word (i >> 5), and its complement.
* BFS: brute-force all-pairs unit distances (Floyd-Warshall) plus the
  minimum-id parent rule, and closed forms (path, star, complete graph,
  2-D grid, binary tree, directed chain for the edge direction).
"""
from __future__ import annotations

import numpy as np
import scipy.sparse as sp

import oracle
import workloads as wl

SHAPES = [(1, 1), (5, 17), (17, 5), (16, 16), (33, 48), (96, 95), (64, 1), (1, 64), (40, 40)]
DENSITIES = [0.0, 0.05, 0.3, 1.0]


def _om(a: wl.CSR, lib_path):
    return oracle.OracleMatrix(a.m, a.n, a.row_ptr, a.col_idx, a.vals, lib_path=lib_path)


def _x_support(n, rng, kind):
    if kind == "empty":
        return np.zeros(0, dtype=np.int32)
    if kind == "all":
        return np.arange(n, dtype=np.int32)
    k = int(rng.integers(1, n + 1))
    return rng.permutation(n)[:k].astype(np.int32)  # unsorted on purpose


def _dense_ref(a: wl.CSR, idx, val):
    D = a.dense()
    P = (D != 0) | _pattern(a)
    x = np.zeros(a.n)
    x[idx] = val
    xp = np.zeros(a.n, dtype=np.int64)
    xp[idx] = 1
    y = D @ x
    S = np.abs(D) @ np.abs(x)
    pat = (P.astype(np.int64) @ xp) > 0
    return y, S, pat


def _pattern(a: wl.CSR):
    P = np.zeros((a.m, a.n), dtype=bool)
    rows = np.repeat(np.arange(a.m), np.diff(a.row_ptr))
    P[rows, a.col_idx] = True
    return P


def check_dense_matvec(lib_path=None):
    case = 0
    for (m, n) in SHAPES:
        for d in DENSITIES:
            for kind in ("empty", "some", "all"):
                case += 1
                a = wl.random_csr(m, n, d, key=(11, case))
                rng = wl.rng_for(wl.W_RAND, 12, case)
                idx = _x_support(n, rng, kind)
                val = rng.uniform(-1, 1, idx.size).astype(np.float32)
                om = _om(a, lib_path)
                yi, yv, ys = om.spmspv(idx, val)
                y, S, pat = _dense_ref(a, idx, val.astype(np.float64))
                exp_idx = np.nonzero(pat)[0]
                assert np.array_equal(yi, exp_idx), (m, n, d, kind, "pattern")
                assert np.all(np.abs(yv - y[yi]) <= 1e-12 * S[yi]), (m, n, d, kind, "values")
                assert np.allclose(ys, S[yi], rtol=1e-12, atol=0), (m, n, d, kind, "S")
                # rows outside the pattern are exactly zero in the dense product
                off = np.ones(m, dtype=bool)
                off[yi] = False
                assert np.all(y[off] == 0.0)


def check_bool(lib_path=None):
    case = 0
    for (m, n) in SHAPES:
        for d in DENSITIES:
            case += 1
            a = wl.random_csr(m, n, d, key=(13, case), dtype=None)
            rng = wl.rng_for(wl.W_RAND, 14, case)
            idx = _x_support(n, rng, "some")
            om = _om(a, lib_path)
            yi = om.spmspv_bool(idx)
            xp = np.zeros(n, dtype=np.int64)
            xp[idx] = 1
            exp = np.nonzero((_pattern(a).astype(np.int64) @ xp) > 0)[0]
            assert np.array_equal(yi, exp), (m, n, d)


def check_special_cases(lib_path=None):
    rng = wl.rng_for(wl.W_RAND, 15, 0)
    n = 77
    # identity: y = x exactly
    eye = wl.csr_from_coo(n, n, np.arange(n), np.arange(n), np.ones(n, dtype=np.float32))
    idx = rng.permutation(n)[:30].astype(np.int32)
    val = rng.uniform(-1, 1, 30).astype(np.float32)
    yi, yv, _ = _om(eye, lib_path).spmspv(idx, val)
    order = np.argsort(idx)
    assert np.array_equal(yi, idx[order])
    assert np.array_equal(yv, val[order].astype(np.float64))
    # permutation: P[pi(j), j] = 1 -> y[pi(j)] = x[j]
    pi = rng.permutation(n)
    P = wl.csr_from_coo(n, n, pi, np.arange(n), np.ones(n, dtype=np.float32))
    yi, yv, _ = _om(P, lib_path).spmspv(idx, val)
    exp_i = pi[idx]
    o = np.argsort(exp_i)
    assert np.array_equal(yi, exp_i[o])
    assert np.array_equal(yv, val[o].astype(np.float64))
    # non-square, non-symmetric matrix; unit vector e_j picks column j exactly
    a = wl.random_csr(50, 70, 0.2, key=(15, 1))
    D = a.dense()
    om = _om(a, lib_path)
    for j in (0, 13, 69):
        xj = np.float32(0.75)
        yi, yv, _ = om.spmspv(np.array([j], dtype=np.int32), np.array([xj]))
        col = D[:, j]
        assert np.array_equal(yi, np.nonzero(col)[0])
        assert np.array_equal(yv, col[yi] * np.float64(xj))
    # full x = SpMV (scipy CSR matvec)
    x = rng.uniform(-1, 1, 70)
    yi, yv, ys = om.spmspv(np.arange(70, dtype=np.int32), x)
    A = sp.csr_matrix((a.vals.astype(np.float64), a.col_idx, a.row_ptr), shape=(50, 70))
    ysp = A @ x
    rows_nz = np.nonzero(np.diff(a.row_ptr))[0]
    assert np.array_equal(yi, rows_nz)
    assert np.all(np.abs(yv - ysp[yi]) <= 1e-12 * ys)
    # linearity over disjoint supports: y(x1 + x2) = y(x1) + y(x2)
    perm = rng.permutation(70).astype(np.int32)
    i1, i2 = perm[:30], perm[30:55]
    v1 = rng.uniform(-1, 1, 30)
    v2 = rng.uniform(-1, 1, 25)
    ya = np.zeros(50)
    for ii, vv in ((i1, v1), (i2, v2)):
        yi_, yv_, _ = om.spmspv(ii, vv)
        ya[yi_] += yv_
    yi, yv, ys = om.spmspv(np.concatenate([i1, i2]), np.concatenate([v1, v2]))
    assert np.all(np.abs(yv - ya[yi]) <= 1e-12 * ys)


def check_masks(lib_path=None):
    a = wl.random_csr(90, 60, 0.15, key=(16, 0))
    om = _om(a, lib_path)
    rng = wl.rng_for(wl.W_RAND, 16, 1)
    idx = rng.permutation(60)[:25].astype(np.int32)
    val = rng.uniform(-1, 1, 25)
    yi, yv, ys = om.spmspv(idx, val)
    words = (90 + 31) // 32
    allm = np.full(words, 0xFFFFFFFF, dtype=np.uint32)
    nonem = np.zeros(words, dtype=np.uint32)
    r = om.spmspv(idx, val, mask=allm)
    assert np.array_equal(r[0], yi) and np.array_equal(r[1], yv)
    assert om.spmspv(idx, val, mask=nonem)[0].size == 0
    r = om.spmspv(idx, val, mask=nonem, complement=True)
    assert np.array_equal(r[0], yi)
    bits = rng.random(90) < 0.5
    mask = np.zeros(words, dtype=np.uint32)
    for i in np.nonzero(bits)[0]:
        mask[i // 32] |= np.uint32(1) << np.uint32(i % 32)
    r = om.spmspv(idx, val, mask=mask)
    keep = bits[yi]
    assert np.array_equal(r[0], yi[keep]) and np.array_equal(r[1], yv[keep])
    r = om.spmspv(idx, val, mask=mask, complement=True)
    assert np.array_equal(r[0], yi[~keep]) and np.array_equal(r[1], yv[~keep])
    rb = om.spmspv_bool(idx, mask=mask, complement=True)
    assert np.array_equal(rb, yi[~keep])


# ------------------------------------------------------------------ BFS
def _graph(n, edges, symmetric=True):
    """CSR pattern with A[v][u] stored for every edge u -> v."""
    ent = set()
    for u, v in edges:
        if u == v:
            continue
        ent.add((v, u))
        if symmetric:
            ent.add((u, v))
    if ent:
        r, c = zip(*sorted(ent))
    else:
        r, c = (), ()
    return wl.csr_from_coo(n, n, np.array(r, dtype=np.int64), np.array(c, dtype=np.int64))


def _brute_bfs(a: wl.CSR, s):
    n = a.n
    P = _pattern(a)  # P[v][u]: edge u -> v
    INF = 10 ** 9
    dist = np.full((n, n), INF, dtype=np.int64)
    np.fill_diagonal(dist, 0)
    dist[P.T] = np.minimum(dist[P.T], 1)  # dist[u][v] = 1 for edge u -> v
    np.fill_diagonal(dist, 0)
    for k in range(n):
        dist = np.minimum(dist, dist[:, k:k + 1] + dist[k:k + 1, :])
    lvl = dist[s].copy()
    level = np.where(lvl >= INF, -1, lvl).astype(np.int32)
    parent = np.full(n, -1, dtype=np.int32)
    parent[s] = s
    for v in range(n):
        if v == s or level[v] < 0:
            continue
        cands = [u for u in range(n) if level[u] == level[v] - 1 and P[v, u]]
        parent[v] = min(cands)
    return level, parent


def check_bfs_bruteforce(lib_path=None):
    for case in range(24):
        rng = wl.rng_for(wl.W_RAND, 17, case)
        n = int(rng.integers(1, 65))
        p = float(rng.choice([0.02, 0.05, 0.1, 0.3]))
        sym = bool(case % 2 == 0)
        edges = [(u, v) for u in range(n) for v in range(n) if rng.random() < p]
        a = _graph(n, edges, symmetric=sym)
        om = _om(a, lib_path)
        for s in sorted(set([0, n - 1, int(rng.integers(0, n))])):
            level, parent, _ = om.bfs(s)
            el, ep = _brute_bfs(a, s)
            assert np.array_equal(level, el), (case, s, "level")
            assert np.array_equal(parent, ep), (case, s, "parent")


def check_bfs_closed_forms(lib_path=None):
    # path 0-1-...-(n-1): level = |v - s|, parent = neighbour toward s
    n = 50
    a = _graph(n, [(i, i + 1) for i in range(n - 1)])
    for s in (0, 17, 49):
        level, parent, nl = _om(a, lib_path).bfs(s)
        v = np.arange(n)
        assert np.array_equal(level, np.abs(v - s))
        exp = np.where(v < s, v + 1, np.where(v > s, v - 1, s))
        assert np.array_equal(parent, exp)
        assert nl == max(s, n - 1 - s) + 1
    # star centred at 0
    a = _graph(n, [(0, i) for i in range(1, n)])
    level, parent, _ = _om(a, lib_path).bfs(5)
    exp_l = np.full(n, 2)
    exp_l[5] = 0
    exp_l[0] = 1
    exp_p = np.zeros(n, dtype=np.int32)
    exp_p[5] = 5
    exp_p[0] = 5
    assert np.array_equal(level, exp_l) and np.array_equal(parent, exp_p)
    # complete graph: every other vertex at level 1 with parent s
    k = 20
    a = _graph(k, [(u, v) for u in range(k) for v in range(u + 1, k)])
    level, parent, _ = _om(a, lib_path).bfs(7)
    assert np.array_equal(level, np.where(np.arange(k) == 7, 0, 1))
    assert np.all(parent == 7)
    # 2-D grid R x C: level = Manhattan distance; parent = smallest-id
    # neighbour one step closer (up before left since ids grow row-major)
    R, C = 9, 13
    vid = lambda r, c: r * C + c  # noqa: E731
    edges = [(vid(r, c), vid(r, c + 1)) for r in range(R) for c in range(C - 1)]
    edges += [(vid(r, c), vid(r + 1, c)) for r in range(R - 1) for c in range(C)]
    a = _graph(R * C, edges)
    sr, sc = 4, 6
    level, parent, _ = _om(a, lib_path).bfs(vid(sr, sc))
    for r in range(R):
        for c in range(C):
            assert level[vid(r, c)] == abs(r - sr) + abs(c - sc)
            if (r, c) == (sr, sc):
                continue
            closer = []
            for dr, dc in ((-1, 0), (1, 0), (0, -1), (0, 1)):
                rr, cc = r + dr, c + dc
                if 0 <= rr < R and 0 <= cc < C and abs(rr - sr) + abs(cc - sc) == level[vid(r, c)] - 1:
                    closer.append(vid(rr, cc))
            assert parent[vid(r, c)] == min(closer)
    # complete binary tree rooted at 0: level = depth, parent = (v-1)//2
    n = 127
    a = _graph(n, [((v - 1) // 2, v) for v in range(1, n)])
    level, parent, _ = _om(a, lib_path).bfs(0)
    v = np.arange(n)
    assert np.array_equal(level, np.floor(np.log2(v + 1)).astype(np.int32))
    assert np.array_equal(parent[1:], (v[1:] - 1) // 2) and parent[0] == 0
    # directed chain u -> u+1 (A[u+1][u] stored): reached forward only
    a = _graph(30, [(i, i + 1) for i in range(29)], symmetric=False)
    level, parent, _ = _om(a, lib_path).bfs(0)
    assert np.array_equal(level, np.arange(30))
    level, parent, _ = _om(a, lib_path).bfs(29)
    assert level[29] == 0 and np.all(level[:29] == -1) and np.all(parent[:29] == -1)
    # isolated source
    a = _graph(10, [(1, 2)])
    level, parent, nl = _om(a, lib_path).bfs(5)
    assert nl == 1 and level[5] == 0 and parent[5] == 5 and np.sum(level >= 0) == 1


def check_decode(lib_path=None):
    w = wl.random_csr(40, 64, 0.5, key=(18, 0), dtype=np.float16)
    om = _om(w, lib_path)
    rng = wl.rng_for(wl.W_RAND, 18, 1)
    a = np.zeros(64, dtype=np.float16)
    pos = rng.choice(64, 9, replace=False)
    a[pos] = np.abs(rng.standard_normal(9)).astype(np.float16) + np.float16(0.01)
    a[3] = np.float16(-0.0)  # signed zero is inactive
    y64, S, y16 = oracle.decode_linear(om, a)
    D = w.dense()
    ref = D @ a.astype(np.float64)
    assert np.all(np.abs(y64 - ref) <= 1e-12 * S)
    assert np.array_equal(y16, ref.astype(np.float16))


def check_fp16_rounding(lib_path=None):
    """The fp16 reference is IEEE round-to-nearest-even straight from fp64
    (values from the IEEE 754 definition, not from any implementation)."""
    cases = [
        (1 + 2 ** -11, 1.0),                       # tie -> even (1.0)
        (1 + 3 * 2 ** -11, 1 + 2 ** -9),           # tie -> even (up)
        (1 + 2 ** -11 + 2 ** -40, 1 + 2 ** -10),   # above the tie: no double rounding via fp32
        (2049.0, 2048.0), (2051.0, 2052.0),
        (-(1 + 2 ** -11), -1.0),
        (65519.0, 65504.0), (65520.0, np.inf),
        (2 ** -25, 0.0), (3 * 2 ** -25, 2 ** -23),  # subnormal ties
    ]
    for v, e in cases:
        with np.errstate(over="ignore"):
            got = np.float64(v).astype(np.float16)
        assert float(got) == e, (v, float(got), e)
    # decode_linear's fp16 output follows that rounding of its fp64 sum
    w = wl.csr_from_coo(1, 2, np.array([0, 0]), np.array([0, 1]),
                        np.array([1.0, 2 ** -11], dtype=np.float16))
    om = _om(w, lib_path)
    y64, S, y16 = oracle.decode_linear(om, np.array([1.0, 1.0], dtype=np.float16))
    assert y64[0] == 1 + 2 ** -11 and float(y16[0]) == 1.0


def check_within_tol(fn=None):
    """The acceptance rule of every value comparison against the oracle.

    Values with exact binary forms put each case exactly on, or one double
    beyond, the bound rel * S, so that a strict comparison, a dropped abs, a
    bound of rel + S or rel * |y_ref|, or a NaN accepted against a number each
    flips at least one verdict.
    """
    fn = fn or oracle.within_tol
    tol1 = 1e-5 * 1.0  # the bound for S = 1 at the default rel, as the rule computes it
    up = np.nextafter
    cases = [
        # (y_gpu, y_ref, S, accept)
        (tol1, 0.0, 1.0, True),                       # exactly on the bound
        (-tol1, 0.0, 1.0, True),                      # below the reference by the bound
        (up(tol1, np.inf), 0.0, 1.0, False),          # one double beyond
        (-up(tol1, np.inf), 0.0, 1.0, False),
        (-2.0 * tol1, 0.0, 1.0, False),               # far below (a dropped abs accepts it)
        (0.0, 0.0, 0.0, True),                        # S = 0: exact equality only
        (5e-324, 0.0, 0.0, False),                    # smallest subnormal off
        (1e-6, 0.0, 0.0, False),
        (0.5 + 5e-4, 0.5, 100.0, True),               # cancellation: S >> |y_ref|
        (0.5 + 2e-3, 0.5, 100.0, False),
        (1e30 * (1 + 0.5e-5), 1e30, 1e30, True),      # relative at large scale
        (1e30 * (1 + 2e-5), 1e30, 1e30, False),
        (np.nan, 1.0, 1.0, False),                    # NaN result, number expected
        (1.0, np.nan, np.nan, False),                 # number result, NaN expected
        (np.nan, np.nan, np.nan, True),               # NaN where the reference is NaN
        (np.inf, np.inf, np.inf, True),
        (-np.inf, np.inf, np.inf, False),
        (1.0, np.inf, np.inf, False),                 # an infinite reference demands it exactly
        (np.inf, 1.0, 1.0, False),
        (-0.0, 0.0, 0.0, True),                       # the sign of an exact zero sum is free
    ]
    g = np.array([c[0] for c in cases], dtype=np.float64)
    r = np.array([c[1] for c in cases], dtype=np.float64)
    s = np.array([c[2] for c in cases], dtype=np.float64)
    want = np.array([c[3] for c in cases])
    got = np.asarray(fn(g, r, s))
    assert got.shape == want.shape, ("within_tol shape", got.shape)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, ("within_tol verdicts", [cases[i] for i in bad])
    # element-wise: one verdict per element, in order, for float32 inputs too
    g32 = np.array([1.0, 1.5, 2.0], dtype=np.float32)
    r64 = np.array([1.0, 1.0, 2.0 + 1e-9], dtype=np.float64)
    s64 = np.array([1.0, 1.0, 1.0], dtype=np.float64)
    assert np.array_equal(np.asarray(fn(g32, r64, s64)), [True, False, True])
    # another rel scales the bound; with rel and S powers of two the bound
    # 2^-17 * 8 = 2^-14 is exact at any magnitude of the reference
    assert np.array_equal(np.asarray(fn(np.array([1.0 + 2.0 ** -14, up(1.0 + 2.0 ** -14, 2.0), 1.0 - 2.0 ** -14]),
                                        np.ones(3), np.full(3, 8.0), 2.0 ** -17)), [True, False, True])
    assert np.array_equal(np.asarray(fn(np.array([1e-3, 2e-3]), np.zeros(2), np.ones(2), 1e-3)), [True, False])
    # arrays of different shapes are an error, not a broadcast
    for shapes in (((3,), (2,), (2,)), ((3,), (1,), (1,)), ((3,), (3,), ())):
        try:
            fn(*(np.zeros(sh) for sh in shapes))
        except ValueError:
            pass
        else:
            raise AssertionError(f"within_tol accepted arrays of shapes {shapes}")


ALL_CHECKS = [check_fp16_rounding, check_dense_matvec, check_bool, check_special_cases, check_masks,
              check_bfs_bruteforce, check_bfs_closed_forms, check_decode]
