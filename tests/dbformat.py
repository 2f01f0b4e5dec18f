"""Independent Python reader of the DB format described in include/dbspmspv.h.

Used by the CPU tests to check the C++ builder: decode every block record back
into (row, col, value) triples, recompute the block classifier, the block-CSC
view and the pull segments from their definitions (Sec. 3.2.1, 3.3.2).
"""
from __future__ import annotations

import numpy as np

COO, DENSE, FCSR, FCSC, CSR = range(5)
WEIGHT = {DENSE: 4, FCSR: 2, FCSC: 2, CSR: 2, COO: 1}


def desc_fields(d):
    d = int(d)
    return d >> 16, ((d >> 8) & 0xFF) + 1, d & 7


def desc_inline(d):
    return (int(d) >> 3) & 1 == 1


def inline_capacity(vb):
    return 48 // (8 + 8 * vb)


def seg_fields(s):
    s = int(s)
    return s & 0xFFFFFFFF, (s >> 32) & 0x7FFFFFF, ((s >> 59) & 0xF) + 1, (s >> 63) & 1


def _vals(pay, at, count, vb):
    if vb == 0:
        return [None] * count
    raw = pay[at: at + count * vb].tobytes()
    return list(np.frombuffer(raw, dtype=np.float32 if vb == 4 else np.uint16))


def _u16(pay, at):
    return int(pay[at]) | (int(pay[at + 1]) << 8)


def decode_block(pay, d, vb):
    """Returns a list of (local row, local col, value or None) in row-major order."""
    off, nnz, t = desc_fields(d)
    out = []
    if desc_inline(d):
        assert t == COO and nnz <= inline_capacity(vb)
        d = int(d)
        for e in range(nnz):
            sh = 16 + e * (8 + 8 * vb)
            cd = (d >> sh) & 0xFF
            v = None
            if vb == 4:
                v = np.uint32((d >> (sh + 8)) & 0xFFFFFFFF).view(np.float32)
            elif vb == 2:
                v = np.uint16((d >> (sh + 8)) & 0xFFFF)
            out.append((cd >> 4, cd & 15, v))
        return out
    if t == COO:
        vals = _vals(pay, off, nnz, vb)
        for k in range(nnz):
            cd = int(pay[off + vb * nnz + k])
            out.append((cd >> 4, cd & 15, vals[k]))
    elif t == DENSE:
        vals = _vals(pay, off + 32, 256, vb)
        for r in range(16):
            rm = _u16(pay, off + 2 * r)
            for c in range(16):
                if (rm >> c) & 1:
                    out.append((r, c, vals[r * 16 + c]))
    elif t == FCSR:
        vals = _vals(pay, off + 48, nnz, vb)
        for r in range(16):
            rm = _u16(pay, off + 2 * r)
            start = int(pay[off + 32 + r])
            cols = [c for c in range(16) if (rm >> c) & 1]
            for k, c in enumerate(cols):
                out.append((r, c, vals[start + k]))
    elif t == FCSC:
        vals = _vals(pay, off + 48, nnz, vb)
        for c in range(16):
            cm = _u16(pay, off + 2 * c)
            start = int(pay[off + 32 + c])
            rows = [r for r in range(16) if (cm >> r) & 1]
            for k, r in enumerate(rows):
                out.append((r, c, vals[start + k]))
        out.sort(key=lambda e: (e[0], e[1]))
    elif t == CSR:
        vstart = off + 64 + (nnz + 15) // 16 * 16
        vals = _vals(pay, vstart, nnz, vb)
        rstart = [int(pay[off + 32 + r]) for r in range(16)]
        cstart = [int(pay[off + 48 + c]) for c in range(16)] + [nnz]
        row_view = []
        for r in range(16):
            rm = _u16(pay, off + 2 * r)
            cols = [c for c in range(16) if (rm >> c) & 1]
            for k, c in enumerate(cols):
                row_view.append((r, c, vals[rstart[r] + k]))
        # the column view (col_start + row_idx_csc2csr) must describe the same entries
        col_view = []
        for c in range(16):
            for q in range(cstart[c], cstart[c + 1]):
                rc = int(pay[off + 64 + q])
                r, rank = rc >> 4, rc & 15
                col_view.append((r, c, vals[rstart[r] + rank]))
        col_view.sort(key=lambda e: (e[0], e[1]))
        assert [(r, c) for r, c, _ in col_view] == [(r, c) for r, c, _ in row_view], "csc2csr view mismatch"
        for (_, _, a), (_, _, b) in zip(col_view, row_view):
            assert (a is None and b is None) or a == b
        out = row_view
    else:
        raise AssertionError(f"bad block type {t}")
    assert len(out) == nnz, (t, len(out), nnz)
    return out


def to_csr(arrs, info, vb):
    """Decodes the whole format back to sorted COO triples."""
    m, n = info["m"], info["n"]
    rows, cols, vals = [], [], []
    rb = arrs["rb_ptr"]
    for R in range(info["nbr"]):
        for b in range(rb[R], rb[R + 1]):
            J = int(arrs["cb_col"][b])
            for r, c, v in decode_block(arrs["payload"], arrs["desc"][b], vb):
                i, j = R * 16 + r, J * 16 + c
                assert i < m and j < n
                rows.append(i)
                cols.append(j)
                vals.append(v)
    order = np.lexsort((np.array(cols, dtype=np.int64), np.array(rows, dtype=np.int64))) if rows else []
    rows = np.array(rows, dtype=np.int64)[order] if len(rows) else np.zeros(0, np.int64)
    cols = np.array(cols, dtype=np.int64)[order] if len(cols) else np.zeros(0, np.int64)
    vals = [vals[i] for i in order] if len(vals) else []
    return rows, cols, vals


def expected_type(rc, cc, nnz, th0=32, th1=128, th2=2.0):
    """The classifier of Sec. 3.2.1 from its definition (epsilon cancels)."""
    if nnz < th0:
        return COO
    if nnz > th1:
        return DENSE
    eps = 1e-9
    skew_r = max(rc) / (nnz / 16 + eps)
    skew_c = max(cc) / (nnz / 16 + eps)
    if skew_c / skew_r > th2:
        return FCSC
    if skew_r / skew_c > th2:
        return FCSR
    return CSR


def expected_segments(types_per_row, seg_close=16):
    """Segments per block row: close once the accumulated weight reaches
    seg_close (or 16 blocks); never span block rows (Sec. 3.3.2)."""
    segs = []
    base = 0
    for R, types in enumerate(types_per_row):
        row = []
        w = cnt = 0
        start = 0
        for k, t in enumerate(types):
            w += WEIGHT[t]
            cnt += 1
            if w >= seg_close or cnt == 16:
                row.append((base + start, R, cnt))
                start = k + 1
                w = cnt = 0
        if cnt:
            row.append((base + start, R, cnt))
        single = 1 if len(row) == 1 else 0
        segs += [(f, r, c, single) for f, r, c in row]
        base += len(types)
    return segs
