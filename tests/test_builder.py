"""CPU tests of the offline DB conversion (Sec. 3.1, 3.2.1, 3.3.2) and of the
C-ABI library's exports.  No GPU is needed: only host functions are called."""
import json
import os
import re

import numpy as np
import pytest

import dbformat as dbf
import paper_2608_16308_amd as dbs
import workloads as wl
from paper_2608_16308_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(ROOT, "tests", "golden")


def test_library_exports_every_declared_symbol():
    header = open(os.path.join(ROOT, "include", "dbspmspv.h")).read()
    declared = set(re.findall(r"^[A-Za-z_][\w\s\*]*?\b(dbs_\w+)\s*\(", header, flags=re.M))
    assert len(declared) >= 20
    lib = _lib.load()
    missing = [s for s in sorted(declared) if not hasattr(lib, s)]
    assert not missing, missing
    assert set(_lib.EXPORTED) == declared


def _vb(vals):
    return 0 if vals is None else vals.dtype.itemsize


def _check_roundtrip(a: wl.CSR, opts=None):
    hm = dbs.HostMatrix.from_csr(a.m, a.n, a.row_ptr, a.col_idx, a.vals, opts)
    info = hm.info()
    arrs = hm.arrays()
    rows, cols, vals = dbf.to_csr(arrs, info, _vb(a.vals))
    er = np.repeat(np.arange(a.m), np.diff(a.row_ptr))
    order = np.lexsort((a.col_idx, er))
    assert np.array_equal(rows, er[order])
    assert np.array_equal(cols, a.col_idx[order].astype(np.int64))
    if a.vals is not None:
        got = np.array(vals)
        exp = a.vals[order]
        if a.vals.dtype == np.float16:
            exp = exp.view(np.uint16)
        assert np.array_equal(got, exp), "values not bit-exact"
    return hm, info, arrs


def _block_stats(a: wl.CSR):
    """Per block (R, J): entries, row counts, col counts -- from the CSR."""
    er = np.repeat(np.arange(a.m), np.diff(a.row_ptr))
    blocks = {}
    for i, j in zip(er, a.col_idx):
        key = (int(i) // 16, int(j) // 16)
        rc, cc, cnt = blocks.setdefault(key, [[0] * 16, [0] * 16, [0]])
        rc[i % 16] += 1
        cc[j % 16] += 1
        cnt[0] += 1
    return blocks


CASES = {
    "crafted_f32": lambda: wl.crafted(np.float32),
    "crafted_f16": lambda: wl.crafted(np.float16, key=1),
    "crafted_pattern": lambda: wl.crafted(None, key=2),
    "random_ragged": lambda: wl.random_csr(77, 131, 0.08, key=(1, 1)),
    "random_dense": lambda: wl.random_csr(50, 45, 0.7, key=(1, 2)),
    "empty": lambda: wl.random_csr(20, 30, 0.0, key=(1, 3)),
    "one_by_one": lambda: wl.random_csr(1, 1, 1.0, key=(1, 4)),
    "tiny_config": lambda: wl.tiny(),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_roundtrip_types_views_segments(case):
    a = CASES[case]()
    hm, info, arrs = _check_roundtrip(a)
    # classifier recomputed from its definition
    stats = _block_stats(a)
    assert info["nblk"] == len(stats)
    rb = arrs["rb_ptr"]
    types_per_row = []
    for R in range(info["nbr"]):
        tr = []
        prevJ = -1
        for b in range(rb[R], rb[R + 1]):
            J = int(arrs["cb_col"][b])
            assert J > prevJ, "block columns must ascend within a block row"
            prevJ = J
            rc, cc, cnt = stats[(R, J)]
            _, nnz, t = dbf.desc_fields(arrs["desc"][b])
            assert nnz == cnt[0]
            assert t == dbf.expected_type(rc, cc, cnt[0]), (R, J, rc, cc)
            tr.append(t)
        types_per_row.append(tr)
    counts = [sum(t == k for tr in types_per_row for t in tr) for k in range(5)]
    assert counts == [info["blocks_by_type"][n] for n in _lib.BLOCK_TYPE_NAMES]
    # block-CSC view and csc2csr against the block-CSR view
    cb = arrs["cb_ptr"]
    assert cb[-1] == info["nblk"]
    row_of = np.repeat(np.arange(info["nbr"]), np.diff(rb))
    for J in range(info["nbc"]):
        prevR = -1
        for q in range(cb[J], cb[J + 1]):
            b = int(arrs["csc2csr"][q])
            assert int(arrs["cb_col"][b]) == J
            assert int(arrs["csc_row"][q]) == int(row_of[b])
            assert int(arrs["csc_row"][q]) > prevR
            prevR = int(arrs["csc_row"][q])
    assert sorted(arrs["csc2csr"].tolist()) == list(range(info["nblk"]))
    # segments
    got = [dbf.seg_fields(s) for s in arrs["seg"]]
    assert got == dbf.expected_segments(types_per_row)
    assert info["nseg"] == len(got)


def test_crafted_covers_every_format_and_boundary():
    a = wl.crafted(np.float32)
    info = dbs.HostMatrix.from_csr(a.m, a.n, a.row_ptr, a.col_idx, a.vals).info()
    assert all(v > 0 for v in info["blocks_by_type"].values()), info["blocks_by_type"]


@pytest.mark.parametrize("force", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("dtype", [np.float32, np.float16, None])
@pytest.mark.parametrize("inline", [1, 0])
def test_forced_formats_roundtrip(force, dtype, inline):
    a = wl.crafted(dtype, key=3)
    opts = dbs.default_opts(force_type=force, inline_small=inline)
    hm, info, arrs = _check_roundtrip(a, opts)
    assert info["blocks_by_type"][_lib.BLOCK_TYPE_NAMES[force]] == info["nblk"]
    n_inline = sum(dbf.desc_inline(d) for d in arrs["desc"])
    if not inline or force != 0:
        assert n_inline == 0
    else:
        cap = dbf.inline_capacity(_vb(a.vals))
        small = sum(dbf.desc_fields(d)[1] <= cap for d in arrs["desc"])
        assert n_inline == small > 0


def test_inline_blocks_take_no_payload():
    a = wl.random_csr(300, 300, 0.004, key=(1, 9))  # almost only 1-entry blocks
    on = dbs.HostMatrix.from_csr(a.m, a.n, a.row_ptr, a.col_idx, a.vals).info()
    off = dbs.HostMatrix.from_csr(a.m, a.n, a.row_ptr, a.col_idx, a.vals, dbs.default_opts(inline_small=0)).info()
    assert on["payload_bytes"] < off["payload_bytes"]


@pytest.mark.parametrize("seg_close", [1, 4, 16, 64])
def test_segment_close_option(seg_close):
    a = wl.crafted(np.float32, key=4)
    opts = dbs.default_opts(seg_close=seg_close)
    hm = dbs.HostMatrix.from_csr(a.m, a.n, a.row_ptr, a.col_idx, a.vals, opts)
    arrs = hm.arrays()
    info = hm.info()
    rb = arrs["rb_ptr"]
    types = [[dbf.desc_fields(arrs["desc"][b])[2] for b in range(rb[R], rb[R + 1])] for R in range(info["nbr"])]
    assert [dbf.seg_fields(s) for s in arrs["seg"]] == dbf.expected_segments(types, seg_close)


def test_fig5_row_mask_bit_order():
    """Fig. 5: row_mask 10 = 0b1010 marks local columns 1 and 3."""
    g = json.load(open(os.path.join(GOLDEN, "fig5_row_mask.json")))
    cols = g["columns"]
    # one block row whose first row holds exactly those columns, stored as
    # ForceCSR (row masks) and as Dense (row masks + values)
    for force in (dbf.FCSR, dbf.DENSE, dbf.CSR):
        a = wl.csr_from_coo(16, 16, np.array([0] * len(cols)), np.array(cols),
                            np.ones(len(cols), dtype=np.float32))
        hm = dbs.HostMatrix.from_csr(16, 16, a.row_ptr, a.col_idx, a.vals, dbs.default_opts(force_type=force))
        arrs = hm.arrays()
        off = int(arrs["desc"][0]) >> 16
        pay = arrs["payload"]
        assert int(pay[off]) | (int(pay[off + 1]) << 8) == g["row_mask"]


def test_tab4_storage_convention():
    g = json.load(open(os.path.join(GOLDEN, "tab4_storage.json")))
    for mat in g["matrices"]:
        csr, both = dbs.storage_model(mat["rows"], mat["rows"], mat["nnz"], g["value_bytes"])
        assert round(csr / 2 ** 20, 2) == mat["csr_mb"], mat["name"]
        assert round(both / 2 ** 20, 2) == mat["csr_csc_mb"], mat["name"]


def test_build_rejects_bad_input():
    a = wl.random_csr(20, 20, 0.3, key=(2, 1))
    col = a.col_idx.copy()
    col[3] = col[2]  # duplicate within a row
    with pytest.raises(dbs.DbsError) as e:
        dbs.HostMatrix.from_csr(a.m, a.n, a.row_ptr, col, a.vals)
    assert e.value.status == _lib.DBS_ERR_ARG and "duplicate" in str(e.value)
    col = a.col_idx.copy()
    col[0] = 20
    with pytest.raises(dbs.DbsError) as e:
        dbs.HostMatrix.from_csr(a.m, a.n, a.row_ptr, col, a.vals)
    assert e.value.status == _lib.DBS_ERR_ARG
    rp = a.row_ptr.copy()
    rp[5], rp[6] = rp[6], rp[5] - 1
    with pytest.raises(dbs.DbsError):
        dbs.HostMatrix.from_csr(a.m, a.n, rp, a.col_idx, a.vals)
    with pytest.raises(dbs.DbsError):
        dbs.HostMatrix.from_csr(a.m, a.n, a.row_ptr, a.col_idx, a.vals, dbs.default_opts(force_type=7))


def test_info_accounting():
    a = wl.crafted(np.float32)
    info = dbs.HostMatrix.from_csr(a.m, a.n, a.row_ptr, a.col_idx, a.vals).info()
    assert sum(info["blocks_by_type"].values()) == info["nblk"]
    assert info["csr_bytes"] == 8 * a.nnz + 4 * (a.m + 1)
    assert info["csr_csc_bytes"] == info["csr_bytes"] + 8 * a.nnz + 4 * (a.n + 1)
    assert info["db_bytes"] > info["payload_bytes"] > 0


def test_device_calls_fail_cleanly_without_gpu():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    a = wl.random_csr(20, 20, 0.3, key=(2, 2))
    hm = dbs.HostMatrix.from_csr(a.m, a.n, a.row_ptr, a.col_idx, a.vals)
    with pytest.raises(dbs.DbsError) as e:
        dbs.Matrix.upload(hm)
    assert e.value.status == _lib.DBS_ERR_DEVICE


def test_basic_baseline_checks_input_before_any_device_call():
    import torch
    a = wl.random_csr(20, 20, 0.3, key=(2, 3))
    col = a.col_idx.copy()
    col[0] = 20
    with pytest.raises(dbs.DbsError) as e:
        dbs.BasicMatrix(a.m, a.n, a.row_ptr, col, a.vals)
    assert e.value.status == _lib.DBS_ERR_ARG
    rp = a.row_ptr.copy()
    rp[5], rp[6] = rp[6], rp[5] - 1
    with pytest.raises(dbs.DbsError) as e:
        dbs.BasicMatrix(a.m, a.n, rp, a.col_idx, a.vals)
    assert e.value.status == _lib.DBS_ERR_ARG
    if not torch.cuda.is_available():
        with pytest.raises(dbs.DbsError) as e:
            dbs.BasicMatrix(a.m, a.n, a.row_ptr, a.col_idx, a.vals)
        assert e.value.status == _lib.DBS_ERR_DEVICE
