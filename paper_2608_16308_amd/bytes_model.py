"""Algorithmic bytes of one SpMSpV call on the DB format (measurement only).

Replays, on the host and from the same inputs, the decisions the kernels
take -- the global path (s_b = N_nzblk / N_blk < th3, Sec. 3.3.1), which
blocks are visited, the microkernel of each visited block (format x vector
block mask, Sec. 3.3.3) -- and counts the bytes each step must move, every
distinct element once per kernel that needs it:

  blocker   k indices + k values read, k values written to the dense x,
            4 B mask word update per index
  scan      2 B mask per vector block, and per active vector block 8 B of
            block-CSC pointers read + a 16 B work item (first task, vector
            block, block-CSC base) written
  push      per active vector block its 16 B work item; per visited block
            4 B block row + 8 B descriptor (both in block-CSC order) + the
            record bytes its microkernel reads; 8 B per (block, row) fp64
            accumulator update; 4 B structure-mask update per block with hits
  pull      4 B per segment + 4 B block column per segment slot (16 per
            segment, padding included) + 2 B x-mask per scanned block; per
            block with an active vector block 8 B descriptor + record bytes;
            8 B per (segment, row) accumulator write; 4 B mask update per
            segment with hits
  x values  V bytes per nonzero of x (read once from the dense x)
  finalize  2 B structure mask per block row; per y entry 8 B accumulator
            read + 8 B reset + 4 B index + V value written; 4 B mask reset
            per active vector block

Record bytes read per visited block (V = value bytes):
  COO   nnz coordinates + V per matching entry (none when held inline in the
        descriptor)
  Dense 32 B masks + 256 V
  ForceCSR / ForceCSC / row-wise patched CSR   48 B header + V per matching entry
  column-wise patched CSR (fewer than 8 active columns)
        64 B header + (1 + V) per matching entry
"""
from __future__ import annotations

import numpy as np

COO, DENSE, FCSR, FCSC, CSR = range(5)
_POPC16 = np.array([bin(i).count("1") for i in range(1 << 16)], dtype=np.int32)


class BytesModel:
    def __init__(self, m, n, row_ptr, col_idx, arrays: dict, info: dict, vbytes: int):
        self.m, self.n, self.V = int(m), int(n), int(vbytes)
        self.nblk, self.nseg = int(info["nblk"]), int(info["nseg"])
        self.nbr, self.nbc = int(info["nbr"]), int(info["nbc"])
        self.nnz = int(row_ptr[-1])
        desc = arrays["desc"]
        self.btype = (desc & np.uint64(7)).astype(np.int8)
        self.binline = ((desc >> np.uint64(3)) & np.uint64(1)).astype(bool)
        self.bnnz = (((desc >> np.uint64(8)) & np.uint64(0xFF)) + np.uint64(1)).astype(np.int32)
        self.bcol = arrays["cb_col"].astype(np.int64)
        rb = arrays["rb_ptr"].astype(np.int64)
        self.brow = np.repeat(np.arange(self.nbr, dtype=np.int64), np.diff(rb))
        seg = arrays["seg"]
        seg_first = (seg & np.uint64(0xFFFFFFFF)).astype(np.int64)
        seg_nb = (((seg >> np.uint64(59)) & np.uint64(0xF)) + np.uint64(1)).astype(np.int64)
        self.bseg = np.repeat(np.arange(self.nseg, dtype=np.int64), seg_nb)
        assert self.bseg.size == self.nblk and (seg_first.size == 0 or seg_first[0] == 0)
        # entry -> primary block id, local row
        er = np.repeat(np.arange(self.m, dtype=np.int64), np.diff(np.asarray(row_ptr, dtype=np.int64)))
        ec = np.asarray(col_idx, dtype=np.int64)
        key_e = (er >> 4) * self.nbc + (ec >> 4)
        key_b = self.brow * self.nbc + self.bcol  # ascending in primary order
        ukeys, eb = np.unique(key_e, return_inverse=True)
        assert np.array_equal(ukeys, key_b), "blocks do not match the CSR"
        self.eb = eb.astype(np.int64).reshape(-1)
        self.er_local = (er & 15).astype(np.int64)
        self.ec = ec
        self.col_nnz = np.bincount(ec, minlength=self.n)

    def call(self, x_idx, path: str, th3: float = 0.01) -> dict:
        V = self.V
        x_idx = np.asarray(x_idx, dtype=np.int64)
        k = int(x_idx.size)
        xact = np.zeros(self.n, dtype=bool)
        xact[x_idx] = True
        xm = np.zeros(self.nbc, dtype=np.int64)
        np.bitwise_or.at(xm, x_idx >> 4, np.left_shift(1, x_idx & 15))
        active_vb = np.nonzero(xm)[0]
        N = int(active_vb.size)
        if path == "auto":
            path = "push" if N < th3 * self.nbc else "pull"
        mx_b = xm[self.bcol]
        act_b = mx_b != 0
        em = xact[self.ec]
        eb_m = self.eb[em]
        match_b = np.bincount(eb_m, minlength=self.nblk)
        t = self.btype
        # record bytes the kernels read per active block: stored COO blocks and,
        # in push, every format are taken entry-parallel (all coordinates and
        # values; the 48-byte mask + start header for the non-COO formats, 32
        # bytes of row masks for Dense); pull takes Dense with 4 lanes per row
        # (masks + all 256 values) and the other formats entry-parallel.
        rec = np.zeros(self.nblk, dtype=np.int64)
        nnz_b = self.bnnz
        sel = act_b & (t == COO) & ~self.binline   # inline blocks live in the descriptor
        rec[sel] = (1 + V) * nnz_b[sel]
        sel = act_b & ((t == FCSR) | (t == FCSC) | (t == CSR))
        rec[sel] = 48 + V * nnz_b[sel]
        sel = act_b & (t == DENSE)
        rec[sel] = 32 + 256 * V
        rec_pull = int(rec.sum())
        rec[sel] = 32 + V * nnz_b[sel]
        rec_push = int(rec.sum())
        nact_blocks = int(act_b.sum())
        # y structure
        row_key_blk = np.unique(eb_m * 16 + self.er_local[em])
        blk_rows = int(row_key_blk.size)                     # (block, row) pairs hit
        blks_hit = int(np.unique(eb_m).size)
        seg_rows = int(np.unique(self.bseg[eb_m] * 16 + self.er_local[em]).size)
        segs_hit = int(np.unique(self.bseg[eb_m]).size)
        y_nnz = int(np.unique(self.brow[eb_m] * 16 + self.er_local[em]).size)
        useful = int(em.sum())

        blocker = k * (4 + V) + k * V + 4 * k
        scan = 2 * self.nbc + 24 * N
        if path == "push":
            main = 16 * N + nact_blocks * (4 + 8) + rec_push + 8 * blk_rows + 4 * blks_hit
        else:
            main = 4 * self.nseg + 64 * self.nseg + 2 * self.nblk + 8 * nact_blocks + rec_pull \
                + 8 * seg_rows + 4 * segs_hit
        main += V * k
        finalize = 2 * self.nbr + y_nnz * (8 + 8 + 4 + V) + 4 * N
        total = blocker + scan + main + finalize
        compulsory = useful * (V + 1) + 8 * k + (4 + V) * y_nnz
        return {"path": path, "k": k, "n_nzblk": N, "visited_blocks": nact_blocks,
                "useful_nnz": useful, "y_nnz": y_nnz, "bytes_blocker": blocker, "bytes_scan": scan,
                "bytes_main": int(main), "bytes_finalize": finalize, "bytes_total": int(total),
                "bytes_compulsory": int(compulsory)}

    def call_dense(self, x_idx, path: str, th3: float = 0.01) -> dict:
        """The same for a dense activation and a dense y (decoding, Sec. 4.1):
        the blocker reads all n values, writes the padded dense x and the
        n-bit mask; the finalize reads every fp64 accumulator, writes y (V
        bytes per row) and resets the accumulators, the y and x masks and
        the dense x.  x_idx are the nonzero positions of the activation.
        (When pull is known on the host, the scan-free pass writes no dense
        x or masks and runs no scan: it moves about 2 V n + 2 nbc bytes
        fewer than charged here, under 0.1% of a decode layer's bytes.)"""
        r = self.call(x_idx, path, th3)
        V, m, n = self.V, self.m, self.n
        r["bytes_blocker"] = 2 * V * n + n // 8
        r["bytes_finalize"] = m * (8 + 8 + V) + m // 8 + n // 8 + V * n
        r["bytes_total"] = r["bytes_blocker"] + r["bytes_scan"] + r["bytes_main"] + r["bytes_finalize"]
        r["bytes_compulsory"] = r["useful_nnz"] * (V + 1) + V * n + V * m
        return r
