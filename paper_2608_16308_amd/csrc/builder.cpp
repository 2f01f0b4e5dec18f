// Offline CSR -> dual-view blocked (DB) conversion on the host (Sec. 3.1,
// 3.2.1, 3.3.2).  Runs once per matrix; the result is reused across SpMSpV
// calls, BFS levels and decoding tokens (Sec. 5.5).
//
// Steps, all O(nnz log(entries per block row)):
//  1. per 16-row block row, gather the entries, sort them by
//     (block column, local row, local column), reject duplicates;
//  2. classify every nonzero block (Sec. 3.2.1): nnz < th0 -> COO,
//     nnz > th1 -> Dense, otherwise the row/column skew ratio decides
//     ForceCSC / ForceCSR / patched CSR;
//  3. size the block records, segments and block counts per block row,
//     prefix-sum them, then write the records in primary (block-CSR) order;
//  4. derive the block-CSC view and csc2csr by a counting sort over blocks.
// Block rows are processed by a pool of host threads.
#include <algorithm>
#include <array>
#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <thread>

#include "internal.hpp"

using namespace dbs;

static thread_local std::string g_last_error;

dbs_status dbs_fail(dbs_status st, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

extern "C" const char *dbs_last_error(void) { return g_last_error.c_str(); }
extern "C" const char *dbs_version(void) { return "dbspmspv-gfx950 0.1"; }

extern "C" void dbs_build_opts_default(dbs_build_opts *o)
{
    if (!o) return;
    o->th0 = 32;
    o->th1 = 128;
    o->th2 = 2.0f;
    o->seg_close = 16;
    o->force_type = -1;
    o->inline_small = 1;
}

namespace {

struct Entry {
    uint64_t key;  // block column << 8 | local row << 4 | local column
    int64_t p;     // position in the input CSR
};

int build_threads()
{
    if (const char *e = std::getenv("DBS_BUILD_THREADS")) {
        int t = std::atoi(e);
        if (t > 0) return t;
    }
    unsigned hc = std::thread::hardware_concurrency();
    int t = hc ? (int)hc : 4;
    return std::min(t, 16);
}

template <class F>
void parallel_chunks(int64_t n, int64_t chunk, F &&f)
{
    int nt = build_threads();
    if (n <= chunk || nt <= 1) {
        for (int64_t s = 0; s < n; s += chunk) f(0, s, std::min(n, s + chunk));
        return;
    }
    std::atomic<int64_t> next{0};
    std::vector<std::thread> pool;
    for (int t = 0; t < nt; ++t) {
        pool.emplace_back([&, t]() {
            for (;;) {
                int64_t s = next.fetch_add(chunk);
                if (s >= n) break;
                f(t, s, std::min(n, s + chunk));
            }
        });
    }
    for (auto &th : pool) th.join();
}

struct Failure {
    std::mutex mu;
    std::atomic<bool> failed{false};
    dbs_status st = DBS_OK;
    std::string msg;
    void set(dbs_status s, const std::string &m)
    {
        std::lock_guard<std::mutex> g(mu);
        if (!failed.load()) {
            st = s;
            msg = m;
            failed.store(true);
        }
    }
};

// Gathers and sorts the entries of block row R.  Returns false on a
// duplicate or an out-of-range column.
bool gather_block_row(int32_t R, int32_t m, int32_t n, const int64_t *row_ptr,
                      const int32_t *col_idx, std::vector<Entry> &ents, Failure &fail)
{
    ents.clear();
    int32_t i0 = R * BS, i1 = std::min(m, i0 + BS);
    for (int32_t i = i0; i < i1; ++i) {
        for (int64_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) {
            int32_t j = col_idx[p];
            if (j < 0 || j >= n) {
                char b[128];
                snprintf(b, sizeof b, "column index %d out of range at row %d", j, i);
                fail.set(DBS_ERR_ARG, b);
                return false;
            }
            uint64_t key = ((uint64_t)(uint32_t)(j >> 4) << 8) | ((uint64_t)(i & 15) << 4) |
                           (uint64_t)(j & 15);
            ents.push_back({key, p});
        }
    }
    std::sort(ents.begin(), ents.end(), [](const Entry &a, const Entry &b) { return a.key < b.key; });
    for (size_t k = 1; k < ents.size(); ++k) {
        if (ents[k].key == ents[k - 1].key) {
            char b[128];
            int32_t r = (int32_t)((ents[k].key >> 4) & 15), c = (int32_t)(ents[k].key & 15);
            int64_t J = (int64_t)(ents[k].key >> 8);
            snprintf(b, sizeof b, "duplicate entry (%d, %lld)", R * BS + r, (long long)(J * BS + c));
            fail.set(DBS_ERR_ARG, b);
            return false;
        }
    }
    return true;
}

// Format classifier (Sec. 3.2.1).  With B_r = B_c = 16 the epsilon of the
// skew definition cancels: skew_c / skew_r = max column count / max row count.
uint32_t classify(const Entry *e, uint32_t nnz, const dbs_build_opts &o)
{
    if (o.force_type >= 0) return (uint32_t)o.force_type;
    if ((int64_t)nnz < o.th0) return T_COO;
    if ((int64_t)nnz > o.th1) return T_DENSE;
    uint32_t rc[BS] = {0}, cc[BS] = {0};
    for (uint32_t k = 0; k < nnz; ++k) {
        rc[(e[k].key >> 4) & 15]++;
        cc[e[k].key & 15]++;
    }
    uint32_t mr = *std::max_element(rc, rc + BS), mc = *std::max_element(cc, cc + BS);
    if ((float)mc > o.th2 * (float)mr) return T_FCSC;
    if ((float)mr > o.th2 * (float)mc) return T_FCSR;
    return T_CSR;
}

void put_value(uint8_t *dst, const void *vals, int64_t p, uint32_t vb)
{
    if (vb) std::memcpy(dst, (const uint8_t *)vals + p * vb, vb);
}

// Writes one block record at dst (zero-filled beforehand).  Entries are in
// row-major order within the block.
void write_record(uint8_t *dst, uint32_t type, const Entry *e, uint32_t nnz, const void *vals,
                  uint32_t vb)
{
    uint16_t mask[BS] = {0};
    uint32_t rcnt[BS] = {0}, ccnt[BS] = {0};
    for (uint32_t k = 0; k < nnz; ++k) {
        rcnt[(e[k].key >> 4) & 15]++;
        ccnt[e[k].key & 15]++;
    }
    uint32_t rstart[BS], cstart[BS];
    uint32_t s = 0;
    for (int r = 0; r < BS; ++r) { rstart[r] = s; s += rcnt[r]; }
    s = 0;
    for (int c = 0; c < BS; ++c) { cstart[c] = s; s += ccnt[c]; }
    switch (type) {
    case T_COO:
        for (uint32_t k = 0; k < nnz; ++k) {
            put_value(dst + (size_t)k * vb, vals, e[k].p, vb);
            dst[(size_t)vb * nnz + k] = (uint8_t)(e[k].key & 0xFF);
        }
        break;
    case T_DENSE:
        for (uint32_t k = 0; k < nnz; ++k) {
            uint32_t r = (e[k].key >> 4) & 15, c = e[k].key & 15;
            mask[r] |= (uint16_t)(1u << c);
            put_value(dst + HDR_START + (size_t)(r * BS + c) * vb, vals, e[k].p, vb);
        }
        std::memcpy(dst + HDR_MASK, mask, sizeof mask);
        break;
    case T_FCSR:
        for (uint32_t k = 0; k < nnz; ++k) {
            uint32_t r = (e[k].key >> 4) & 15, c = e[k].key & 15;
            mask[r] |= (uint16_t)(1u << c);
            put_value(dst + HDR_START2 + (size_t)k * vb, vals, e[k].p, vb);
        }
        std::memcpy(dst + HDR_MASK, mask, sizeof mask);
        for (int r = 0; r < BS; ++r) dst[HDR_START + r] = (uint8_t)rstart[r];
        break;
    case T_FCSC: {
        uint32_t fill[BS] = {0};
        for (uint32_t k = 0; k < nnz; ++k) {
            uint32_t r = (e[k].key >> 4) & 15, c = e[k].key & 15;
            mask[c] |= (uint16_t)(1u << r);
            uint32_t pos = cstart[c] + fill[c]++;  // rows ascend in row-major order
            put_value(dst + HDR_START2 + (size_t)pos * vb, vals, e[k].p, vb);
        }
        std::memcpy(dst + HDR_MASK, mask, sizeof mask);
        for (int c = 0; c < BS; ++c) dst[HDR_START + c] = (uint8_t)cstart[c];
        break;
    }
    default: {  // patched CSR
        uint32_t fill[BS] = {0};
        uint32_t voff = HDR_RCSC + round_up(nnz, 16);
        for (uint32_t k = 0; k < nnz; ++k) {
            uint32_t r = (e[k].key >> 4) & 15, c = e[k].key & 15;
            mask[r] |= (uint16_t)(1u << c);
            uint32_t rank = k - rstart[r];
            uint32_t pos = cstart[c] + fill[c]++;
            dst[HDR_RCSC + pos] = (uint8_t)((r << 4) | rank);
            put_value(dst + voff + (size_t)k * vb, vals, e[k].p, vb);
        }
        std::memcpy(dst + HDR_MASK, mask, sizeof mask);
        for (int r = 0; r < BS; ++r) dst[HDR_START + r] = (uint8_t)rstart[r];
        for (int c = 0; c < BS; ++c) dst[HDR_START2 + c] = (uint8_t)cstart[c];
        break;
    }
    }
}

// Descriptor of a COO block small enough to live inline (bit 3 set).
uint64_t inline_desc(const Entry *e, uint32_t nnz, const void *vals, uint32_t vb)
{
    uint64_t d = ((uint64_t)(nnz - 1) << 8) | DESC_INLINE | (uint64_t)T_COO;
    for (uint32_t k = 0; k < nnz; ++k) {
        const uint32_t sh = inline_shift(k, vb);
        d |= (uint64_t)(e[k].key & 0xFF) << sh;
        if (vb) {
            uint64_t bits = 0;
            std::memcpy(&bits, (const uint8_t *)vals + e[k].p * vb, vb);
            d |= bits << (sh + 8);
        }
    }
    return d;
}

struct RowBlockSizes {
    int64_t nblk = 0, bytes = 0, nseg = 0;
};

// Walks the sorted entries of one block row, calling on_block(first entry
// index, nnz, type, record offset) for every nonzero block and
// on_segment(first block index within the row, blocks) for every segment.
// Returns the sizes.
template <class OnBlock, class OnSeg>
RowBlockSizes walk_block_row(const std::vector<Entry> &ents, const dbs_build_opts &o,
                             uint32_t vb, OnBlock &&on_block, OnSeg &&on_seg)
{
    RowBlockSizes rs;
    uint64_t cursor = 0;
    uint32_t seg_w = 0, seg_cnt = 0;
    int64_t seg_start = 0;
    size_t k = 0;
    while (k < ents.size()) {
        uint64_t J = ents[k].key >> 8;
        size_t e = k;
        while (e < ents.size() && (ents[e].key >> 8) == J) ++e;
        uint32_t nnz = (uint32_t)(e - k);
        uint32_t type = classify(&ents[k], nnz, o);
        const bool inl = o.inline_small && type == T_COO && nnz <= inline_capacity(vb);
        if (!inl)
            cursor = (cursor + record_align(type, vb) - 1) / record_align(type, vb) * record_align(type, vb);
        on_block(k, nnz, type, inl ? ~0ull : cursor, (int32_t)J);
        if (!inl) cursor += record_bytes(type, nnz, vb);
        seg_w += seg_weight(type);
        seg_cnt += 1;
        if ((int32_t)seg_w >= o.seg_close || seg_cnt == (uint32_t)MAX_SEG_BLOCKS) {
            on_seg(seg_start, seg_cnt);
            rs.nseg++;
            seg_start += seg_cnt;
            seg_w = 0;
            seg_cnt = 0;
        }
        rs.nblk++;
        k = e;
    }
    if (seg_cnt) {
        on_seg(seg_start, seg_cnt);
        rs.nseg++;
    }
    rs.bytes = (int64_t)round_up((uint32_t)0, 1) + (int64_t)((cursor + 15) / 16 * 16);
    return rs;
}

}  // namespace

void fill_info(const dbs_host_matrix &h, dbs_matrix_info *out)
{
    std::memset(out, 0, sizeof *out);
    out->m = h.m;
    out->n = h.n;
    out->nnz = h.nnz;
    out->dtype = h.dtype;
    out->nbr = h.nbr;
    out->nbc = h.nbc;
    out->nblk = h.nblk;
    out->nseg = h.nseg;
    for (int t = 0; t < DBS_NUM_BLOCK_TYPES; ++t) out->blocks_by_type[t] = h.by_type[t];
    out->payload_bytes = (int64_t)h.payload.size();
    out->db_bytes = 4 * (int64_t)(h.nbr + 1) + 4 * h.nblk + 4 * (int64_t)(h.nbc + 1) + 8 * h.nblk +
                    8 * h.nblk + (int64_t)h.payload.size() + 8 * h.nseg;
    dbs_storage_model(h.m, h.n, h.nnz, (int32_t)dtype_bytes(h.dtype), &out->csr_bytes,
                      &out->csr_csc_bytes);
}

extern "C" dbs_status dbs_storage_model(int64_t rows, int64_t cols, int64_t nnz,
                                        int32_t value_bytes, int64_t *csr_bytes,
                                        int64_t *csr_csc_bytes)
{
    if (rows < 0 || cols < 0 || nnz < 0 || value_bytes < 0)
        return dbs_fail(DBS_ERR_ARG, "dbs_storage_model: negative argument");
    int64_t csr = (int64_t)(value_bytes + 4) * nnz + 4 * (rows + 1);
    int64_t csc = (int64_t)(value_bytes + 4) * nnz + 4 * (cols + 1);
    if (csr_bytes) *csr_bytes = csr;
    if (csr_csc_bytes) *csr_csc_bytes = csr + csc;
    return DBS_OK;
}

extern "C" dbs_status dbs_host_build_csr(int32_t m, int32_t n, int64_t nnz, const int64_t *row_ptr,
                                         const int32_t *col_idx, const void *vals, dbs_dtype vt,
                                         const dbs_build_opts *opts, dbs_host_matrix **out)
{
    if (!out) return dbs_fail(DBS_ERR_ARG, "dbs_host_build_csr: out is NULL");
    *out = nullptr;
    if (m < 0 || n < 0 || nnz < 0) return dbs_fail(DBS_ERR_ARG, "negative shape or nnz");
    if (vt != DBS_F32 && vt != DBS_F16 && vt != DBS_PATTERN)
        return dbs_fail(DBS_ERR_ARG, "unknown dtype %d", (int)vt);
    if (!row_ptr) return dbs_fail(DBS_ERR_ARG, "row_ptr is NULL");
    if (nnz > 0 && !col_idx) return dbs_fail(DBS_ERR_ARG, "col_idx is NULL");
    if (nnz > 0 && vt != DBS_PATTERN && !vals) return dbs_fail(DBS_ERR_ARG, "vals is NULL");
    dbs_build_opts o;
    dbs_build_opts_default(&o);
    if (opts) o = *opts;
    if (o.th0 < 0 || o.th1 < 0 || !(o.th2 > 0.0f) || o.seg_close < 1 || o.force_type < -1 ||
        o.force_type >= DBS_NUM_BLOCK_TYPES || (o.inline_small != 0 && o.inline_small != 1))
        return dbs_fail(DBS_ERR_ARG, "invalid build options");
    if (row_ptr[0] != 0 || row_ptr[m] != nnz)
        return dbs_fail(DBS_ERR_ARG, "row_ptr[0] must be 0 and row_ptr[m] must equal nnz");
    for (int32_t i = 0; i < m; ++i)
        if (row_ptr[i + 1] < row_ptr[i])
            return dbs_fail(DBS_ERR_ARG, "row_ptr decreases at row %d", i);

    dbs_host_matrix *h = new (std::nothrow) dbs_host_matrix();
    if (!h) return dbs_fail(DBS_ERR_ALLOC, "host allocation failed");
    h->m = m;
    h->n = n;
    h->nnz = nnz;
    h->dtype = vt;
    h->opts = o;
    h->nbr = (int32_t)(((int64_t)m + BS - 1) / BS);
    h->nbc = (int32_t)(((int64_t)n + BS - 1) / BS);
    const uint32_t vb = dtype_bytes(vt);
    const int32_t nbr = h->nbr;

    try {
        // ---- pass 1: sizes per block row ----
        std::vector<int64_t> rb_nblk(nbr + 1, 0), rb_bytes(nbr + 1, 0), rb_nseg(nbr + 1, 0);
        Failure fail;
        int nt = build_threads();
        std::vector<std::vector<Entry>> scratch(nt);
        std::vector<std::array<int64_t, DBS_NUM_BLOCK_TYPES>> tcount(nt);
        for (auto &a : tcount) a.fill(0);
        parallel_chunks(nbr, 64, [&](int t, int64_t s, int64_t e) {
            for (int64_t R = s; R < e && !fail.failed.load(); ++R) {
                if (!gather_block_row((int32_t)R, m, n, row_ptr, col_idx, scratch[t], fail)) return;
                RowBlockSizes rs = walk_block_row(
                    scratch[t], o, vb,
                    [&](size_t, uint32_t, uint32_t type, uint64_t, int32_t) { tcount[t][type]++; },
                    [](int64_t, uint32_t) {});
                rb_nblk[R + 1] = rs.nblk;
                rb_bytes[R + 1] = rs.bytes;
                rb_nseg[R + 1] = rs.nseg;
            }
        });
        if (fail.failed.load()) {
            delete h;
            return dbs_fail(fail.st, "%s", fail.msg.c_str());
        }
        for (int32_t R = 0; R < nbr; ++R) {
            rb_nblk[R + 1] += rb_nblk[R];
            rb_bytes[R + 1] += rb_bytes[R];
            rb_nseg[R + 1] += rb_nseg[R];
        }
        const int64_t nblk = rb_nblk[nbr];
        if (nblk >= ((int64_t)1 << 31) - 1) {
            delete h;
            return dbs_fail(DBS_ERR_UNSUPPORTED, "%lld nonzero blocks exceed 2^31-1", (long long)nblk);
        }
        if (rb_bytes[nbr] >= ((int64_t)1 << 47)) {
            delete h;
            return dbs_fail(DBS_ERR_UNSUPPORTED, "payload too large");
        }
        h->nblk = nblk;
        h->nseg = rb_nseg[nbr];
        for (auto &a : tcount)
            for (int ty = 0; ty < DBS_NUM_BLOCK_TYPES; ++ty) h->by_type[ty] += a[ty];
        h->rb_ptr.resize(nbr + 1);
        for (int32_t R = 0; R <= nbr; ++R) h->rb_ptr[R] = (int32_t)rb_nblk[R];
        // row i is bit i % 16 of block row i / 16's mask, i.e. bit i % 32 of
        // word i / 32
        h->row_occ.assign((size_t)(nbr + 1) / 2, 0u);
        for (int32_t i = 0; i < m; ++i)
            if (row_ptr[i + 1] > row_ptr[i]) h->row_occ[(size_t)(i >> 5)] |= 1u << (i & 31);
        h->cb_col.resize(nblk);
        h->desc.resize(nblk);
        h->seg.resize(h->nseg);
        h->payload.assign((size_t)rb_bytes[nbr], 0);

        // ---- pass 2: write records, block columns, descriptors, segments ----
        parallel_chunks(nbr, 64, [&](int t, int64_t s, int64_t e) {
            for (int64_t R = s; R < e; ++R) {
                if (!gather_block_row((int32_t)R, m, n, row_ptr, col_idx, scratch[t], fail)) return;
                const std::vector<Entry> &ents = scratch[t];
                int64_t b = rb_nblk[R];
                const uint64_t base = (uint64_t)rb_bytes[R];
                int64_t sidx = rb_nseg[R];
                const bool single = (rb_nseg[R + 1] - rb_nseg[R]) == 1;
                walk_block_row(
                    ents, o, vb,
                    [&](size_t k, uint32_t nnz, uint32_t type, uint64_t off, int32_t J) {
                        h->cb_col[b] = J;
                        if (off == ~0ull) {
                            h->desc[b] = inline_desc(&ents[k], nnz, vals, vb);
                        } else {
                            write_record(h->payload.data() + base + off, type, &ents[k], nnz, vals, vb);
                            h->desc[b] = desc_make(base + off, nnz, type);
                        }
                        ++b;
                    },
                    [&](int64_t first_local, uint32_t cnt) {
                        h->seg[sidx++] = seg_make((uint32_t)(rb_nblk[R] + first_local), (uint32_t)R,
                                                  cnt, single);
                    });
            }
        });
        if (fail.failed.load()) {
            delete h;
            return dbs_fail(fail.st, "%s", fail.msg.c_str());
        }

        // ---- block-CSC view by a counting sort over blocks ----
        const int32_t nbc = h->nbc;
        h->cb_ptr.assign(nbc + 1, 0);
        for (int64_t b = 0; b < nblk; ++b) h->cb_ptr[h->cb_col[b] + 1]++;
        for (int32_t J = 0; J < nbc; ++J) h->cb_ptr[J + 1] += h->cb_ptr[J];
        h->csc_row.resize(nblk);
        h->csc2csr.resize(nblk);
        std::vector<int32_t> next(h->cb_ptr.begin(), h->cb_ptr.end() - (nbc >= 0 ? 1 : 0));
        for (int32_t R = 0; R < nbr; ++R) {
            for (int32_t b = h->rb_ptr[R]; b < h->rb_ptr[R + 1]; ++b) {
                int32_t q = next[h->cb_col[b]]++;
                h->csc_row[q] = R;
                h->csc2csr[q] = b;
            }
        }
    } catch (const std::bad_alloc &) {
        delete h;
        return dbs_fail(DBS_ERR_ALLOC, "host allocation failed during build");
    }
    *out = h;
    return DBS_OK;
}

extern "C" dbs_status dbs_host_info(const dbs_host_matrix *h, dbs_matrix_info *out)
{
    if (!h || !out) return dbs_fail(DBS_ERR_ARG, "dbs_host_info: NULL argument");
    fill_info(*h, out);
    return DBS_OK;
}

extern "C" dbs_status dbs_host_arrays_get(const dbs_host_matrix *h, dbs_host_arrays *out)
{
    if (!h || !out) return dbs_fail(DBS_ERR_ARG, "dbs_host_arrays_get: NULL argument");
    out->rb_ptr = h->rb_ptr.data();
    out->cb_col = h->cb_col.data();
    out->cb_ptr = h->cb_ptr.data();
    out->csc_row = h->csc_row.data();
    out->csc2csr = h->csc2csr.data();
    out->desc = h->desc.data();
    out->payload = h->payload.data();
    out->payload_bytes = (int64_t)h->payload.size();
    out->seg = h->seg.data();
    out->nseg = h->nseg;
    return DBS_OK;
}

extern "C" void dbs_host_destroy(dbs_host_matrix *h) { delete h; }
