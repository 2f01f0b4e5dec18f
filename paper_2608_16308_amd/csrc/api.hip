// C ABI of the library: device matrix upload, per-stream contexts, and the
// SpMSpV / dense-activation / BFS entry points (argument checks, launches,
// optional statistics and HIP-event timing).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <cstring>
#include <new>
#include <vector>

#include "internal.hpp"
#include "kernels.hpp"
#include "matrix.hpp"

using namespace dbs;

namespace {

dbs_status hip_fail(hipError_t e, const char *what)
{
    return dbs_fail(DBS_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                          \
    do {                                             \
        hipError_t e_ = (expr);                      \
        if (e_ != hipSuccess) return hip_fail(e_, what); \
    } while (0)

dbs_status check_device()
{
    int cnt = 0;
    hipError_t e = hipGetDeviceCount(&cnt);
    if (e != hipSuccess || cnt <= 0) return dbs_fail(DBS_ERR_DEVICE, "no HIP device available");
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev), "hipGetDevice");
    hipDeviceProp_t prop;
    HIP_TRY(hipGetDeviceProperties(&prop, dev), "hipGetDeviceProperties");
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return dbs_fail(DBS_ERR_DEVICE, "device %d is %s; this library is built for gfx950 only", dev,
                        prop.gcnArchName);
    return DBS_OK;
}

// pad: zeroed bytes after the data (the payload gets 16, so that a 16-byte
// load of the chunk holding a record's last byte stays inside the allocation)
template <class T>
dbs_status dev_upload(std::vector<void *> &allocs, const std::vector<T> &h, const T **out, size_t pad = 0)
{
    const size_t data = h.size() * sizeof(T);
    size_t bytes = std::max<size_t>(data + pad, 16);
    void *p = nullptr;
    HIP_TRY(hipMalloc(&p, bytes), "hipMalloc (matrix)");
    allocs.push_back(p);
    if (bytes > data) HIP_TRY(hipMemset((char *)p + data, 0, bytes - data), "hipMemset (matrix)");
    if (!h.empty()) HIP_TRY(hipMemcpy(p, h.data(), data, hipMemcpyHostToDevice), "hipMemcpy (matrix)");
    *out = (const T *)p;
    return DBS_OK;
}

template <class T>
dbs_status dev_zeros(std::vector<void *> &allocs, size_t count, T **out, int byte = 0)
{
    size_t bytes = std::max<size_t>(count * sizeof(T), 16);
    void *p = nullptr;
    HIP_TRY(hipMalloc(&p, bytes), "hipMalloc (context)");
    allocs.push_back(p);
    HIP_TRY(hipMemset(p, byte, bytes), "hipMemset (context)");
    *out = (T *)p;
    return DBS_OK;
}

}  // namespace


struct TimedLaunch {
    int cls;
    hipEvent_t a, b;
};

struct dbs_ctx {
    int32_t max_m = 0, max_n = 0, max_nbr = 0, max_nbc = 0;
    int64_t max_nblk = 0;
    hipStream_t stream = nullptr;
    DevCtx c;
    std::vector<void *> allocs;
    int32_t *h_counters = nullptr;  // pinned
    bool timing = false;
    std::vector<TimedLaunch> pending;
    std::vector<hipEvent_t> pool;
    double ms[DBS_K_COUNT] = {0};
    int64_t launches[DBS_K_COUNT] = {0};
    bool broken = false;
    bool single = false;  // one launch per call for short index lists (fused_fits)
    // batched dense activations: DBS_MAX_BATCH padded x copies and
    // accumulator sets, allocated by the first batched call
    void *xdb = nullptr;
    double *yaccb = nullptr;
};

namespace {

void free_all(std::vector<void *> &allocs)
{
    for (void *p : allocs) (void)hipFree(p);
    allocs.clear();
}

hipEvent_t take_event(dbs_ctx *ctx)
{
    if (!ctx->pool.empty()) {
        hipEvent_t e = ctx->pool.back();
        ctx->pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// Brackets one kernel launch with an event pair when timing is on.
struct Timer {
    dbs_ctx *ctx;
    int cls;
    hipEvent_t a = nullptr, b = nullptr;
    Timer(dbs_ctx *c, int k) : ctx(c), cls(k)
    {
        if (ctx->timing) {
            a = take_event(ctx);
            b = take_event(ctx);
            if (a) (void)hipEventRecord(a, ctx->stream);
        }
    }
    ~Timer()
    {
        if (ctx->timing && a && b) {
            (void)hipEventRecord(b, ctx->stream);
            ctx->pending.push_back({cls, a, b});
        }
    }
};

dbs_status sync_counters(dbs_ctx *ctx)
{
    HIP_TRY(hipMemcpyAsync(ctx->h_counters, ctx->c.counters, sizeof(int32_t) * C_COUNT,
                           hipMemcpyDeviceToHost, ctx->stream),
            "hipMemcpyAsync (counters)");
    HIP_TRY(hipStreamSynchronize(ctx->stream), "hipStreamSynchronize");
    return DBS_OK;
}

dbs_status check_ctx(dbs_ctx *ctx, const dbs_matrix *A)
{
    if (!ctx || !A) return dbs_fail(DBS_ERR_ARG, "NULL context or matrix");
    if (ctx->broken) return dbs_fail(DBS_ERR_STATE, "context unusable after an earlier device error");
    if (A->d.m > ctx->max_m || A->d.n > ctx->max_n || A->d.nblk > ctx->max_nblk)
        return dbs_fail(DBS_ERR_ARG, "matrix %dx%d with %lld blocks exceeds the context's %dx%d / %lld",
                        A->d.m, A->d.n, (long long)A->d.nblk, ctx->max_m, ctx->max_n,
                        (long long)ctx->max_nblk);
    return DBS_OK;
}

#define LAUNCH(ctx, cls, expr)                                   \
    do {                                                         \
        Timer t_(ctx, cls);                                      \
        hipError_t e_ = (expr);                                  \
        if (e_ != hipSuccess) {                                  \
            (ctx)->broken = true;                                \
            return hip_fail(e_, "kernel launch");                \
        }                                                        \
    } while (0)

}  // namespace

// ---------------------------------------------------------------------------
// matrix
// ---------------------------------------------------------------------------
extern "C" dbs_status dbs_matrix_upload(const dbs_host_matrix *h, dbs_matrix **out)
{
    if (!h || !out) return dbs_fail(DBS_ERR_ARG, "dbs_matrix_upload: NULL argument");
    *out = nullptr;
    dbs_status st = check_device();
    if (st != DBS_OK) return st;
    if ((int64_t)h->nbc > MAX_BLOCK_COLS)
        return dbs_fail(DBS_ERR_UNSUPPORTED, "n = %d: the device format holds at most 2^26 block columns", h->n);
    dbs_matrix *A = new (std::nothrow) dbs_matrix();
    if (!A) return dbs_fail(DBS_ERR_ALLOC, "host allocation failed");
    DevMatrix &d = A->d;
    d.m = h->m;
    d.n = h->n;
    d.nbr = h->nbr;
    d.nbc = h->nbc;
    d.nblk = h->nblk;
    d.nseg = h->nseg;
    d.dtype = h->dtype;
    // primary order -> pull-segment slots (see DevMatrix)
    std::vector<int32_t> sl_col, hv_col, hv_cstart, hv_crow, hv_rowchunks;
    std::vector<uint64_t> sl_desc, hv_desc, csc_desc;
    std::vector<uint32_t> seg_rs;
    std::vector<int32_t> task_order;
    try {
        const size_t nslots = (size_t)16 * (size_t)h->nseg;
        sl_col.assign(nslots, -1);
        sl_desc.assign(nslots, 0ull);
        seg_rs.resize((size_t)h->nseg);
        // stored COO entries per group of 16 segments (the work of the
        // segment loop's entry-parallel pass), for the task order below
        std::vector<int64_t> gent((size_t)((h->nseg + 15) / 16), 0);
        for (int64_t s = 0; s < h->nseg; ++s) {
            const uint64_t sg = h->seg[s];
            const uint32_t first = seg_first(sg), nb = seg_nb(sg);
            for (uint32_t i = 0; i < nb; ++i) {
                const size_t slot = (size_t)16 * s + i;
                const uint64_t dd = h->desc[first + i];
                sl_col[slot] = slot_word(h->cb_col[first + i], dd);
                sl_desc[slot] = dd;
                if (desc_type(dd) == T_COO && !desc_inline(dd)) gent[(size_t)(s / 16)] += desc_nnz(dd);
                if (desc_type(dd) != T_COO) {
                    // pulled from the non-COO list (flagged in the slot by the
                    // sign bit of its word); a new chunk starts at a new block
                    // row or after HV_CHUNK blocks
                    const int32_t brow = (int32_t)seg_brow(sg);
                    if (hv_crow.empty() || hv_crow.back() != brow ||
                        (int64_t)hv_col.size() - hv_cstart.back() == HV_CHUNK) {
                        hv_cstart.push_back((int32_t)hv_col.size());
                        hv_crow.push_back(brow);
                    }
                    hv_col.push_back(h->cb_col[first + i]);
                    hv_desc.push_back(dd);
                }
            }
            seg_rs[s] = seg_brow(sg);
        }
        // segment-loop tasks by decreasing cost: a wave iteration per group
        // plus one per 256 stored entries (a window of the entry-parallel
        // pass); ties keep segment order
        const int64_t ntask = (h->nseg + PULL_TASK_SEGS - 1) / PULL_TASK_SEGS;
        std::vector<int64_t> tcost((size_t)ntask, 0);
        for (size_t g = 0; g < gent.size(); ++g)
            tcost[g / (PULL_TASK_SEGS / 16)] += 1 + (gent[g] + 255) / 256;
        task_order.resize((size_t)ntask);
        for (int64_t t = 0; t < ntask; ++t) task_order[(size_t)t] = (int32_t)t;
        std::stable_sort(task_order.begin(), task_order.end(),
                         [&](int32_t x, int32_t y) { return tcost[(size_t)x] > tcost[(size_t)y]; });
        hv_cstart.push_back((int32_t)hv_col.size());
        hv_rowchunks.assign((size_t)std::max(h->nbr, 1), 0);
        for (const int32_t R : hv_crow) ++hv_rowchunks[(size_t)R];
        csc_desc.resize((size_t)h->nblk);
        for (int64_t q = 0; q < h->nblk; ++q) csc_desc[q] = h->desc[h->csc2csr[q]];
    } catch (const std::bad_alloc &) {
        delete A;
        return dbs_fail(DBS_ERR_ALLOC, "host allocation failed during upload");
    }
    if ((int64_t)16 * h->nseg >= ((int64_t)1 << 31)) {
        delete A;
        return dbs_fail(DBS_ERR_UNSUPPORTED, "%lld pull segments exceed the 2^31 slot limit", (long long)h->nseg);
    }
    dbs_status s2 = DBS_OK;
    if ((s2 = dev_upload(A->allocs, sl_col, &d.sl_col)) != DBS_OK ||
        (s2 = dev_upload(A->allocs, sl_desc, &d.sl_desc)) != DBS_OK ||
        (s2 = dev_upload(A->allocs, seg_rs, &d.seg_rs)) != DBS_OK ||
        (s2 = dev_upload(A->allocs, h->cb_ptr, &d.cb_ptr)) != DBS_OK ||
        (s2 = dev_upload(A->allocs, h->csc_row, &d.csc_row)) != DBS_OK ||
        (s2 = dev_upload(A->allocs, csc_desc, &d.csc_desc)) != DBS_OK ||
        (s2 = dev_upload(A->allocs, hv_col, &d.hv_col)) != DBS_OK ||
        (s2 = dev_upload(A->allocs, hv_desc, &d.hv_desc)) != DBS_OK ||
        (s2 = dev_upload(A->allocs, hv_cstart, &d.hv_cstart)) != DBS_OK ||
        (s2 = dev_upload(A->allocs, hv_crow, &d.hv_crow)) != DBS_OK ||
        (s2 = dev_upload(A->allocs, hv_rowchunks, &d.hv_rowchunks)) != DBS_OK ||
        (s2 = dev_upload(A->allocs, h->payload, &d.pay, 16)) != DBS_OK ||
        (s2 = dev_upload(A->allocs, task_order, &d.task_order)) != DBS_OK ||
        (s2 = dev_upload(A->allocs, h->row_occ, &d.row_occ)) != DBS_OK) {
        free_all(A->allocs);
        delete A;
        return s2;
    }
    d.nheavy = (int64_t)hv_col.size();
    d.nchunk = (int64_t)hv_crow.size();
    d.ntask = (int32_t)task_order.size();
    fill_info(*h, &A->info);
    *out = A;
    return DBS_OK;
}

extern "C" dbs_status dbs_matrix_build_csr(int32_t m, int32_t n, int64_t nnz, const int64_t *row_ptr,
                                           const int32_t *col_idx, const void *vals, dbs_dtype vt,
                                           const dbs_build_opts *opts, dbs_matrix **out)
{
    dbs_host_matrix *h = nullptr;
    dbs_status st = dbs_host_build_csr(m, n, nnz, row_ptr, col_idx, vals, vt, opts, &h);
    if (st != DBS_OK) return st;
    st = dbs_matrix_upload(h, out);
    dbs_host_destroy(h);
    return st;
}

extern "C" dbs_status dbs_matrix_info_get(const dbs_matrix *A, dbs_matrix_info *out)
{
    if (!A || !out) return dbs_fail(DBS_ERR_ARG, "dbs_matrix_info_get: NULL argument");
    *out = A->info;
    return DBS_OK;
}

extern "C" dbs_status dbs_matrix_layout_get(const dbs_matrix *A, dbs_matrix_layout *out)
{
    if (!A || !out) return dbs_fail(DBS_ERR_ARG, "dbs_matrix_layout_get: NULL argument");
    std::memset(out, 0, sizeof *out);
    out->nslots = 16 * A->d.nseg;
    out->nseg = A->d.nseg;
    out->nblk = A->d.nblk;
    out->nbc = A->d.nbc;
    out->nheavy = A->d.nheavy;
    out->nchunk = A->d.nchunk;
    out->payload_bytes = A->info.payload_bytes;
    return DBS_OK;
}

extern "C" dbs_status dbs_matrix_download(const dbs_matrix *A, dbs_matrix_arrays *out)
{
    if (!A || !out) return dbs_fail(DBS_ERR_ARG, "dbs_matrix_download: NULL argument");
    const DevMatrix &d = A->d;
    auto get = [](void *dst, const void *src, size_t bytes) -> hipError_t {
        if (!dst || !bytes) return hipSuccess;
        return hipMemcpy(dst, src, bytes, hipMemcpyDeviceToHost);
    };
    const size_t ns = (size_t)(16 * d.nseg), nb = (size_t)d.nblk, nh = (size_t)d.nheavy, nc = (size_t)d.nchunk;
    HIP_TRY(get(out->sl_col, d.sl_col, ns * 4), "hipMemcpy (slots)");
    HIP_TRY(get(out->sl_desc, d.sl_desc, ns * 8), "hipMemcpy (slots)");
    HIP_TRY(get(out->seg_rs, d.seg_rs, (size_t)d.nseg * 4), "hipMemcpy (segments)");
    HIP_TRY(get(out->cb_ptr, d.cb_ptr, ((size_t)d.nbc + 1) * 4), "hipMemcpy (block-CSC)");
    HIP_TRY(get(out->csc_row, d.csc_row, nb * 4), "hipMemcpy (block-CSC)");
    HIP_TRY(get(out->csc_desc, d.csc_desc, nb * 8), "hipMemcpy (block-CSC)");
    HIP_TRY(get(out->hv_col, d.hv_col, nh * 4), "hipMemcpy (non-COO list)");
    HIP_TRY(get(out->hv_desc, d.hv_desc, nh * 8), "hipMemcpy (non-COO list)");
    HIP_TRY(get(out->hv_cstart, d.hv_cstart, (nc + 1) * 4), "hipMemcpy (non-COO list)");
    HIP_TRY(get(out->hv_crow, d.hv_crow, nc * 4), "hipMemcpy (non-COO list)");
    HIP_TRY(get(out->payload, d.pay, (size_t)A->info.payload_bytes), "hipMemcpy (payload)");
    return DBS_OK;
}

extern "C" void dbs_matrix_destroy(dbs_matrix *A)
{
    if (!A) return;
    free_all(A->allocs);
    delete A;
}

// ---------------------------------------------------------------------------
// context
// ---------------------------------------------------------------------------
extern "C" dbs_status dbs_ctx_create(const dbs_matrix *sizing, void *stream, dbs_ctx **out)
{
    if (!sizing || !out) return dbs_fail(DBS_ERR_ARG, "dbs_ctx_create: NULL argument");
    *out = nullptr;
    dbs_status st = check_device();
    if (st != DBS_OK) return st;
    dbs_ctx *ctx = new (std::nothrow) dbs_ctx();
    if (!ctx) return dbs_fail(DBS_ERR_ALLOC, "host allocation failed");
    ctx->max_m = sizing->d.m;
    ctx->max_n = sizing->d.n;
    ctx->max_nbr = sizing->d.nbr;
    ctx->max_nbc = sizing->d.nbc;
    ctx->max_nblk = sizing->d.nblk;
    ctx->stream = (hipStream_t)stream;
    DevCtx &c = ctx->c;
    const int32_t nbr = std::max(ctx->max_nbr, 1), nbc = std::max(ctx->max_nbc, 1);
    // BFS reuses the vector-block masks as row-block masks, so size both by
    // the larger of the two.
    const int32_t nb = std::max(nbr, nbc);
    c.nxwords = (nb + 1) / 2 + 2;
    c.nywords = (nbr + 1) / 2 + 2;
    c.n_st_scan = scan_tiles(nbc) + 1;
    c.n_st_fin = finalize_tiles(nbr) + 1;
    uint32_t *xmask = nullptr, *ybits = nullptr, *visited = nullptr, *nextm = nullptr;
    float *xd = nullptr;
    // densified x: all-ones bits mark absent entries (fp32 and fp16 views)
    if ((st = dev_zeros(ctx->allocs, (size_t)16 * nb, &xd, 0xFF)) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)c.nxwords, &xmask)) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)(nb + 31) / 32 + 64, &c.xbits)) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)nbc + 2, &c.items)) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)16 * nbr, &c.yacc)) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)c.nywords, &ybits)) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)c.nxwords, &visited)) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)c.nxwords, &nextm)) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)C_COUNT, &c.counters)) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)nbr, &c.rdone)) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)c.n_st_scan, &c.st_scan[0])) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)c.n_st_scan, &c.st_scan[1])) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)c.n_st_fin, &c.st_fin[0])) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)c.n_st_fin, &c.st_fin[1])) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)compact_list_entries(sizing->d.nseg), &c.clist)) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)compact_list_regions(), &c.ccount)) != DBS_OK ||
        (st = dev_zeros(ctx->allocs, (size_t)SYNC_WORDS, &c.sync)) != DBS_OK) {
        free_all(ctx->allocs);
        delete ctx;
        return st;
    }
    c.clist_cap = compact_list_entries(sizing->d.nseg);
    c.xd = xd;
    c.xmask = xmask;
    c.ybits = ybits;
    c.visited = visited;
    c.nextm = nextm;
    hipError_t e = hipHostMalloc((void **)&ctx->h_counters, sizeof(int32_t) * C_COUNT, hipHostMallocDefault);
    if (e != hipSuccess) {
        free_all(ctx->allocs);
        delete ctx;
        return hip_fail(e, "hipHostMalloc");
    }
    *out = ctx;
    return DBS_OK;
}

extern "C" dbs_status dbs_ctx_set_stream(dbs_ctx *ctx, void *stream)
{
    if (!ctx) return dbs_fail(DBS_ERR_ARG, "NULL context");
    ctx->stream = (hipStream_t)stream;
    return DBS_OK;
}

extern "C" void dbs_ctx_destroy(dbs_ctx *ctx)
{
    if (!ctx) return;
    (void)hipStreamSynchronize(ctx->stream);
    for (auto &p : ctx->pending) {
        (void)hipEventDestroy(p.a);
        (void)hipEventDestroy(p.b);
    }
    for (auto e : ctx->pool) (void)hipEventDestroy(e);
    free_all(ctx->allocs);
    if (ctx->xdb) (void)hipFree(ctx->xdb);
    if (ctx->yaccb) (void)hipFree(ctx->yaccb);
    if (ctx->h_counters) (void)hipHostFree(ctx->h_counters);
    delete ctx;
}

extern "C" dbs_status dbs_ctx_set_single_launch(dbs_ctx *ctx, int enable)
{
    if (!ctx) return dbs_fail(DBS_ERR_ARG, "NULL context");
    ctx->single = enable != 0;
    return DBS_OK;
}

extern "C" dbs_status dbs_ctx_enable_timing(dbs_ctx *ctx, int enable)
{
    if (!ctx) return dbs_fail(DBS_ERR_ARG, "NULL context");
    ctx->timing = enable != 0;
    return DBS_OK;
}

extern "C" dbs_status dbs_ctx_read_timing(dbs_ctx *ctx, dbs_timing *out)
{
    if (!ctx || !out) return dbs_fail(DBS_ERR_ARG, "NULL argument");
    HIP_TRY(hipStreamSynchronize(ctx->stream), "hipStreamSynchronize");
    for (auto &p : ctx->pending) {
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
            ctx->ms[p.cls] += ms;
            ctx->launches[p.cls] += 1;
        }
        ctx->pool.push_back(p.a);
        ctx->pool.push_back(p.b);
    }
    ctx->pending.clear();
    for (int k = 0; k < DBS_K_COUNT; ++k) {
        out->ms[k] = ctx->ms[k];
        out->launches[k] = ctx->launches[k];
        ctx->ms[k] = 0;
        ctx->launches[k] = 0;
    }
    return DBS_OK;
}

// ---------------------------------------------------------------------------
// SpMSpV
// ---------------------------------------------------------------------------
static float norm_th3(float th3) { return th3 > 0.f ? th3 : DBS_TH3_DEFAULT; }
// the spread rule's threshold: with the default th3 only
static double spread_th3(float th3) { return th3 > 0.f ? 0.0 : (double)DBS_TH3_SPREAD; }

namespace {

// Argument checks of one SpMSpV call shared by the context and no-allocation
// entry points; sets the kernel mode.
dbs_status spmspv_check_args(const dbs_matrix *A, dbs_semiring sr, int32_t x_nnz, const int32_t *d_x_idx,
                             const void *d_x_val, dbs_path path, int32_t *d_y_idx, void *d_y_val,
                             int32_t *d_y_nnz, int *mode)
{
    if (sr != DBS_PLUS_TIMES && sr != DBS_OR_AND) return dbs_fail(DBS_ERR_ARG, "unknown semiring");
    if (path < DBS_PATH_AUTO || path > DBS_PATH_PULL) return dbs_fail(DBS_ERR_ARG, "unknown path");
    if (x_nnz < 0 || x_nnz > A->d.n)
        return dbs_fail(DBS_ERR_ARG, "x_nnz %d outside [0, n=%d]", x_nnz, A->d.n);
    if (x_nnz > 0 && !d_x_idx) return dbs_fail(DBS_ERR_ARG, "d_x_idx is NULL");
    if (!d_y_idx || !d_y_nnz) return dbs_fail(DBS_ERR_ARG, "d_y_idx / d_y_nnz is NULL");
    if (sr == DBS_OR_AND) {
        *mode = M_BOOL;
    } else {
        if (A->d.dtype == DBS_PATTERN)
            return dbs_fail(DBS_ERR_ARG, "a pattern matrix supports only the OR-AND semiring");
        if (x_nnz > 0 && !d_x_val) return dbs_fail(DBS_ERR_ARG, "d_x_val is NULL");
        if (!d_y_val) return dbs_fail(DBS_ERR_ARG, "d_y_val is NULL");
        *mode = A->d.dtype == DBS_F16 ? M_F16 : M_F32;
    }
    return DBS_OK;
}

// The kernel launches of one SpMSpV call on the scratch buffers c (argument
// checks done).  run(kernel class, launcher) issues one launch and maps its
// error.
template <class Run>
dbs_status spmspv_launches(const dbs_matrix *A, DevCtx &c, hipStream_t s, int mode, dbs_semiring sr,
                           int32_t x_nnz, const int32_t *d_x_idx, const void *d_x_val, const uint32_t *d_mask,
                           int complement_mask, dbs_path path, float th3, int32_t *d_y_idx, void *d_y_val,
                           int32_t *d_y_nnz, bool single, Run &&run)
{
    if (single && fused_fits(A->d, x_nnz)) {
        // a short index list: the whole call in one launch (the device
        // chooses the path; pull takes the segment loop)
        return run(DBS_K_FUSED, [&] {
            return launch_fused(A->d, c, mode, x_nnz, d_x_idx, d_x_val, d_mask, complement_mask ? 1 : 0, (int)path,
                                (double)norm_th3(th3), spread_th3(th3), d_y_idx,
                                sr == DBS_OR_AND ? nullptr : d_y_val, d_y_nnz, s);
        });
    }
    // The automatic choice (push iff N_nzblk < th3 N_blk) is made on the
    // device, so both traversal kernels are launched and one returns at once.
    // Often k alone settles it: N_nzblk <= k, and N_nzblk >= ceil(k / 16)
    // when the k indices are distinct and in range (with invalid x, which is
    // flagged, the other path may be taken; y is the same).  Then only that
    // kernel is launched.
    int launch_path = (int)path;
    if (path == DBS_PATH_AUTO) {
        // (the spread rule can take push up to its own threshold: push when
        // N_nzblk < lim_s and the k distinct indices number fewer than 2 N_nzblk)
        const double lim = (double)norm_th3(th3) * (double)A->d.nbc;
        const double lim_s = spread_th3(th3) * (double)A->d.nbc;
        const double lim_any = std::max(lim, lim_s);
        const int64_t nlo = (x_nnz + 15) / 16, nhi = std::min<int64_t>(x_nnz, A->d.nbc);
        // the smallest N_nzblk the paper's rule leaves to pull
        const int64_t a = std::max<int64_t>(nlo, (int64_t)std::ceil(lim));
        if ((double)x_nnz < lim) launch_path = DBS_PATH_PUSH;
        else if ((double)nlo >= lim_any) launch_path = DBS_PATH_PULL;
        else if ((double)nhi < lim_s && 2 * a > x_nnz) launch_path = DBS_PATH_PUSH;  // spread for every such N
    }
    dbs_status st;
    if (small_x_fits(A->d, (int32_t)x_nnz)) {
        // a short index list: blocker and scan in one workgroup
        st = run(DBS_K_SCAN, [&] {
            return launch_small_x(A->d, c, mode, (int32_t)x_nnz, d_x_idx, d_x_val, launch_path,
                                  (double)norm_th3(th3), spread_th3(th3), s);
        });
        if (st != DBS_OK) return st;
    } else {
        st = run(DBS_K_SCATTER, [&] { return launch_scatter(A->d, c, mode, x_nnz, d_x_idx, d_x_val, s); });
        if (st != DBS_OK) return st;
        st = run(DBS_K_SCAN,
                 [&] { return launch_scan(A->d, c, launch_path, (double)norm_th3(th3), spread_th3(th3), s); });
        if (st != DBS_OK) return st;
    }
    st = run(DBS_K_MAIN, [&] {
        return launch_main(A->d, c, mode, c.xd, d_mask, complement_mask ? 1 : 0, nullptr, launch_path, s);
    });
    if (st != DBS_OK) return st;
    return run(DBS_K_FINALIZE, [&] {
        return launch_finalize(A->d, c, mode, d_y_idx, sr == DBS_OR_AND ? nullptr : d_y_val, d_y_nnz, d_x_idx,
                               x_nnz, s);
    });
}

}  // namespace

extern "C" dbs_status dbs_spmspv(dbs_ctx *ctx, const dbs_matrix *A, dbs_semiring sr, int32_t x_nnz,
                                 const int32_t *d_x_idx, const void *d_x_val, const uint32_t *d_mask,
                                 int complement_mask, dbs_path path, float th3, int32_t *d_y_idx,
                                 void *d_y_val, int32_t *d_y_nnz, dbs_call_stats *stats)
{
    dbs_status st = check_ctx(ctx, A);
    if (st != DBS_OK) return st;
    int mode = 0;
    st = spmspv_check_args(A, sr, x_nnz, d_x_idx, d_x_val, path, d_y_idx, d_y_val, d_y_nnz, &mode);
    if (st != DBS_OK) return st;
    st = spmspv_launches(A, ctx->c, ctx->stream, mode, sr, x_nnz, d_x_idx, d_x_val, d_mask, complement_mask, path,
                         th3, d_y_idx, d_y_val, d_y_nnz, ctx->single, [ctx](int cls, auto &&launch) -> dbs_status {
                             Timer t_(ctx, cls);
                             const hipError_t e = launch();
                             if (e != hipSuccess) {
                                 ctx->broken = true;
                                 return hip_fail(e, "kernel launch");
                             }
                             return DBS_OK;
                         });
    if (st != DBS_OK) return st;
    if (stats) {
        if ((st = sync_counters(ctx)) != DBS_OK) return st;
        const int32_t *h = ctx->h_counters;
        std::memset(stats, 0, sizeof *stats);
        stats->path = h[C_PATH];
        stats->n_nzblk = h[C_NZBLK];
        stats->n_blk = A->d.nbc;
        stats->y_nnz = h[C_YNNZ];
        stats->tasks = h[C_PATH] == PATH_PUSH ? (int64_t)h[C_TASKS] : A->d.nseg;
        stats->error_flags = h[C_ERR_LAST];
    }
    return DBS_OK;
}

extern "C" dbs_status dbs_spmspv_dense(dbs_ctx *ctx, const dbs_matrix *A, const void *d_x_dense,
                                       dbs_path path, float th3, void *d_y_dense, float *d_y_f32,
                                       dbs_call_stats *stats)
{
    dbs_status st = check_ctx(ctx, A);
    if (st != DBS_OK) return st;
    if (A->d.dtype == DBS_PATTERN) return dbs_fail(DBS_ERR_ARG, "dense activation needs a valued matrix");
    if (path < DBS_PATH_AUTO || path > DBS_PATH_PULL) return dbs_fail(DBS_ERR_ARG, "unknown path");
    if (!d_x_dense || !d_y_dense) return dbs_fail(DBS_ERR_ARG, "NULL activation or output");
    const int mode = A->d.dtype == DBS_F16 ? M_F16 : M_F32;
    const hipStream_t s = ctx->stream;
    // a matrix without COO blocks (a decode layer) under the default
    // selector: pull, without launching the push kernel for the device's
    // choice (see DBS_TH3_DEFAULT)
    int p = (int)path;
    if (p == DBS_PATH_AUTO && !(th3 > 0.f) && A->d.nblk > 0 && A->d.nheavy == A->d.nblk) p = DBS_PATH_PULL;
    if (p == DBS_PATH_PULL && rows_dx_fits(A->d, d_x_dense)) {
        // pull known on the host: the non-COO pass reads the activation
        // itself, without a scan, and writes y itself
        LAUNCH(ctx, DBS_K_MAIN, launch_rows_dx(A->d, ctx->c, mode, d_x_dense, d_y_dense, d_y_f32, s));
    } else {
        if (scan_takes_dense(A->d, d_x_dense)) {
            LAUNCH(ctx, DBS_K_SCAN,
                   launch_scan_dense(A->d, ctx->c, mode, d_x_dense, p, (double)norm_th3(th3), spread_th3(th3), s));
        } else {
            LAUNCH(ctx, DBS_K_SCATTER, launch_ballot(A->d, ctx->c, mode, d_x_dense, s));
            LAUNCH(ctx, DBS_K_SCAN, launch_scan(A->d, ctx->c, p, (double)norm_th3(th3), spread_th3(th3), s));
        }
        LAUNCH(ctx, DBS_K_MAIN, launch_main(A->d, ctx->c, mode, ctx->c.xd, nullptr, 0, nullptr, p, s));
        LAUNCH(ctx, DBS_K_FINALIZE, launch_finalize_dense(A->d, ctx->c, mode, d_y_dense, d_y_f32, s));
    }
    if (stats) {
        if ((st = sync_counters(ctx)) != DBS_OK) return st;
        const int32_t *h = ctx->h_counters;
        std::memset(stats, 0, sizeof *stats);
        stats->path = h[C_PATH];
        stats->n_nzblk = h[C_NZBLK];
        stats->n_blk = A->d.nbc;
        stats->y_nnz = A->d.m;
        stats->tasks = h[C_PATH] == PATH_PUSH ? (int64_t)h[C_TASKS] : A->d.nseg;
        stats->error_flags = h[C_ERR_LAST];
    }
    return DBS_OK;
}

extern "C" dbs_status dbs_spmm_dense(dbs_ctx *ctx, const dbs_matrix *A, int32_t nb, const void *d_x,
                                     void *d_y, float *d_y_f32, dbs_call_stats *stats)
{
    dbs_status st = check_ctx(ctx, A);
    if (st != DBS_OK) return st;
    if (A->d.dtype == DBS_PATTERN) return dbs_fail(DBS_ERR_ARG, "dense activations need a valued matrix");
    if (nb < 1 || nb > DBS_MAX_BATCH) return dbs_fail(DBS_ERR_ARG, "nb = %d outside [1, %d]", nb, DBS_MAX_BATCH);
    if (!d_x || !d_y) return dbs_fail(DBS_ERR_ARG, "NULL activations or outputs");
    const int mode = A->d.dtype == DBS_F16 ? M_F16 : M_F32;
    const size_t vb = A->d.dtype == DBS_F16 ? 2 : 4;
    if (nb == 1 || A->d.nheavy < A->d.nblk || A->d.nblk == 0) {
        // one vector, or a matrix with COO blocks (their segment loop is
        // single-vector): one dense-activation call per vector
        for (int32_t b = 0; b < nb; ++b) {
            st = dbs_spmspv_dense(ctx, A, (const char *)d_x + (size_t)b * A->d.n * vb, DBS_PATH_AUTO, 0.f,
                                  (char *)d_y + (size_t)b * A->d.m * vb, d_y_f32 ? d_y_f32 + (size_t)b * A->d.m : nullptr,
                                  b + 1 == nb ? stats : nullptr);
            if (st != DBS_OK) return st;
        }
        return DBS_OK;
    }
    if (!ctx->xdb) {
        const size_t xb = (size_t)DBS_MAX_BATCH * BS * ctx->max_nbc * 4;
        const size_t yb = (size_t)DBS_MAX_BATCH * BS * ctx->max_nbr * sizeof(double);
        HIP_TRY(hipMalloc(&ctx->xdb, xb), "hipMalloc (batched x)");
        HIP_TRY(hipMemset(ctx->xdb, 0, xb), "hipMemset (batched x)");
        HIP_TRY(hipMalloc((void **)&ctx->yaccb, yb), "hipMalloc (batched y)");
        HIP_TRY(hipMemset(ctx->yaccb, 0, yb), "hipMemset (batched y)");
    }
    const int32_t NB = nb <= 2 ? 2 : nb <= 4 ? 4 : 8;
    const hipStream_t s = ctx->stream;
    LAUNCH(ctx, DBS_K_SCATTER, launch_ballot_batch(A->d, ctx->c, mode, d_x, nb, NB, ctx->xdb, s));
    LAUNCH(ctx, DBS_K_SCAN, launch_scan(A->d, ctx->c, PATH_PULL, 0.0, 0.0, s));
    LAUNCH(ctx, DBS_K_MAIN, launch_rows_batch(A->d, ctx->c, mode, NB, ctx->xdb, ctx->yaccb, s));
    LAUNCH(ctx, DBS_K_FINALIZE, launch_finalize_batch(A->d, ctx->c, mode, nb, NB, ctx->yaccb, d_y, d_y_f32, s));
    if (stats) {
        if ((st = sync_counters(ctx)) != DBS_OK) return st;
        const int32_t *h = ctx->h_counters;
        std::memset(stats, 0, sizeof *stats);
        stats->path = PATH_PULL;
        stats->n_nzblk = h[C_NZBLK];
        stats->n_blk = A->d.nbc;
        stats->y_nnz = A->d.m;
        stats->tasks = A->d.nchunk;
        stats->error_flags = 0;
    }
    return DBS_OK;
}

// ---------------------------------------------------------------------------
// BFS
// ---------------------------------------------------------------------------
extern "C" dbs_status dbs_bfs(dbs_ctx *ctx, const dbs_matrix *A, int32_t source, int32_t *d_level,
                              int32_t *d_parent, dbs_path policy, float th3, dbs_bfs_stats *stats)
{
    dbs_status st = check_ctx(ctx, A);
    if (st != DBS_OK) return st;
    if (A->d.m != A->d.n) return dbs_fail(DBS_ERR_ARG, "BFS needs a square matrix (%dx%d)", A->d.m, A->d.n);
    if (source < 0 || source >= A->d.n) return dbs_fail(DBS_ERR_ARG, "source %d outside [0, %d)", source, A->d.n);
    if (!d_level || !d_parent) return dbs_fail(DBS_ERR_ARG, "NULL level or parent");
    if (policy < DBS_PATH_AUTO || policy > DBS_PATH_PULL) return dbs_fail(DBS_ERR_ARG, "unknown path");
    const hipStream_t s = ctx->stream;
    if (stats) std::memset(stats, 0, sizeof *stats);
    LAUNCH(ctx, DBS_K_OTHER, launch_bfs_init(A->d, ctx->c, source, d_level, d_parent, s));
    int32_t level = 0, reached = 1, frontier = 1;
    for (;;) {
        // BFS levels: with the default th3 push iff the level's push tasks
        // (blocks in the block-CSC lists of the frontier's column blocks) are
        // fewer than DBS_BFS_PUSH_TASKS of the matrix's blocks; an explicit
        // th3 > 0 gives the paper's rule
        const double tasks_max = th3 > 0.f ? -1.0 : (double)DBS_BFS_PUSH_TASKS * (double)A->d.nblk;
        LAUNCH(ctx, DBS_K_SCAN, launch_scan(A->d, ctx->c, (int)policy, (double)norm_th3(th3), 0.0, s, tasks_max));
        if ((st = sync_counters(ctx)) != DBS_OK) {
            ctx->broken = true;
            return st;
        }
        const int32_t *h = ctx->h_counters;
        // the scan's mask popcount is the frontier size
        if (level > 0) {
            frontier = h[C_XPOP];
            reached += frontier;
        }
        if (h[C_NZBLK] == 0) break;
        if (stats && level < DBS_BFS_MAX_LEVEL_STATS) {
            stats->path[level] = h[C_PATH];
            stats->frontier[level] = frontier;
        }
        // the scan's choice is on the host already: launch that kernel only
        LAUNCH(ctx, DBS_K_MAIN,
               launch_main(A->d, ctx->c, M_BFS, nullptr, ctx->c.visited, 1, d_parent, h[C_PATH], s));
        LAUNCH(ctx, DBS_K_BFS_UPDATE, launch_bfs_update(A->d, ctx->c, level + 1, d_level, s));
        ++level;
    }
    LAUNCH(ctx, DBS_K_OTHER, launch_bfs_finish(A->d, d_parent, s));
    if (stats) {
        stats->levels = level;
        stats->reached = reached;
    }
    return DBS_OK;
}

// ---------------------------------------------------------------------------
// SpMSpV without device allocation
// ---------------------------------------------------------------------------
// The scratch of dbs_spmspv_noalloc: the buffers of one call for a matrix of
// up to DBS_NOALLOC_MAX_DIM rows and columns, at fixed 256-byte aligned
// offsets (the layout below).  Each GPU holds its own copy.  In host code
// this name is a host-side stand-in, never a device address: the device
// address of a GPU's copy comes from hipGetSymbolAddress.
static __device__ __align__(256) uint8_t scratch[DBS_NOALLOC_SCRATCH_BYTES];

// Fills `words` 32-bit words at p with v (set-up of the scratch).
static __global__ __launch_bounds__(256) void k_noalloc_fill(uint32_t *p, uint32_t v, int64_t words)
{
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < words; i += (int64_t)gridDim.x * 256) p[i] = v;
}

namespace {

constexpr int32_t NA_NB = (DBS_NOALLOC_MAX_DIM + 15) / 16;  // block rows / block columns at most
constexpr size_t na_round(size_t b) { return (b + 255) / 256 * 256; }
constexpr int32_t NA_NXWORDS = (NA_NB + 1) / 2 + 2;         // mask words (two 16-bit masks each)
constexpr int32_t NA_ST_SCAN = 512, NA_ST_FIN = 1024;       // look-back status words per copy
// byte offsets of the buffers (the roles of a context's scratch)
constexpr size_t NA_XD = 0;                                                     // densified x, 16 NB values
constexpr size_t NA_XMASK = NA_XD + na_round((size_t)16 * NA_NB * 4);           // blk_x_mask words
constexpr size_t NA_XBITS = NA_XMASK + na_round((size_t)NA_NXWORDS * 4);        // activity bits
constexpr size_t NA_ITEMS = NA_XBITS + na_round(((size_t)NA_NB + 31) / 32 * 4 + 256);  // push work items
constexpr size_t NA_YACC = NA_ITEMS + na_round(((size_t)NA_NB + 2) * 16);       // fp64 y accumulators
constexpr size_t NA_YBITS = NA_YACC + na_round((size_t)16 * NA_NB * 8);         // y structure words
constexpr size_t NA_COUNTERS = NA_YBITS + na_round((size_t)NA_NXWORDS * 4);     // counters
constexpr size_t NA_ST = NA_COUNTERS + na_round((size_t)C_COUNT * 4);           // statuses: scan x2, fin x2
constexpr size_t NA_ST_SCAN_BYTES = na_round((size_t)NA_ST_SCAN * 8), NA_ST_FIN_BYTES = na_round((size_t)NA_ST_FIN * 8);
constexpr size_t NA_SYNC = NA_ST + 2 * NA_ST_SCAN_BYTES + 2 * NA_ST_FIN_BYTES;  // single-launch flags
constexpr size_t NA_END = NA_SYNC + na_round((size_t)SYNC_WORDS * 4);
static_assert(NA_END <= DBS_NOALLOC_SCRATCH_BYTES, "the static scratch holds the buffers of a maximal call");

constexpr int NA_MAX_DEVICES = 64;
struct NoAllocDevice {
    uint8_t *ptr = nullptr;  // device address of this GPU's copy of `scratch`
    int scan_parity = 0, fin_parity = 0;
    uint32_t gen = 0;        // number of the last single-launch call
};
NoAllocDevice g_na[NA_MAX_DEVICES];
std::mutex g_na_mu;  // guards g_na (held for the whole host side of a call)

// The current device's scratch, set up on its first use: its address, then
// its initial contents (all-ones bits in the densified x mark absent
// entries, zeros elsewhere), waited for on the stream.
dbs_status noalloc_device(hipStream_t s, NoAllocDevice **out)
{
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev), "hipGetDevice");
    if (dev < 0 || dev >= NA_MAX_DEVICES)
        return dbs_fail(DBS_ERR_UNSUPPORTED, "device %d: the no-allocation path serves devices 0..%d", dev,
                        NA_MAX_DEVICES - 1);
    NoAllocDevice &d = g_na[dev];
    if (!d.ptr) {
        dbs_status st = check_device();
        if (st != DBS_OK) return st;
        if (scan_tiles(NA_NB) + 1 > NA_ST_SCAN || finalize_tiles(NA_NB) + 1 > NA_ST_FIN)
            return dbs_fail(DBS_ERR_UNSUPPORTED, "static scratch: status regions too small");
        void *p = nullptr;
        HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress (static scratch)");
        hipLaunchKernelGGL(k_noalloc_fill, dim3(1024), dim3(256), 0, s, (uint32_t *)p, 0xFFFFFFFFu,
                           (int64_t)(NA_XMASK / 4));
        HIP_TRY(hipGetLastError(), "kernel launch (scratch set-up)");
        hipLaunchKernelGGL(k_noalloc_fill, dim3(1024), dim3(256), 0, s, (uint32_t *)((uint8_t *)p + NA_XMASK), 0u,
                           (int64_t)((NA_END - NA_XMASK) / 4));
        HIP_TRY(hipGetLastError(), "kernel launch (scratch set-up)");
        HIP_TRY(hipStreamSynchronize(s), "hipStreamSynchronize (scratch set-up)");
        d.ptr = (uint8_t *)p;
    }
    *out = &d;
    return DBS_OK;
}

// Context buffers over a device's scratch.
DevCtx noalloc_ctx(const NoAllocDevice &d)
{
    DevCtx c;
    c.xd = d.ptr + NA_XD;
    c.xmask = (uint32_t *)(d.ptr + NA_XMASK);
    c.nxwords = NA_NXWORDS;
    c.xbits = (uint32_t *)(d.ptr + NA_XBITS);
    c.items = (int4 *)(d.ptr + NA_ITEMS);
    c.yacc = (double *)(d.ptr + NA_YACC);
    c.ybits = (uint32_t *)(d.ptr + NA_YBITS);
    c.nywords = NA_NXWORDS;
    c.visited = nullptr;  // (BFS only)
    c.nextm = nullptr;
    c.counters = (int32_t *)(d.ptr + NA_COUNTERS);
    c.st_scan[0] = (uint64_t *)(d.ptr + NA_ST);
    c.st_scan[1] = (uint64_t *)(d.ptr + NA_ST + NA_ST_SCAN_BYTES);
    c.n_st_scan = scan_tiles(NA_NB) + 1;
    c.st_fin[0] = (uint64_t *)(d.ptr + NA_ST + 2 * NA_ST_SCAN_BYTES);
    c.st_fin[1] = (uint64_t *)(d.ptr + NA_ST + 2 * NA_ST_SCAN_BYTES + NA_ST_FIN_BYTES);
    c.n_st_fin = finalize_tiles(NA_NB) + 1;
    c.scan_parity = d.scan_parity;
    c.fin_parity = d.fin_parity;
    c.sync = (uint32_t *)(d.ptr + NA_SYNC);
    c.gen = d.gen;
    // no compaction list: pull takes the segment loop at every activity
    c.clist = nullptr;
    c.clist_cap = 0;
    c.ccount = nullptr;
    return c;
}

}  // namespace

extern "C" dbs_status dbs_spmspv_noalloc(const dbs_matrix *A, dbs_semiring sr, int32_t x_nnz,
                                         const int32_t *d_x_idx, const void *d_x_val, const uint32_t *d_mask,
                                         int complement_mask, dbs_path path, float th3, int32_t *d_y_idx,
                                         void *d_y_val, int32_t *d_y_nnz, void *stream)
{
    if (!A) return dbs_fail(DBS_ERR_ARG, "dbs_spmspv_noalloc: NULL matrix");
    if (A->d.m > DBS_NOALLOC_MAX_DIM || A->d.n > DBS_NOALLOC_MAX_DIM)
        return dbs_fail(DBS_ERR_UNSUPPORTED,
                        "dbs_spmspv_noalloc: matrix %dx%d exceeds the static scratch's limit of %d rows and columns",
                        A->d.m, A->d.n, DBS_NOALLOC_MAX_DIM);
    int mode = 0;
    dbs_status st = spmspv_check_args(A, sr, x_nnz, d_x_idx, d_x_val, path, d_y_idx, d_y_val, d_y_nnz, &mode);
    if (st != DBS_OK) return st;
    const hipStream_t s = (hipStream_t)stream;
    std::lock_guard<std::mutex> lock(g_na_mu);
    NoAllocDevice *d = nullptr;
    if ((st = noalloc_device(s, &d)) != DBS_OK) return st;
    DevCtx c = noalloc_ctx(*d);
    st = spmspv_launches(A, c, s, mode, sr, x_nnz, d_x_idx, d_x_val, d_mask, complement_mask, path, th3, d_y_idx,
                         d_y_val, d_y_nnz, false, [](int, auto &&launch) -> dbs_status {
                             const hipError_t e = launch();
                             return e == hipSuccess ? DBS_OK : hip_fail(e, "kernel launch");
                         });
    d->scan_parity = c.scan_parity;
    d->fin_parity = c.fin_parity;
    d->gen = c.gen;
    return st;
}
