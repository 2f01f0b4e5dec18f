// GPU-side conversion (the offline step of Sec. 3.1 / 3.2.1 / 3.3.2, done on
// the device): a dense matrix already in device memory -- a pruned weight
// matrix as decoding loads it (Sec. 4.3) -- becomes a device DB matrix, the
// same arrays, byte for byte, that the host builder and dbs_matrix_upload
// produce from the CSR of its nonzero entries.
//
//   1. k_conv_tiles: a wave per 16x16 tile finds its row masks (entry stored
//      iff its value is nonzero), its nnz and format (Sec. 3.2.1 classifier);
//   2. k_conv_rows: a thread per block row walks its tiles in block-column
//      order like the host walk: record offsets and alignment, block index,
//      pull-segment closure (weights 4/2/1 closing at seg_close or 16
//      blocks), index in the non-COO list;
//   3. the per-row totals are prefix-summed on the host (nbr values), the
//      device arrays are allocated at their exact sizes;
//   4. k_conv_write: a wave per nonzero tile writes its record (Dense,
//      ForceCSR, ForceCSC, patched CSR or COO; or the inline COO descriptor),
//      its slot and its non-COO list entry; k_conv_segs the segment words and
//      non-COO chunks; k_conv_csc_* the block-CSC view by a count, a host
//      scan and an in-order fill per block column.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <new>
#include <vector>

#include "device_common.hpp"
#include "matrix.hpp"

using namespace dbs;

namespace {

constexpr int CTPB = 256;             // 4 waves per workgroup, one tile each
constexpr int RS = 10;                // per-row statistics, see k_conv_rows
constexpr int PRE = 5;                // per-row prefixes: blocks, bytes, segments, non-COO, chunks

dbs_status conv_fail(hipError_t e, const char *what)
{
    return dbs_fail(DBS_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}
#define CONV_TRY(expr, what)                             \
    do {                                                 \
        hipError_t e_ = (expr);                          \
        if (e_ != hipSuccess) return conv_fail(e_, what); \
    } while (0)

// Raw bits of element (row, col) of the dense input (0 outside the matrix).
template <int VB>
__device__ __forceinline__ uint32_t elem_bits(const void *w, int64_t ld, int32_t m, int32_t n, int64_t row,
                                              int64_t col)
{
    if (row >= m || col >= n) return 0u;
    if constexpr (VB == 4) return ((const uint32_t *)w)[row * ld + col];
    else return ((const uint16_t *)w)[row * ld + col];
}
// Stored iff the value is nonzero (-0 is zero; NaN is stored).
template <int VB>
__device__ __forceinline__ bool stored_bits(uint32_t b)
{
    return VB == 4 ? (b & 0x7FFFFFFFu) != 0u : (b & 0x7FFFu) != 0u;
}

// One wave, one tile: lane l covers row l / 4, columns 4 (l % 4) .. + 3.
// Loads the lane's four elements and leaves the tile's 16 row masks in rm.
template <int VB>
__device__ __forceinline__ uint32_t tile_lane(const void *w, int64_t ld, int32_t m, int32_t n, int32_t R,
                                              int32_t J, uint32_t (&bits)[4], uint16_t *rm)
{
    const int lane = lane_id(), r = lane >> 2, c0 = (lane & 3) * 4;
    uint32_t nib = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        bits[q] = elem_bits<VB>(w, ld, m, n, (int64_t)R * BS + r, (int64_t)J * BS + c0 + q);
        nib |= (stored_bits<VB>(bits[q]) ? 1u : 0u) << q;
    }
    uint32_t row = nib << c0;
    row |= (uint32_t)__shfl_xor((int)row, 1, WAVE);
    row |= (uint32_t)__shfl_xor((int)row, 2, WAVE);
    if ((lane & 3) == 0) rm[r] = (uint16_t)row;
    wave_lds_sync();
    return nib;
}

// Sec. 3.2.1 classifier on the row masks, as the host builder applies it.
__device__ __forceinline__ uint32_t classify_masks(const uint16_t *rm, uint32_t nnz, int32_t th0, int32_t th1,
                                                   float th2, int32_t force_type)
{
    if (force_type >= 0) return (uint32_t)force_type;
    if ((int64_t)nnz < th0) return T_COO;
    if ((int64_t)nnz > th1) return T_DENSE;
    uint32_t mr = 0, mc = 0;
#pragma unroll
    for (int t = 0; t < BS; ++t) mr = max(mr, (uint32_t)__popc(rm[t]));
#pragma unroll
    for (int c = 0; c < BS; ++c) {
        uint32_t cc = 0;
#pragma unroll
        for (int t = 0; t < BS; ++t) cc += (rm[t] >> c) & 1u;
        mc = max(mc, cc);
    }
    if ((float)mc > th2 * (float)mr) return T_FCSC;
    if ((float)mr > th2 * (float)mc) return T_FCSR;
    return T_CSR;
}

// Per tile: nnz | type << 16 | inline << 24 (0 for an empty tile).
template <int VB>
__global__ __launch_bounds__(CTPB) void k_conv_tiles(const void *w, int64_t ld, int32_t m, int32_t n, int32_t nbc,
                                                     int64_t ntiles, int32_t th0, int32_t th1, float th2,
                                                     int32_t force_type, int32_t inline_small, uint32_t *tinfo)
{
    __shared__ uint16_t rms[CTPB / WAVE][BS];
    const int wv = threadIdx.x >> 6;
    const int64_t tile = (int64_t)blockIdx.x * (CTPB / WAVE) + wv;
    if (tile >= ntiles) return;
    const int32_t R = (int32_t)(tile / nbc), J = (int32_t)(tile % nbc);
    uint32_t bits[4];
    uint16_t *rm = rms[wv];
    tile_lane<VB>(w, ld, m, n, R, J, bits, rm);
    uint32_t nnz = 0;
#pragma unroll
    for (int t = 0; t < BS; ++t) nnz += (uint32_t)__popc(rm[t]);
    if (lane_id() != 0) return;
    if (nnz == 0) {
        tinfo[tile] = 0u;
        return;
    }
    const uint32_t type = classify_masks(rm, nnz, th0, th1, th2, force_type);
    const uint32_t inl = (inline_small && type == T_COO && nnz <= inline_capacity((uint32_t)VB)) ? 1u : 0u;
    tinfo[tile] = nnz | (type << 16) | (inl << 24);
}

// A thread per block row: the host walk over its nonzero tiles.  Per tile:
// record offset within the row (all ones: inline), block index within the
// row | position in its segment << 28, segment index within the row, index
// among the row's non-COO blocks.  Per row (RS int64): blocks, payload bytes
// (16-byte multiple), segments, non-COO blocks, nnz, blocks by type.
__global__ __launch_bounds__(CTPB) void k_conv_rows(const uint32_t *tinfo, int32_t nbr, int32_t nbc,
                                                    int32_t seg_close, uint32_t vb, uint32_t *toff, uint32_t *tb,
                                                    uint32_t *tseg, uint32_t *thv, int64_t *rstat)
{
    const int32_t R = (int32_t)(blockIdx.x * CTPB + threadIdx.x);
    if (R >= nbr) return;
    uint64_t cursor = 0;
    uint32_t seg_w = 0, seg_cnt = 0, nseg = 0, nblk = 0, heavy = 0;
    int64_t nnz_sum = 0, bytype[DBS_NUM_BLOCK_TYPES] = {0, 0, 0, 0, 0};
    for (int32_t J = 0; J < nbc; ++J) {
        const int64_t tile = (int64_t)R * nbc + J;
        const uint32_t t = tinfo[tile];
        const uint32_t nnz = t & 0xFFFFu;
        if (nnz == 0) continue;
        const uint32_t type = (t >> 16) & 0xFFu, inl = (t >> 24) & 1u;
        if (!inl) {
            const uint32_t al = record_align(type, vb);
            cursor = (cursor + al - 1) / al * al;
        }
        toff[tile] = inl ? 0xFFFFFFFFu : (uint32_t)cursor;
        if (!inl) cursor += record_bytes(type, nnz, vb);
        tb[tile] = nblk | (seg_cnt << 28);
        tseg[tile] = nseg;
        thv[tile] = heavy;
        if (type != T_COO) ++heavy;
        seg_w += seg_weight(type);
        seg_cnt += 1;
        if ((int32_t)seg_w >= seg_close || seg_cnt == (uint32_t)MAX_SEG_BLOCKS) {
            ++nseg;
            seg_w = 0;
            seg_cnt = 0;
        }
        ++nblk;
        nnz_sum += nnz;
        bytype[type]++;
    }
    if (seg_cnt) ++nseg;
    int64_t *o = rstat + (int64_t)R * RS;
    o[0] = nblk;
    o[1] = (int64_t)((cursor + 15) / 16 * 16);
    o[2] = nseg;
    o[3] = heavy;
    o[4] = nnz_sum;
#pragma unroll
    for (int t = 0; t < DBS_NUM_BLOCK_TYPES; ++t) o[5 + t] = bytype[t];
}

struct ConvOut {
    uint8_t *pay;
    int32_t *sl_col;
    uint64_t *sl_desc;
    int32_t *hv_col;
    uint64_t *hv_desc;
    uint64_t *blk_desc;  // descriptor per primary block (for the CSC fill)
};

// A wave per nonzero tile: record, descriptor, slot, non-COO list entry.
template <int VB>
__global__ __launch_bounds__(CTPB) void k_conv_write(const void *w, int64_t ld, int32_t m, int32_t n, int32_t nbc,
                                                     int64_t ntiles, const uint32_t *tinfo, const uint32_t *toff,
                                                     const uint32_t *tb, const uint32_t *tseg,
                                                     const uint32_t *thv, const int64_t *pre, ConvOut out)
{
    __shared__ uint16_t rms[CTPB / WAVE][BS];
    __shared__ uint16_t cms[CTPB / WAVE][BS];
    const int wv = threadIdx.x >> 6, lane = lane_id();
    const int64_t tile = (int64_t)blockIdx.x * (CTPB / WAVE) + wv;
    if (tile >= ntiles) return;
    const uint32_t t = tinfo[tile];
    const uint32_t nnz = t & 0xFFFFu;
    if (nnz == 0) return;
    const uint32_t type = (t >> 16) & 0xFFu, inl = (t >> 24) & 1u;
    const int32_t R = (int32_t)(tile / nbc), J = (int32_t)(tile % nbc);
    uint32_t bits[4];
    uint16_t *rm = rms[wv], *cm = cms[wv];
    const uint32_t nib = tile_lane<VB>(w, ld, m, n, R, J, bits, rm);
    // column masks (bit r of column c), by lanes 0..15
    if (lane < BS) {
        uint32_t c = 0;
#pragma unroll
        for (int q = 0; q < BS; ++q) c |= ((rm[q] >> lane) & 1u) << q;
        cm[lane] = (uint16_t)c;
    }
    wave_lds_sync();
    const int r = lane >> 2, c0 = (lane & 3) * 4;
    const uint32_t myrow = rm[r];
    uint32_t rstart = 0;
#pragma unroll
    for (int q = 0; q < BS; ++q) rstart += q < r ? (uint32_t)__popc(rm[q]) : 0u;
    const int64_t *P = pre + (int64_t)R * PRE;
    const uint32_t vb = (uint32_t)VB;
    const uint64_t off = (uint64_t)P[1] + (inl ? 0ull : (uint64_t)toff[tile]);
    uint8_t *rec = out.pay + off;
    uint64_t dpart = 0;  // inline descriptor bits of this lane's entries
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        if (!((nib >> q) & 1u)) continue;
        const uint32_t c = (uint32_t)(c0 + q);
        const uint32_t k = rstart + (uint32_t)__popc(myrow & ((1u << c) - 1u));  // row-major rank
        uint32_t cstart = 0;
#pragma unroll
        for (int u = 0; u < BS; ++u) cstart += (uint32_t)u < c ? (uint32_t)__popc(cm[u]) : 0u;
        const uint32_t pos = cstart + (uint32_t)__popc(cm[c] & ((1u << r) - 1u));  // column-major rank
        const uint8_t cd = (uint8_t)((r << 4) | c);
        if (inl) {
            const uint32_t sh = inline_shift(k, vb);
            dpart |= ((uint64_t)cd << sh) | ((uint64_t)bits[q] << (sh + 8));
            continue;
        }
        uint64_t vo = 0;
        switch (type) {
        case T_COO:
            vo = (uint64_t)k * vb;
            rec[(uint64_t)vb * nnz + k] = cd;
            break;
        case T_DENSE: vo = HDR_START + (uint64_t)(r * BS + c) * vb; break;
        case T_FCSR: vo = HDR_START2 + (uint64_t)k * vb; break;
        case T_FCSC: vo = HDR_START2 + (uint64_t)pos * vb; break;
        default:
            rec[HDR_RCSC + pos] = (uint8_t)((r << 4) | (k - rstart));
            vo = HDR_RCSC + round_up(nnz, 16) + (uint64_t)k * vb;
            break;
        }
        if constexpr (VB == 4) *(uint32_t *)(rec + vo) = bits[q];
        else *(uint16_t *)(rec + vo) = (uint16_t)bits[q];
    }
    // headers: row masks (column masks for ForceCSC) and group starts
    if (!inl && type != T_COO) {
        if (type == T_FCSC) {
            if (lane < BS) {
                uint32_t cs = 0;
#pragma unroll
                for (int u = 0; u < BS; ++u) cs += u < lane ? (uint32_t)__popc(cm[u]) : 0u;
                *(uint16_t *)(rec + HDR_MASK + 2 * lane) = cm[lane];
                rec[HDR_START + lane] = (uint8_t)cs;
            }
        } else if ((lane & 3) == 0) {
            *(uint16_t *)(rec + HDR_MASK + 2 * r) = (uint16_t)myrow;
            if (type != T_DENSE) rec[HDR_START + r] = (uint8_t)rstart;
        }
        if (type == T_CSR && lane < BS) {
            uint32_t cs = 0;
#pragma unroll
            for (int u = 0; u < BS; ++u) cs += u < lane ? (uint32_t)__popc(cm[u]) : 0u;
            rec[HDR_START2 + lane] = (uint8_t)cs;
        }
    }
    // descriptor (inline: the wave's entries OR-ed together)
    uint64_t d;
    if (inl) {
        uint64_t acc = dpart;
#pragma unroll
        for (int o = 1; o < WAVE; o <<= 1) {
            const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)acc, o, WAVE);
            const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(acc >> 32), o, WAVE);
            acc |= ((uint64_t)hi << 32) | lo;
        }
        d = acc | ((uint64_t)(nnz - 1) << 8) | DESC_INLINE | (uint64_t)T_COO;
    } else {
        d = desc_make(off, nnz, type);
    }
    if (lane == 0) {
        const uint32_t bl = tb[tile] & 0x0FFFFFFFu, pi = tb[tile] >> 28;
        const int64_t b = P[0] + bl;
        const int64_t slot = (P[2] + (int64_t)tseg[tile]) * 16 + pi;
        out.sl_col[slot] = slot_word(J, d);
        out.sl_desc[slot] = d;
        out.blk_desc[b] = d;
        if (type != T_COO) {
            const int64_t hv = P[3] + (int64_t)thv[tile];
            out.hv_col[hv] = J;
            out.hv_desc[hv] = d;
        }
    }
}

// A thread per block row: its segment words (the block row) and non-COO
// chunks (at most HV_CHUNK consecutive blocks of the row each).
// Chunks of each block row (the count array starts at zero).
__global__ __launch_bounds__(CTPB) void k_conv_rowchunks(int64_t nchunk, const int32_t *hv_crow, int32_t *rowchunks)
{
    const int64_t c = (int64_t)blockIdx.x * CTPB + threadIdx.x;
    if (c < nchunk) atomicAdd(&rowchunks[hv_crow[c]], 1);
}

__global__ __launch_bounds__(CTPB) void k_conv_segs(int32_t nbr, const int64_t *pre, uint32_t *seg_rs,
                                                    int32_t *hv_cstart, int32_t *hv_crow)
{
    const int32_t R = (int32_t)(blockIdx.x * CTPB + threadIdx.x);
    if (R >= nbr) return;
    const int64_t *P = pre + (int64_t)R * PRE, *Q = P + PRE;
    const int64_t nseg = Q[2] - P[2], nch = Q[4] - P[4];
    for (int64_t s = 0; s < nseg; ++s) seg_rs[P[2] + s] = (uint32_t)R;
    for (int64_t c = 0; c < nch; ++c) {
        hv_cstart[P[4] + c] = (int32_t)(P[3] + c * HV_CHUNK);
        hv_crow[P[4] + c] = R;
    }
}

// A thread per block column: its nonzero tiles.
__global__ __launch_bounds__(CTPB) void k_conv_csc_count(const uint32_t *tinfo, int32_t nbr, int32_t nbc,
                                                         int32_t *cnt)
{
    const int32_t J = (int32_t)(blockIdx.x * CTPB + threadIdx.x);
    if (J >= nbc) return;
    int32_t c = 0;
    for (int32_t R = 0; R < nbr; ++R) c += (tinfo[(int64_t)R * nbc + J] & 0xFFFFu) ? 1 : 0;
    cnt[J] = c;
}

// A thread per block column: its blocks in block-row order.
__global__ __launch_bounds__(CTPB) void k_conv_csc_fill(const uint32_t *tinfo, const uint32_t *tb,
                                                        const int64_t *pre, int32_t nbr, int32_t nbc,
                                                        const int32_t *cb_ptr, const uint64_t *blk_desc,
                                                        int32_t *csc_row, uint64_t *csc_desc)
{
    const int32_t J = (int32_t)(blockIdx.x * CTPB + threadIdx.x);
    if (J >= nbc) return;
    int32_t q = cb_ptr[J];
    for (int32_t R = 0; R < nbr; ++R) {
        const int64_t tile = (int64_t)R * nbc + J;
        if (!(tinfo[tile] & 0xFFFFu)) continue;
        const int64_t b = pre[(int64_t)R * PRE] + (tb[tile] & 0x0FFFFFFFu);
        csc_row[q] = R;
        csc_desc[q] = blk_desc[b];
        ++q;
    }
}

// Device allocation owned by the matrix (at least 16 bytes), cleared to
// `byte` on the stream.
template <class T>
dbs_status conv_alloc(std::vector<void *> &allocs, size_t count, T **out, int byte, hipStream_t s, size_t pad = 0)
{
    const size_t bytes = std::max<size_t>(count * sizeof(T) + pad, 16);
    void *p = nullptr;
    CONV_TRY(hipMalloc(&p, bytes), "hipMalloc (conversion)");
    allocs.push_back(p);
    CONV_TRY(hipMemsetAsync(p, byte, bytes, s), "hipMemsetAsync (conversion)");
    *out = (T *)p;
    return DBS_OK;
}

// Temporary device buffers of one conversion; the stream is drained before
// they are freed (also on an error return).
struct Scratch {
    hipStream_t s;
    std::vector<void *> p;
    ~Scratch()
    {
        (void)hipStreamSynchronize(s);
        for (void *q : p) (void)hipFree(q);
    }
};

template <int VB>
dbs_status convert(int32_t m, int32_t n, const void *d_w, int64_t ld, const dbs_build_opts &o, hipStream_t s,
                   dbs_matrix *A)
{
    DevMatrix &d = A->d;
    const int32_t nbr = (int32_t)(((int64_t)m + BS - 1) / BS), nbc = (int32_t)(((int64_t)n + BS - 1) / BS);
    const int64_t ntiles = (int64_t)nbr * nbc;
    const uint32_t vb = (uint32_t)VB;
    Scratch tmp{s, {}};
    uint32_t *tinfo = nullptr, *toff = nullptr, *tb = nullptr, *tseg = nullptr, *thv = nullptr;
    int64_t *rstat = nullptr, *pre_d = nullptr;
    auto scratch = [&](size_t bytes, void **out) -> hipError_t {
        hipError_t e = hipMalloc(out, std::max<size_t>(bytes, 16));
        if (e == hipSuccess) tmp.p.push_back(*out);
        return e;
    };
    CONV_TRY(scratch(ntiles * 4, (void **)&tinfo), "hipMalloc (tiles)");
    CONV_TRY(scratch(ntiles * 4, (void **)&toff), "hipMalloc (tiles)");
    CONV_TRY(scratch(ntiles * 4, (void **)&tb), "hipMalloc (tiles)");
    CONV_TRY(scratch(ntiles * 4, (void **)&tseg), "hipMalloc (tiles)");
    CONV_TRY(scratch(ntiles * 4, (void **)&thv), "hipMalloc (tiles)");
    CONV_TRY(scratch((size_t)nbr * RS * 8, (void **)&rstat), "hipMalloc (rows)");
    CONV_TRY(scratch((size_t)(nbr + 1) * PRE * 8, (void **)&pre_d), "hipMalloc (rows)");
    const int64_t tgrid = (ntiles + (CTPB / WAVE) - 1) / (CTPB / WAVE);
    if (ntiles > 0) {
        hipLaunchKernelGGL(k_conv_tiles<VB>, dim3((unsigned)tgrid), dim3(CTPB), 0, s, d_w, ld, m, n, nbc, ntiles,
                           o.th0, o.th1, o.th2, o.force_type, o.inline_small, tinfo);
        CONV_TRY(hipGetLastError(), "k_conv_tiles");
        hipLaunchKernelGGL(k_conv_rows, dim3((unsigned)((nbr + CTPB - 1) / CTPB)), dim3(CTPB), 0, s, tinfo, nbr,
                           nbc, o.seg_close, vb, toff, tb, tseg, thv, rstat);
        CONV_TRY(hipGetLastError(), "k_conv_rows");
    }
    // per-row totals -> prefixes (host)
    std::vector<int64_t> rs((size_t)nbr * RS), pre((size_t)(nbr + 1) * PRE, 0);
    if (nbr > 0 && ntiles > 0) {
        CONV_TRY(hipMemcpyAsync(rs.data(), rstat, rs.size() * 8, hipMemcpyDeviceToHost, s), "hipMemcpy (rows)");
        CONV_TRY(hipStreamSynchronize(s), "hipStreamSynchronize");
    }
    int64_t nnz = 0, by_type[DBS_NUM_BLOCK_TYPES] = {0, 0, 0, 0, 0};
    for (int32_t R = 0; R < nbr; ++R) {
        const int64_t *x = rs.data() + (size_t)R * RS;
        int64_t *p = pre.data() + (size_t)R * PRE, *q = p + PRE;
        q[0] = p[0] + x[0];
        q[1] = p[1] + x[1];
        q[2] = p[2] + x[2];
        q[3] = p[3] + x[3];
        q[4] = p[4] + (x[3] + HV_CHUNK - 1) / HV_CHUNK;
        nnz += x[4];
        for (int t = 0; t < DBS_NUM_BLOCK_TYPES; ++t) by_type[t] += x[5 + t];
    }
    const int64_t *tot = pre.data() + (size_t)nbr * PRE;
    const int64_t nblk = tot[0], bytes = tot[1], nseg = tot[2], nheavy = tot[3], nchunk = tot[4];
    if (nblk >= ((int64_t)1 << 31) - 1)
        return dbs_fail(DBS_ERR_UNSUPPORTED, "%lld nonzero blocks exceed 2^31-1", (long long)nblk);
    if (bytes >= ((int64_t)1 << 47)) return dbs_fail(DBS_ERR_UNSUPPORTED, "payload too large");
    if ((int64_t)16 * nseg >= ((int64_t)1 << 31))
        return dbs_fail(DBS_ERR_UNSUPPORTED, "%lld pull segments exceed the 2^31 slot limit", (long long)nseg);
    CONV_TRY(hipMemcpyAsync(pre_d, pre.data(), pre.size() * 8, hipMemcpyHostToDevice, s), "hipMemcpy (prefixes)");

    int32_t *sl_col = nullptr, *cb_ptr = nullptr, *csc_row = nullptr, *hv_col = nullptr, *hv_cstart = nullptr,
            *hv_crow = nullptr, *hv_rowchunks = nullptr;
    uint64_t *sl_desc = nullptr, *csc_desc = nullptr, *hv_desc = nullptr, *blk_desc = nullptr;
    uint32_t *seg_rs = nullptr;
    uint8_t *pay = nullptr;
    dbs_status st = DBS_OK;
    if ((st = conv_alloc(A->allocs, (size_t)(16 * nseg), &sl_col, 0xFF, s)) != DBS_OK ||
        (st = conv_alloc(A->allocs, (size_t)(16 * nseg), &sl_desc, 0, s)) != DBS_OK ||
        (st = conv_alloc(A->allocs, (size_t)nseg, &seg_rs, 0, s)) != DBS_OK ||
        (st = conv_alloc(A->allocs, (size_t)nbc + 1, &cb_ptr, 0, s)) != DBS_OK ||
        (st = conv_alloc(A->allocs, (size_t)nblk, &csc_row, 0, s)) != DBS_OK ||
        (st = conv_alloc(A->allocs, (size_t)nblk, &csc_desc, 0, s)) != DBS_OK ||
        (st = conv_alloc(A->allocs, (size_t)nheavy, &hv_col, 0, s)) != DBS_OK ||
        (st = conv_alloc(A->allocs, (size_t)nheavy, &hv_desc, 0, s)) != DBS_OK ||
        (st = conv_alloc(A->allocs, (size_t)nchunk + 1, &hv_cstart, 0, s)) != DBS_OK ||
        (st = conv_alloc(A->allocs, (size_t)nchunk, &hv_crow, 0, s)) != DBS_OK ||
        (st = conv_alloc(A->allocs, (size_t)std::max<int64_t>(nbr, 1), &hv_rowchunks, 0, s)) != DBS_OK ||
        (st = conv_alloc(A->allocs, (size_t)bytes, &pay, 0, s, 16)) != DBS_OK)
        return st;
    CONV_TRY(scratch((size_t)nblk * 8, (void **)&blk_desc), "hipMalloc (descriptors)");
    int32_t *ccnt = nullptr;
    CONV_TRY(scratch((size_t)nbc * 4, (void **)&ccnt), "hipMalloc (column counts)");
    if (nblk > 0) {
        ConvOut out{pay, sl_col, sl_desc, hv_col, hv_desc, blk_desc};
        hipLaunchKernelGGL(k_conv_write<VB>, dim3((unsigned)tgrid), dim3(CTPB), 0, s, d_w, ld, m, n, nbc, ntiles,
                           tinfo, toff, tb, tseg, thv, pre_d, out);
        CONV_TRY(hipGetLastError(), "k_conv_write");
        hipLaunchKernelGGL(k_conv_segs, dim3((unsigned)((nbr + CTPB - 1) / CTPB)), dim3(CTPB), 0, s, nbr, pre_d,
                           seg_rs, hv_cstart, hv_crow);
        CONV_TRY(hipGetLastError(), "k_conv_segs");
        if (nchunk > 0) {
            hipLaunchKernelGGL(k_conv_rowchunks, dim3((unsigned)((nchunk + CTPB - 1) / CTPB)), dim3(CTPB), 0, s,
                               nchunk, hv_crow, hv_rowchunks);
            CONV_TRY(hipGetLastError(), "k_conv_rowchunks");
        }
    }
    const int32_t nheavy32 = (int32_t)nheavy;
    CONV_TRY(hipMemcpyAsync(hv_cstart + nchunk, &nheavy32, 4, hipMemcpyHostToDevice, s), "hipMemcpy (chunks)");
    // block-CSC view: counts, host scan, in-order fill
    std::vector<int32_t> cnt((size_t)nbc, 0), ptr((size_t)nbc + 1, 0);
    if (nblk > 0) {
        hipLaunchKernelGGL(k_conv_csc_count, dim3((unsigned)((nbc + CTPB - 1) / CTPB)), dim3(CTPB), 0, s, tinfo,
                           nbr, nbc, ccnt);
        CONV_TRY(hipGetLastError(), "k_conv_csc_count");
        CONV_TRY(hipMemcpyAsync(cnt.data(), ccnt, (size_t)nbc * 4, hipMemcpyDeviceToHost, s), "hipMemcpy (csc)");
        CONV_TRY(hipStreamSynchronize(s), "hipStreamSynchronize");
    }
    for (int32_t J = 0; J < nbc; ++J) ptr[J + 1] = ptr[J] + cnt[J];
    CONV_TRY(hipMemcpyAsync(cb_ptr, ptr.data(), ptr.size() * 4, hipMemcpyHostToDevice, s), "hipMemcpy (csc)");
    if (nblk > 0) {
        hipLaunchKernelGGL(k_conv_csc_fill, dim3((unsigned)((nbc + CTPB - 1) / CTPB)), dim3(CTPB), 0, s, tinfo, tb,
                           pre_d, nbr, nbc, cb_ptr, blk_desc, csc_row, csc_desc);
        CONV_TRY(hipGetLastError(), "k_conv_csc_fill");
    }
    // the scratch is freed on return: finish first (host vectors are read
    // by the asynchronous copies above as well)
    CONV_TRY(hipStreamSynchronize(s), "hipStreamSynchronize");

    d.m = m;
    d.n = n;
    d.nbr = nbr;
    d.nbc = nbc;
    d.nblk = nblk;
    d.nseg = nseg;
    d.sl_col = sl_col;
    d.sl_desc = sl_desc;
    d.seg_rs = seg_rs;
    d.cb_ptr = cb_ptr;
    d.csc_row = csc_row;
    d.csc_desc = csc_desc;
    d.hv_col = hv_col;
    d.hv_desc = hv_desc;
    d.hv_cstart = hv_cstart;
    d.hv_crow = hv_crow;
    d.hv_rowchunks = hv_rowchunks;
    d.nheavy = nheavy;
    d.nchunk = nchunk;
    d.pay = pay;
    dbs_matrix_info &I = A->info;
    std::memset(&I, 0, sizeof I);
    I.m = m;
    I.n = n;
    I.nnz = nnz;
    I.dtype = d.dtype;
    I.nbr = nbr;
    I.nbc = nbc;
    I.nblk = nblk;
    I.nseg = nseg;
    for (int t = 0; t < DBS_NUM_BLOCK_TYPES; ++t) I.blocks_by_type[t] = by_type[t];
    I.payload_bytes = bytes;
    I.db_bytes = 4 * (int64_t)(nbr + 1) + 4 * nblk + 4 * (int64_t)(nbc + 1) + 8 * nblk + 8 * nblk + bytes + 8 * nseg;
    dbs_storage_model(m, n, nnz, (int32_t)vb, &I.csr_bytes, &I.csr_csc_bytes);
    return DBS_OK;
}

}  // namespace

extern "C" dbs_status dbs_matrix_build_dense(int32_t m, int32_t n, const void *d_w, int64_t ld, dbs_dtype vt,
                                             const dbs_build_opts *opts, void *stream, dbs_matrix **out)
{
    if (!out) return dbs_fail(DBS_ERR_ARG, "dbs_matrix_build_dense: out is NULL");
    *out = nullptr;
    if (m < 0 || n < 0) return dbs_fail(DBS_ERR_ARG, "negative shape");
    if (vt != DBS_F32 && vt != DBS_F16) return dbs_fail(DBS_ERR_ARG, "dense conversion takes DBS_F32 or DBS_F16");
    if (ld < n) return dbs_fail(DBS_ERR_ARG, "ld (%lld) < n (%d)", (long long)ld, n);
    if ((int64_t)m * n > 0 && !d_w) return dbs_fail(DBS_ERR_ARG, "d_w is NULL");
    // record offsets within a block row are 32-bit: n < 2^26
    if (n >= (1 << 26)) return dbs_fail(DBS_ERR_UNSUPPORTED, "n = %d too large for the dense conversion", n);
    dbs_build_opts o;
    dbs_build_opts_default(&o);
    if (opts) o = *opts;
    if (o.th0 < 0 || o.th1 < 0 || !(o.th2 > 0.0f) || o.seg_close < 1 || o.force_type < -1 ||
        o.force_type >= DBS_NUM_BLOCK_TYPES || (o.inline_small != 0 && o.inline_small != 1))
        return dbs_fail(DBS_ERR_ARG, "invalid build options");
    int cnt = 0;
    if (hipGetDeviceCount(&cnt) != hipSuccess || cnt <= 0) return dbs_fail(DBS_ERR_DEVICE, "no HIP device available");
    dbs_matrix *A = new (std::nothrow) dbs_matrix();
    if (!A) return dbs_fail(DBS_ERR_ALLOC, "host allocation failed");
    A->d.dtype = (int32_t)vt;
    const hipStream_t s = (hipStream_t)stream;
    dbs_status st = vt == DBS_F32 ? convert<4>(m, n, d_w, ld, o, s, A) : convert<2>(m, n, d_w, ld, o, s, A);
    if (st != DBS_OK) {
        (void)hipStreamSynchronize(s);
        for (void *p : A->allocs) (void)hipFree(p);
        delete A;
        return st;
    }
    *out = A;
    return DBS_OK;
}
