// gfx950 kernels of the dual-view blocked SpMSpV (DB-SpMSpV).
//
// One call of y = A x runs four kernels on the context's stream:
//   k_scatter / k_ballot  vector blocker (Sec. 3.2.2, 4.1): dense x values and
//                         the 16-bit blk_x_mask of every 16-element vector block
//   k_scan                single-pass look-back scan over vector blocks: the
//                         ascending list of nonzero vector blocks, N_nzblk, the
//                         push task offsets, and the global push/pull choice
//                         s_b = N_nzblk / N_blk < th3 (Sec. 3.3.1)
//   k_main                push (block tasks flattened over the block-CSC lists
//                         of the active column blocks, fetched grid-stride) or
//                         pull (weighted row-block segments), with a per-block
//                         microkernel chosen from the block format and the
//                         vector-block mask (Sec. 3.3.2, 3.3.3, Alg. 2-5) and
//                         hierarchical writeback through LDS (Sec. 3.3.3)
//   k_finalize            look-back compaction of the touched rows into an
//                         ascending sparse y, and reset of the scratch it used
//
// Wave64 mapping (differs from the paper's warp-32 kernels):
//  * a hypersparse COO block is processed by ONE lane (a quarter-wave of 16
//    lanes covers the <= 16 blocks of a pull segment; a full wave covers 64
//    push tasks); blocks of the other formats are processed by the whole wave,
//    one at a time, picked by a ballot.
//  * Dense / ForceCSR / patched-CSR row kernels use 4 lanes per block row
//    (16 rows x 4 = 64 lanes); ForceCSC uses 16 row lanes x 4 column quarters.
//  * fp32 partial sums per row block go through LDS atomics (ds_add_f32), and
//    are committed to an fp64 accumulator per row: a plain store when the
//    block row has one segment, a global fp64 atomic otherwise.
#include <climits>

#include "device_common.hpp"
#include "kernels.hpp"

namespace dbs {

constexpr int TPB = 256;            // threads per workgroup (4 waves)
constexpr int SCAN_ITEMS = 4;       // items per thread in the look-back scans
constexpr int SCAN_TILE = TPB * SCAN_ITEMS;
constexpr int MAX_MAIN_GRID = 2048; // 256 CUs x 8 workgroups

constexpr uint64_t ST_AGG = 1ull << 62, ST_INC = 2ull << 62, ST_PAYLOAD = (1ull << 62) - 1;

// ---------------------------------------------------------------------------
// value access
// ---------------------------------------------------------------------------
template <int MODE> struct VT;
template <> struct VT<M_F32> {
    static constexpr uint32_t VB = 4;
    __device__ static float load(const uint8_t *p, uint32_t i) { return ((const float *)p)[i]; }
    __device__ static float x(const void *xd, int64_t j) { return ((const float *)xd)[j]; }
};
template <> struct VT<M_F16> {
    static constexpr uint32_t VB = 2;
    __device__ static float load(const uint8_t *p, uint32_t i) { return h2f(((const uint16_t *)p)[i]); }
    __device__ static float x(const void *xd, int64_t j) { return h2f(((const uint16_t *)xd)[j]); }
};
template <> struct VT<M_BOOL> {
    static constexpr uint32_t VB = 0;
    __device__ static float load(const uint8_t *, uint32_t) { return 0.f; }
    __device__ static float x(const void *, int64_t) { return 0.f; }
};
template <> struct VT<M_BFS> : VT<M_BOOL> {};

template <int MODE> constexpr bool valued() { return MODE == M_F32 || MODE == M_F16; }

// ---------------------------------------------------------------------------
// decoupled look-back (run by wave 0 of a workgroup)
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint64_t st_load(const uint64_t *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_store(uint64_t *p, uint64_t v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Exclusive prefix (sum of payloads) of all tiles before `tile`.  Every
// predecessor eventually publishes an aggregate or inclusive status, and
// lower tiles are dispatched first, so the wait always ends.
__device__ uint64_t lookback(const uint64_t *status, int tile)
{
    const int lane = lane_id();
    uint64_t excl = 0;
    int pred = tile - 1;
    for (;;) {
        int idx = pred - lane;
        uint64_t s = ST_INC;  // virtual tile before the first: inclusive 0
        if (idx >= 0) {
            do {
                s = st_load(&status[idx]);
            } while ((s >> 62) == 0);
        }
        uint64_t incm = ballot((s >> 62) == 2);
        int first = incm ? ctz64(incm) : WAVE;
        uint64_t v = lane <= first ? (s & ST_PAYLOAD) : 0;
        excl += wave_sum(v);
        if (incm) break;
        pred -= WAVE;
    }
    return excl;
}

// Workgroup exclusive scan of one uint64 per thread; returns the exclusive
// value and writes the workgroup total to *total (all threads).
__device__ uint64_t block_exclusive_scan(uint64_t v, uint64_t *total, uint64_t *lds4)
{
    const int lane = lane_id(), w = threadIdx.x >> 6;
    uint64_t inc = v;
#pragma unroll
    for (int o = 1; o < WAVE; o <<= 1) {
        uint64_t t = __shfl_up(inc, o, WAVE);
        if (lane >= o) inc += t;
    }
    if (lane == WAVE - 1) lds4[w] = inc;
    __syncthreads();
    uint64_t before = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < TPB / WAVE; ++i) {
        uint64_t t = lds4[i];
        if (i < w) before += t;
        tot += t;
    }
    __syncthreads();
    *total = tot;
    return before + inc - v;
}

// ---------------------------------------------------------------------------
// vector blocker
// ---------------------------------------------------------------------------
template <int MODE>
__global__ __launch_bounds__(TPB) void k_scatter(const int32_t *__restrict__ xi,
                                                 const void *__restrict__ xv, int32_t k, int32_t n,
                                                 void *__restrict__ xd, uint32_t *__restrict__ xmask,
                                                 int32_t *__restrict__ counters)
{
    int32_t t = blockIdx.x * TPB + threadIdx.x;
    if (t >= k) return;
    int32_t j = xi[t];
    if (j < 0 || j >= n) {
        atomicOr(&counters[C_ERR], 1);
        return;
    }
    if constexpr (MODE == M_F32) ((float *)xd)[j] = ((const float *)xv)[t];
    if constexpr (MODE == M_F16) ((uint16_t *)xd)[j] = ((const uint16_t *)xv)[t];
    uint32_t J = (uint32_t)j >> 4;
    uint32_t bit = 1u << ((J & 1) * 16 + (j & 15));
    uint32_t old = atomicOr(&xmask[J >> 1], bit);
    if (old & bit) atomicOr(&counters[C_ERR], 2);
}

// Dense activation (Sec. 4.1): each wave reads 64 consecutive entries and
// one 64-bit ballot of "value != 0" gives the masks of 4 vector blocks.  The
// values are copied into the padded dense-x scratch so that the block
// microkernels never read past the caller's n entries.
template <int MODE>
__global__ __launch_bounds__(TPB) void k_ballot(const void *__restrict__ x, int32_t n,
                                                void *__restrict__ xd,
                                                uint32_t *__restrict__ xmask, int32_t nwords)
{
    int64_t j = (int64_t)blockIdx.x * TPB + threadIdx.x;
    bool nz = false;
    if (j < n) {
        if constexpr (MODE == M_F16) {
            uint16_t v = ((const uint16_t *)x)[j];
            ((uint16_t *)xd)[j] = v;
            nz = (v & 0x7FFFu) != 0;
        } else {
            uint32_t v = ((const uint32_t *)x)[j];
            ((uint32_t *)xd)[j] = v;
            nz = (v & 0x7FFFFFFFu) != 0;
        }
    }
    uint64_t b = ballot(nz);
    if (lane_id() == 0) {
        int64_t w = (j - lane_id()) >> 5;
        if (w < nwords) xmask[w] = (uint32_t)b;
        if (w + 1 < nwords) xmask[w + 1] = (uint32_t)(b >> 32);
    }
}

// Active vector blocks, their push task offsets and the path choice.
__global__ __launch_bounds__(TPB) void k_scan(const uint32_t *__restrict__ xmask,
                                              const int32_t *__restrict__ cb_ptr, int32_t nbc,
                                              int32_t *__restrict__ act, int32_t *__restrict__ task_off,
                                              int32_t *__restrict__ counters, uint64_t *status,
                                              uint64_t *next_status, int32_t n_status,
                                              int32_t forced_path, double th3)
{
    __shared__ uint64_t lds4[TPB / WAVE];
    __shared__ uint64_t s_prefix;
    // clear the other copy of the status words for the next scan
    for (int32_t i = blockIdx.x * TPB + threadIdx.x; i < n_status; i += gridDim.x * TPB)
        next_status[i] = 0;
    const int tile = blockIdx.x;
    const int32_t base = tile * SCAN_TILE + threadIdx.x * SCAN_ITEMS;
    uint32_t am[SCAN_ITEMS];
    uint32_t len[SCAN_ITEMS];
    uint64_t mine = 0;
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
        int32_t J = base + k;
        am[k] = J < nbc ? mask16(xmask, J) : 0u;
        len[k] = am[k] ? (uint32_t)(cb_ptr[J + 1] - cb_ptr[J]) : 0u;
        if (am[k]) mine += (1ull << 34) + len[k];
    }
    uint64_t total;
    uint64_t excl = block_exclusive_scan(mine, &total, lds4);
    if (threadIdx.x < WAVE) {
        uint64_t prefix = 0;
        if (tile == 0) {
            if (threadIdx.x == 0) st_store(&status[0], ST_INC | total);
        } else {
            if (threadIdx.x == 0) st_store(&status[tile], ST_AGG | total);
            prefix = lookback(status, tile);
            if (threadIdx.x == 0) st_store(&status[tile], ST_INC | (prefix + total));
        }
        if (threadIdx.x == 0) s_prefix = prefix;
    }
    __syncthreads();
    uint64_t pos = s_prefix + excl;
    int64_t idx = (int64_t)(pos >> 34);
    int64_t off = (int64_t)(pos & ((1ull << 34) - 1));
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
        if (am[k]) {
            act[idx] = base + k;
            task_off[idx] = (int32_t)off;
            ++idx;
            off += len[k];
        }
    }
    if (tile == (int)gridDim.x - 1 && threadIdx.x == 0) {
        uint64_t all = s_prefix + total;
        int32_t N = (int32_t)(all >> 34);
        int32_t T = (int32_t)(all & ((1ull << 34) - 1));
        counters[C_NZBLK] = N;
        counters[C_TASKS] = T;
        task_off[N] = T;
        int path = forced_path;
        if (path == 0) path = ((double)N < th3 * (double)nbc) ? PATH_PUSH : PATH_PULL;
        counters[C_PATH] = path;
    }
}

// ---------------------------------------------------------------------------
// block microkernels
// ---------------------------------------------------------------------------

// One lane, one COO block (packed 4-bit row | 4-bit column coordinates,
// entries in row-major order).  Adds the products of entries whose column is
// active and whose row is admitted into dst16[row] (LDS), merging runs of
// one row first; for BFS records the smallest active column per row (the
// first one met, since columns ascend within a row).  Returns the rows hit.
template <int MODE>
__device__ __forceinline__ uint32_t coo_block(const uint8_t *__restrict__ pay, uint32_t vb, uint64_t d,
                                              int32_t J, uint32_t mx, uint32_t am,
                                              const void *__restrict__ xd, float *dst16,
                                              int32_t *pdst16)
{
    const uint32_t nnz = desc_nnz(d);
    const uint8_t *rec = pay + desc_off(d);
    const uint8_t *crd = rec + vb * nnz;  // coordinates follow the matrix's values
    uint32_t hit = 0;
    int cur = -1;
    float acc = 0.f;
    for (uint32_t e = 0; e < nnz; ++e) {
        uint32_t cd = crd[e];
        uint32_t r = cd >> 4, c = cd & 15u;
        if (!((mx >> c) & (am >> r) & 1u)) continue;
        if constexpr (valued<MODE>()) {
            float prod = VT<MODE>::load(rec, e) * VT<MODE>::x(xd, (int64_t)J * BS + c);
            if ((int)r != cur) {
                if (cur >= 0) atomicAdd(&dst16[cur], acc);
                cur = (int)r;
                acc = prod;
            } else {
                acc += prod;
            }
        }
        if constexpr (MODE == M_BFS) {
            if (!((hit >> r) & 1u)) atomicMin(&pdst16[r], J * BS + (int32_t)c);
        }
        hit |= 1u << r;
    }
    if constexpr (valued<MODE>()) {
        if (cur >= 0) atomicAdd(&dst16[cur], acc);
    }
    return hit;
}

// Same COO block, committing straight to global memory (push path).
template <int MODE>
__device__ __forceinline__ uint32_t coo_block_push(const uint8_t *__restrict__ pay, uint32_t vb,
                                                   uint64_t d, int32_t J, int32_t R, uint32_t mx,
                                                   uint32_t am, const void *__restrict__ xd,
                                                   double *yacc, int32_t *parent)
{
    const uint32_t nnz = desc_nnz(d);
    const uint8_t *rec = pay + desc_off(d);
    const uint8_t *crd = rec + vb * nnz;
    uint32_t hit = 0;
    int cur = -1;
    float acc = 0.f;
    for (uint32_t e = 0; e < nnz; ++e) {
        uint32_t cd = crd[e];
        uint32_t r = cd >> 4, c = cd & 15u;
        if (!((mx >> c) & (am >> r) & 1u)) continue;
        if constexpr (valued<MODE>()) {
            float prod = VT<MODE>::load(rec, e) * VT<MODE>::x(xd, (int64_t)J * BS + c);
            if ((int)r != cur) {
                if (cur >= 0) atomicAdd(&yacc[(int64_t)R * BS + cur], (double)acc);
                cur = (int)r;
                acc = prod;
            } else {
                acc += prod;
            }
        }
        if constexpr (MODE == M_BFS) {
            if (!((hit >> r) & 1u)) atomicMin(&parent[(int64_t)R * BS + r], J * BS + (int32_t)c);
        }
        hit |= 1u << r;
    }
    if constexpr (valued<MODE>()) {
        if (cur >= 0) atomicAdd(&yacc[(int64_t)R * BS + cur], (double)acc);
    }
    return hit;
}

// i-th set bit of v (i >= 0), or -1.
__device__ __forceinline__ int nth_set_bit(uint32_t v, int i)
{
    for (int k = 0; k < i && v; ++k) v &= v - 1;
    return v ? ctz32(v) : -1;
}

// Whole wave, one block of a non-COO format.  Adds the row sums of the
// admitted rows into dst16 (LDS); for BFS records the smallest active
// column per row in pdst16.  Returns the rows hit (uniform).
template <int MODE>
__device__ uint32_t heavy_block(const uint8_t *__restrict__ pay, uint64_t d, int32_t J,
                                uint32_t mx, uint32_t am, const void *__restrict__ xd, float *dst16,
                                int32_t *pdst16)
{
    const int lane = lane_id();
    const uint32_t type = desc_type(d), nnz = desc_nnz(d);
    const uint8_t *rec = pay + desc_off(d);
    const uint16_t *msk = (const uint16_t *)(rec + HDR_MASK);
    const uint8_t *st = rec + HDR_START;
    const int64_t xb = (int64_t)J * BS;

    if constexpr (!valued<MODE>()) {
        // Boolean propagation (Alg. 5): per row lane, the active columns with a
        // stored entry; the first one is the smallest candidate parent.
        const int r = lane & 15;
        uint32_t cand = 0;
        if (lane < 16) {
            if (type == T_FCSC) {
                uint32_t a = mx;
                while (a) {
                    int c = ctz32(a);
                    if ((msk[c] >> r) & 1u) { cand = 1u << c; break; }  // first hit ends the scan
                    a &= a - 1;
                }
            } else {
                cand = msk[r] & mx;
            }
        }
        bool h = lane < 16 && cand != 0 && ((am >> r) & 1u);
        uint32_t hits = (uint32_t)ballot(h) & 0xFFFFu;
        if constexpr (MODE == M_BFS) {
            if (h) atomicMin(&pdst16[r], (int32_t)xb + ctz32(cand));
        }
        return hits;
    } else {
        const uint32_t VB = VT<MODE>::VB;
        if (type == T_DENSE) {
            // Alg. 4 on wave64: 4 lanes per row, 4 consecutive columns each,
            // one coalesced 1 KB (fp32) / 512 B (fp16) read of the block.
            const int r = lane >> 2, c0 = (lane & 3) * 4;
            const uint8_t *vrow = rec + HDR_START + (uint32_t)(r * BS + c0) * VB;
            float s = 0.f;
            if constexpr (MODE == M_F32) {
                float4 v = *(const float4 *)vrow;
                float4 x = *(const float4 *)((const float *)xd + xb + c0);
                if ((mx >> (c0 + 0)) & 1u) s = fmaf(v.x, x.x, s);
                if ((mx >> (c0 + 1)) & 1u) s = fmaf(v.y, x.y, s);
                if ((mx >> (c0 + 2)) & 1u) s = fmaf(v.z, x.z, s);
                if ((mx >> (c0 + 3)) & 1u) s = fmaf(v.w, x.w, s);
            } else {
                uint2 v = *(const uint2 *)vrow;
                uint2 x = *(const uint2 *)((const uint16_t *)xd + xb + c0);
                uint16_t vv[4] = {(uint16_t)v.x, (uint16_t)(v.x >> 16), (uint16_t)v.y, (uint16_t)(v.y >> 16)};
                uint16_t xx[4] = {(uint16_t)x.x, (uint16_t)(x.x >> 16), (uint16_t)x.y, (uint16_t)(x.y >> 16)};
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    if ((mx >> (c0 + k)) & 1u) s = fmaf(h2f(vv[k]), h2f(xx[k]), s);
            }
            s += __shfl_xor(s, 1, WAVE);
            s += __shfl_xor(s, 2, WAVE);
            const int rr = lane & 15;
            float srow = __shfl(s, rr * 4, WAVE);
            bool h = lane < 16 && (msk[rr] & mx) != 0 && ((am >> rr) & 1u);
            uint32_t hits = (uint32_t)ballot(h) & 0xFFFFu;
            if (h) atomicAdd(&dst16[rr], srow);
            return hits;
        }
        const bool rowwise = type == T_FCSR || (type == T_CSR && __popc(mx) >= 8);
        if (rowwise) {
            // Alg. 2 on wave64: 4 lanes per row take every 4th active column.
            const uint8_t *vals = rec + values_at(type, nnz);
            const int r = lane >> 2, sub = lane & 3;
            const uint32_t rm = msk[r];
            uint32_t a = rm & mx;
            const uint32_t start = st[r];
            float s = 0.f;
            int k = 0;
            while (a) {
                int c = ctz32(a);
                if ((k & 3) == sub) {
                    uint32_t p = start + __popc(rm & ((1u << c) - 1u));
                    s = fmaf(VT<MODE>::load(vals, p), VT<MODE>::x(xd, xb + c), s);
                }
                a &= a - 1;
                ++k;
            }
            s += __shfl_xor(s, 1, WAVE);
            s += __shfl_xor(s, 2, WAVE);
            const int rr = lane & 15;
            float srow = __shfl(s, rr * 4, WAVE);
            bool h = lane < 16 && (msk[rr] & mx) != 0 && ((am >> rr) & 1u);
            uint32_t hits = (uint32_t)ballot(h) & 0xFFFFu;
            if (h) atomicAdd(&dst16[rr], srow);
            return hits;
        }
        if (type == T_FCSC) {
            // Alg. 3 on wave64: lane = row, 4 column quarters per wave.
            const uint8_t *vals = rec + HDR_START2;
            const int r = lane & 15, part = lane >> 4;
            uint32_t a = mx & (0xFu << (4 * part));
            float s = 0.f;
            uint32_t found = 0;
            while (a) {
                int c = ctz32(a);
                uint32_t cm = msk[c];
                if ((cm >> r) & 1u) {
                    uint32_t p = st[c] + __popc(cm & ((1u << r) - 1u));
                    s = fmaf(VT<MODE>::load(vals, p), VT<MODE>::x(xd, xb + c), s);
                    found = 1;
                }
                a &= a - 1;
            }
            s += __shfl_xor(s, 16, WAVE);
            s += __shfl_xor(s, 32, WAVE);
            found |= __shfl_xor(found, 16, WAVE);
            found |= __shfl_xor(found, 32, WAVE);
            bool h = lane < 16 && found && ((am >> r) & 1u);
            uint32_t hits = (uint32_t)ballot(h) & 0xFFFFu;
            if (h) atomicAdd(&dst16[r], s);
            return hits;
        }
        // Patched CSR with a sparse vector block: push by columns through
        // col_start and row_idx_csc2csr (row << 4 | rank in row), reading only
        // the entries of the active columns; 4 columns x 16 entries per pass.
        {
            const uint8_t *cs = rec + HDR_START2;
            const uint8_t *rcsc = rec + HDR_RCSC;
            const uint8_t *vals = rec + values_at(type, nnz);
            const int slot = lane >> 4, k = lane & 15;
            uint32_t cols = mx;
            uint32_t hl = 0;
            while (cols) {
                int c = nth_set_bit(cols, slot);
                if (c >= 0) {
                    uint32_t b0 = cs[c], b1 = c == 15 ? nnz : cs[c + 1];
                    if ((uint32_t)k < b1 - b0) {
                        uint32_t rc = rcsc[b0 + k];
                        uint32_t row = rc >> 4, rank = rc & 15u;
                        if ((am >> row) & 1u) {
                            uint32_t p = st[row] + rank;
                            atomicAdd(&dst16[row], VT<MODE>::load(vals, p) * VT<MODE>::x(xd, xb + c));
                            hl |= 1u << row;
                        }
                    }
                }
                for (int q = 0; q < 4 && cols; ++q) cols &= cols - 1;
            }
            hl |= __shfl_xor(hl, 1, WAVE);
            hl |= __shfl_xor(hl, 2, WAVE);
            hl |= __shfl_xor(hl, 4, WAVE);
            hl |= __shfl_xor(hl, 8, WAVE);
            hl |= __shfl_xor(hl, 16, WAVE);
            hl |= __shfl_xor(hl, 32, WAVE);
            return hl;
        }
    }
}

// ---------------------------------------------------------------------------
// main traversal kernel
// ---------------------------------------------------------------------------
struct MainArgs {
    const int32_t *cb_col;
    const uint64_t *desc;
    const uint8_t *pay;
    uint32_t vb;            // value bytes of the matrix (4, 2 or 0)
    const int32_t *cb_ptr;
    const int32_t *csc_row;
    const int32_t *csc2csr;
    const uint64_t *seg;
    int64_t nseg;
    const void *xd;
    const uint32_t *xmask;
    const int32_t *act;
    const int32_t *task_off;
    int32_t *counters;
    const uint32_t *omask;  // output mask bitmap (NULL = none); BFS: visited
    int32_t complement;
    double *yacc;
    uint32_t *ybits;        // y structure; BFS: next-frontier bitmap
    int32_t *parent;        // BFS only
};

template <int MODE>
__device__ __forceinline__ uint32_t row_admit(const MainArgs &a, int32_t R)
{
    return allowed16(a.omask, a.complement, R);
}

// Pull (Sec. 3.3.2): one quarter-wave per row-block segment, 4 segments per
// wave, grid-stride over segments.
template <int MODE>
__device__ void pull_loop(const MainArgs &a, int gw, int nw, float *sy, int32_t *sp)
{
    const int lane = lane_id(), q = lane >> 4, i = lane & 15;
    const int64_t units = (a.nseg + 3) / 4;
    for (int64_t u = gw; u < units; u += nw) {
        const int64_t sid = u * 4 + q;
        const bool vs = sid < a.nseg;
        const uint64_t s = vs ? a.seg[sid] : 0ull;
        const int32_t R = (int32_t)seg_brow(s);
        const uint32_t nb = seg_nb(s);
        const bool single = seg_single(s);
        const uint32_t am = vs ? row_admit<MODE>(a, R) : 0u;
        bool act = vs && (uint32_t)i < nb && am != 0;
        const int32_t b = (int32_t)seg_first(s) + i;
        int32_t J = 0;
        uint32_t mx = 0;
        uint64_t d = 0;
        if (act) {
            J = a.cb_col[b];
            mx = mask16(a.xmask, J);
            act = mx != 0;
        }
        if (act) d = a.desc[b];
        const uint32_t type = desc_type(d);
        uint32_t hit = 0;
        if (act && type == T_COO)
            hit = coo_block<MODE>(a.pay, a.vb, d, J, mx, am, a.xd, sy + q * 16, sp + q * 16);
        uint64_t hv = ballot(act && type != T_COO);
        while (hv) {
            const int L = ctz64(hv);
            hv &= hv - 1;
            const uint64_t dL = readlane_u64(d, L);
            const int32_t JL = (int32_t)readlane_u32((uint32_t)J, L);
            const uint32_t mxL = readlane_u32(mx, L), amL = readlane_u32(am, L);
            const int qL = L >> 4;
            uint32_t h = heavy_block<MODE>(a.pay, dL, JL, mxL, amL, a.xd, sy + qL * 16, sp + qL * 16);
            if (lane == L) hit |= h;
        }
        wave_lds_sync();
        const uint32_t hq = or16_in_quarter(hit);
        if (vs && ((hq >> i) & 1u)) {
            const int64_t row = (int64_t)R * BS + i;
            if constexpr (valued<MODE>()) {
                const float v = sy[lane];
                if (single) a.yacc[row] = (double)v;
                else atomicAdd(&a.yacc[row], (double)v);
            }
            if constexpr (MODE == M_BFS) {
                const int32_t p = sp[lane];
                if (single) a.parent[row] = p;
                else atomicMin(&a.parent[row], p);
            }
        }
        if (vs && i == 0 && hq) or_mask16(a.ybits, R, hq);
        if constexpr (valued<MODE>()) sy[lane] = 0.f;
        if constexpr (MODE == M_BFS) sp[lane] = INT_MAX;
        wave_lds_sync();
    }
}

// Push (Sec. 3.3.2): block tasks flattened over the block-CSC lists of the
// active column blocks, 64 tasks per wave, grid-stride.
template <int MODE>
__device__ void push_loop(const MainArgs &a, int gw, int nw, float *sy, int32_t *sp)
{
    const int lane = lane_id();
    const int32_t T = a.counters[C_TASKS];
    const int32_t N = a.counters[C_NZBLK];
    const int64_t units = ((int64_t)T + WAVE - 1) / WAVE;
    for (int64_t u = gw; u < units; u += nw) {
        const int64_t t = u * WAVE + lane;
        const bool vt = t < T;
        int32_t J = 0, R = 0, b = 0;
        uint32_t mx = 0, am = 0;
        uint64_t d = 0;
        if (vt) {
            // largest a with task_off[a] <= t
            int32_t lo = 0, hi = N - 1;
            while (lo < hi) {
                int32_t mid = (lo + hi + 1) >> 1;
                if (a.task_off[mid] <= t) lo = mid;
                else hi = mid - 1;
            }
            J = a.act[lo];
            const int32_t p = a.cb_ptr[J] + (int32_t)(t - a.task_off[lo]);
            R = a.csc_row[p];
            b = a.csc2csr[p];
            mx = mask16(a.xmask, J);
            am = row_admit<MODE>(a, R);
        }
        const bool act = vt && am != 0;
        if (act) d = a.desc[b];
        const uint32_t type = desc_type(d);
        uint32_t hit = 0;
        if (act && type == T_COO)
            hit = coo_block_push<MODE>(a.pay, a.vb, d, J, R, mx, am, a.xd, a.yacc, a.parent);
        uint64_t hv = ballot(act && type != T_COO);
        while (hv) {
            const int L = ctz64(hv);
            hv &= hv - 1;
            const uint64_t dL = readlane_u64(d, L);
            const int32_t JL = (int32_t)readlane_u32((uint32_t)J, L);
            const int32_t RL = (int32_t)readlane_u32((uint32_t)R, L);
            const uint32_t mxL = readlane_u32(mx, L), amL = readlane_u32(am, L);
            uint32_t h = heavy_block<MODE>(a.pay, dL, JL, mxL, amL, a.xd, sy, sp);
            wave_lds_sync();
            if (lane < 16) {
                const int64_t row = (int64_t)RL * BS + lane;
                if ((h >> lane) & 1u) {
                    if constexpr (valued<MODE>()) atomicAdd(&a.yacc[row], (double)sy[lane]);
                    if constexpr (MODE == M_BFS) atomicMin(&a.parent[row], sp[lane]);
                }
                if constexpr (valued<MODE>()) sy[lane] = 0.f;
                if constexpr (MODE == M_BFS) sp[lane] = INT_MAX;
            }
            wave_lds_sync();
            if (lane == L) hit |= h;
        }
        if (act && hit) or_mask16(a.ybits, R, hit);
    }
}

template <int MODE>
__global__ __launch_bounds__(TPB) void k_main(MainArgs a)
{
    __shared__ float s_y[TPB / WAVE][WAVE];
    __shared__ int32_t s_p[TPB / WAVE][WAVE];
    if (MODE == M_BFS && blockIdx.x == 0 && threadIdx.x == 0) a.counters[C_FRONTIER] = 0;
    if (a.counters[C_NZBLK] == 0) return;
    const int w = threadIdx.x >> 6, lane = lane_id();
    float *sy = s_y[w];
    int32_t *sp = s_p[w];
    sy[lane] = 0.f;
    sp[lane] = INT_MAX;
    wave_lds_sync();
    const int gw = blockIdx.x * (TPB / WAVE) + w, nw = gridDim.x * (TPB / WAVE);
    if (a.counters[C_PATH] == PATH_PUSH) push_loop<MODE>(a, gw, nw, sy, sp);
    else pull_loop<MODE>(a, gw, nw, sy, sp);
}

// ---------------------------------------------------------------------------
// finalize: ascending sparse y from the row-block structure masks
// ---------------------------------------------------------------------------
// A tile is 256 structure words (8192 rows).  Thread t first owns word t
// (its popcount enters the tile scan and the look-back); the rows are then
// written in 32 rounds where thread t handles row t + 256 r of the tile, so
// consecutive lanes touch consecutive accumulators and output slots.
constexpr int FIN_WORDS = TPB;

template <int MODE>
__global__ __launch_bounds__(TPB) void k_finalize(uint32_t *__restrict__ ybits, int32_t nywords,
                                                  double *__restrict__ yacc, int32_t m,
                                                  int32_t *__restrict__ y_idx, void *__restrict__ y_val,
                                                  int32_t *__restrict__ y_nnz,
                                                  int32_t *__restrict__ counters, uint64_t *status,
                                                  uint64_t *next_status, int32_t n_status,
                                                  uint32_t *__restrict__ xmask,
                                                  const int32_t *__restrict__ act)
{
    __shared__ uint64_t lds4[TPB / WAVE];
    __shared__ uint64_t s_prefix;
    __shared__ uint32_t s_word[FIN_WORDS];
    __shared__ uint32_t s_wpos[FIN_WORDS];
    for (int32_t i = blockIdx.x * TPB + threadIdx.x; i < n_status; i += gridDim.x * TPB)
        next_status[i] = 0;
    // clear blk_x_mask of this call's active vector blocks
    const int32_t N = counters[C_NZBLK];
    for (int32_t i = blockIdx.x * TPB + threadIdx.x; i < N; i += gridDim.x * TPB)
        xmask[act[i] >> 1] = 0u;
    const int tile = blockIdx.x;
    const int32_t w = tile * FIN_WORDS + threadIdx.x;
    const uint32_t word = w < nywords ? ybits[w] : 0u;
    uint64_t total;
    const uint64_t excl = block_exclusive_scan((uint64_t)__popc(word), &total, lds4);
    s_word[threadIdx.x] = word;
    s_wpos[threadIdx.x] = (uint32_t)excl;
    if (threadIdx.x < WAVE) {
        uint64_t prefix = 0;
        if (tile == 0) {
            if (threadIdx.x == 0) st_store(&status[0], ST_INC | total);
        } else {
            if (threadIdx.x == 0) st_store(&status[tile], ST_AGG | total);
            prefix = lookback(status, tile);
            if (threadIdx.x == 0) st_store(&status[tile], ST_INC | (prefix + total));
        }
        if (threadIdx.x == 0) s_prefix = prefix;
    }
    __syncthreads();
    if (word) ybits[w] = 0u;
    const int64_t base_pos = (int64_t)s_prefix;
    const int64_t row0 = (int64_t)tile * FIN_WORDS * 32;
#pragma unroll 4
    for (int r = 0; r < 32; ++r) {
        const int lr = r * TPB + threadIdx.x;  // row within the tile
        const uint32_t wd = s_word[lr >> 5];
        const uint32_t bit = lr & 31;
        if (!((wd >> bit) & 1u)) continue;
        const int64_t pos = base_pos + s_wpos[lr >> 5] + __popc(wd & ((1u << bit) - 1u));
        const int64_t i = row0 + lr;
        y_idx[pos] = (int32_t)i;
        if constexpr (MODE == M_F32) {
            ((float *)y_val)[pos] = (float)yacc[i];
            yacc[i] = 0.0;
        }
        if constexpr (MODE == M_F16) {
            ((uint16_t *)y_val)[pos] = f64_to_f16_rne(yacc[i]);
            yacc[i] = 0.0;
        }
    }
    if (tile == (int)gridDim.x - 1 && threadIdx.x == 0) {
        int32_t tot = (int32_t)(s_prefix + total);
        *y_nnz = tot;
        counters[C_YNNZ] = tot;
        counters[C_ERR_LAST] = counters[C_ERR];
        counters[C_ERR] = 0;
    }
    (void)m;
}

// Dense output (decoding): every row, converted from the fp64 accumulator.
template <int MODE>
__global__ __launch_bounds__(TPB) void k_finalize_dense(double *__restrict__ yacc, int32_t m,
                                                        void *__restrict__ y, float *__restrict__ y32,
                                                        uint32_t *__restrict__ ybits, int32_t nywords,
                                                        uint32_t *__restrict__ xmask, int32_t nxwords,
                                                        int32_t *__restrict__ counters)
{
    const int64_t stride = (int64_t)gridDim.x * TPB;
    for (int64_t i = (int64_t)blockIdx.x * TPB + threadIdx.x; i < m; i += stride) {
        double v = yacc[i];
        if constexpr (MODE == M_F32) ((float *)y)[i] = (float)v;
        else ((uint16_t *)y)[i] = f64_to_f16_rne(v);
        if (y32) y32[i] = (float)v;
        yacc[i] = 0.0;
    }
    for (int64_t i = (int64_t)blockIdx.x * TPB + threadIdx.x; i < nywords; i += stride) ybits[i] = 0u;
    for (int64_t i = (int64_t)blockIdx.x * TPB + threadIdx.x; i < nxwords; i += stride) xmask[i] = 0u;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        counters[C_YNNZ] = m;
        counters[C_ERR_LAST] = counters[C_ERR];
        counters[C_ERR] = 0;
    }
}

// ---------------------------------------------------------------------------
// BFS (Sec. 4.2)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(TPB) void k_bfs_init(int32_t n, int32_t source, int32_t *__restrict__ level,
                                                  int32_t *__restrict__ parent,
                                                  uint32_t *__restrict__ visited,
                                                  uint32_t *__restrict__ nextm,
                                                  uint32_t *__restrict__ xmask, int32_t nwords)
{
    const int64_t stride = (int64_t)gridDim.x * TPB;
    for (int64_t v = (int64_t)blockIdx.x * TPB + threadIdx.x; v < n; v += stride) {
        level[v] = v == source ? 0 : -1;
        parent[v] = v == source ? source : INT_MAX;
    }
    const int32_t sw = source >> 5;
    const uint32_t sb = 1u << (source & 31);
    for (int64_t w = (int64_t)blockIdx.x * TPB + threadIdx.x; w < nwords; w += stride) {
        visited[w] = w == sw ? sb : 0u;
        xmask[w] = w == sw ? sb : 0u;
        nextm[w] = 0u;
    }
}

// Next frontier -> current frontier masks, visited |= next, level of the
// newly reached vertices, frontier size.
__global__ __launch_bounds__(TPB) void k_bfs_update(int32_t nwords, int32_t next_level,
                                                    int32_t *__restrict__ level,
                                                    uint32_t *__restrict__ visited,
                                                    uint32_t *__restrict__ nextm,
                                                    uint32_t *__restrict__ xmask,
                                                    int32_t *__restrict__ counters)
{
    int32_t w = blockIdx.x * TPB + threadIdx.x;
    uint32_t cnt = 0;
    if (w < nwords) {
        uint32_t nm = nextm[w];
        xmask[w] = nm;
        if (nm) {
            visited[w] |= nm;
            nextm[w] = 0u;
            cnt = __popc(nm);
            while (nm) {
                int b = ctz32(nm);
                nm &= nm - 1;
                level[(int64_t)w * 32 + b] = next_level;
            }
        }
    }
    uint32_t tot = wave_sum(cnt);
    if (lane_id() == 0 && tot) atomicAdd(&counters[C_FRONTIER], (int32_t)tot);
}

__global__ __launch_bounds__(TPB) void k_bfs_finish(int32_t n, int32_t *__restrict__ parent)
{
    const int64_t stride = (int64_t)gridDim.x * TPB;
    for (int64_t v = (int64_t)blockIdx.x * TPB + threadIdx.x; v < n; v += stride)
        if (parent[v] == INT_MAX) parent[v] = -1;
}

// ---------------------------------------------------------------------------
// host launch wrappers
// ---------------------------------------------------------------------------
static inline int grid_for(int64_t items, int per_block, int cap)
{
    int64_t g = (items + per_block - 1) / per_block;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (int)g;
}

int main_grid(const DevMatrix &A)
{
    int64_t pull_waves = (A.nseg + 3) / 4;
    int64_t push_waves = (A.nblk + WAVE - 1) / WAVE;
    int64_t waves = pull_waves > push_waves ? pull_waves : push_waves;
    return grid_for(waves, TPB / WAVE, MAX_MAIN_GRID);
}

hipError_t launch_scatter(const DevMatrix &A, const DevCtx &C, int mode, int32_t k,
                          const int32_t *x_idx, const void *x_val, hipStream_t s)
{
    if (k <= 0) return hipSuccess;
    dim3 g(grid_for(k, TPB, INT_MAX)), b(TPB);
    switch (mode) {
    case M_F32: hipLaunchKernelGGL(k_scatter<M_F32>, g, b, 0, s, x_idx, x_val, k, A.n, C.xd, C.xmask, C.counters); break;
    case M_F16: hipLaunchKernelGGL(k_scatter<M_F16>, g, b, 0, s, x_idx, x_val, k, A.n, C.xd, C.xmask, C.counters); break;
    default: hipLaunchKernelGGL(k_scatter<M_BOOL>, g, b, 0, s, x_idx, x_val, k, A.n, C.xd, C.xmask, C.counters); break;
    }
    return hipGetLastError();
}

hipError_t launch_ballot(const DevMatrix &A, const DevCtx &C, int mode, const void *x_dense,
                         hipStream_t s)
{
    int64_t lanes = ((int64_t)A.n + WAVE - 1) / WAVE * WAVE;
    dim3 g(grid_for(lanes, TPB, INT_MAX)), b(TPB);
    if (mode == M_F16) hipLaunchKernelGGL(k_ballot<M_F16>, g, b, 0, s, x_dense, A.n, C.xd, C.xmask, C.nxwords);
    else hipLaunchKernelGGL(k_ballot<M_F32>, g, b, 0, s, x_dense, A.n, C.xd, C.xmask, C.nxwords);
    return hipGetLastError();
}

hipError_t launch_scan(const DevMatrix &A, DevCtx &C, int forced_path, double th3, hipStream_t s)
{
    dim3 g(grid_for(A.nbc, SCAN_TILE, INT_MAX)), b(TPB);
    const int p = C.scan_parity;
    hipLaunchKernelGGL(k_scan, g, b, 0, s, C.xmask, A.cb_ptr, A.nbc, C.act, C.task_off, C.counters,
                       C.st_scan[p], C.st_scan[1 - p], C.n_st_scan, forced_path, th3);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) C.scan_parity = 1 - p;
    return e;
}

hipError_t launch_main(const DevMatrix &A, const DevCtx &C, int mode, const void *xd,
                       const uint32_t *omask, int complement, int32_t *parent, hipStream_t s)
{
    MainArgs a;
    a.cb_col = A.cb_col;
    a.desc = A.desc;
    a.pay = A.pay;
    a.vb = A.dtype == 0 ? 4u : (A.dtype == 1 ? 2u : 0u);
    a.cb_ptr = A.cb_ptr;
    a.csc_row = A.csc_row;
    a.csc2csr = A.csc2csr;
    a.seg = A.seg;
    a.nseg = A.nseg;
    a.xd = xd;
    a.xmask = C.xmask;
    a.act = C.act;
    a.task_off = C.task_off;
    a.counters = C.counters;
    a.omask = omask;
    a.complement = complement;
    a.yacc = C.yacc;
    a.ybits = mode == M_BFS ? C.nextm : C.ybits;
    a.parent = parent;
    dim3 g(main_grid(A)), b(TPB);
    switch (mode) {
    case M_F32: hipLaunchKernelGGL(k_main<M_F32>, g, b, 0, s, a); break;
    case M_F16: hipLaunchKernelGGL(k_main<M_F16>, g, b, 0, s, a); break;
    case M_BOOL: hipLaunchKernelGGL(k_main<M_BOOL>, g, b, 0, s, a); break;
    default: hipLaunchKernelGGL(k_main<M_BFS>, g, b, 0, s, a); break;
    }
    return hipGetLastError();
}

hipError_t launch_finalize(const DevMatrix &A, DevCtx &C, int mode, int32_t *y_idx, void *y_val,
                           int32_t *y_nnz, hipStream_t s)
{
    int32_t nyw = (A.nbr + 1) / 2;
    dim3 g(grid_for(nyw, FIN_WORDS, INT_MAX)), b(TPB);
    const int p = C.fin_parity;
    uint64_t *st = C.st_fin[p], *nx = C.st_fin[1 - p];
    const int32_t ns = C.n_st_fin;
    switch (mode) {
    case M_F32: hipLaunchKernelGGL(k_finalize<M_F32>, g, b, 0, s, C.ybits, nyw, C.yacc, A.m, y_idx, y_val, y_nnz, C.counters, st, nx, ns, C.xmask, C.act); break;
    case M_F16: hipLaunchKernelGGL(k_finalize<M_F16>, g, b, 0, s, C.ybits, nyw, C.yacc, A.m, y_idx, y_val, y_nnz, C.counters, st, nx, ns, C.xmask, C.act); break;
    default: hipLaunchKernelGGL(k_finalize<M_BOOL>, g, b, 0, s, C.ybits, nyw, C.yacc, A.m, y_idx, y_val, y_nnz, C.counters, st, nx, ns, C.xmask, C.act); break;
    }
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) C.fin_parity = 1 - p;
    return e;
}

hipError_t launch_finalize_dense(const DevMatrix &A, const DevCtx &C, int mode, void *y, float *y32,
                                 hipStream_t s)
{
    int32_t nyw = (A.nbr + 1) / 2;
    int64_t items = A.m > C.nxwords ? A.m : C.nxwords;
    dim3 g(grid_for(items, TPB, 4096)), b(TPB);
    if (mode == M_F16)
        hipLaunchKernelGGL(k_finalize_dense<M_F16>, g, b, 0, s, C.yacc, A.m, y, y32, C.ybits, nyw, C.xmask, C.nxwords, C.counters);
    else
        hipLaunchKernelGGL(k_finalize_dense<M_F32>, g, b, 0, s, C.yacc, A.m, y, y32, C.ybits, nyw, C.xmask, C.nxwords, C.counters);
    return hipGetLastError();
}

hipError_t launch_bfs_init(const DevMatrix &A, const DevCtx &C, int32_t source, int32_t *level,
                           int32_t *parent, hipStream_t s)
{
    int32_t nwords = (A.nbr + 1) / 2;
    dim3 g(grid_for(A.n, TPB, 4096)), b(TPB);
    hipLaunchKernelGGL(k_bfs_init, g, b, 0, s, A.n, source, level, parent, C.visited, C.nextm, C.xmask, nwords);
    return hipGetLastError();
}

hipError_t launch_bfs_update(const DevMatrix &A, const DevCtx &C, int32_t next_level, int32_t *level,
                             hipStream_t s)
{
    int32_t nwords = (A.nbr + 1) / 2;
    dim3 g(grid_for(nwords, TPB, INT_MAX)), b(TPB);
    hipLaunchKernelGGL(k_bfs_update, g, b, 0, s, nwords, next_level, level, C.visited, C.nextm, C.xmask,
                       C.counters);
    return hipGetLastError();
}

hipError_t launch_bfs_finish(const DevMatrix &A, int32_t *parent, hipStream_t s)
{
    dim3 g(grid_for(A.n, TPB, 4096)), b(TPB);
    hipLaunchKernelGGL(k_bfs_finish, g, b, 0, s, A.n, parent);
    return hipGetLastError();
}

}  // namespace dbs
