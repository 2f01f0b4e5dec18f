// gfx950 kernels of the dual-view blocked SpMSpV (DB-SpMSpV).
//
// One call of y = A x runs these kernels on the context's stream:
//   k_scatter / k_ballot  vector blocker (Sec. 3.2.2, 4.1): dense x values and
//                         the 16-bit blk_x_mask of every 16-element vector block
//   k_scan                single-pass look-back scan over vector blocks: the
//                         list of nonzero vector blocks, N_nzblk, the push
//                         task offsets, and the global push/pull choice
//                         s_b = N_nzblk / N_blk < th3 (Sec. 3.3.1; BFS levels:
//                         the push task count against a share of the blocks)
//   (k_small_x            both of the above in one workgroup, for short index
//                         lists)
//   k_traverse            pull (weighted row-block segments, or below an
//                         activity threshold a compaction of the segments'
//                         active slots), then push (block tasks flattened over
//                         the block-CSC lists of the active column blocks,
//                         fetched grid-stride; or the walk of the compacted
//                         slots), with a per-block microkernel chosen from the
//                         block format and the vector-block mask (Sec. 3.3.2,
//                         3.3.3, Alg. 2-5) and hierarchical writeback through
//                         LDS (Sec. 3.3.3); the kernel the device choice does
//                         not need returns at once
//   k_finalize            look-back compaction of the touched rows into an
//                         ascending sparse y, and reset of the scratch it used
//
// Wave64 mapping (differs from the paper's warp-32 kernels):
//  * pull: a quarter-wave (16 lanes) per segment, one block per lane, four
//    segments per lane in flight; blocks whose vector block is empty are
//    dropped by an activity bitmap in LDS before anything is gathered.
//  * a COO block whose entries sit in its descriptor is taken by one lane
//    (one x gather, which also tells whether x_j is stored); COO blocks with
//    a record are taken entry-parallel by the whole wave (flat_pass), as are
//    all record blocks in push.  Pull takes the other formats from an
//    upload-time list ahead of the segment loop, in chunks of up to 16
//    blocks of one block row, with one lane per row (pull_rows).
//  * fp32 partial sums per row block go through LDS atomics (ds_add_f32), and
//    are committed to an fp64 accumulator per row with a global fp64 atomic,
//    once per run of segments of one block row that a quarter-wave takes.
//  * wave scans and row reductions use DPP row shifts and broadcasts.
#include <algorithm>
#include <climits>

#include "device_common.hpp"
#include "kernels.hpp"

namespace dbs {

constexpr int TPB = 256;            // threads per workgroup (4 waves)
constexpr int SCAN_ITEMS = SCAN_ITEMS_PER_THREAD;  // vector blocks per thread in the scan
#ifndef SCAN_TPB
#define SCAN_TPB 256
#endif
constexpr int STPB = SCAN_TPB;                  // threads per scan workgroup
constexpr int SCAN_TILE = STPB * SCAN_ITEMS;
static_assert(SCAN_ITEMS == 1 || SCAN_ITEMS == 2 || SCAN_ITEMS == 4, "scan items");
constexpr int MAX_MAIN_GRID = 4096; // upper bound: 256 CUs x 16 workgroups

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
template <int NTH = TPB>
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
    for (int i = 0; i < NTH / WAVE; ++i) {
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
// Sparse x: scatter the values into the dense scratch and set the mask bits
// (Sec. 3.2.2).  Out-of-range indices are counted and skipped.  N_nzblk
// (Sec. 3.3.1) and the number of distinct indices (which exposes duplicates)
// are counted afterwards by the scan from the masks.
template <int MODE>
__global__ __launch_bounds__(TPB) void k_scatter(const int32_t *__restrict__ xi,
                                                 const void *__restrict__ xv, int32_t k, int32_t n,
                                                 void *__restrict__ xd, uint32_t *__restrict__ xmask,
                                                 int32_t *__restrict__ counters)
{
    const int32_t t = blockIdx.x * TPB + threadIdx.x;
    const int lane = lane_id();
    bool bad = false;
    int32_t w = -1;     // mask word of the entry (-1: none)
    uint32_t bits = 0;  // its bit in that word
    if (t < k) {
        const int32_t j = xi[t];
        if (j < 0 || j >= n) {
            bad = true;
        } else {
            // an input equal to the absent-entry marker becomes the canonical NaN
            if constexpr (MODE == M_F32) {
                const uint32_t v = ((const uint32_t *)xv)[t];
                ((uint32_t *)xd)[j] = v == 0xFFFFFFFFu ? 0x7FC00000u : v;
            }
            if constexpr (MODE == M_F16) {
                const uint16_t v = ((const uint16_t *)xv)[t];
                ((uint16_t *)xd)[j] = v == 0xFFFFu ? (uint16_t)0x7E00u : v;
            }
            w = j >> 5;
            bits = 1u << (j & 31);
        }
    }
    // Segmented OR over runs of lanes with the same mask word (sorted or
    // clustered indices form long runs), then one non-returning atomic per
    // run.  Duplicates and the nonzero vector blocks are counted by the scan.
#pragma unroll
    for (int o = 1; o < WAVE; o <<= 1) {
        const uint32_t vb = (uint32_t)__shfl_up((int)bits, o, WAVE);
        const int32_t vw = __shfl_up(w, o, WAVE);
        if (lane >= o && vw == w) bits |= vb;
    }
    const int32_t nextw = __shfl_down(w, 1, WAVE);
    if (w >= 0 && (lane == WAVE - 1 || nextw != w)) atomicOr(&xmask[w], bits);
    const uint64_t bm = ballot(bad);
    if (lane == 0 && bm) atomicAdd(&counters[C_XBAD], (int32_t)__popcll(bm));
}

// Dense activation (Sec. 4.1): each wave reads 64 consecutive entries and
// one 64-bit ballot of "value != 0" gives the masks of 4 vector blocks.  The
// values are copied into the padded dense-x scratch so that the block
// microkernels never read past the caller's n entries.
template <int MODE>
__global__ __launch_bounds__(TPB) void k_ballot(const void *__restrict__ x, int32_t n,
                                                void *__restrict__ xd,
                                                uint32_t *__restrict__ xmask, int32_t nwords,
                                                int32_t *__restrict__ counters)
{
    int64_t j = (int64_t)blockIdx.x * TPB + threadIdx.x;
    bool nz = false;
    if (j < n) {
        // zero entries are not stored: they keep the absent-entry marker
        if constexpr (MODE == M_F16) {
            uint16_t v = ((const uint16_t *)x)[j];
            nz = (v & 0x7FFFu) != 0;
            ((uint16_t *)xd)[j] = !nz ? (uint16_t)0xFFFFu : v == 0xFFFFu ? (uint16_t)0x7E00u : v;
        } else {
            uint32_t v = ((const uint32_t *)x)[j];
            nz = (v & 0x7FFFFFFFu) != 0;
            ((uint32_t *)xd)[j] = !nz ? 0xFFFFFFFFu : v == 0xFFFFFFFFu ? 0x7FC00000u : v;
        }
    }
    uint64_t b = ballot(nz);
    if (lane_id() == 0) {
        int64_t w = (j - lane_id()) >> 5;
        if (w < nwords) xmask[w] = (uint32_t)b;
        if (w + 1 < nwords) xmask[w + 1] = (uint32_t)(b >> 32);
        (void)counters;
    }
}

// Single-pass scan over vector blocks.  Every nonzero vector block J whose
// block column holds matrix blocks becomes one push work item
//   items[a] = {first task, J, pbase = cb_ptr[J] - first task, 0}
// so that task t of item a visits block-CSC position pbase + t.  The last
// tile fixes N_nzblk (counted by the blocker), the task totals and the
// global path: push iff N_nzblk < th3 N_blk (Sec. 3.3.1), or, with th3s > 0,
// also when x is spread (fewer than two indices per nonzero vector block)
// and N_nzblk < th3s N_blk; with tasks_max >= 0 (BFS levels) instead push iff
// the push tasks (blocks in the block-CSC lists of the nonzero vector
// blocks) number fewer than tasks_max.
// DX (dense activation, MODE fp32 or fp16, n a multiple of 16, x 16-byte
// aligned): the blocker is folded into the scan's front end -- each thread
// reads the x of its vector blocks, writes their densified copy and masks.
template <bool DX, int MODE>
__global__ __launch_bounds__(STPB) void k_scan(uint32_t *__restrict__ xmask, const void *__restrict__ xdense,
                                              void *__restrict__ xd,
                                              const int32_t *__restrict__ cb_ptr, int32_t nbc,
                                              int4 *__restrict__ items,
                                              uint32_t *__restrict__ xbits,
                                              int32_t *__restrict__ counters, uint64_t *status,
                                              uint64_t *next_status, int32_t n_status,
                                              int32_t forced_path, double th3, double th3s, double tasks_max)
{
    __shared__ uint64_t lds4[STPB / WAVE];
    __shared__ uint64_t s_cnt[STPB / WAVE];
    __shared__ uint64_t s_prefix;
    // clear the other copy of the status words for the next scan
    for (int32_t i = blockIdx.x * STPB + threadIdx.x; i < n_status; i += gridDim.x * STPB)
        next_status[i] = 0;
    const int tile = blockIdx.x;
    const int32_t base = tile * SCAN_TILE + threadIdx.x * SCAN_ITEMS;
    int32_t start[SCAN_ITEMS];
    uint32_t len[SCAN_ITEMS];
    uint64_t mine = 0;
    uint32_t nib = 0;  // activity of this thread's 4 vector blocks
    uint32_t pop = 0;  // stored x entries in them
    uint32_t amk[SCAN_ITEMS];
    // the block-column pointers of all the thread's vector blocks, active or
    // not, go out with the masks (a dependent load would add a round trip)
    int32_t cbv[SCAN_ITEMS + 1];
#pragma unroll
    for (int k = 0; k <= SCAN_ITEMS; ++k) cbv[k] = base + k <= nbc ? cb_ptr[base + k] : 0;
    if constexpr (DX) {
        // 16 entries per vector block: the marker for zeros, the canonical
        // NaN for an entry equal to the marker
        constexpr int PER = MODE == M_F16 ? 8 : 4;  // entries per 16 bytes
#pragma unroll
        for (int k = 0; k < SCAN_ITEMS; ++k) {
            const int32_t J = base + k;
            uint32_t msk = 0;
            if (J < nbc) {
                const uint4 *src = (const uint4 *)xdense + (int64_t)J * (16 / PER);
                uint4 *dst = (uint4 *)xd + (int64_t)J * (16 / PER);
#pragma unroll
                for (int q = 0; q < 16 / PER; ++q) {
                    const uint4 v = src[q];
                    uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        if constexpr (MODE == M_F16) {
#pragma unroll
                            for (int h = 0; h < 2; ++h) {
                                const uint32_t hv = (w[e] >> (16 * h)) & 0xFFFFu;
                                const bool nz = (hv & 0x7FFFu) != 0;
                                const uint32_t o = !nz ? 0xFFFFu : hv == 0xFFFFu ? 0x7E00u : hv;
                                w[e] = (w[e] & ~(0xFFFFu << (16 * h))) | (o << (16 * h));
                                msk |= (nz ? 1u : 0u) << (q * 8 + e * 2 + h);
                            }
                        } else {
                            const bool nz = (w[e] & 0x7FFFFFFFu) != 0;
                            msk |= (nz ? 1u : 0u) << (q * 4 + e);
                            w[e] = !nz ? 0xFFFFFFFFu : w[e] == 0xFFFFFFFFu ? 0x7FC00000u : w[e];
                        }
                    }
                    dst[q] = make_uint4(w[0], w[1], w[2], w[3]);
                }
            }
            amk[k] = msk;
        }
        // the masks of two consecutive vector blocks share a word
#pragma unroll
        for (int k = 0; k < SCAN_ITEMS; k += 2)
            if (base + k < nbc) xmask[(base + k) >> 1] = amk[k] | (base + k + 1 < nbc ? amk[k + 1] << 16 : 0u);
    } else {
#pragma unroll
        for (int k = 0; k < SCAN_ITEMS; ++k) {
            const int32_t J = base + k;
            amk[k] = J < nbc ? mask16(xmask, J) : 0u;
        }
    }
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
        const uint32_t am = amk[k];
        nib |= (am ? 1u : 0u) << k;
        pop += __popc(am);
        start[k] = am ? cbv[k] : 0;
        len[k] = am ? (uint32_t)(cbv[k + 1] - cbv[k]) : 0u;
        if (len[k]) mine += (1ull << 34) + len[k];
    }
    // one activity bit per vector block: 32 / SCAN_ITEMS threads form a word
    {
        constexpr int LPW = 32 / SCAN_ITEMS;
        uint32_t word = nib << (SCAN_ITEMS * (lane_id() & (LPW - 1)));
#pragma unroll
        for (int o = 1; o < LPW; o <<= 1) word |= __shfl_xor(word, o, WAVE);
        const int32_t wi = base >> 5;
        if ((lane_id() & (LPW - 1)) == 0 && base < nbc) xbits[wi] = word;
    }
    // nonzero vector blocks and stored x entries of the tile (low / high
    // 32 bits), reduced alongside the scan
    uint64_t cnt2 = wave_sum(((uint64_t)pop << 32) | (uint64_t)__popc(nib));
    if (lane_id() == 0) s_cnt[threadIdx.x >> 6] = cnt2;
    uint64_t total;
    uint64_t excl = block_exclusive_scan<STPB>(mine, &total, lds4);
    // the tile's counts (thread 0; a single tile keeps them for itself)
    uint64_t c = 0;
    if (threadIdx.x < WAVE) {
        uint64_t prefix = 0;
        if (threadIdx.x == 0) {
#pragma unroll
            for (int i = 0; i < STPB / WAVE; ++i) c += s_cnt[i];
            // counted before the tile's status is published: a tile that
            // has seen every earlier status (directly or through an
            // inclusive one) also sees their counts
            if (gridDim.x > 1) {
                if ((uint32_t)c) atomicAdd(&counters[C_NZACC], (int32_t)(uint32_t)c);
                if (c >> 32) atomicAdd(&counters[C_XPOP], (int32_t)(c >> 32));
                __threadfence();
            }
        }
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
    const uint64_t pos = s_prefix + excl;
    int64_t idx = (int64_t)(pos >> 34);
    int64_t off = (int64_t)(pos & ((1ull << 34) - 1));
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
        if (len[k]) {
            items[idx] = make_int4((int32_t)off, base + k, start[k] - (int32_t)off, 0);
            ++idx;
            off += len[k];
        }
    }
    if (tile == (int)gridDim.x - 1 && threadIdx.x == 0) {
        const uint64_t all = s_prefix + total;
        const int32_t NT = (int32_t)(all >> 34);
        const int32_t T = (int32_t)(all & ((1ull << 34) - 1));
        int32_t N, pop;
        if (gridDim.x > 1) {
            __threadfence();
            N = __hip_atomic_load(&counters[C_NZACC], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            counters[C_NZACC] = 0;
            pop = __hip_atomic_load(&counters[C_XPOP], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else {
            // one tile: no other counts to wait for (the distinct-index total
            // still goes to the counter, where the compaction reads it)
            N = (int32_t)(uint32_t)c;
            pop = (int32_t)(c >> 32);
            counters[C_XPOP] = pop;
        }
        counters[C_NZBLK] = N;
        counters[C_NTB] = NT;
        counters[C_TASKS] = T;
        items[NT] = make_int4(T, 0, 0, 0);
        int path = forced_path;
        if (path == 0 && tasks_max >= 0.0) {
            path = (double)T < tasks_max ? PATH_PUSH : PATH_PULL;
        } else if (path == 0) {
            const bool spread = th3s > 0.0 && (int64_t)pop < 2 * (int64_t)N && (double)N < th3s * (double)nbc;
            path = ((double)N < th3 * (double)nbc || spread) ? PATH_PUSH : PATH_PULL;
        }
        counters[C_PATH] = path;
    }
}

// Blocker and scan in one workgroup for a short index list (k <= SMALL_X_MAX
// and an activity bitmap of at most SMALL_X_WORDS words), in place of
// k_scatter + k_scan, whose grid walks every vector block and whose tiles
// wait on each other's look-back status.  Each thread takes up to two
// indices: the value goes into the dense scratch and the index's mask bit is
// set with a returning atomic, whose old word tells whether the index was
// already stored (the distinct indices are counted from that).  The vector
// blocks are deduplicated in an LDS hash table (after runs of equal blocks
// in consecutive lanes); each first occurrence loads
// its block-column extent, sets its bit in an LDS copy of the activity
// bitmap, and becomes a push work item (in hash-arrival order, not ascending
// J: push needs only increasing first tasks).  The counters, the path choice
// and the whole bitmap are then written as k_scan writes them.
constexpr int SX_TPB = 1024;
constexpr int SX_HASH_LOG = 12;
constexpr int SX_HASH = 1 << SX_HASH_LOG;      // hash slots: twice the indices
static_assert(SX_HASH == 2 * SMALL_X_MAX, "small-x hash table");

__device__ __forceinline__ bool sx_insert(uint32_t *tab, uint32_t key)
{
    // multiplicative hashing, linear probing; the table is never more than
    // half full, so a free slot is always found
    uint32_t h = (key * 2654435761u) >> (32 - SX_HASH_LOG);
    for (;;) {
        const uint32_t old = atomicCAS(&tab[h], 0xFFFFFFFFu, key);
        if (old == 0xFFFFFFFFu) return true;
        if (old == key) return false;
        h = (h + 1u) & (uint32_t)(SX_HASH - 1);
    }
}

// The work of one workgroup of NTH threads (SMALL_X_MAX / NTH indices per
// thread) over LDS scratch s_hash[SX_HASH], s_bits[(nbc + 31) / 32] and
// lds4[NTH / 64]; ends with every global write issued (not fenced).
template <int MODE, int NTH>
__device__ __forceinline__ void small_x_body(const int32_t *__restrict__ xi, const void *__restrict__ xv,
                                             int32_t k, int32_t n, void *__restrict__ xd,
                                             uint32_t *__restrict__ xmask, const int32_t *__restrict__ cb_ptr,
                                             int32_t nbc, int4 *__restrict__ items, uint32_t *__restrict__ xbits,
                                             int32_t *__restrict__ counters, int32_t forced_path, double th3,
                                             double th3s, uint32_t *s_hash, uint32_t *s_bits, uint64_t *lds4)
{
    constexpr int PER = SMALL_X_MAX / NTH;
    static_assert(PER * NTH == SMALL_X_MAX, "small-x tile");
    const int t = threadIdx.x;
    const int32_t nwords = (nbc + 31) >> 5;
    int32_t j[PER];
    uint32_t v[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        const int32_t i = e * NTH + t;
        j[e] = i < k ? xi[i] : -1;
        v[e] = 0;
        if constexpr (MODE == M_F32) v[e] = i < k ? ((const uint32_t *)xv)[i] : 0u;
        if constexpr (MODE == M_F16) v[e] = i < k ? ((const uint16_t *)xv)[i] : 0u;
    }
    for (int32_t i = t; i < SX_HASH; i += NTH) s_hash[i] = 0xFFFFFFFFu;
    for (int32_t i = t; i < nwords; i += NTH) s_bits[i] = 0u;
    uint32_t bad = 0, pop = 0, own = 0;
    int32_t cs[PER], ce[PER];
    uint32_t bits[PER], old[PER];
    // every memory operation that depends only on the index goes out at
    // once: the value's scatter, the mask atomic (its old word is used only
    // for the final counts) and the block-column extent of the index's
    // vector block (kept by the lane that owns the block below)
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        const int32_t i = e * NTH + t;
        const bool valid = i < k && j[e] >= 0 && j[e] < n;
        if (i < k && !valid) ++bad;
        if (!valid) j[e] = -1;
        cs[e] = ce[e] = 0;
        bits[e] = 0u;
        old[e] = 0xFFFFFFFFu;
        if (!ballot(i < k)) continue;  // (wave-uniform) no index left for this wave
        // an input equal to the absent-entry marker becomes the canonical NaN
        if (valid) {
            if constexpr (MODE == M_F32) ((uint32_t *)xd)[j[e]] = v[e] == 0xFFFFFFFFu ? 0x7FC00000u : v[e];
            if constexpr (MODE == M_F16)
                ((uint16_t *)xd)[j[e]] = v[e] == 0xFFFFu ? (uint16_t)0x7E00u : (uint16_t)v[e];
        }
        // runs of lanes with one mask word (sorted or clustered indices) are
        // merged first: one returning atomic per run, whose old word tells
        // which of the run's bits were already stored
        const int32_t w = valid ? j[e] >> 5 : -1;
        bits[e] = wave_run_or(valid ? 1u << (j[e] & 31) : 0u, (uint32_t)w);
        const int32_t nextw = (int32_t)dpp_mov<dppc::WF_SL1>(~(uint32_t)w, (uint32_t)w);
        const bool last = w >= 0 && nextw != w;
        if (last) old[e] = atomicOr(&xmask[w], bits[e]);
        if (valid) {
            const int32_t J = j[e] >> 4;
            cs[e] = cb_ptr[J];
            ce[e] = cb_ptr[J + 1];
        }
    }
    __syncthreads();
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        // likewise the vector blocks: the first lane of a run inserts
        const int32_t J = j[e] >= 0 ? j[e] >> 4 : -1;
        const int32_t prevJ = (int32_t)dpp_mov<dppc::WF_SR1>(~(uint32_t)J, (uint32_t)J);
        if (J >= 0 && prevJ != J && sx_insert(s_hash, (uint32_t)J)) {
            own |= 1u << e;
            atomicOr(&s_bits[J >> 5], 1u << (J & 31));
        }
    }
#pragma unroll
    for (int e = 0; e < PER; ++e) pop += __popc(bits[e] & ~old[e]);
    uint64_t mine = 0;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        const uint32_t len = (uint32_t)(ce[e] - cs[e]);
        if (((own >> e) & 1u) && len) mine += (1ull << 34) + len;
    }
    uint64_t total, ctot;
    const uint64_t excl = block_exclusive_scan<NTH>(mine, &total, lds4);
    // block totals of (distinct indices, bad indices, distinct vector blocks)
    block_exclusive_scan<NTH>(((uint64_t)pop << 32) | ((uint64_t)bad << 16) | (uint64_t)__popc(own), &ctot,
                                 lds4);
    int64_t idx = (int64_t)(excl >> 34);
    int64_t off = (int64_t)(excl & ((1ull << 34) - 1));
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        const int32_t len = ce[e] - cs[e];
        if (((own >> e) & 1u) && len) {
            items[idx] = make_int4((int32_t)off, j[e] >> 4, cs[e] - (int32_t)off, 0);
            ++idx;
            off += len;
        }
    }
    // (the scans' barriers have completed the LDS bitmap)
    for (int32_t i = t; i < nwords; i += NTH) xbits[i] = s_bits[i];
    if (t == 0) {
        const int32_t NT = (int32_t)(total >> 34);
        const int32_t T = (int32_t)(total & ((1ull << 34) - 1));
        const int32_t N = (int32_t)(ctot & 0xFFFFu);
        const int32_t nbad = (int32_t)((ctot >> 16) & 0xFFFFu);
        const int32_t npop = (int32_t)(ctot >> 32);
        items[NT] = make_int4(T, 0, 0, 0);
        counters[C_NZBLK] = N;
        counters[C_NTB] = NT;
        counters[C_TASKS] = T;
        if (npop) atomicAdd(&counters[C_XPOP], npop);
        if (nbad) atomicAdd(&counters[C_XBAD], nbad);
        int path = forced_path;
        if (path == 0) {
            const bool spread = th3s > 0.0 && (int64_t)npop < 2 * (int64_t)N && (double)N < th3s * (double)nbc;
            path = ((double)N < th3 * (double)nbc || spread) ? PATH_PUSH : PATH_PULL;
        }
        counters[C_PATH] = path;
    }
}

template <int MODE>
__global__ __launch_bounds__(SX_TPB) void k_small_x(const int32_t *__restrict__ xi, const void *__restrict__ xv,
                                                   int32_t k, int32_t n, void *__restrict__ xd,
                                                   uint32_t *__restrict__ xmask,
                                                   const int32_t *__restrict__ cb_ptr, int32_t nbc,
                                                   int4 *__restrict__ items, uint32_t *__restrict__ xbits,
                                                   int32_t *__restrict__ counters, int32_t forced_path,
                                                   double th3, double th3s)
{
    __shared__ uint32_t s_hash[SX_HASH];
    __shared__ uint32_t s_bits[SMALL_X_WORDS];
    __shared__ uint64_t lds4[SX_TPB / WAVE];
    small_x_body<MODE, SX_TPB>(xi, xv, k, n, xd, xmask, cb_ptr, nbc, items, xbits, counters, forced_path, th3, th3s,
                               s_hash, s_bits, lds4);
}

// ---------------------------------------------------------------------------
// block microkernels
// ---------------------------------------------------------------------------

// Coordinate bytes (row << 4 | col) of a COO block held in its descriptor
// (at most 6 entries), byte e of the result for entry e.
__device__ __forceinline__ uint64_t inline_coords(uint64_t d, uint32_t vb, uint32_t nnz)
{
    if (nnz == 1) return (d >> 16) & 0xFFull;  // the common hypersparse case
    uint64_t c = 0;
    for (uint32_t e = 0; e < nnz; ++e) c |= ((d >> inline_shift(e, vb)) & 0xFFull) << (8 * e);
    return c;
}

// Value of entry e of a COO block held in its descriptor.
template <int MODE>
__device__ __forceinline__ float inline_value(uint64_t d, uint32_t vb, uint32_t e)
{
    const uint32_t bits = (uint32_t)(d >> (inline_shift(e, vb) + 8));
    if constexpr (MODE == M_F32) return __uint_as_float(bits);
    else if constexpr (MODE == M_F16) return h2f((uint16_t)bits);
    else return 0.f;
}

// Bit e set for every entry e of a COO block whose column is active in the
// vector-block mask and whose row is admitted.
__device__ __forceinline__ uint32_t coo_matches(uint64_t cds, uint32_t nnz, uint32_t mx, uint32_t am)
{
    uint32_t mm = 0;
    for (uint32_t e = 0; e < nnz; ++e) {
        const uint32_t cd = (uint32_t)(cds >> (8 * e)) & 0xFFu;
        mm |= ((mx >> (cd & 15u)) & (am >> (cd >> 4)) & 1u) << e;
    }
    return mm;
}

// One lane, one COO block whose entries sit in its descriptor (entries in
// row-major order), committing straight to global memory (push path): the
// products of the matching entries are added to the row accumulators,
// merging runs of one row first; for BFS the smallest active column per row
// is kept (the first match met, columns ascend within a row).  Returns the
// rows hit.
template <int MODE>
__device__ __forceinline__ uint32_t inline_block_push(uint32_t vb, uint64_t d, int32_t J, int32_t R,
                                                      uint32_t mx, uint32_t am, const void *__restrict__ xd,
                                                      double *yacc, int32_t *parent)
{
    const uint32_t nnz = desc_nnz(d);
    const uint64_t cds = inline_coords(d, vb, nnz);
    uint32_t mm = coo_matches(cds, nnz, mx, am);
    uint32_t hit = 0;
    int cur = -1;
    float acc = 0.f;
    while (mm) {
        const uint32_t e = ctz32(mm);
        mm &= mm - 1;
        const uint32_t cd = (uint32_t)(cds >> (8 * e)) & 0xFFu, r = cd >> 4, c = cd & 15u;
        if constexpr (valued<MODE>()) {
            const float prod = inline_value<MODE>(d, vb, e) * VT<MODE>::x(xd, (int64_t)J * BS + c);
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

// COO blocks whose entries sit in the descriptor are processed by one lane
// (no payload loads); COO blocks with a payload record are processed
// entry-parallel by the whole wave (flat_pass); in pull, the other formats
// row-per-lane from their own list (pull_rows).
__device__ __forceinline__ bool lane_coo(uint64_t d) { return desc_inline(d); }
__device__ __forceinline__ bool flat_coo(uint64_t d) { return !desc_inline(d) && desc_type(d) == T_COO; }

// Densified x (valued modes): absent entries hold all-ones bits in either
// element width, so the gather of x_j also tells whether x_j is stored.  The
// scatter kernel maps an input whose bits equal the marker to the canonical
// NaN.  Boolean modes test the vector-block mask instead.
constexpr uint32_t X_ABSENT32 = 0xFFFFFFFFu;
constexpr uint32_t X_ABSENT16 = 0xFFFFu;

template <int MODE>
__device__ __forceinline__ bool x_present(uint32_t raw, int32_t J, uint32_t c)
{
    if constexpr (MODE == M_F32) return raw != X_ABSENT32;
    else if constexpr (MODE == M_F16) return raw != X_ABSENT16;
    else return (raw >> ((J & 1) * 16 + c)) & 1u;
}
template <int MODE>
__device__ __forceinline__ float x_value(uint32_t raw)
{
    if constexpr (MODE == M_F32) return __uint_as_float(raw);
    else if constexpr (MODE == M_F16) return h2f((uint16_t)raw);
    else return 0.f;
}

// Gathered x words held per inline COO block: one per entry for valued
// modes (capacity 1 fp32 / 2 fp16 entries), the block's mask word otherwise.
template <int MODE> constexpr int inline_max() { return MODE == M_F32 ? 1 : MODE == M_F16 ? 2 : 1; }
__device__ __forceinline__ uint32_t inline_cd(uint64_t d, int e, uint32_t vb)
{
    return (uint32_t)(d >> inline_shift((uint32_t)e, vb)) & 0xFFu;
}


// The 16 group masks at the head of a Dense, ForceCSR, ForceCSC or patched-CSR
// record (row masks; column masks for ForceCSC), read with two 16-byte loads
// (records of these formats are 16-byte aligned).
struct Masks16 {
    uint32_t m[8];
};
__device__ __forceinline__ Masks16 load_masks(const uint8_t *rec)
{
    const uint4 a = ((const uint4 *)(rec + HDR_MASK))[0], b = ((const uint4 *)(rec + HDR_MASK))[1];
    return Masks16{{a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w}};
}
// (t is a constant after unrolling: no dynamic register indexing)
__device__ __forceinline__ uint32_t mask_at(const Masks16 &h, int t) { return (h.m[t >> 1] >> ((t & 1) * 16)) & 0xFFFFu; }

// Position of the k-th (0-based) set bit of a 16-bit v, by halving.
__device__ __forceinline__ uint32_t nth_bit16(uint32_t v, uint32_t k)
{
    uint32_t pos = 0;
#pragma unroll
    for (int step = 8; step > 0; step >>= 1) {
        const uint32_t c = __popc(v & ((1u << step) - 1u));
        if (k >= c) {
            k -= c;
            v >>= step;
            pos += (uint32_t)step;
        }
    }
    return pos;
}

// Push stages a stored COO block whose vector-block mask leaves some columns
// out with this tag in place of its format, when the wave iteration's COO
// records hold more than COO_LIVE_WAVE entries: the staged mask word then
// holds the block's matching entries (column active, row admitted), read
// from its coordinates at staging, and the entry-parallel pass walks those
// only (a chunk of hub blocks otherwise loads every stored entry, most of
// which miss a sparse x, in a dozen serial windows).
constexpr uint32_t T_COO_LIVE = 5;
#ifndef COO_LIVE_WAVE
#define COO_LIVE_WAVE 256
#endif
#ifndef COO_LIVE_MAX
#define COO_LIVE_MAX 32
#endif
static_assert(COO_LIVE_MAX <= 32, "one 32-bit mask per block");

// Matching entries (bit e: entry e) of a COO record of nnz <= COO_LIVE_MAX
// fp32 entries: its coordinate bytes follow the 4 nnz value bytes, so they
// start 4-byte aligned.
__device__ __forceinline__ uint32_t coo_live_mask(const uint8_t *rec, uint32_t nnz, uint32_t mx, uint32_t am)
{
    constexpr int NW = (COO_LIVE_MAX + 3) / 4;
    const uint32_t *cw = (const uint32_t *)(rec + 4u * nnz);
    uint32_t w[NW];
#pragma unroll
    for (int q = 0; q < NW; ++q) w[q] = (uint32_t)(4 * q) < nnz ? cw[q] : 0u;
    uint32_t m = 0;
#pragma unroll
    for (int e = 0; e < COO_LIVE_MAX; ++e) {
        const uint32_t cd = (w[e >> 2] >> ((e & 3) * 8)) & 0xFFu;
        const bool hit = (uint32_t)e < nnz && ((mx >> (cd & 15u)) & 1u) && ((am >> (cd >> 4)) & 1u);
        m |= (hit ? 1u : 0u) << e;
    }
    return m;
}

// The e-th set bit of a 32-bit mask (e below its population count).
__device__ __forceinline__ uint32_t nth_bit32(uint32_t v, uint32_t e)
{
    const uint32_t lo = __popc(v & 0xFFFFu);
    return e < lo ? nth_bit16(v & 0xFFFFu, e) : 16u + nth_bit16(v >> 16, e - lo);
}

// Group t's mask restricted to the entries one push task has to multiply
// (Sec. 3.3.3: the block's structure against blk_x_mask): entries whose column
// is active in the vector-block mask mx and whose row is admitted (am).  The
// groups of the row view are rows (bits: columns); ForceCSC groups are columns
// (bits: rows).
__device__ __forceinline__ uint32_t group_live(uint32_t type, int t, uint32_t gm, uint32_t mx, uint32_t am)
{
    if (type == T_FCSC) return ((mx >> t) & 1u) ? (gm & am) : 0u;
    return ((am >> t) & 1u) ? (gm & mx) : 0u;
}

// Number of live entries of a record with the given masks.
__device__ __forceinline__ uint32_t live_count(const Masks16 &h, uint32_t type, uint32_t mx, uint32_t am)
{
    uint32_t n = 0;
#pragma unroll
    for (int t = 0; t < 16; ++t) n += __popc(group_live(type, t, mask_at(h, t), mx, am));
    return n;
}

// Live entry e (in record order: row-major, column-major for ForceCSC) of a
// Dense, ForceCSR, ForceCSC or patched-CSR record: its local row and column
// and the index of its value in the record's value array (Dense: r * 16 + c
// over all 256 values; the others: the group's start plus the entry's rank in
// the group's stored mask).
__device__ __forceinline__ void live_entry(const uint8_t *rec, uint32_t type, uint32_t e, uint32_t mx, uint32_t am,
                                           uint32_t &r, uint32_t &c, uint32_t &vi)
{
    const Masks16 h = load_masks(rec);
    const uint4 st = *(const uint4 *)(rec + HDR_START);  // group starts (not read for Dense)
    uint32_t before = 0, g = 0, gb = 0, gl = 0, gm = 0;
#pragma unroll
    for (int t = 0; t < 16; ++t) {
        const uint32_t m = mask_at(h, t), l = group_live(type, t, m, mx, am);
        if (l != 0u && before <= e) {
            g = (uint32_t)t;
            gb = before;
            gl = l;
            gm = m;
        }
        before += __popc(l);
    }
    const uint32_t o = nth_bit16(gl, e - gb);
    r = type == T_FCSC ? o : g;
    c = type == T_FCSC ? g : o;
    if (type == T_DENSE) {
        vi = r * BS + c;
    } else {
        const uint32_t w = g < 8u ? (g < 4u ? st.x : st.y) : (g < 12u ? st.z : st.w);
        vi = ((w >> ((g & 3u) * 8u)) & 0xFFu) + __popc(gm & ((1u << o) - 1u));
    }
}

template <int MODE>
__device__ __forceinline__ uint32_t xd_raw(const void *xd, int64_t j)
{
    if constexpr (MODE == M_F32) return ((const uint32_t *)xd)[j];
    else return ((const uint16_t *)xd)[j];
}

// ---------------------------------------------------------------------------
// main traversal kernel
// ---------------------------------------------------------------------------
struct MainArgs {
    const int32_t *sl_col;   // pull-segment slots: block column (-1 padding, sign bit: listed)
    const uint64_t *sl_desc; // pull-segment slots: descriptor
    const uint32_t *seg_rs;  // per segment: its block row
    const uint8_t *pay;
    uint32_t vb;            // value bytes of the matrix (4, 2 or 0)
    int32_t nbc;
    const int32_t *csc_row;
    const uint64_t *csc_desc;
    const int32_t *hv_col;     // the non-COO list and its chunks (see DevMatrix)
    const uint64_t *hv_desc;
    const int32_t *hv_cstart;
    const int32_t *hv_crow;
    int64_t nchunk;
    int64_t nseg;
    const void *xd;
    int64_t xstride;        // batched pull: elements between the dense x of consecutive vectors
    const uint32_t *xmask;
    const uint32_t *xbits;       // one activity bit per vector block (global copy)
    const int4 *items;           // push work items (see k_scan)
    int32_t *counters;
    const uint32_t *omask;  // output mask bitmap (NULL = none); BFS: visited
    int32_t complement;
    double *yacc;
    int64_t ystride;        // batched pull: accumulators between consecutive vectors
    uint32_t *ybits;        // y structure; BFS: next-frontier bitmap
    int32_t *parent;        // BFS only
    int32_t *clist;         // compacted pull: per-wave regions of active slot ids (NULL: not used)
    uint32_t *ccount;       // compacted pull: entries per region
    int64_t clist_cap;      // entries the list holds
    int32_t nreg;           // compacted pull: regions (waves of the second kernel's grid)
    int32_t cpw;            // non-COO pass: chunks per workgroup round (1..16)
    int32_t cpm;            // compacted pull below N_nzblk / N_blk = cpm / 1000
    int32_t creg;           // compacted pull: regions the list's counts have room for
    const int32_t *torder;  // segment-loop tasks by decreasing cost (NULL: segment order)
    int32_t ntask;          // tasks in torder
    // dense output written by the non-COO pass itself (k_rows_dx): the
    // chunks of each block row, the per-call count of its committed chunks,
    // the outputs (y in the matrix's value type, optional fp32 copy), m
    const int32_t *rowchunks;
    int32_t *rdone;
    void *ydense;
    float *y32;
    int32_t m;
};

// Independent work units per lane and loop iteration: four segments per
// quarter-wave (pull) or four 64-task chunks per wave (push), so that four
// dependent load chains are in flight per lane instead of one.
constexpr int SLOTS = 4;

__device__ __forceinline__ uint32_t row_admit(const MainArgs &a, int32_t R)
{
    return allowed16(a.omask, a.complement, R);
}

// Gathers the word that holds x_j for j = 16 J + c: the value bits (valued
// modes) or the vector-block mask word (boolean modes).
template <int MODE>
__device__ __forceinline__ uint32_t x_gather(const MainArgs &a, int32_t J, uint32_t c)
{
    const int64_t j = (int64_t)J * BS + c;
    if constexpr (MODE == M_F32) return ((const uint32_t *)a.xd)[j];
    else if constexpr (MODE == M_F16) return ((const uint16_t *)a.xd)[j];
    else return a.xmask[J >> 1];
}

// One lane, one COO block whose entries sit in its descriptor, with the x
// words already gathered (pull path): the products of the entries whose x is
// stored and whose row is admitted are added to dst16[row] (LDS), merging
// runs of one row first; for BFS the smallest active column per row is kept
// in pdst16 (the first match met, columns ascend within a row).  Returns the
// rows hit.
template <int MODE>
__device__ __forceinline__ uint32_t inline_block(const MainArgs &a, uint64_t d, int32_t J, uint32_t am,
                                                 const uint32_t (&xr)[inline_max<MODE>()], float *dst16,
                                                 int32_t *pdst16)
{
    constexpr int CAP = valued<MODE>() ? inline_max<MODE>() : 6;
    const uint32_t nnz = desc_nnz(d), vb = a.vb;
    uint32_t hit = 0;
    int cur = -1;
    float acc = 0.f;
#pragma unroll
    for (int e = 0; e < CAP; ++e) {
        if ((uint32_t)e >= nnz) break;
        const uint32_t cd = inline_cd(d, e, vb), r = cd >> 4, c = cd & 15u;
        const uint32_t raw = xr[valued<MODE>() ? e : 0];
        if (!x_present<MODE>(raw, J, c) || !((am >> r) & 1u)) continue;
        if constexpr (valued<MODE>()) {
            const float prod = inline_value<MODE>(d, vb, (uint32_t)e) * x_value<MODE>(raw);
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

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int l)
{
    const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)v, l, WAVE);
    const uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(v >> 32), l, WAVE);
    return ((uint64_t)hi << 32) | lo;
}

// Entries per lane in one window of the entry-parallel pass (a window is
// FLAT_E * 64 consecutive entries; lane l takes entries FLAT_E l .. FLAT_E l
// + FLAT_E - 1), so that FLAT_E record loads, then FLAT_E x gathers, are in
// flight per lane.
constexpr int FLAT_E = 4;
constexpr int FLAT_W = FLAT_E * WAVE;
static_assert(FLAT_E == 4, "the mark reads below take 4 marks per lane");

// Blocks staged for whole-wave processing: slot-major, one entry per lane
// (entry k * 64 + lane for slot k).  After an entry is processed its J word
// carries the rows hit back to the lane that staged it.  Stored COO blocks
// for the entry-parallel pass use the same entries, with the descriptor
// replaced by flat_word.  About 4.4 KB per wave (5.3 KB with the block rows
// and per-block hits push needs), so that the traversal kernels' LDS, with
// the pull kernel's activity bitmap, allows five workgroups per compute unit.
template <bool PUSH>
struct HeavyStage {
    uint64_t d[SLOTS * WAVE];
    int32_t J[SLOTS * WAVE];      // block column; rows hit once processed
    uint32_t mxam[SLOTS * WAVE];  // vector-block mask | admitted rows << 16
    alignas(8) uint16_t mark[FLAT_W];  // entry-parallel pass: 1 + block starting at each window entry
    uint32_t hitw[PUSH ? SLOTS * WAVE : SLOTS * 4];  // entry-parallel pass: rows hit per block
                                                     // (push) or per slot quarter (pull)
    int32_t R[PUSH ? SLOTS * WAVE : 1];
    __device__ __forceinline__ void stage(int e, uint64_t dd, int32_t j, uint32_t mx, uint32_t am, int32_t r)
    {
        d[e] = dd;
        J[e] = j;
        if constexpr (PUSH) R[e] = r;
        mxam[e] = mx | (am << 16);
    }
};

// Staged word of a stored COO block in the entry-parallel pass: payload
// offset, entry count and the number of entries before the block.  The
// payload offset keeps 39 bits (512 GB), the count 8 and the start 17
// (at most SLOTS * 64 blocks of at most 256 entries).
__device__ __forceinline__ uint64_t flat_word(uint64_t d, uint32_t excl)
{
    return (desc_off(d) << 25) | ((uint64_t)(desc_nnz(d) - 1) << 17) | excl;
}


// One lane's entries of a window (the block's column and masks are read
// again from the staging area when the entry is finished).
struct FlatEntries {
    uint32_t ocd[FLAT_E];   // staging entry of the block (slot * 64 + lane) << 8 | coordinate byte;
                            // bit 31: valid
    float val[FLAT_E];      // value (valued modes)
};

// Finds the blocks of this lane's entries of the window starting at base
// and issues their coordinate and value loads.  carry: 1 + the block of the
// last entry of the previous window.
template <int MODE, bool PUSH, bool ANYTYPE>
__device__ __forceinline__ FlatEntries flat_issue(const MainArgs &a, HeavyStage<PUSH> *hs,
                                                  const uint32_t (&cnt)[SLOTS], const uint32_t (&excl)[SLOTS],
                                                  uint32_t tot, uint32_t base, uint32_t &carry)
{
    const int lane = lane_id();
    // marks: 1 + block index at the window position of each block's first entry
    *(uint64_t *)&hs->mark[lane * FLAT_E] = 0ull;
    wave_lds_sync();
#pragma unroll
    for (int k = 0; k < SLOTS; ++k)
        if (cnt[k] && excl[k] >= base && excl[k] < base + FLAT_W)
            hs->mark[excl[k] - base] = (uint16_t)(k * WAVE + lane + 1);
    wave_lds_sync();
    const uint64_t mw = *(const uint64_t *)&hs->mark[lane * FLAT_E];
    uint32_t m[FLAT_E];
#pragma unroll
    for (int j = 0; j < FLAT_E; ++j) m[j] = (uint32_t)(mw >> (16 * j)) & 0xFFFFu;
#pragma unroll
    for (int j = 1; j < FLAT_E; ++j) m[j] = max(m[j], m[j - 1]);
    // blocks start in ascending entry order: the block of an entry is the
    // largest mark at or before it (max-scan over the lanes, then carry)
    const uint32_t inc = wave_incl_max(m[FLAT_E - 1]);
    const uint32_t cin = max(wave_shr1(inc), carry);
    carry = max(carry, readlane_u32(inc, WAVE - 1));
    FlatEntries f;
#pragma unroll
    for (int j = 0; j < FLAT_E; ++j) {
        const uint32_t g = base + (uint32_t)(lane * FLAT_E + j);
        const bool valid = g < tot;
        const uint32_t own = max(cin, m[j]);
        const uint32_t o = own ? own - 1 : 0u;
        const uint64_t w = hs->d[o];
        const uint64_t off = w >> 25;
        const uint32_t nnz = (uint32_t)((w >> 17) & 0xFFu) + 1u, e = g - (uint32_t)(w & 0x1FFFFu);
        uint32_t cd = 0;
        f.val[j] = 0.f;
        const uint32_t type = ANYTYPE ? ((uint32_t)hs->J[o] >> 28) : (uint32_t)T_COO;
        if (type == T_COO) {
            cd = valid ? a.pay[off + (uint64_t)a.vb * nnz + e] : 0u;
            if constexpr (valued<MODE>()) f.val[j] = valid ? VT<MODE>::load(a.pay + off, e) : 0.f;
        } else if (ANYTYPE && type == T_COO_LIVE) {
            // the e-th matching entry of the record
            const uint32_t ei = nth_bit32(hs->mxam[o], e);
            cd = valid ? a.pay[off + (uint64_t)a.vb * nnz + ei] : 0u;
            if constexpr (valued<MODE>()) f.val[j] = valid ? VT<MODE>::load(a.pay + off, ei) : 0.f;
        } else if constexpr (ANYTYPE) {
            // the other formats: the e-th live entry, located from the header
            if (valid) {
                uint32_t r, c, vi;
                const uint32_t ma = hs->mxam[o];
                live_entry(a.pay + off, type, e, ma & 0xFFFFu, ma >> 16, r, c, vi);
                cd = (r << 4) | c;
                if constexpr (valued<MODE>()) f.val[j] = VT<MODE>::load(a.pay + off + values_at(type, nnz), vi);
            }
        }
        f.ocd[j] = (valid ? 0x80000000u : 0u) | (o << 8) | cd;
    }
    return f;
}

// Gathers x for the entries and adds their products (see flat_pass).  MXK:
// the staged word holds the block's vector-block mask, which then answers
// the boolean modes' presence test without a gather.
template <int MODE, bool PUSH, bool MXK, bool RUNS>
__device__ __forceinline__ void flat_finish(const MainArgs &a, HeavyStage<PUSH> *hs, FlatEntries f,
                                            float *sy, int32_t *sp)
{
    static_assert(!RUNS || PUSH, "the run destination uses the staged block rows");
    constexpr bool known = MXK && !valued<MODE>();
    uint32_t raw[FLAT_E];
#pragma unroll
    for (int j = 0; j < FLAT_E; ++j) {
        const uint32_t o = (f.ocd[j] >> 8) & 0xFFu, r = (f.ocd[j] >> 4) & 15u, c = f.ocd[j] & 15u;
        // with the vector-block mask staged, an entry whose column it lacks
        // needs no gather
        // (a COO_LIVE block stages only matching entries, its mask word
        // holding which)
        const bool live = PUSH && ((uint32_t)hs->J[o] >> 28) == T_COO_LIVE;
        const bool adm = (f.ocd[j] >> 31) &&
                         (live || (((hs->mxam[o] >> (16 + r)) & 1u) && (!MXK || ((hs->mxam[o] >> c) & 1u))));
        raw[j] = (adm && !known) ? x_gather<MODE>(a, hs->J[o] & 0x0FFFFFFF, c) : 0u;
        if (!adm) f.ocd[j] = 0u;
    }
#pragma unroll
    for (int j = 0; j < FLAT_E; ++j) {
        const uint32_t o = (f.ocd[j] >> 8) & 0xFFu, r = (f.ocd[j] >> 4) & 15u, c = f.ocd[j] & 15u;
        const int32_t J = hs->J[o] & 0x0FFFFFFF;
        const bool present = known ? ((hs->mxam[o] >> c) & 1u) != 0 : x_present<MODE>(raw[j], J, c);
        if ((f.ocd[j] >> 31) && present) {
            const int ko = (int)(o >> 6), lo = (int)(o & (WAVE - 1));
            if constexpr (RUNS) {
                const int at = hs->R[o] * 16 + (int)r;
                if constexpr (valued<MODE>()) atomicAdd(&sy[at], f.val[j] * x_value<MODE>(raw[j]));
                if constexpr (MODE == M_BFS) atomicMin(&sp[at], J * BS + (int32_t)c);
                atomicOr(&hs->hitw[o], 1u << r);
            } else if constexpr (PUSH) {
                const int64_t row = (int64_t)hs->R[o] * BS + r;
                if constexpr (valued<MODE>()) atomicAdd(&a.yacc[row], (double)(f.val[j] * x_value<MODE>(raw[j])));
                if constexpr (MODE == M_BFS) atomicMin(&a.parent[row], J * BS + (int32_t)c);
                atomicOr(&hs->hitw[o], 1u << r);
            } else {
                const int at = ko * WAVE + (lo >> 4) * 16 + (int)r;
                if constexpr (valued<MODE>()) atomicAdd(&sy[at], f.val[j] * x_value<MODE>(raw[j]));
                if constexpr (MODE == M_BFS) atomicMin(&sp[at], J * BS + (int32_t)c);
                atomicOr(&hs->hitw[ko * 4 + (lo >> 4)], 1u << r);
            }
        }
    }
}

// Entry-parallel pass over the stored COO blocks of one wave iteration
// (Sec. 3.3.3's COO microkernel, re-mapped to wave64).  The entries of the
// blocks staged with cnt[k] > 0 are numbered in slot-major order by wave
// prefix sums; the wave walks them FLAT_W at a time, FLAT_E consecutive
// entries per lane.  Each window, the blocks that start inside it mark their
// first entry; a max-scan over the marks then gives every lane the blocks of
// its entries (blocks start in ascending entry order).  The coordinate and
// value loads of all lanes go out together, then the x gathers.
//   pull: products are added to the owner's quarter of its slot's LDS rows;
//         BFS keeps the smallest active column per row there; rows hit are
//         collected per slot quarter in hitw[slot * 4 + quarter].
//   push: products go straight to the fp64 accumulators of the owner's
//         block row; rows hit are collected per block in hitw[entry].
//   runs (compacted pull): the staged row word is the owner's run; products
//         go to the run's LDS rows, rows hit per block in hitw[entry].
template <int MODE, bool PUSH, bool MXK, bool ANYTYPE, bool RUNS, class Between>
__device__ __forceinline__ void flat_pass(const MainArgs &a, HeavyStage<PUSH> *hs, const uint32_t (&cnt)[SLOTS],
                          const uint64_t (&d)[SLOTS], float *sy, int32_t *sp, Between &&between)
{
    const int lane = lane_id();
    uint32_t excl[SLOTS];
    uint32_t tot = 0;
#pragma unroll
    for (int k = 0; k < SLOTS; ++k) {
        const uint32_t incl = wave_incl_add(cnt[k]);
        excl[k] = tot + incl - cnt[k];
        tot += readlane_u32(incl, WAVE - 1);
    }
#pragma unroll
    for (int k = 0; k < SLOTS; ++k)
        if (cnt[k]) hs->d[k * WAVE + lane] = flat_word(d[k], excl[k]);
    if constexpr (PUSH) {
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) hs->hitw[k * WAVE + lane] = 0u;
    } else {
        if (lane < SLOTS * 4) hs->hitw[lane] = 0u;
    }
    uint32_t carry = 0;
    // the first window is peeled: its record loads are in flight while the
    // caller's inline products are formed
    FlatEntries f = flat_issue<MODE, PUSH, ANYTYPE>(a, hs, cnt, excl, tot, 0u, carry);
    between();
    flat_finish<MODE, PUSH, MXK, RUNS>(a, hs, f, sy, sp);
    for (uint32_t base = FLAT_W; base < tot; base += FLAT_W) {
        f = flat_issue<MODE, PUSH, ANYTYPE>(a, hs, cnt, excl, tot, base, carry);
        flat_finish<MODE, PUSH, MXK, RUNS>(a, hs, f, sy, sp);
    }
    wave_lds_sync();
}


// Pull (Sec. 3.3.2): a quarter-wave per row-block segment (<= 16 blocks,
// one block per lane); a quarter takes SLOTS consecutive segments per
// iteration, consecutive slots of one block row are folded in registers
// before the commit (Sec. 3.3.3's local aggregation), grid-stride over
// segment groups.  Blocks that need the whole wave (non-COO formats, long
// COO blocks) are staged in LDS and processed one by one after the
// lane-parallel COO work, from a single call site.
// Activity bitmap of the pull kernel (one bit per vector block), written by
// the scan: up to 16 KB (131072 vector blocks) it is copied into the LDS of
// every workgroup and tested before the vector-block mask is gathered.  A
// larger bitmap is not used (a global lookup would add a dependent load in
// front of the mask gather).
constexpr int32_t LDS_BITMAP_WORDS = 4096;
extern __shared__ uint32_t lds_bits[];

__device__ __forceinline__ bool block_active(int32_t J) { return (lds_bits[J >> 5] >> (J & 31)) & 1u; }

// Pull: the non-COO blocks (Dense, ForceCSR, ForceCSC, patched CSR), listed
// at upload in block-CSR order and cut into chunks of at most HV_CHUNK
// consecutive blocks of one block row, taken a.cpw (at most 16) chunks per
// workgroup and round ahead of the segment loop:
//  1. thread t (chunk t / 16 if below a.cpw, block t % 16 of it) loads its block's metadata
//     (block column, activity, descriptor), then its record header (row
//     masks and starts, or column masks and starts for ForceCSC) and its
//     vector-block mask into LDS; the active blocks of the round are listed
//     in LDS by a workgroup prefix sum;
//  2. the 16 quarter-waves of the workgroup deal the listed blocks out
//     round-robin (a chunk with more active blocks than others does not hold
//     the round up), one lane per row of the block: lane r reads row r's mask
//     and start (ForceCSC: every column's) from LDS, loads the 16 x words of
//     the block's vector block and row r's matching values -- Dense: its 16
//     values; the other formats: entry by entry (fp32), or (fp16) from a copy
//     of the block's value array that the quarter brings into LDS with
//     16-byte loads -- and forms row r's fp32 share of the block (Alg. 2 and 4
//     with a row per lane; Alg. 3's column view for ForceCSC), added to the
//     chunk's fp64 row accumulator in LDS;
//  3. each run of the round's chunks of one block row is summed in LDS and
//     committed with one fp64 atomic per row (the segments of such a block
//     row commit with atomics as well).
constexpr int HV_WORDS = 16;       // LDS words per staged block: 8 mask words, 4 start words,
                                   // x mask | admitted rows << 16, block column, descriptor
constexpr int HV_VAL_BYTES = 256;  // per quarter: LDS copy of one fp16 block's value array

// LDS layout of the non-COO pass (32-bit words)
template <int MODE, int NB = 1> struct RowsLds {
    static constexpr int NT = TPB;                 // staged blocks: one per thread
    static constexpr int NQ = TPB / 16;            // quarter-waves = chunks per round
    static constexpr int ST = 0;                                          // staged entries
    static constexpr int VB = ST + NT * HV_WORDS;                         // fp16 value buffers
    static constexpr int AC = VB + (MODE == M_F16 ? NQ * HV_VAL_BYTES / 4 : 0);  // fp64 [vector][chunk][row]
    static constexpr int HM = AC + NB * NQ * 16 * 2;  // rows hit per chunk
    static constexpr int CR = HM + NQ;             // block row per chunk (-1: none)
    static constexpr int NI = CR + NQ;             // active blocks per wave: Dense, then the others
    static constexpr int IT = NI + 2 * (NT / WAVE);  // listed blocks (staging index, one byte each)
    static constexpr int XQ = IT + NT / 4;         // fp16, one vector: x of the quarter's block (fp32)
    static constexpr int WORDS = XQ + (MODE == M_F16 && NB == 1 ? NQ * 16 : 0);
};

// Raw bits of value i of a record's value array, and the per-lane value
// words of pull_rows (fp32: one per column; fp16: two per word).
typedef _Float16 h2_t __attribute__((ext_vector_type(2)));  // packed fp16 pair

template <int MODE>
__device__ __forceinline__ uint32_t value_raw(const uint8_t *vals, uint32_t i)
{
    if constexpr (MODE == M_F32) return ((const uint32_t *)vals)[i];
    else return ((const uint16_t *)vals)[i];
}
template <int MODE, int N>
__device__ __forceinline__ void put_value(uint32_t (&v)[N], int c, uint32_t raw)
{
    if constexpr (MODE == M_F32) v[c] = raw;
    else if ((c & 1) == 0) v[c >> 1] = raw;
    else v[c >> 1] |= raw << 16;
}
template <int MODE, int N>
__device__ __forceinline__ float get_value(const uint32_t (&v)[N], int c)
{
    if constexpr (MODE == M_F32) return __uint_as_float(v[c]);
    else return h2f((uint16_t)(v[c >> 1] >> ((c & 1) * 16)));
}

// Row r's matching values of a ForceCSR / patched-CSR (row view) or
// ForceCSC (column view, header hs in LDS) block from its value array.
template <int MODE, int N>
__device__ __forceinline__ void row_values(const uint8_t *vals, bool colview, const uint32_t *hs, uint32_t rm,
                                           uint32_t rs, uint32_t mx, uint32_t r, bool on, uint32_t (&v)[N])
{
    if (colview) {
#pragma unroll
        for (int c = 0; c < 16; ++c) {
            const uint32_t m = (hs[c >> 1] >> ((c & 1) * 16)) & 0xFFFFu;
            const uint32_t st = (hs[8 + (c >> 2)] >> ((c & 3) * 8)) & 0xFFu;
            const bool ld = on && (((mx >> c) & (m >> r)) & 1u);
            put_value<MODE>(v, c, ld ? value_raw<MODE>(vals, st + __popc(m & ((1u << r) - 1u))) : 0u);
        }
    } else {
#pragma unroll
        for (int c = 0; c < 16; ++c) {
            const bool ld = on && (((rm & mx) >> c) & 1u);
            put_value<MODE>(v, c, ld ? value_raw<MODE>(vals, rs + __popc(rm & ((1u << c) - 1u))) : 0u);
        }
    }
}

// A round's chunk bounds and block row for thread t (chunk c0 + t / 16 of
// the round starting at chunk c0), so that a caller can issue the first
// round's loads before anything else it waits for.
struct RowsPre {
    int32_t h0, h1, R;
    bool valid;
};
__device__ __forceinline__ RowsPre rows_pre(const MainArgs &a, int64_t c0)
{
    const int cs = threadIdx.x >> 4;
    const int64_t ch = c0 + cs;
    RowsPre p;
    p.valid = cs < a.cpw && ch < a.nchunk;
    p.h0 = p.valid ? a.hv_cstart[ch] : 0;
    p.h1 = p.valid ? a.hv_cstart[ch + 1] : 0;
    p.R = p.valid ? a.hv_crow[ch] : 0;
    return p;
}

// NB > 1 (valued modes): NB vectors at once (batched decoding): the blocks
// active for any of them are visited, each row value is loaded once and
// multiplied with the NB dense x (zeros where a vector has no entry), and
// the NB sums go to NB accumulator sets (x and accumulators NB-strided).
// XL: the vector-block masks come from an LDS table (16 bits per vector
// block, after the activity bitmap: see k_rows_dx) instead of xmask.
// DOUT: the pass also writes the dense output (see k_rows_dx).
template <int MODE, bool LDSBITS, int NB = 1, bool XL = false, bool DOUT = false>
__device__ __forceinline__ void pull_rows(const MainArgs &a, uint32_t *L, const RowsPre *first = nullptr)
{
    using Y = RowsLds<MODE, NB>;
    static_assert(NB == 1 || valued<MODE>(), "batched pull is for valued modes");
    const int t = threadIdx.x, lane = lane_id(), wv = t >> 6, cs = t >> 4;
    const uint32_t r = (uint32_t)t & 15u;
    double *acc = (double *)(L + Y::AC);
    int32_t *pacc = (int32_t *)(L + Y::AC);
    uint8_t *items = (uint8_t *)(L + Y::IT);
    uint8_t *qvals = (uint8_t *)(L + Y::VB) + cs * HV_VAL_BYTES;
    constexpr int VW = MODE == M_F16 ? 8 : 16;
    for (int64_t c0 = (int64_t)blockIdx.x * a.cpw; c0 < a.nchunk; c0 += (int64_t)gridDim.x * a.cpw) {
        // 1. metadata, headers and x masks of the round's blocks; the list of the active ones
        const RowsPre rp = (first && c0 == (int64_t)blockIdx.x * a.cpw) ? *first : rows_pre(a, c0);
        const bool valid = rp.valid;
        const int32_t h0 = rp.h0, h1 = rp.h1, R = rp.R;
        const uint32_t am = valid ? row_admit(a, R) : 0u;
        const int32_t h = h0 + (int32_t)r;
        bool act = h < h1 && am != 0;
        // block column and descriptor together (one round trip)
        const int32_t J = act ? a.hv_col[h] : 0;
        const uint64_t d = act ? a.hv_desc[h] : 0ull;
        if constexpr (LDSBITS) act = act && block_active(J);
        uint32_t mx = 0u;
        if constexpr (XL) mx = act ? (uint32_t)((const uint16_t *)(lds_bits + ((a.nbc + 31) >> 5)))[J] : 0u;
        else mx = act ? mask16(a.xmask, J) : 0u;
        // with the activity bitmap in LDS an active block's mask is nonzero,
        // so its header loads go out with the mask's
        if constexpr (!LDSBITS) act = act && mx != 0;
        if (act) {
            const uint4 *hp = (const uint4 *)(a.pay + desc_off(d));
            const uint4 m0 = hp[0], m1 = hp[1];
            const uint4 st = desc_type(d) == T_DENSE ? make_uint4(0, 0, 0, 0) : hp[2];
            uint32_t *dst = L + Y::ST + t * HV_WORDS;
            dst[0] = m0.x; dst[1] = m0.y; dst[2] = m0.z; dst[3] = m0.w;
            dst[4] = m1.x; dst[5] = m1.y; dst[6] = m1.z; dst[7] = m1.w;
            dst[8] = st.x; dst[9] = st.y; dst[10] = st.z; dst[11] = st.w;
            dst[12] = mx | (am << 16);
            dst[13] = (uint32_t)J;
            dst[14] = (uint32_t)d;
            dst[15] = (uint32_t)(d >> 32);
        }
        if constexpr (valued<MODE>()) {
#pragma unroll
            for (int b = 0; b < NB; ++b) acc[b * TPB + t] = 0.0;
        } else {
            pacc[t] = INT_MAX;
        }
        if (r == 0) {
            L[Y::HM + cs] = 0u;
            L[Y::CR + cs] = valid ? (uint32_t)R : 0xFFFFFFFFu;
        }
        // the list holds the Dense blocks first, so that the four quarters of
        // a wave mostly take blocks of one kind at a time (the Dense and the
        // other formats' code paths are not both run)
        const bool dn = desc_type(d) == T_DENSE;
        const uint64_t bmd = ballot(act && dn), bmo = ballot(act && !dn);
        if (lane == 0) {
            L[Y::NI + wv] = (uint32_t)__popcll(bmd);
            L[Y::NI + TPB / WAVE + wv] = (uint32_t)__popcll(bmo);
        }
        __syncthreads();
        uint32_t based = 0, baseo = 0, totd = 0, total = 0;
#pragma unroll
        for (int w = 0; w < TPB / WAVE; ++w) {
            const uint32_t cd = L[Y::NI + w], co = L[Y::NI + TPB / WAVE + w];
            based += w < wv ? cd : 0u;
            baseo += w < wv ? co : 0u;
            totd += cd;
            total += cd + co;
        }
        const uint64_t below = (1ull << lane) - 1ull;
        if (act) items[dn ? based + __popcll(bmd & below) : totd + baseo + __popcll(bmo & below)] = (uint8_t)t;
        __syncthreads();
        // 2. the listed blocks, round-robin over the quarter-waves
        for (uint32_t it = (uint32_t)cs; ballot(it < total); it += Y::NQ) {
            const bool blk = it < total;  // the quarter has a block
            const int src = blk ? items[it] : 0;
            const uint32_t *hs = L + Y::ST + src * HV_WORDS;
            const int csB = src >> 4;
            const uint32_t mxB = hs[12] & 0xFFFFu;
            const bool on = blk && ((hs[12] >> (16 + r)) & 1u);  // and lane r's row is admitted
            const int32_t JB = (int32_t)hs[13];
            const uint64_t dB = (uint64_t)hs[14] | ((uint64_t)hs[15] << 32);
            const uint32_t type = desc_type(dB), nnz = desc_nnz(dB);
            const uint32_t rm = (hs[r >> 1] >> ((r & 1) * 16)) & 0xFFFFu;   // row r's mask
            const uint32_t rs = (hs[8 + (r >> 2)] >> ((r & 3) * 8)) & 0xFFu;  // row r's start
            const bool colview = type == T_FCSC;
            uint32_t w[16], v[VW];
            bool staged = false;
            float sb1 = 0.f;  // fp16, one vector: row r's share, formed below
            if constexpr (MODE == M_F16 && NB == 1) {
                const uint8_t *rec = a.pay + desc_off(dB);
                const uint8_t *vals = rec + values_at(type, nnz);
                const uint4 *xp = (const uint4 *)((const uint8_t *)a.xd + (int64_t)JB * BS * 2);
                if (type == T_DENSE) {
                    // 16 values of row r against the 16 x, the pairs outside
                    // the stored entries with a stored x masked to 0, two
                    // products per packed dot instruction
                    const uint32_t cm = rm & mxB;
                    const uint4 *vp = (const uint4 *)(rec + HDR_START + r * BS * 2);
#pragma unroll
                    for (int k = 0; k < 2; ++k) {
                        const uint4 z = on ? xp[k] : make_uint4(0, 0, 0, 0);
                        const uint4 u = on ? vp[k] : make_uint4(0, 0, 0, 0);
                        w[4 * k] = z.x; w[4 * k + 1] = z.y; w[4 * k + 2] = z.z; w[4 * k + 3] = z.w;
                        v[4 * k] = u.x; v[4 * k + 1] = u.y; v[4 * k + 2] = u.z; v[4 * k + 3] = u.w;
                    }
#pragma unroll
                    for (int p2 = 0; p2 < 8; ++p2) {
                        const uint32_t keep = (((cm >> (2 * p2)) & 1u) ? 0x0000FFFFu : 0u) |
                                              (((cm >> (2 * p2 + 1)) & 1u) ? 0xFFFF0000u : 0u);
                        sb1 = __builtin_amdgcn_fdot2(__builtin_bit_cast(h2_t, v[p2] & keep),
                                                     __builtin_bit_cast(h2_t, w[p2] & keep), sb1, false);
                    }
                } else if (nnz * 2 <= HV_VAL_BYTES) {
                    // the block's value array and its 16 x into the quarter's
                    // LDS buffers (every lane of the quarter helps); then lane
                    // r walks its matching entries only
                    const uint32_t nq = (nnz * 2 + 15) / 16;
                    if (blk && r < nq) ((uint4 *)qvals)[r] = ((const uint4 *)vals)[r];
                    if (blk) {
                        const uint16_t xr = ((const uint16_t *)xp)[r];
                        ((float *)(L + Y::XQ))[cs * 16 + r] = ((mxB >> r) & 1u) ? h2f(xr) : 0.f;
                    }
                    staged = true;
                } else {
                    constexpr int NX = 2;
#pragma unroll
                    for (int k = 0; k < NX; ++k) {
                        const uint4 z = on ? xp[k] : make_uint4(0, 0, 0, 0);
                        w[4 * k] = z.x; w[4 * k + 1] = z.y; w[4 * k + 2] = z.z; w[4 * k + 3] = z.w;
                    }
                    row_values<MODE>(vals, colview, hs, rm, rs, mxB, r, on, v);
                    uint32_t cand = rm & mxB;
                    if (colview) {
                        cand = 0;
#pragma unroll
                        for (int c = 0; c < 16; ++c) {
                            const uint32_t m = (hs[c >> 1] >> ((c & 1) * 16)) & 0xFFFFu;
                            cand |= (((mxB >> c) & (m >> r)) & 1u) << c;
                        }
                    }
#pragma unroll
                    for (int c = 0; c < 16; ++c)
                        if ((cand >> c) & 1u) sb1 = fmaf(get_value<MODE>(v, c), get_value<MODE>(w, c), sb1);
                }
                if (ballot(staged)) {
                    wave_lds_sync();
                    if (staged && on) {
                        const uint16_t *q16 = (const uint16_t *)qvals;
                        const float *xq = (const float *)(L + Y::XQ) + cs * 16;
                        if (colview) {
                            // ForceCSC: row r's entry in each matching column
#pragma unroll 1
                            for (uint32_t mm = mxB; mm;) {
                                const uint32_t c = ctz32(mm);
                                mm &= mm - 1u;
                                const uint32_t m = (hs[c >> 1] >> ((c & 1) * 16)) & 0xFFFFu;
                                if ((m >> r) & 1u) {
                                    const uint32_t st = (hs[8 + (c >> 2)] >> ((c & 3) * 8)) & 0xFFu;
                                    sb1 = fmaf(h2f(q16[st + __popc(m & ((1u << r) - 1u))]), xq[c], sb1);
                                }
                            }
                        } else {
#pragma unroll 1
                            for (uint32_t mm = rm & mxB; mm;) {
                                const uint32_t c = ctz32(mm);
                                mm &= mm - 1u;
                                sb1 = fmaf(h2f(q16[rs + __popc(rm & ((1u << c) - 1u))]), xq[c], sb1);
                            }
                        }
                    }
                    wave_lds_sync();  // the buffers are refilled for the next block
                }
            } else if constexpr (valued<MODE>()) {
                const uint8_t *rec = a.pay + desc_off(dB);
                constexpr int NX = MODE == M_F32 ? 4 : 2;
                const uint4 *xp = (const uint4 *)((const uint8_t *)a.xd + (int64_t)JB * BS * VT<MODE>::VB);
#pragma unroll
                for (int k = 0; k < NX; ++k) {
                    const uint4 z = on ? xp[k] : make_uint4(0, 0, 0, 0);
                    w[4 * k] = z.x; w[4 * k + 1] = z.y; w[4 * k + 2] = z.z; w[4 * k + 3] = z.w;
                }
                const uint8_t *vals = rec + values_at(type, nnz);
                if (type == T_DENSE) {
                    const uint4 *vp = (const uint4 *)(rec + HDR_START + r * BS * VT<MODE>::VB);
#pragma unroll
                    for (int k = 0; k < VW / 4; ++k) {
                        const uint4 z = on ? vp[k] : make_uint4(0, 0, 0, 0);
                        v[4 * k] = z.x; v[4 * k + 1] = z.y; v[4 * k + 2] = z.z; v[4 * k + 3] = z.w;
                    }
                } else if (MODE == M_F16 && nnz * 2 <= HV_VAL_BYTES) {
                    // the block's value array into the quarter's LDS buffer,
                    // 16 bytes per lane (every lane of the quarter helps)
                    const uint32_t nq = (nnz * 2 + 15) / 16;
                    if (blk && r < nq) ((uint4 *)qvals)[r] = ((const uint4 *)vals)[r];
                    staged = true;
                } else {
                    row_values<MODE>(vals, colview, hs, rm, rs, mxB, r, on, v);
                }
                if (ballot(staged)) {
                    wave_lds_sync();
                    if (staged) row_values<MODE>(qvals, colview, hs, rm, rs, mxB, r, on, v);
                    wave_lds_sync();  // the buffer is refilled for the next block
                }
            }
            if (on) {
                uint32_t cand = rm & mxB;
                if (colview) {
                    cand = 0;
#pragma unroll
                    for (int c = 0; c < 16; ++c) {
                        const uint32_t m = (hs[c >> 1] >> ((c & 1) * 16)) & 0xFFFFu;
                        cand |= (((mxB >> c) & (m >> r)) & 1u) << c;
                    }
                }
                if (cand) {
                    atomicOr(&L[Y::HM + csB], 1u << r);
                    if constexpr (MODE == M_F16 && NB == 1) {
                        atomicAdd(&acc[csB * 16 + r], (double)sb1);
                    } else if constexpr (valued<MODE>()) {
#pragma unroll
                        for (int b = 0; b < NB; ++b) {
                            if (b > 0) {
                                // vector b's x words (vector 0's were loaded with the values)
                                constexpr int NX = MODE == M_F32 ? 4 : 2;
                                const uint4 *xp = (const uint4 *)((const uint8_t *)a.xd +
                                                                  ((int64_t)b * a.xstride + (int64_t)JB * BS) *
                                                                      VT<MODE>::VB);
#pragma unroll
                                for (int k = 0; k < NX; ++k) {
                                    const uint4 z = xp[k];
                                    w[4 * k] = z.x; w[4 * k + 1] = z.y; w[4 * k + 2] = z.z; w[4 * k + 3] = z.w;
                                }
                            }
                            float sb = 0.f;
#pragma unroll
                            for (int c = 0; c < 16; ++c)
                                if ((cand >> c) & 1u) sb = fmaf(get_value<MODE>(v, c), get_value<MODE>(w, c), sb);
                            atomicAdd(&acc[(b * Y::NQ + csB) * 16 + r], (double)sb);
                        }
                    }
                    if constexpr (MODE == M_BFS) atomicMin(&pacc[csB * 16 + r], JB * BS + (int32_t)ctz32(cand));
                }
            }
        }
        __syncthreads();
        // 3. one commit per row and run of the round's chunks of one block row
        {
            const int c = cs;
            const uint32_t rr = r;
            const int32_t Rc = (int32_t)L[Y::CR + c];
            if (Rc >= 0 && (c == 0 || (int32_t)L[Y::CR + c - 1] != Rc)) {
                double sum[NB];
#pragma unroll
                for (int b = 0; b < NB; ++b) sum[b] = 0.0;
                int32_t pm = INT_MAX;
                uint32_t run = 0;
                int32_t nrun = 0;  // chunks in the run
                // the run's chunks CG at a time, their LDS reads issued together
                constexpr int CG = NB == 1 ? 4 : 1;
                bool in = true;
                for (int c0 = c; in && c0 < Y::NQ; c0 += CG) {
                    int32_t crs[CG];
                    uint32_t hms[CG];
                    double vs[NB][CG];
                    int32_t pms[CG];
#pragma unroll
                    for (int j = 0; j < CG; ++j) {
                        const int cc = c0 + j;
                        const bool ok = cc < Y::NQ;
                        crs[j] = ok ? (int32_t)L[Y::CR + cc] : -1;
                        hms[j] = ok ? L[Y::HM + cc] : 0u;
                        if constexpr (valued<MODE>()) {
#pragma unroll
                            for (int b = 0; b < NB; ++b) vs[b][j] = ok ? acc[(b * Y::NQ + cc) * 16 + rr] : 0.0;
                        } else {
                            pms[j] = ok ? pacc[cc * 16 + rr] : INT_MAX;
                        }
                    }
#pragma unroll
                    for (int j = 0; j < CG; ++j) {
                        in = in && crs[j] == Rc;
                        if (!in) break;
                        ++nrun;
                        run |= hms[j];
                        if ((hms[j] >> rr) & 1u) {
                            if constexpr (valued<MODE>()) {
#pragma unroll
                                for (int b = 0; b < NB; ++b) sum[b] += vs[b][j];
                            } else {
                                pm = min(pm, pms[j]);
                            }
                        }
                    }
                }
                if ((run >> rr) & 1u) {
                    const int64_t row = (int64_t)Rc * BS + rr;
                    if constexpr (valued<MODE>()) {
#pragma unroll
                        for (int b = 0; b < NB; ++b) atomicAdd(&a.yacc[(int64_t)b * a.ystride + row], sum[b]);
                    }
                    if constexpr (MODE == M_BFS) atomicMin(&a.parent[row], pm);
                }
                if constexpr (DOUT) {
                    // Count the run's chunks once its adds have completed:
                    // they are device-scope atomics, complete when the wave's
                    // memory counter drains, so no cache write-back (a
                    // release fence) is needed.  The workgroup that
                    // completes the block row converts its rows, taking each
                    // sum and clearing it in one atomic exchange (performed
                    // where the adds were), and clears the count.
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
                    __builtin_amdgcn_s_waitcnt(0);
                    uint32_t last = 0;
                    if (rr == 0) last = atomicAdd(&a.rdone[Rc], nrun) + nrun == a.rowchunks[Rc] ? 1u : 0u;
                    last = (uint32_t)__shfl((int)last, lane & ~15, WAVE);
                    if (last) {
                        const int64_t row = (int64_t)Rc * BS + rr;
                        if (row < a.m) {
                            const double v = atomicExch(&a.yacc[row], 0.0);
                            if constexpr (MODE == M_F32) ((float *)a.ydense)[row] = (float)v;
                            else ((uint16_t *)a.ydense)[row] = f64_to_f16_rne(v);
                            if (a.y32) a.y32[row] = (float)v;
                        }
                        if (rr == 0) atomicExch(&a.rdone[Rc], 0);
                    }
                } else {
                    if (rr == 0 && run) or_mask16(a.ybits, Rc, run);
                }
            }
        }
        __syncthreads();  // the next round overwrites the staging
    }
}

// Segment loop tasks.  An iteration of a wave takes 4 spq consecutive
// segments, spq per quarter (SLOTS when there is enough work to keep every
// wave busy with that many, else 1), so that the wave reads one contiguous
// stretch of slots; a wave task is G consecutive iterations' worth, tasks
// dealt out grid-stride.  Each quarter follows the block row of its segments
// through the task and folds the segments of one row in registers, so that a
// row is committed (fp64 atomics: other quarters, tasks and the non-COO pass
// add to the same rows) once per quarter and stretch of the task it covers.
// G is at most PULL_TASK_ITERS and leaves every wave about
// PULL_TASKS_PER_WAVE tasks: longer tasks fold more but balance the waves
// worse (R-MAT workloads concentrate their heavy segments in a few block
// rows).  The Boolean modes keep G = 1: a BFS level commits few rows, and
// longer tasks only unbalanced its levels.
#ifndef PULL_TASK_ITERS
#define PULL_TASK_ITERS 2
#endif
#ifndef PULL_TASKS_PER_WAVE
#define PULL_TASKS_PER_WAVE 4
#endif

#ifndef ORDER_MODES
#define ORDER_MODES(M) valued<M>()
#endif
template <int MODE, bool LDSBITS>
__device__ __forceinline__ void pull_loop(const MainArgs &a, int gw, int nw, float *sy, int32_t *sp, HeavyStage<false> *hs,
                          bool spec)
{
    const int lane = lane_id(), q = lane >> 4, i = lane & 15;
    constexpr int IM = inline_max<MODE>();
    // (segment ids fit 32 bits: the upload keeps 16 nseg below 2^31)
    const int32_t nseg = (int32_t)a.nseg;
    static_assert(PULL_TASK_SEGS % (4 * SLOTS) == 0, "a task is whole iterations");
    const int32_t spq = nseg >= nw * 4 * SLOTS * 2 ? SLOTS : 1, W = 4 * spq;
    // the matrix's task order (tasks of PULL_TASK_SEGS segments) when an
    // iteration takes 4 SLOTS segments; else G iterations per task in
    // segment order
    const bool ordered = ORDER_MODES(MODE) && a.torder != nullptr && spq == SLOTS;
    int32_t G, ntask;
    if (ordered) {
        G = PULL_TASK_SEGS / W;
        ntask = a.ntask;
    } else {
        G = nseg / (nw * W * PULL_TASKS_PER_WAVE);
        constexpr int32_t GMAX = valued<MODE>() ? PULL_TASK_ITERS : 1;
        G = G < 1 ? 1 : (G > GMAX ? GMAX : G);
        ntask = (nseg + G * W - 1) / (G * W);
    }
    // Boolean modes with an output mask and one 16-segment iteration per
    // task (BFS levels, masked OR-AND calls): a wave first reads the block
    // rows of the segments of its next PRE_TASKS tasks and their admitted
    // rows, four consecutive segments per lane (lane 4 j + p: segments
    // 4 p .. 4 p + 3 of the j-th task), and then skips the tasks none of whose
    // rows is admitted without reading their slots; in the other tasks a
    // segment without admitted rows reads no slot.  Once most rows have been
    // reached (the BFS levels after the largest), most segments belong to
    // such block rows.
    constexpr int32_t PRE_TASKS = WAVE / 4;
    const bool pre = !valued<MODE>() && a.omask != nullptr && !ordered && G == 1 && spq == SLOTS;
    uint32_t pre_am01 = 0u, pre_am23 = 0u;  // admitted rows of the lane's segments, two per word
    uint64_t pre_live = 0ull;               // bit 4 j + p: one of lane 4 j + p's segments has some
    // ordered tasks are dealt out by rank in snake order: round j gives rank
    // j nw + nw - 1 - gw to wave gw for even j and j nw + gw for odd j (the
    // first workgroups also take the first chunks of the non-COO pass);
    // tasks in segment order grid-stride
    for (int32_t r0 = 0; r0 < ntask; r0 += nw) {
        const int32_t pj = (r0 / nw) % PRE_TASKS;
        if (pre && pj == 0) {
            const int32_t rj = r0 + (lane >> 2) * nw + gw;
            const int64_t sid = (int64_t)rj * 16 + (lane & 3) * 4;
            uint32_t rs[4] = {0u, 0u, 0u, 0u};
            if (rj < ntask) {
                if (sid + 4 <= nseg) {
                    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
                    const u32x4 v = __builtin_nontemporal_load((const u32x4 *)(a.seg_rs + sid));
                    rs[0] = v.x;
                    rs[1] = v.y;
                    rs[2] = v.z;
                    rs[3] = v.w;
                } else {
#pragma unroll
                    for (int k = 0; k < 4; ++k) rs[k] = sid + k < nseg ? a.seg_rs[sid + k] : 0u;
                }
            }
            uint32_t am4[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) am4[k] = (rj < ntask && sid + k < nseg) ? row_admit(a, (int32_t)rs[k]) : 0u;
            pre_am01 = am4[0] | (am4[1] << 16);
            pre_am23 = am4[2] | (am4[3] << 16);
            pre_live = ballot((pre_am01 | pre_am23) != 0u);
        }
        const int32_t r = r0 + ((!ordered || ((r0 / nw) & 1)) ? gw : nw - 1 - gw);
        if (r >= ntask) continue;
        if (pre && ((pre_live >> (pj * 4)) & 0xFull) == 0ull) continue;
        const int32_t task = ordered ? a.torder[r] : r;
        const int32_t ts = task * G * W + q * spq;
        // the open run of the quarter: its block row, lane i's share of row
        // i (fp64 across segments) and the rows hit
        int32_t Rc = -1;
        double racc = 0.0;
        int32_t pacc = INT_MAX;
        uint32_t hc = 0;
        auto commit = [&]() {
            if (Rc < 0) return;
            if ((hc >> i) & 1u) {
                const int64_t row = (int64_t)Rc * BS + i;
                if constexpr (valued<MODE>()) atomicAdd(&a.yacc[row], racc);
                if constexpr (MODE == M_BFS) atomicMin(&a.parent[row], pacc);
            }
            if (i == 0 && hc) or_mask16(a.ybits, Rc, hc);
        };
        for (int32_t it = 0; it < G; ++it) {
            uint32_t s[SLOTS];
            uint64_t d[SLOTS];
            bool vs[SLOTS], act[SLOTS];
            int32_t b[SLOTS], J[SLOTS];
            uint32_t am[SLOTS], mx[SLOTS];
            // segment word, block column and (spec) descriptor: independent
            // loads, non-temporal (each slot is read once per call), so that
            // the stream does not push x out of the L2
            uint32_t a01 = 0u, a23 = 0u;
            if (pre) {
                a01 = (uint32_t)__shfl((int)pre_am01, pj * 4 + q, WAVE);
                a23 = (uint32_t)__shfl((int)pre_am23, pj * 4 + q, WAVE);
            }
#pragma unroll
            for (int k = 0; k < SLOTS; ++k) {
                const int32_t sid = ts + it * W + k;
                vs[k] = k < spq && sid < nseg;
                bool live = vs[k];
                s[k] = vs[k] ? __builtin_nontemporal_load(&a.seg_rs[sid]) : 0u;
                if (pre) {
                    // segment 4 q + k of the task: lane 4 pj + q above, its k-th
                    const uint32_t w2 = k < 2 ? a01 : a23;
                    am[k] = (k & 1) ? (w2 >> 16) : (w2 & 0xFFFFu);
                    live = live && am[k] != 0u;
                }
                b[k] = sid * 16 + i;
                const int32_t w = live ? __builtin_nontemporal_load(&a.sl_col[b[k]]) : SLOT_PAD;
                J[k] = w >= 0 ? slot_col(w) : -1;
                d[k] = (live && spec) ? __builtin_nontemporal_load(&a.sl_desc[b[k]]) : 0ull;
            }
            // block activity: the LDS bitmap when it fits, else the
            // vector-block mask (gathered here then, and kept for the
            // whole-wave blocks)
#pragma unroll
            for (int k = 0; k < SLOTS; ++k) {
                if (!pre) am[k] = vs[k] ? row_admit(a, (int32_t)s[k]) : 0u;
                act[k] = J[k] >= 0 && am[k] != 0;
                if constexpr (LDSBITS) act[k] = act[k] && block_active(J[k]);
            }
            if constexpr (!LDSBITS) {
#pragma unroll
                for (int k = 0; k < SLOTS; ++k) {
                    mx[k] = act[k] ? mask16(a.xmask, J[k]) : 0u;
                    act[k] = act[k] && mx[k] != 0;
                }
            }
            if (!spec) {
#pragma unroll
                for (int k = 0; k < SLOTS; ++k) d[k] = act[k] ? __builtin_nontemporal_load(&a.sl_desc[b[k]]) : 0ull;
            }
            // with nothing to multiply anywhere in the wave the LDS rows stay
            // untouched; the runs are still followed
            const bool any = ballot(act[0] || act[1] || act[2] || act[3]) != 0;
            uint32_t hq[SLOTS];
            if (any) {
                // Issue every gather that depends only on the descriptors at
                // once: x of the entries of the inline COO blocks (one lane
                // each) and (in flat_pass) the records of the stored COO
                // blocks; the inline products are formed while the record
                // loads are in flight.  Blocks of the other formats are not in
                // the slots' work (negative block column): pull_rows takes them.
                uint32_t hit[SLOTS], cnt[SLOTS];
                uint32_t xr[SLOTS][IM];
#pragma unroll
                for (int k = 0; k < SLOTS; ++k) {
                    const bool inl = act[k] && desc_inline(d[k]);
                    const uint32_t nnz = desc_nnz(d[k]);
                    if constexpr (!LDSBITS && !valued<MODE>()) {
                        // the vector-block mask is already here: it is the x word
                        xr[k][0] = mx[k] << ((J[k] & 1) * 16);
                    } else {
#pragma unroll
                        for (int e = 0; e < IM; ++e)
                            xr[k][e] = (inl && (uint32_t)e < nnz)
                                           ? x_gather<MODE>(a, J[k], inline_cd(d[k], e, a.vb) & 15u)
                                           : 0u;
                    }
                    const bool flat = act[k] && flat_coo(d[k]);
                    cnt[k] = flat ? nnz : 0u;
                    if (flat) hs->stage(k * WAVE + lane, d[k], J[k], LDSBITS ? 0u : mx[k], am[k], 0);
                }
                auto inline_products = [&]() {
#pragma unroll
                    for (int k = 0; k < SLOTS; ++k) {
                        hit[k] = 0;
                        if (act[k] && desc_inline(d[k]))
                            hit[k] = inline_block<MODE>(a, d[k], J[k], am[k], xr[k], sy + k * WAVE + q * 16,
                                                        sp + k * WAVE + q * 16);
                    }
                };
                if (ballot(cnt[0] | cnt[1] | cnt[2] | cnt[3])) {
                    wave_lds_sync();
                    flat_pass<MODE, false, !LDSBITS, false, false>(a, hs, cnt, d, sy, sp, inline_products);
#pragma unroll
                    for (int k = 0; k < SLOTS; ++k) hit[k] |= hs->hitw[k * 4 + q];
                } else {
                    inline_products();
                }
                wave_lds_sync();
#pragma unroll
                for (int k = 0; k < SLOTS; ++k) hq[k] = or16_in_quarter(hit[k]);
            }
            // follow the runs: a new block row commits the open run and opens
            // the next one
#pragma unroll
            for (int k = 0; k < SLOTS; ++k) {
                if (vs[k]) {
                    const int32_t R = (int32_t)s[k];
                    if (R != Rc) {
                        commit();
                        Rc = R;
                        racc = 0.0;
                        pacc = INT_MAX;
                        hc = 0;
                    }
                    if (any) {
                        hc |= hq[k];
                        if constexpr (valued<MODE>()) racc += (double)sy[k * WAVE + lane];
                        if constexpr (MODE == M_BFS) pacc = min(pacc, sp[k * WAVE + lane]);
                    }
                }
                if (any) {
                    if constexpr (valued<MODE>()) sy[k * WAVE + lane] = 0.f;
                    if constexpr (MODE == M_BFS) sp[k * WAVE + lane] = INT_MAX;
                }
            }
            if (any) wave_lds_sync();
        }
        commit();
    }
}

// Compacted pull.  Below an activity threshold most slots of a segment have
// nothing to multiply, and the segment loop pays its full chain of dependent
// loads for a few useful lanes.  Instead, the pull kernel compacts the slots
// with work into a list (pull_compact; k_pull_compact when the bitmap is too
// large for the pull kernel's LDS copy) alongside the non-COO blocks, and the
// push kernel runs the same block work over the list (pull_active), 256
// active slots per wave and round, with the products summed per run of one
// block row in LDS before the commit.  Used while
// N_nzblk / N_blk is below PULL_COMPACT_PERMILLE / 1000 (the slot activity
// roughly follows it; PULL_COMPACT_PERMILLE_BOOL for the Boolean modes).
#ifndef PULL_COMPACT_PERMILLE
#define PULL_COMPACT_PERMILLE 400
#endif
// Boolean modes (BFS levels) do less per active slot, so the segment loop
// stays ahead of the list down to a lower activity
#ifndef PULL_COMPACT_PERMILLE_BOOL
#define PULL_COMPACT_PERMILLE_BOOL 150
#endif
// The compaction tests activity in an LDS copy of the bitmap; without one
// (more vector blocks than this many bits) the segment loop is used.
constexpr int32_t COMPACT_BITMAP_WORDS = 8192;
// The segments are cut into nr regions of L = rcap / 16 consecutive
// segments (L a multiple of 64, so that a compaction round of one segment per
// lane never straddles two regions; as short as the count array, creg
// entries, and WALK_MAX_REGIONS regions per walk wave allow); a region holds
// up to rcap entries.  Wave w of the compaction fills regions w, w + nreg, ..;
// wave w of the walk takes the same regions, concatenated (they follow one
// another in slot order).  R-MAT matrices put most of their stored entries in
// a few block rows: short strided regions spread such a stretch over many
// waves of the walk instead of leaving it to one (R-MAT 20, regions of 64
// instead of 305 segments: 1% uniform 119 -> 106 us, 10% clustered 120 -> 110
// us, 1% clustered 59 -> 61 us).  False when the list is absent or too small.
#ifndef WALK_MAX_REGIONS
#define WALK_MAX_REGIONS 8
#endif
__device__ __forceinline__ bool compact_pull(const MainArgs &a, int32_t N, int64_t &rcap, int32_t &nr)
{
    const int64_t nw = a.nreg;
    const int64_t most = min((int64_t)a.creg, nw * WALK_MAX_REGIONS);
    const int64_t L = most > 0 ? 64 * ((a.nseg + 64 * most - 1) / (64 * most)) : 0;
    rcap = L * 16;
    nr = L > 0 ? (int32_t)((a.nseg + L - 1) / L) : 0;
    return a.clist != nullptr && a.nseg > 0 && nw > 0 && (int64_t)N * 1000 < (int64_t)a.nbc * a.cpm &&
           ((a.nbc + 31) >> 5) <= COMPACT_BITMAP_WORDS && (int64_t)nr * rcap <= a.clist_cap;
}

// First half: a wave takes the segments of region gw, one segment per lane
// and round (its 16 slot words by four 16-byte loads), and appends the slots
// that hold work -- a COO block (the listed
// non-COO blocks carry the sign bit) whose vector block is active, in an
// admitted block row -- to its region of the list, in slot order.  When x is
// spread (fewer than 4 indices per nonzero vector block on average, so that
// most single entries miss), a block whose single entry is held inline is
// listed only if x stores that entry's column (tested from the local column
// in the slot word against the vector block's mask).  The region's entry
// count goes to ccount[gw].  The activity bitmap is copied into LDS when it
// fits.
template <bool LDSBITS>
__device__ __forceinline__ void pull_compact(const MainArgs &a, int gw, int64_t rcap, int32_t N, int32_t xpop)
{
    const int lane = lane_id();
    const bool exact = (int64_t)xpop < 4 * (int64_t)N;
    const int64_t s0 = (int64_t)gw * (rcap / 16);
    const int64_t s1 = min(a.nseg, s0 + rcap / 16);
    int32_t *out = a.clist + s0 * 16;
    uint32_t n = 0;
    for (int64_t base = s0; base < s1; base += WAVE) {
        const int64_t sid = base + lane;
        uint32_t f = 0;
        if (sid < s1) {
            const int4 *p = (const int4 *)(a.sl_col + sid * 16);
            const int4 c0 = p[0], c1 = p[1], c2 = p[2], c3 = p[3];
            const uint32_t am = row_admit(a, (int32_t)a.seg_rs[sid]);
            const int32_t col[16] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w,
                                     c2.x, c2.y, c2.z, c2.w, c3.x, c3.y, c3.z, c3.w};
            if (am) {
                uint32_t one = 0;
                uint32_t m16[LDSBITS ? 1 : 16];
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int32_t J = slot_col(col[i]);
                    bool on = col[i] >= 0;
                    if constexpr (LDSBITS) {
                        on = on && block_active(J);
                    } else {
                        m16[i] = on ? mask16(a.xmask, J) : 0u;
                        on = m16[i] != 0u;
                    }
                    f |= (on ? 1u : 0u) << i;
                    one |= (exact && on && slot_one(col[i]) ? 1u : 0u) << i;
                }
                if (one) {
                    // (with the bitmap in LDS, the masks of all such slots of
                    // the segment are gathered together)
                    uint32_t mw[16];
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        if constexpr (LDSBITS) mw[i] = ((one >> i) & 1u) ? mask16(a.xmask, slot_col(col[i])) : 0u;
                        else mw[i] = m16[i];
                    }
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        if (((one >> i) & 1u) && !((mw[i] >> slot_c(col[i])) & 1u)) f &= ~(1u << i);
                }
            }
        }
        const uint32_t cnt = __popc(f), incl = wave_incl_add(cnt);
        uint32_t pos = n + incl - cnt;
        while (f) {
            const int i = ctz32(f);
            f &= f - 1;
            out[pos++] = (int32_t)(sid * 16 + i);
        }
        n += readlane_u32(incl, WAVE - 1);
    }
    if (lane == 0) a.ccount[gw] = n;
}

// The compaction as a kernel of its own, for activity bitmaps of more than
// LDS_BITMAP_WORDS words (the pull kernel then returns at once): it also
// takes the non-COO blocks (pull_rows), so that their chains overlap the
// compaction instead of preceding it.
template <int MODE>
__global__ __launch_bounds__(TPB) void k_pull_compact(MainArgs a)
{
    __shared__ __align__(16) uint32_t rows_lds[RowsLds<MODE, 1>::WORDS];
    const int32_t N = a.counters[C_NZBLK], xpop = a.counters[C_XPOP];
    int64_t rcap;
    int32_t nr;
    if (N == 0 || a.counters[C_PATH] != PATH_PULL || !compact_pull(a, N, rcap, nr)) return;
    // every wave of the grid (its resident size, more waves than the walk's
    // when this kernel's registers allow) takes regions gw, gw + nw, ..
    const int gw = blockIdx.x * (TPB / WAVE) + (threadIdx.x >> 6), nw = gridDim.x * (TPB / WAVE);
    const int32_t nwords = (a.nbc + 31) >> 5;
    if (nwords <= COMPACT_BITMAP_WORDS) {  // (always, by compact_pull)
        for (int32_t t = threadIdx.x; t < nwords; t += TPB) lds_bits[t] = a.xbits[t];
        __syncthreads();
        pull_rows<MODE, true>(a, rows_lds);
        for (int32_t r = gw; r < nr; r += nw) pull_compact<true>(a, r, rcap, N, xpop);
    } else {
        pull_rows<MODE, false>(a, rows_lds);
        for (int32_t r = gw; r < nr; r += nw) pull_compact<false>(a, r, rcap, N, xpop);
    }
}

// For each of SLOTS wave-uniform targets, the largest a in [0, n) with
// arr[a] <= target (arr increasing, arr[0] = 0 <= target): a 64-ary search in
// which the whole wave probes 64 positions per round (log64 n rounds), the
// SLOTS searches interleaved so that their loads overlap.  With WIDTH > 1 it
// stops at a window [res, res + WIDTH) that holds the answer.
template <int STRIDE, int WIDTH = 1>
__device__ __forceinline__ void wave_search(const int32_t *__restrict__ arr, int32_t n,
                                            const int32_t (&target)[SLOTS], const bool (&valid)[SLOTS],
                                            int32_t (&res)[SLOTS])
{
    const int lane = lane_id();
    int32_t lo[SLOTS], hi[SLOTS];
#pragma unroll
    for (int k = 0; k < SLOTS; ++k) {
        lo[k] = 0;
        hi[k] = valid[k] ? n : 1;  // an unused slot needs no search
    }
    for (;;) {
        bool more = false;
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) more |= hi[k] - lo[k] > WIDTH;
        if (!more) break;
        int32_t v[SLOTS], step[SLOTS], pi[SLOTS];
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) {
            step[k] = (hi[k] - lo[k] + WAVE - 1) / WAVE;
            pi[k] = lo[k] + lane * step[k];
            v[k] = (hi[k] - lo[k] > WIDTH && pi[k] < hi[k]) ? arr[(int64_t)pi[k] * STRIDE] : INT_MAX;
        }
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) {
            if (hi[k] - lo[k] <= WIDTH) continue;
            const uint64_t m = ballot(v[k] <= target[k]);  // lane 0 probes lo: always set
            const int L = 63 - __builtin_clzll(m);
            lo[k] += L * step[k];
            hi[k] = min(hi[k], lo[k] + step[k]);
        }
    }
#pragma unroll
    for (int k = 0; k < SLOTS; ++k) res[k] = lo[k];
}

// Push (Sec. 3.3.2): block tasks flattened over the block-CSC lists of the
// active column blocks; chunks of 64 consecutive tasks, one task per lane,
// up to SLOTS chunks per wave iteration, grid-stride.  The chunk's first
// work item comes from a wave search over the item starts (its last step
// taken on a loaded window of items); a lane then finds its own item by a
// 6-step binary search over the next 64 item starts, held one per lane and
// read by shuffles.
template <int MODE>
__device__ __forceinline__ void push_loop(const MainArgs &a, int gw, int nw, float *sy, int32_t *sp, HeavyStage<true> *hs,
                                          int32_t T, int32_t NT)
{
    const int lane = lane_id();
    const int64_t nchunks = ((int64_t)T + WAVE - 1) / WAVE;
    const int cpw = nchunks >= (int64_t)nw * SLOTS * 2 ? SLOTS : 1;
    for (int64_t u = gw; u * cpw < nchunks; u += nw) {
        int32_t t[SLOTS], a0[SLOTS], B[SLOTS], tgt[SLOTS];  // B: first task of the lane's item
        bool vt[SLOTS], vc[SLOTS];
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) {
            const int64_t c = u * cpw + k;
            vc[k] = k < cpw && c < nchunks;
            t[k] = (int32_t)(c * WAVE + lane);
            vt[k] = vc[k] && t[k] < T;
            tgt[k] = vc[k] ? (int32_t)(c * WAVE) : 0;
        }
        // the search narrows to a window of at most 64 items holding the
        // chunk's first item; the window and the 64 items after it are then
        // loaded whole (one round trip for the last search step and the
        // items), the first item a0 found among them, and lane l takes item
        // a0 + l (at most 63 further items start inside the chunk) by shuffles
        int32_t lo[SLOTS];
        wave_search<4, WAVE>((const int32_t *)a.items, NT, tgt, vc, lo);
        int32_t BJ[SLOTS], Bp[SLOTS];
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) {
            const int32_t w0 = lo[k] + lane, w1 = w0 + WAVE;
            const int4 i0 = (vc[k] && w0 < NT) ? a.items[w0] : make_int4(INT_MAX, 0, 0, 0);
            const int4 i1 = (vc[k] && w1 < NT) ? a.items[w1] : make_int4(INT_MAX, 0, 0, 0);
            const uint64_t m = ballot(i0.x <= tgt[k]);  // lane 0 (item lo) is always set for a valid chunk
            const int L = m ? 63 - __builtin_clzll(m) : 0;
            a0[k] = lo[k] + L;
            const int src = (L + lane) & (WAVE - 1);
            const bool hi = L + lane >= WAVE;
            const int32_t x0 = __shfl(i0.x, src, WAVE), x1 = __shfl(i1.x, src, WAVE);
            const int32_t y0 = __shfl(i0.y, src, WAVE), y1 = __shfl(i1.y, src, WAVE);
            const int32_t z0 = __shfl(i0.z, src, WAVE), z1 = __shfl(i1.z, src, WAVE);
            B[k] = hi ? x1 : x0;
            BJ[k] = hi ? y1 : y0;
            Bp[k] = hi ? z1 : z0;
        }
        int32_t J[SLOTS], p[SLOTS];
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) {
            int lo = 0;
#pragma unroll
            for (int st = 32; st > 0; st >>= 1) {
                const int32_t v = __shfl(B[k], (lo + st) & (WAVE - 1), WAVE);
                if (lo + st < WAVE && v <= t[k]) lo += st;
            }
            J[k] = __shfl(BJ[k], lo, WAVE);
            p[k] = __shfl(Bp[k], lo, WAVE) + t[k];
            if (!vt[k]) {
                J[k] = 0;
                p[k] = 0;
            }
        }
        int32_t R[SLOTS];
        uint32_t mx[SLOTS], am[SLOTS];
        bool act[SLOTS];
        uint64_t d[SLOTS];
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) {
            R[k] = vt[k] ? a.csc_row[p[k]] : 0;
            d[k] = vt[k] ? a.csc_desc[p[k]] : 0ull;
            mx[k] = vt[k] ? mask16(a.xmask, J[k]) : 0u;
        }
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) {
            am[k] = vt[k] ? row_admit(a, R[k]) : 0u;
            act[k] = vt[k] && am[k] != 0;
            if (!act[k]) d[k] = 0ull;
        }
        uint32_t hit[SLOTS], cnt[SLOTS];
        // the matching entries of stored COO blocks are read from their
        // coordinates (one more dependent load) only when the iteration's
        // COO records hold more than one window of the entry-parallel pass
        bool coo_live = false;
        if constexpr (MODE == M_F32) {
            uint32_t ce = 0;
#pragma unroll
            for (int k = 0; k < SLOTS; ++k)
                ce += (act[k] && !desc_inline(d[k]) && desc_type(d[k]) == T_COO) ? desc_nnz(d[k]) : 0u;
            coo_live = wave_sum(ce) > (uint32_t)COO_LIVE_WAVE;
        }
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) {
            hit[k] = 0;
            const bool lanework = act[k] && lane_coo(d[k]);
            if (lanework)
                hit[k] = inline_block_push<MODE>(a.vb, d[k], J[k], R[k], mx[k], am[k], a.xd, a.yacc, a.parent);
            // every block with a payload record (stored COO and the other
            // formats) goes to the entry-parallel pass; the block column
            // carries the format in its top bits there.  A COO record is
            // walked whole; of the others only the live entries, counted
            // from the record's masks
            const bool flat = act[k] && !desc_inline(d[k]);
            cnt[k] = flat ? desc_nnz(d[k]) : 0u;
            uint32_t tag = desc_type(d[k]), mword = mx[k] | (am[k] << 16);
            if (flat && desc_type(d[k]) != T_COO)
                cnt[k] = live_count(load_masks(a.pay + desc_off(d[k])), desc_type(d[k]), mx[k], am[k]);
            if constexpr (MODE == M_F32) {
                if (coo_live && flat && desc_type(d[k]) == T_COO && cnt[k] <= COO_LIVE_MAX && __popc(mx[k]) < 16) {
                    mword = coo_live_mask(a.pay + desc_off(d[k]), cnt[k], mx[k], am[k]);
                    cnt[k] = __popc(mword);
                    tag = T_COO_LIVE;
                }
            }
            if (cnt[k]) {
                hs->stage(k * WAVE + lane, d[k], J[k] | (int32_t)(tag << 28), 0u, 0u, R[k]);
                hs->mxam[k * WAVE + lane] = mword;
            }
        }
        if (ballot(cnt[0] | cnt[1] | cnt[2] | cnt[3])) {
            wave_lds_sync();
            flat_pass<MODE, true, true, true, false>(a, hs, cnt, d, sy, sp, [] {});
#pragma unroll
            for (int k = 0; k < SLOTS; ++k) if (cnt[k]) hit[k] |= hs->hitw[k * WAVE + lane];
            wave_lds_sync();
        }
#pragma unroll
        for (int k = 0; k < SLOTS; ++k)
            if (act[k] && hit[k]) or_mask16(a.ybits, R[k], hit[k]);
    }
}

// Second half of the compacted pull (run by the push kernel, whose grid has
// a wave per region: wave gw walks region gw).  A round takes the next 256
// entries, entry base + 64 k + lane in slot k of a lane, and numbers the runs of one block
// row among them (the list is in slot order, so block rows do not
// decrease); a round ends early at the first entry of run RUN_CAP.  Inline
// COO blocks are taken by their lane, stored COO blocks entry-parallel
// (flat_pass), both adding into the run's 16 LDS rows; then every run's rows
// hit are committed with one fp64 atomic each (grouped: the 16 lanes of a
// run cover one block row).
constexpr int RUN_CAP = 32;
struct ActiveLds {
    uint32_t acc[RUN_CAP * 16];  // per run: 16 row sums (fp32) or BFS minimum parents
    uint32_t hm[RUN_CAP];        // rows hit per run
    int32_t runR[RUN_CAP];       // block row of each run
    HeavyStage<true> hs;
};

template <int MODE>
__device__ __forceinline__ void pull_active(const MainArgs &a, ActiveLds &L, int gw, int64_t rcap, int32_t nr,
                                            int32_t N, int32_t xpop)
{
    const int lane = lane_id();
    float *sy = (float *)L.acc;
    int32_t *sp = (int32_t *)L.acc;
    constexpr uint32_t ACC0 = MODE == M_BFS ? (uint32_t)INT_MAX : 0u;
    for (int t = lane; t < RUN_CAP * 16; t += WAVE) L.acc[t] = ACC0;
    if (lane < RUN_CAP) L.hm[lane] = 0u;
    wave_lds_sync();
    // the wave's regions, concatenated (they follow one another in slot
    // order): entry e lies in region j with pre[j] <= e < pre[j + 1]
    constexpr int RPW = WALK_MAX_REGIONS;
    uint32_t pre[RPW + 1];
    pre[0] = 0;
#pragma unroll
    for (int j = 0; j < RPW; ++j) pre[j + 1] = pre[j] + (gw + j * a.nreg < nr ? a.ccount[gw + j * a.nreg] : 0u);
    const uint32_t cnt = pre[RPW];
    auto list_at = [&](uint32_t e) {
        int j = 0;
#pragma unroll
        for (int t = 1; t < RPW; ++t) j += e >= pre[t] ? 1 : 0;
        uint32_t pj = pre[0];
#pragma unroll
        for (int t = 1; t < RPW; ++t) pj = j == t ? pre[t] : pj;
        return a.clist[(int64_t)(gw + j * a.nreg) * rcap + (e - pj)];
    };
    constexpr int IM = inline_max<MODE>();
    // spread x (fewer than 4 indices per nonzero vector block on average):
    // a stored COO block's entries are tested against its vector block's
    // mask before x is gathered (the mask words are L2-resident, and most
    // entries then miss); the mask gathers go out with the inline blocks' x
    // gathers and are waited for only once the records' loads are in flight
    constexpr bool MXV = valued<MODE>();
    const bool mxf = MXV && (int64_t)xpop < 4 * (int64_t)N;
    for (uint32_t base = 0; base < cnt;) {
        bool v[SLOTS];
        int32_t slot[SLOTS];
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) {
            const uint32_t e = base + (uint32_t)(k * WAVE + lane);
            v[k] = e < cnt;
            slot[k] = v[k] ? list_at(e) : 0;
        }
        int32_t J[SLOTS], R[SLOTS];
        uint64_t d[SLOTS];
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) {
            J[k] = v[k] ? slot_col(a.sl_col[slot[k]]) : -1;  // (listed slots are COO blocks)
            d[k] = v[k] ? a.sl_desc[slot[k]] : 0ull;
            R[k] = v[k] ? (int32_t)a.seg_rs[slot[k] >> 4] : -1;
        }
        // runs of one block row, in entry order (k major)
        uint32_t run[SLOTS];
        uint32_t nr = 0;
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) {
            const uint32_t last = k ? readlane_u32((uint32_t)R[k - 1], WAVE - 1) : 0xFFFFFFFFu;
            uint32_t prev = wave_shr1((uint32_t)R[k]);
            if (lane == 0) prev = last;
            const uint32_t fl = (v[k] && (uint32_t)R[k] != prev) ? 1u : 0u;
            const uint32_t inc = wave_incl_add(fl);
            run[k] = nr + inc - 1u;
            nr += readlane_u32(inc, WAVE - 1);
            // the first entry of each run records the run's block row
            if (fl && run[k] < (uint32_t)RUN_CAP) L.runR[run[k]] = R[k];
        }
        // the round ends before the first entry of run RUN_CAP
        uint32_t cut = SLOTS * WAVE;
#pragma unroll
        for (int k = SLOTS - 1; k >= 0; --k) {
            const uint64_t b = ballot(v[k] && run[k] >= (uint32_t)RUN_CAP);
            if (b) cut = (uint32_t)(k * WAVE + ctz64(b));
        }
        uint32_t am[SLOTS];
        bool act[SLOTS];
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) {
            v[k] = v[k] && (uint32_t)(k * WAVE + lane) < cut;
            am[k] = v[k] ? row_admit(a, R[k]) : 0u;
            act[k] = v[k] && am[k] != 0u && J[k] >= 0;
        }
        const uint32_t nruns = nr < (uint32_t)RUN_CAP ? nr : (uint32_t)RUN_CAP;
        uint32_t xr[SLOTS][IM];
        uint32_t cnf[SLOTS], mxg[SLOTS];
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) {
            const bool inl = act[k] && desc_inline(d[k]);
            const uint32_t nnz = desc_nnz(d[k]);
#pragma unroll
            for (int e = 0; e < IM; ++e)
                xr[k][e] = (inl && (uint32_t)e < nnz)
                               ? x_gather<MODE>(a, J[k], valued<MODE>() ? (inline_cd(d[k], e, a.vb) & 15u) : 0u)
                               : 0u;
            const bool flat = act[k] && flat_coo(d[k]);
            cnf[k] = flat ? nnz : 0u;
            mxg[k] = (MXV && flat && mxf) ? a.xmask[J[k] >> 1] : 0u;
            if (flat) L.hs.stage(k * WAVE + lane, d[k], J[k], MXV ? 0xFFFFu : 0u, am[k], (int32_t)run[k]);
        }
        auto inline_products = [&]() {
            if constexpr (MXV) {
                if (mxf) {
#pragma unroll
                    for (int k = 0; k < SLOTS; ++k)
                        if (cnf[k]) L.hs.mxam[k * WAVE + lane] = ((mxg[k] >> ((J[k] & 1) * 16)) & 0xFFFFu) | (am[k] << 16);
                    wave_lds_sync();
                }
            }
#pragma unroll
            for (int k = 0; k < SLOTS; ++k) {
                if (act[k] && desc_inline(d[k])) {
                    const uint32_t h = inline_block<MODE>(a, d[k], J[k], am[k], xr[k], sy + run[k] * 16,
                                                          sp + run[k] * 16);
                    if (h) atomicOr(&L.hm[run[k]], h);
                }
            }
        };
        if (ballot(cnf[0] | cnf[1] | cnf[2] | cnf[3])) {
            wave_lds_sync();
            flat_pass<MODE, true, MXV, false, true>(a, &L.hs, cnf, d, sy, sp, inline_products);
#pragma unroll
            for (int k = 0; k < SLOTS; ++k) {
                const uint32_t h = cnf[k] ? L.hs.hitw[k * WAVE + lane] : 0u;
                if (h) atomicOr(&L.hm[run[k]], h);
            }
        } else {
            inline_products();
        }
        wave_lds_sync();
        // commit: four runs at a time, lane i of a run's 16 lanes takes row i
        for (uint32_t rb = 0; rb < nruns; rb += 4) {
            const uint32_t r = rb + (uint32_t)(lane >> 4), i = (uint32_t)(lane & 15);
            if (r < nruns) {
                const uint32_t h = L.hm[r];
                const int32_t Rr = L.runR[r];
                if ((h >> i) & 1u) {
                    const int64_t row = (int64_t)Rr * BS + i;
                    if constexpr (valued<MODE>()) atomicAdd(&a.yacc[row], (double)sy[r * 16 + i]);
                    if constexpr (MODE == M_BFS) atomicMin(&a.parent[row], sp[r * 16 + i]);
                }
                if (i == 0 && h) or_mask16(a.ybits, Rr, h);
                L.acc[r * 16 + i] = ACC0;
            }
        }
        wave_lds_sync();
        if (lane < RUN_CAP) L.hm[lane] = 0u;
        wave_lds_sync();
        base += cut;
    }
}

// LDS of one wave: per-slot row accumulators and the staged whole-wave blocks.
template <bool PUSH>
struct WaveLds {
    uint32_t acc[SLOTS * WAVE];  // row accumulators: fp32 sums, or BFS minimum parents
    HeavyStage<PUSH> hs;
};

// LDS of a traversal kernel: the waves' slices, or (pull, before the
// segment loop) the non-COO pass's layout over the same bytes
template <int MODE, int PATH>
constexpr size_t traverse_lds_bytes()
{
    const size_t waves = (TPB / WAVE) * sizeof(WaveLds<PATH == PATH_PUSH>);
    const size_t other = PATH == PATH_PULL ? RowsLds<MODE>::WORDS * sizeof(uint32_t)
                                           : (TPB / WAVE) * sizeof(ActiveLds);
    return waves > other ? waves : other;
}


// The traversal kernels, launched pull kernel first.  Each reads the path
// the scan chose on the device and returns at once when it has no part in it:
//   pull kernel: above the compaction threshold the non-COO pass and the
//                segment loop; below it the non-COO pass and the compaction
//                of the COO segments (k_pull_compact instead, when the
//                activity bitmap exceeds this kernel's LDS copy)
//   push kernel: push, or the compacted pull's walk of the regions -- one
//                launch for the two, so that an automatic path choice costs
//                two traversal launches, not four.
// Pull is held to 128 registers (four waves per SIMD, no spills: measured
// faster than five waves with 96 registers and a few spills); push keeps its
// registers.  In the Boolean modes k_pull_compact always takes the
// compaction (inside the pull kernel it pushed the BFS kernel's arrays out
// to scratch memory under the earlier 96-register limit).
template <int MODE> constexpr bool pull_takes_compaction() { return valued<MODE>(); }
// activity bitmap words per thread that the pull kernel loads before it reads
// the device choice (the rest after)
#ifndef PULL_PRE_WORDS
#define PULL_PRE_WORDS 8
#endif

template <int MODE, int PATH>
__global__ __launch_bounds__(TPB, PATH == PATH_PULL ? 4 : 1) void k_traverse(MainArgs a)
{
    __shared__ __align__(16) uint8_t lds_raw[traverse_lds_bytes<MODE, PATH>()];
    WaveLds<PATH == PATH_PUSH> *lds = (WaveLds<PATH == PATH_PUSH> *)lds_raw;
    // pull: the first activity bitmap words this thread copies into LDS go
    // out with the device choice (they do not depend on it)
    const int32_t nwords = (a.nbc + 31) >> 5;
    constexpr int PRE_WORDS = PATH == PATH_PULL ? PULL_PRE_WORDS : 1;
    uint32_t xbw[PRE_WORDS];
    if constexpr (PATH == PATH_PULL) {
        const bool cp = nwords <= LDS_BITMAP_WORDS;
#pragma unroll
        for (int k = 0; k < PRE_WORDS; ++k) {
            const int32_t i = (int32_t)threadIdx.x + k * TPB;
            xbw[k] = (cp && i < nwords) ? a.xbits[i] : 0u;
        }
    }
    // the scan's counts, read together
    const int32_t N = a.counters[C_NZBLK];
    const int32_t path = a.counters[C_PATH];
    const int32_t xpop = a.counters[C_XPOP];
    const int32_t T = PATH == PATH_PUSH ? a.counters[C_TASKS] : 0;
    const int32_t NT = PATH == PATH_PUSH ? a.counters[C_NTB] : 0;
    if (N == 0) return;
    const int w = threadIdx.x >> 6, lane = lane_id();
    if constexpr (PATH == PATH_PUSH) {
        if (path == PATH_PULL) {
            int64_t rcap;
            int32_t nr;
            const int gw = blockIdx.x * (TPB / WAVE) + w;
            if (a.nreg > 0 && compact_pull(a, N, rcap, nr) && gw < a.nreg)
                pull_active<MODE>(a, ((ActiveLds *)lds_raw)[w], gw, rcap, nr, N, xpop);
            return;
        }
    }
    if (path != PATH) return;
    WaveLds<PATH == PATH_PUSH> &L = lds[w];
    float *sy = (float *)L.acc;
    int32_t *sp = (int32_t *)L.acc;
    auto init_acc = [&]() {
#pragma unroll
        for (int k = 0; k < SLOTS; ++k) L.acc[k * WAVE + lane] = MODE == M_BFS ? (uint32_t)INT_MAX : 0u;
    };
    const int gw = blockIdx.x * (TPB / WAVE) + w, nw = gridDim.x * (TPB / WAVE);
    if constexpr (PATH == PATH_PUSH) {
        init_acc();
        wave_lds_sync();
        push_loop<MODE>(a, gw, nw, sy, sp, &L.hs, T, NT);
    } else {
        // with an eighth or more of the vector blocks active, enough visited
        // blocks are used to load their descriptors together with their block
        // columns (measured: a quarter was 1.5% slower at 1% uniform x)
        const bool spec = (int64_t)N * 8 >= (int64_t)a.nbc;
        // below the compaction threshold: the non-COO blocks and the
        // compaction of the segments (the push kernel walks the regions)
        int64_t rcap;
        int32_t nr;
        const bool compact = a.nreg > 0 && compact_pull(a, N, rcap, nr);
        if (!pull_takes_compaction<MODE>() && compact) return;  // k_pull_compact
        if (nwords <= LDS_BITMAP_WORDS) {
#pragma unroll
            for (int k = 0; k < PRE_WORDS; ++k) {
                const int32_t i = (int32_t)threadIdx.x + k * TPB;
                if (i < nwords) lds_bits[i] = xbw[k];
            }
            for (int32_t i = (int32_t)threadIdx.x + PRE_WORDS * TPB; i < nwords; i += TPB) lds_bits[i] = a.xbits[i];
            __syncthreads();
            // the non-COO pass stages its headers over the wave's whole LDS slice
            pull_rows<MODE, true>(a, (uint32_t *)lds_raw);
            if constexpr (pull_takes_compaction<MODE>()) {
                if (compact) {
                    if (gw < a.nreg)
                        for (int32_t r = gw; r < nr; r += a.nreg) pull_compact<true>(a, r, rcap, N, xpop);
                    return;
                }
            }
            init_acc();
            wave_lds_sync();
            pull_loop<MODE, true>(a, gw, nw, sy, sp, &L.hs, spec);
        } else {
            if (compact) return;  // k_pull_compact
            pull_rows<MODE, false>(a, (uint32_t *)lds_raw);
            init_acc();
            wave_lds_sync();
            pull_loop<MODE, false>(a, gw, nw, sy, sp, &L.hs, spec);
        }
    }
}

// Pull for a matrix without COO blocks (every block is in the non-COO list,
// as in a decode layer): the non-COO pass alone, in a kernel of its own so
// that its registers do not compete with the segment loop's; one round per
// workgroup, of as few chunks as keep the grid within one resident round
// (fewer chunks per round leave fewer listed blocks per quarter-wave, hence
// shorter chains of dependent loads).
template <int MODE, int NB>
__global__ __launch_bounds__(TPB) void k_rows(MainArgs a)
{
    __shared__ __align__(16) uint32_t rows_lds[RowsLds<MODE, NB>::WORDS];
    // the first round's chunk bounds and the first bitmap words go out with
    // the device choice (the loads do not depend on it)
    const RowsPre first = rows_pre(a, (int64_t)blockIdx.x * a.cpw);
    const int32_t nwords = (a.nbc + 31) >> 5;
    const int t0 = threadIdx.x;
    const uint32_t xb0 = (nwords <= LDS_BITMAP_WORDS && t0 < nwords) ? a.xbits[t0] : 0u;
    const int32_t N = a.counters[C_NZBLK];
    if (N == 0 || a.counters[C_PATH] != PATH_PULL) return;
    if (nwords <= LDS_BITMAP_WORDS) {
        if (t0 < nwords) lds_bits[t0] = xb0;
        for (int32_t t = t0 + TPB; t < nwords; t += TPB) lds_bits[t] = a.xbits[t];
        __syncthreads();
        pull_rows<MODE, true, NB>(a, rows_lds, &first);
    } else {
        pull_rows<MODE, false, NB>(a, rows_lds, &first);
    }
}

// Dense activation on a matrix without COO blocks (decoding) with the path
// known to be pull: the non-COO pass reads the activation itself, with no
// scan before it.  Each workgroup first forms, from the activation, the
// 16-bit mask of every vector block (an entry is present iff it is nonzero,
// -0 counting as zero, as in the scan) and the activity bitmap, both in LDS
// (the mask table after the bitmap); the blocks' x words are then the
// activation's own (the masks select the products), and nothing of the
// context's x scratch is written.  The pass also writes the dense output:
// the workgroup that commits the last chunk of a block row (a per-call
// count per block row) converts its rows and clears their sums and the
// count, and rows of block rows without chunks are written as zeros, so
// that no kernel follows it.  Workgroup 0 records N_nzblk and the path for
// the call's statistics.
// The table takes (nbc + 1) / 2 words of dynamic LDS: ROWS_DX_MAX_NBC vector
// blocks at most.
constexpr int32_t ROWS_DX_MAX_NBC = 4096;
template <int MODE>
__global__ __launch_bounds__(TPB) void k_rows_dx(MainArgs a)
{
    __shared__ __align__(16) uint32_t rows_lds[RowsLds<MODE, 1>::WORDS];
    // the first round's chunk bounds go out before the mask pass
    const RowsPre first = rows_pre(a, (int64_t)blockIdx.x * a.cpw);
    const int32_t nbc = a.nbc, nwords = (nbc + 31) >> 5;
    uint16_t *lmask = (uint16_t *)(lds_bits + nwords);
    const int t0 = threadIdx.x, lane = lane_id();
    constexpr int PER = MODE == M_F16 ? 8 : 4;  // entries per 16 bytes
    uint32_t cnt = 0;
    // four vector blocks per thread and pass, their loads issued together
    constexpr int XB = 4;
    for (int32_t base = 0; base < nbc; base += XB * TPB) {
        uint4 v[XB][16 / PER];
#pragma unroll
        for (int b = 0; b < XB; ++b) {
            const int32_t J = base + b * TPB + t0;
            const uint4 *src = (const uint4 *)a.xd + (int64_t)J * (16 / PER);
#pragma unroll
            for (int q = 0; q < 16 / PER; ++q) v[b][q] = J < nbc ? src[q] : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int b = 0; b < XB; ++b) {
            if (base + b * TPB >= nbc) break;  // (uniform)
            const int32_t J = base + b * TPB + t0;
            uint32_t msk = 0;
#pragma unroll
            for (int q = 0; q < 16 / PER; ++q) {
                const uint32_t w[4] = {v[b][q].x, v[b][q].y, v[b][q].z, v[b][q].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if constexpr (MODE == M_F16) {
                        msk |= ((w[e] & 0x7FFFu) ? 1u : 0u) << (q * 8 + e * 2);
                        msk |= ((w[e] & 0x7FFF0000u) ? 1u : 0u) << (q * 8 + e * 2 + 1);
                    } else {
                        msk |= ((w[e] & 0x7FFFFFFFu) ? 1u : 0u) << (q * 4 + e);
                    }
                }
            }
            if (J < nbc) lmask[J] = (uint16_t)msk;
            // a wave's 64 consecutive vector blocks fill two bitmap words
            const uint64_t bm = ballot(msk != 0u);
            const int32_t w0 = (base + b * TPB + (t0 & ~(WAVE - 1))) >> 5;
            if (lane == 0 && w0 < nwords) lds_bits[w0] = (uint32_t)bm;
            if (lane == 32 && w0 + 1 < nwords) lds_bits[w0 + 1] = (uint32_t)(bm >> 32);
            cnt += msk ? 1u : 0u;
        }
    }
    // (the staging area of pull_rows serves the count's reduction first)
    if (blockIdx.x == 0) {
        const uint32_t c = wave_sum(cnt);
        if (lane == 0) rows_lds[t0 >> 6] = c;
    }
    __syncthreads();
    if (blockIdx.x == 0 && t0 == 0) {
        uint32_t c = 0;
#pragma unroll
        for (int w = 0; w < TPB / WAVE; ++w) c += rows_lds[w];
        a.counters[C_NZBLK] = (int32_t)c;
        a.counters[C_PATH] = PATH_PULL;
        a.counters[C_YNNZ] = a.m;
        a.counters[C_ERR_LAST] = 0;
    }
    // block rows without chunks: zero rows
    for (int64_t R = (int64_t)blockIdx.x * (TPB / 16) + (t0 >> 4); R < (a.m + 15) / 16;
         R += (int64_t)gridDim.x * (TPB / 16)) {
        const int64_t row = R * BS + (t0 & 15);
        if (a.rowchunks[R] == 0 && row < a.m) {
            if constexpr (MODE == M_F32) ((float *)a.ydense)[row] = 0.f;
            else ((uint16_t *)a.ydense)[row] = 0;
            if (a.y32) a.y32[row] = 0.f;
        }
    }
    __syncthreads();
    pull_rows<MODE, true, 1, true, true>(a, rows_lds, &first);
}

// ---------------------------------------------------------------------------
// finalize: ascending sparse y from the row-block structure masks
// ---------------------------------------------------------------------------
// A tile is 256 structure words (8192 rows).  Thread t first owns word t
// (its popcount enters the tile scan and the look-back); the rows are then
// written in 32 rounds where thread t handles row t + 256 r of the tile, so
// consecutive lanes touch consecutive accumulators and output slots.
#ifndef FINALIZE_TPB
#define FINALIZE_TPB 1024
#endif
constexpr int FTPB = FINALIZE_TPB;                 // threads per compaction workgroup
constexpr int FIN_WORDS = FINALIZE_WORDS;
constexpr int FIN_ROUNDS = FIN_WORDS * 32 / FTPB;  // rows per thread
static_assert(FIN_WORDS <= FTPB && FIN_ROUNDS >= 1 && FIN_WORDS * 32 <= 16 * (FTPB - WAVE), "finalize tile");

template <int MODE>
__global__ __launch_bounds__(FTPB) void k_finalize(uint32_t *__restrict__ ybits, int32_t nywords,
                                                  double *__restrict__ yacc, int32_t m,
                                                  int32_t *__restrict__ y_idx, void *__restrict__ y_val,
                                                  int32_t *__restrict__ y_nnz,
                                                  int32_t *__restrict__ counters, uint64_t *status,
                                                  uint64_t *next_status, int32_t n_status,
                                                  uint32_t *__restrict__ xmask, void *__restrict__ xd,
                                                  const int32_t *__restrict__ x_idx, int32_t k,
                                                  int32_t n)
{
    __shared__ uint64_t lds4[FTPB / WAVE];
    __shared__ uint64_t s_prefix;
    __shared__ uint32_t s_word[FIN_WORDS];
    __shared__ uint32_t s_wpos[FIN_WORDS];
    const int tile = blockIdx.x;
    const int32_t w = tile * FIN_WORDS + threadIdx.x;
    // the tile's structure words first: the scatter stores below then do not
    // delay them
    const uint32_t word = ((int)threadIdx.x < FIN_WORDS && w < nywords) ? ybits[w] : 0u;
    for (int32_t i = blockIdx.x * FTPB + threadIdx.x; i < n_status; i += gridDim.x * FTPB)
        next_status[i] = 0;
    // clear the blk_x_mask words this call's x indices touched, and put the
    // absent-entry marker back into the densified x
    for (int32_t t = blockIdx.x * FTPB + threadIdx.x; t < k; t += gridDim.x * FTPB) {
        const int32_t j = x_idx[t];
        if (j >= 0 && j < n) {
            xmask[j >> 5] = 0u;
            if constexpr (MODE == M_F32) ((uint32_t *)xd)[j] = 0xFFFFFFFFu;
            if constexpr (MODE == M_F16) ((uint16_t *)xd)[j] = (uint16_t)0xFFFFu;
        }
    }
    uint64_t total;
    const uint64_t excl = block_exclusive_scan<FTPB>((uint64_t)__popc(word), &total, lds4);
    if ((int)threadIdx.x < FIN_WORDS) {
        s_word[threadIdx.x] = word;
        s_wpos[threadIdx.x] = (uint32_t)excl;
    }
    __syncthreads();
    // wave 0 runs the look-back while the other waves load the accumulators
    // of the tile's rows (row (t - 64) + (FTPB - 64) u for thread t >= 64),
    // so that the two round trips overlap
    constexpr int RT = FTPB - WAVE, RROUNDS = (FIN_WORDS * 32 + RT - 1) / RT;
    const int64_t row0 = (int64_t)tile * FIN_WORDS * 32;
    double v[RROUNDS];
    uint32_t hm = 0;
    if (threadIdx.x >= WAVE) {
#pragma unroll
        for (int u = 0; u < RROUNDS; ++u) {
            const int lr = u * RT + (int)threadIdx.x - WAVE;
            const bool h = lr < FIN_WORDS * 32 && ((s_word[lr >> 5] >> (lr & 31)) & 1u);
            hm |= (h ? 1u : 0u) << u;
            v[u] = (valued<MODE>() && h) ? yacc[row0 + lr] : 0.0;
        }
    }
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
#pragma unroll
    for (int u = 0; u < RROUNDS; ++u) {
        if (!((hm >> u) & 1u)) continue;
        const int lr = u * RT + (int)threadIdx.x - WAVE;
        const uint32_t wd = s_word[lr >> 5];
        const uint32_t bit = lr & 31;
        const int64_t pos = base_pos + s_wpos[lr >> 5] + __popc(wd & ((1u << bit) - 1u));
        const int64_t i = row0 + lr;
        y_idx[pos] = (int32_t)i;
        if constexpr (MODE == M_F32) ((float *)y_val)[pos] = (float)v[u];
        if constexpr (MODE == M_F16) ((uint16_t *)y_val)[pos] = f64_to_f16_rne(v[u]);
        if constexpr (valued<MODE>()) yacc[i] = 0.0;
    }
    if (tile == (int)gridDim.x - 1 && threadIdx.x == 0) {
        int32_t tot = (int32_t)(s_prefix + total);
        *y_nnz = tot;
        counters[C_YNNZ] = tot;
        // out-of-range indices were counted by the blocker; fewer stored
        // entries than valid indices means a duplicate
        const int32_t bad = counters[C_XBAD], pop = counters[C_XPOP];
        counters[C_ERR_LAST] = (bad ? 1 : 0) | (pop < k - bad ? 2 : 0);
        counters[C_XBAD] = 0;
        counters[C_XPOP] = 0;
    }
    (void)m;
}

// Dense output (decoding): every row, converted from the fp64 accumulator.
template <int MODE>
__global__ __launch_bounds__(TPB) void k_finalize_dense(double *__restrict__ yacc, int32_t m,
                                                        void *__restrict__ y, float *__restrict__ y32,
                                                        uint32_t *__restrict__ ybits, int32_t nywords,
                                                        uint32_t *__restrict__ xmask, int32_t nxwords,
                                                        void *__restrict__ xd, int32_t n,
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
    // every x_j went through the densified x: restore the absent-entry marker
    for (int64_t i = (int64_t)blockIdx.x * TPB + threadIdx.x; i < n; i += stride) {
        if constexpr (MODE == M_F32) ((uint32_t *)xd)[i] = 0xFFFFFFFFu;
        else ((uint16_t *)xd)[i] = (uint16_t)0xFFFFu;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        counters[C_YNNZ] = m;
        counters[C_ERR_LAST] = 0;
        counters[C_XBAD] = 0;
        counters[C_XPOP] = 0;
    }
}

// Batched dense activations (nb vectors of n entries, row-major): the
// NB-strided padded copies (zeros where an entry is zero, past n, or past
// nb) and the union of their vector-block masks.
template <int MODE>
__global__ __launch_bounds__(TPB) void k_ballot_batch(const void *__restrict__ x, int32_t nb, int32_t n,
                                                      int64_t xstride, int32_t NB, void *__restrict__ xdb,
                                                      uint32_t *__restrict__ xmask, int32_t nwords)
{
    const int64_t lanes = (xstride + WAVE - 1) / WAVE * WAVE;  // per vector, whole waves
    const int64_t g = (int64_t)blockIdx.x * TPB + threadIdx.x;
    const int32_t b = (int32_t)(g / lanes);
    const int64_t j = g - (int64_t)b * lanes;
    if (b >= NB) return;  // whole waves: b is wave-uniform
    bool nz = false;
    if (j < xstride) {
        if constexpr (MODE == M_F16) {
            const uint16_t v = (b < nb && j < n) ? ((const uint16_t *)x)[(int64_t)b * n + j] : (uint16_t)0;
            nz = (v & 0x7FFFu) != 0;
            ((uint16_t *)xdb)[(int64_t)b * xstride + j] = nz ? v : (uint16_t)0;
        } else {
            const uint32_t v = (b < nb && j < n) ? ((const uint32_t *)x)[(int64_t)b * n + j] : 0u;
            nz = (v & 0x7FFFFFFFu) != 0;
            ((uint32_t *)xdb)[(int64_t)b * xstride + j] = nz ? v : 0u;
        }
    }
    const uint64_t bits = ballot(nz);
    if (lane_id() == 0 && bits) {
        const int64_t w = (j - lane_id()) >> 5;
        if (w < nwords && (uint32_t)bits) atomicOr(&xmask[w], (uint32_t)bits);
        if (w + 1 < nwords && (uint32_t)(bits >> 32)) atomicOr(&xmask[w + 1], (uint32_t)(bits >> 32));
    }
}

// Batched dense output: vector b < nb of y from its fp64 accumulators (RNE),
// every accumulator set and the masks reset.
template <int MODE>
__global__ __launch_bounds__(TPB) void k_finalize_batch(double *__restrict__ yaccb, int64_t ystride, int32_t nb,
                                                        int32_t NB, int32_t m, void *__restrict__ y,
                                                        float *__restrict__ y32, uint32_t *__restrict__ ybits,
                                                        int32_t nywords, uint32_t *__restrict__ xmask,
                                                        int32_t nxwords, int32_t *__restrict__ counters)
{
    const int64_t stride = (int64_t)gridDim.x * TPB;
    const int64_t tot = (int64_t)NB * m;
    for (int64_t g = (int64_t)blockIdx.x * TPB + threadIdx.x; g < tot; g += stride) {
        const int32_t b = (int32_t)(g / m);
        const int64_t i = g - (int64_t)b * m;
        double *pa = yaccb + (int64_t)b * ystride + i;
        const double v = *pa;
        if (b < nb) {
            if constexpr (MODE == M_F32) ((float *)y)[g] = (float)v;
            else ((uint16_t *)y)[g] = f64_to_f16_rne(v);
            if (y32) y32[g] = (float)v;
        }
        *pa = 0.0;
    }
    for (int64_t i = (int64_t)blockIdx.x * TPB + threadIdx.x; i < nywords; i += stride) ybits[i] = 0u;
    for (int64_t i = (int64_t)blockIdx.x * TPB + threadIdx.x; i < nxwords; i += stride) xmask[i] = 0u;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        counters[C_YNNZ] = m;
        counters[C_ERR_LAST] = 0;
        counters[C_XBAD] = 0;
        counters[C_XPOP] = 0;
    }
}

// ---------------------------------------------------------------------------
// BFS (Sec. 4.2)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(TPB) void k_bfs_init(int32_t n, int32_t source, int32_t *__restrict__ level,
                                                  int32_t *__restrict__ parent,
                                                  uint32_t *__restrict__ visited,
                                                  uint32_t *__restrict__ nextm,
                                                  uint32_t *__restrict__ xmask, int32_t nwords,
                                                  const uint32_t *__restrict__ row_occ,
                                                  int32_t *__restrict__ counters)
{
    const int64_t stride = (int64_t)gridDim.x * TPB;
    // the first scan sums the mask popcounts here
    if (blockIdx.x == 0 && threadIdx.x == 0) counters[C_XPOP] = 0;
    for (int64_t v = (int64_t)blockIdx.x * TPB + threadIdx.x; v < n; v += stride) {
        level[v] = v == source ? 0 : -1;
        parent[v] = v == source ? source : INT_MAX;
    }
    const int32_t sw = source >> 5;
    const uint32_t sb = 1u << (source & 31);
    // rows without entries start as visited (no edge reaches them; their
    // level and parent stay unset): the output mask of every level then
    // excludes them
    for (int64_t w = (int64_t)blockIdx.x * TPB + threadIdx.x; w < nwords; w += stride) {
        visited[w] = (row_occ ? ~row_occ[w] : 0u) | (w == sw ? sb : 0u);
        xmask[w] = w == sw ? sb : 0u;
        nextm[w] = 0u;
    }
}

// Next frontier -> current frontier masks, visited |= next, level of the
// newly reached vertices.  A thread per vertex, so that the level writes of
// a wave are coalesced; the first thread of each 32 vertices updates their
// mask words (the 32 threads read the word before it is cleared: one wave,
// program order).  The frontier size is the next scan's mask popcount
// (C_XPOP): a count here would take an atomic per wave on one counter, and
// same-address atomics serialize.
__global__ __launch_bounds__(TPB) void k_bfs_update(int32_t n, int32_t nwords, int32_t next_level,
                                                    int32_t *__restrict__ level,
                                                    uint32_t *__restrict__ visited,
                                                    uint32_t *__restrict__ nextm,
                                                    uint32_t *__restrict__ xmask,
                                                    int32_t *__restrict__ counters)
{
    const int64_t v = (int64_t)blockIdx.x * TPB + threadIdx.x;
    const int64_t w = v >> 5;
    // the next scan sums the mask popcounts here
    if (v == 0) counters[C_XPOP] = 0;
    const uint32_t nm = (v < n && w < nwords) ? nextm[w] : 0u;
    if ((nm >> (v & 31)) & 1u) level[v] = next_level;
    if ((v & 31) == 0 && v < n && w < nwords) {
        xmask[w] = nm;
        if (nm) {
            visited[w] |= nm;
            nextm[w] = 0u;
        }
    }
}

__global__ __launch_bounds__(TPB) void k_bfs_finish(int32_t n, int32_t *__restrict__ parent)
{
    const int64_t stride = (int64_t)gridDim.x * TPB;
    for (int64_t v = (int64_t)blockIdx.x * TPB + threadIdx.x; v < n; v += stride)
        if (parent[v] == INT_MAX) parent[v] = -1;
}

// ---------------------------------------------------------------------------
// single launch for short index lists (Sec. 4.1: blocker, nonzero-block count
// and path choice inside the SpMSpV launch)
// ---------------------------------------------------------------------------
// One kernel runs the whole call for up to SMALL_X_MAX x indices:
//   1. workgroup 0 runs the blocker and the selector (small_x_body) and then
//      publishes the call's number in the `ready` words; the other
//      workgroups wait for it (one writer, many readers);
//   2. every workgroup takes its share of the chosen traversal (push, or
//      the non-COO pass plus the segment loop of pull) and then publishes
//      the call's number in its own `done` word;
//   3. one wave of workgroup 0 waits until every done word holds it and
//      publishes it in the `all` words; the first nfin workgroups wait for
//      those, then compact y (look-back over tiles of FF_WORDS structure
//      words) and restore the scratch.
// Device-wide barriers built from contended atomic counters cost 4-30
// microseconds on this GPU (the atomics on one address are serialized),
// more than the kernel boundaries they would replace, and so does a done
// word polled by many workgroups; here every word has one writer, a single
// wave polls the done words, and the many readers of `ready` and `all`
// spread over eight copies 4 KB apart.  Only workgroups below nfin ever
// wait on workgroups that may not have started, so the others always
// finish and free their slots.  Every wait is bounded: a wait that runs out
// sets bit 2 of the call's error flags instead of hanging.
#ifndef FUSED_MAX_GRID
#define FUSED_MAX_GRID 512
#endif
static_assert(FUSED_MAX_GRID <= MAX_MAIN_GRID, "one done word per workgroup");
constexpr int FF_WORDS = 2 * TPB;       // y-structure words per compaction tile (2 per thread)
constexpr int FUSED_MAX_FIN = 128;      // compacting workgroups at most
constexpr uint32_t FUSED_SPIN_MAX = 1u << 22;
// sync words: copy c (< 8) of `ready` at 1024 c and of `all` at 1024 c + 512;
// the done word of workgroup g at SYNC_DONE + g
constexpr int SYNC_COPIES = 8, SYNC_STRIDE = 1024, SYNC_ALL = 512, SYNC_DONE = SYNC_COPIES * SYNC_STRIDE;
static_assert(SYNC_WORDS == SYNC_DONE + MAX_MAIN_GRID, "single-launch sync words");

struct FusedArgs {
    const int32_t *x_idx;
    const void *x_val;
    int32_t k, n;
    void *xd;
    uint32_t *xmask;
    uint32_t *xbits;
    int4 *items;
    const int32_t *cb_ptr;
    int32_t forced_path;
    double th3, th3s;
    int32_t *y_idx;
    void *y_val;
    int32_t *y_nnz;
    uint32_t *sync;
    uint32_t gen;            // this call's number (never 0)
    uint64_t *status;        // compaction look-back statuses of this call (zero)
    uint64_t *next_status;   // the other copy, cleared for the next call
    int32_t n_status;
    int32_t nfin;            // compacting workgroups
    int32_t ntiles;          // compaction tiles
    int32_t nywords;
};

// Waits (one lane) until *p == v; false if the bound ran out.
__device__ __forceinline__ bool fused_wait_one(const uint32_t *p, uint32_t v)
{
    for (uint32_t i = 0; i < FUSED_SPIN_MAX; ++i) {
        if (__hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == v) return true;
        __builtin_amdgcn_s_sleep(8);
    }
    return false;
}

// Publishes v in the SYNC_COPIES copies of a word (one lane).
__device__ __forceinline__ void fused_publish(uint32_t *base, uint32_t v)
{
    for (int c = 0; c < SYNC_COPIES; ++c)
        __hip_atomic_store(&base[c * SYNC_STRIDE], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Waits until every memory operation this wave issued has completed (the
// fence keeps the compiler from moving them past the wait).
__device__ __forceinline__ void wave_drain()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_s_waitcnt(0);
}

// Waits (one wave) until the g words at p all hold v.
__device__ __forceinline__ bool fused_wait_all(const uint32_t *p, int32_t g, uint32_t v)
{
    const int lane = lane_id();
    for (uint32_t i = 0; i < FUSED_SPIN_MAX; ++i) {
        bool ok = true;
        for (int32_t q = lane; q < g; q += WAVE)
            ok &= __hip_atomic_load(&p[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == v;
        if (!ballot(!ok)) return true;
        __builtin_amdgcn_s_sleep(8);
    }
    return false;
}

// One compaction tile of the single launch: thread t owns structure words
// 2 t and 2 t + 1 of the tile and writes the rows of their set bits in
// ascending order (the outputs of a short x are sparse, so only set bits
// are visited).
template <int MODE>
__device__ __forceinline__ void fused_finalize_tile(const FusedArgs &f, double *yacc, uint32_t *ybits, int tile, uint64_t *lds4,
                                    uint64_t *s_prefix)
{
    const int t = threadIdx.x;
    const int32_t w0 = tile * FF_WORDS + 2 * t;
    uint32_t wd[2];
    wd[0] = w0 < f.nywords ? __hip_atomic_load(&ybits[w0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
    wd[1] = w0 + 1 < f.nywords ? __hip_atomic_load(&ybits[w0 + 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
    uint64_t total;
    const uint64_t excl = block_exclusive_scan<TPB>((uint64_t)(__popc(wd[0]) + __popc(wd[1])), &total, lds4);
    if (t < WAVE) {
        uint64_t prefix = 0;
        if (tile == 0) {
            if (t == 0) st_store(&f.status[0], ST_INC | total);
        } else {
            if (t == 0) st_store(&f.status[tile], ST_AGG | total);
            prefix = lookback(f.status, tile);
            if (t == 0) st_store(&f.status[tile], ST_INC | (prefix + total));
        }
        if (t == 0) *s_prefix = prefix;
    }
    __syncthreads();
    const int64_t prefix = (int64_t)*s_prefix;
    int64_t pos = prefix + (int64_t)excl;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        uint32_t w = wd[h];
        if (!w) continue;
        ybits[w0 + h] = 0u;
        const int64_t row0 = (int64_t)(w0 + h) * 32;
        while (w) {
            // up to four rows at a time: their accumulator loads go out together
            int64_t r[4];
            double v[4];
            int cnt = 0;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                r[u] = row0 + ctz32(w);
                v[u] = 0.0;
                if (w) {
                    if constexpr (valued<MODE>())
                        v[u] = __hip_atomic_load(&yacc[r[u]], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    w &= w - 1u;
                    cnt = u + 1;
                }
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                if (u >= cnt) break;
                f.y_idx[pos] = (int32_t)r[u];
                if constexpr (MODE == M_F32) ((float *)f.y_val)[pos] = (float)v[u];
                if constexpr (MODE == M_F16) ((uint16_t *)f.y_val)[pos] = f64_to_f16_rne(v[u]);
                if constexpr (valued<MODE>()) yacc[r[u]] = 0.0;
                ++pos;
            }
        }
    }
    if (tile == f.ntiles - 1 && t == 0) {
        const int32_t tot = (int32_t)(prefix + (int64_t)total);
        *f.y_nnz = tot;
    }
    __syncthreads();  // *s_prefix is read again by the next tile
}

// LDS of the single-launch kernel: the traversal's (either path) or the
// blocker's hash table, whichever is larger.
template <int MODE>
constexpr size_t fused_lds_bytes()
{
    const size_t a = traverse_lds_bytes<MODE, PATH_PUSH>(), b = traverse_lds_bytes<MODE, PATH_PULL>();
    const size_t c = (size_t)SX_HASH * sizeof(uint32_t);
    const size_t ab = a > b ? a : b;
    return ab > c ? ab : c;
}

template <int MODE>
__global__ __launch_bounds__(TPB, 3) void k_fused(MainArgs a, FusedArgs f)
{
    __shared__ __align__(16) uint8_t lds_raw[fused_lds_bytes<MODE>()];
    __shared__ uint64_t lds4[TPB / WAVE];
    __shared__ uint64_t s_prefix;
    const int t = threadIdx.x;
    const int copy = (blockIdx.x % SYNC_COPIES) * SYNC_STRIDE;
    uint32_t *ready = f.sync, *all = f.sync + SYNC_ALL, *done = f.sync + SYNC_DONE;
    // 1. blocker and selector (workgroup 0); the others wait for them.
    // Workgroup 0's plain stores reach memory by one release (an L2
    // write-back); the waiting workgroups read nothing of them before the
    // ready word, and the caches held none of these lines at the launch.
    if (blockIdx.x == 0) {
        small_x_body<MODE, TPB>(f.x_idx, f.x_val, f.k, f.n, f.xd, f.xmask, f.cb_ptr, a.nbc, f.items, f.xbits,
                                a.counters, f.forced_path, f.th3, f.th3s, (uint32_t *)lds_raw, lds_bits, lds4);
        wave_drain();
        __syncthreads();
        if (t == 0) {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
            fused_publish(ready, f.gen);
        }
    } else {
        if (t == 0 && !fused_wait_one(ready + copy, f.gen)) atomicOr(&a.counters[C_SYNCERR], 1);
        __syncthreads();
    }
    // 2. traversal
    const int32_t N = __hip_atomic_load(&a.counters[C_NZBLK], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int32_t path = __hip_atomic_load(&a.counters[C_PATH], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int w = t >> 6, lane = lane_id();
    const int gw = blockIdx.x * (TPB / WAVE) + w, nw = gridDim.x * (TPB / WAVE);
    if (N > 0) {
        if (path == PATH_PUSH) {
            WaveLds<true> &L = ((WaveLds<true> *)lds_raw)[w];
#pragma unroll
            for (int q = 0; q < SLOTS; ++q) L.acc[q * WAVE + lane] = 0u;
            wave_lds_sync();
            const int32_t T = __hip_atomic_load(&a.counters[C_TASKS], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            const int32_t NT = __hip_atomic_load(&a.counters[C_NTB], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            push_loop<MODE>(a, gw, nw, (float *)L.acc, (int32_t *)L.acc, &L.hs, T, NT);
        } else {
            const bool spec = (int64_t)N * 8 >= (int64_t)a.nbc;
            const int32_t nwords = (a.nbc + 31) >> 5;
            for (int32_t i = t; i < nwords; i += TPB) lds_bits[i] = a.xbits[i];
            __syncthreads();
            pull_rows<MODE, true>(a, (uint32_t *)lds_raw);
            WaveLds<false> &L = ((WaveLds<false> *)lds_raw)[w];
#pragma unroll
            for (int q = 0; q < SLOTS; ++q) L.acc[q * WAVE + lane] = 0u;
            wave_lds_sync();
            pull_loop<MODE, true>(a, gw, nw, (float *)L.acc, (int32_t *)L.acc, &L.hs, spec);
        }
    }
    // 3. completion.  The traversal's results are device-scope atomics,
    // complete once the wave's memory counter drains, so
    // a done word needs no cache write-back; the compaction reads them with
    // device-coherent loads.
    wave_drain();
    __syncthreads();
    if (t == 0) __hip_atomic_store(&done[blockIdx.x], f.gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if ((int)blockIdx.x >= f.nfin) return;
    if (blockIdx.x == 0) {
        if (t < WAVE) {
            const bool ok = fused_wait_all(done, (int32_t)gridDim.x, f.gen);
            if (t == 0) {
                if (!ok) atomicOr(&a.counters[C_SYNCERR], 1);
                fused_publish(all, f.gen);
            }
        }
    } else if (t == 0 && !fused_wait_one(all + copy, f.gen)) {
        atomicOr(&a.counters[C_SYNCERR], 1);
    }
    __syncthreads();
    const int32_t gstride = f.nfin * TPB;
    for (int32_t i = blockIdx.x * TPB + t; i < f.n_status; i += gstride) f.next_status[i] = 0;
    // clear the blk_x_mask words of this call's x indices and put the
    // absent-entry marker back into the densified x
    for (int32_t q = blockIdx.x * TPB + t; q < f.k; q += gstride) {
        const int32_t j = f.x_idx[q];
        if (j >= 0 && j < f.n) {
            f.xmask[j >> 5] = 0u;
            if constexpr (MODE == M_F32) ((uint32_t *)f.xd)[j] = 0xFFFFFFFFu;
            if constexpr (MODE == M_F16) ((uint16_t *)f.xd)[j] = (uint16_t)0xFFFFu;
        }
    }
    for (int tile = blockIdx.x; tile < f.ntiles; tile += f.nfin)
        fused_finalize_tile<MODE>(f, a.yacc, a.ybits, tile, lds4, &s_prefix);
    if ((int)blockIdx.x == (f.ntiles - 1) % f.nfin && t == 0) {
        // the workgroup of the last tile: the call's counters and error flags
        const int32_t tot = *f.y_nnz;
        a.counters[C_YNNZ] = tot;
        const int32_t bad = a.counters[C_XBAD], pop = a.counters[C_XPOP];
        const int32_t serr = __hip_atomic_load(&a.counters[C_SYNCERR], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        a.counters[C_ERR_LAST] = (bad ? 1 : 0) | (pop < f.k - bad ? 2 : 0) | (serr ? 4 : 0);
        a.counters[C_XBAD] = 0;
        a.counters[C_XPOP] = 0;
        a.counters[C_SYNCERR] = 0;
    }
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

// Resident workgroups of a traversal kernel on the whole device (compute
// units x workgroups per compute unit at its register and LDS use), so that
// the persistent grid is exactly one round of residency.
template <int MODE, int PATH>
static int resident_grid(size_t dyn_lds)
{
    // cached per dynamic LDS size (a handful of distinct sizes occur)
    static size_t cached_lds[8];
    static int cached_grid[8];
    static int ncached = 0;
    for (int i = 0; i < ncached; ++i)
        if (cached_lds[i] == dyn_lds) return cached_grid[i];
    int dev = 0, cus = 0, per_cu = 0, grid = MAX_MAIN_GRID;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_traverse<MODE, PATH>, TPB, dyn_lds) == hipSuccess &&
        cus > 0 && per_cu > 0)
        grid = cus * per_cu;
    if (ncached < 8) {
        cached_lds[ncached] = dyn_lds;
        cached_grid[ncached] = grid;
        ++ncached;
    }
    return grid;
}

// Resident workgroups of k_pull_compact with dyn_lds bytes of dynamic LDS.
template <int MODE>
static int compact_grid(size_t dyn_lds)
{
    static size_t cached_lds[8];
    static int cached_grid[8];
    static int ncached = 0;
    for (int i = 0; i < ncached; ++i)
        if (cached_lds[i] == dyn_lds) return cached_grid[i];
    int dev = 0, cus = 0, per_cu = 0, grid = MAX_MAIN_GRID;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_pull_compact<MODE>, TPB, dyn_lds) == hipSuccess &&
        cus > 0 && per_cu > 0)
        grid = min(cus * per_cu, MAX_MAIN_GRID);
    if (ncached < 8) {
        cached_lds[ncached] = dyn_lds;
        cached_grid[ncached] = grid;
        ++ncached;
    }
    return grid;
}

// Chunks per round for k_rows: the fewest (at most 16) that keep its grid
// within one round of resident workgroups.
template <int MODE, int NB>
static int32_t rows_cpw(int64_t nchunk, size_t dyn)
{
    static int resident[2] = {0, 0};
    const int slot = dyn ? 1 : 0;
    if (resident[slot] == 0) {
        int dev = 0, cus = 0, per_cu = 0;
        resident[slot] = -1;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_rows<MODE, NB>, TPB, dyn) == hipSuccess &&
            cus > 0 && per_cu > 0)
            resident[slot] = cus * per_cu;
    }
    if (resident[slot] <= 0) return TPB / 16;
    const int64_t c = (nchunk + resident[slot] - 1) / resident[slot];
    return (int32_t)std::max<int64_t>(1, std::min<int64_t>(c, TPB / 16));
}

// Launch order: the pull kernel (and k_pull_compact when the bitmap does not
// fit the pull kernel's LDS copy), then the push kernel, which also walks the
// compacted pull's regions.  `forced` is the path known on the host (BFS, a
// forced path, or a choice that the number of x entries already settles);
// 0 launches both, and the device choice makes one of them return at once.
template <int MODE>
static hipError_t launch_paths(const DevMatrix &A, const MainArgs &a, int forced, hipStream_t s)
{
    const bool pull = forced != PATH_PUSH, push = forced != PATH_PULL;
    const int32_t nwords = (A.nbc + 31) >> 5;
    const size_t dyn = nwords <= LDS_BITMAP_WORDS ? (size_t)nwords * 4 : 0;
    MainArgs b = a;
    b.nreg = 0;
    b.cpm = valued<MODE>() ? PULL_COMPACT_PERMILLE : PULL_COMPACT_PERMILLE_BOOL;
    hipError_t e = hipSuccess;
    if (pull && A.nblk > 0 && A.nheavy == A.nblk) {
        // no COO blocks: the non-COO pass alone
        MainArgs r = b;
        r.cpw = rows_cpw<MODE, 1>(A.nchunk, dyn);
        hipLaunchKernelGGL((k_rows<MODE, 1>), dim3(grid_for(A.nchunk, r.cpw, INT_MAX)), dim3(TPB), dyn, s, r);
        e = hipGetLastError();
    } else if (pull) {
        int g = grid_for((A.nseg + 3) / 4, TPB / WAVE, MAX_MAIN_GRID);
        g = min(g, resident_grid<MODE, PATH_PULL>(dyn));
        // compacted pull: as many regions as the push kernel keeps resident,
        // and no more than the pull kernel has waves
        if (a.clist && a.nseg > 0) b.nreg = min(resident_grid<MODE, PATH_PUSH>(0), g) * (TPB / WAVE);
        hipLaunchKernelGGL((k_traverse<MODE, PATH_PULL>), dim3(g), dim3(TPB), dyn, s, b);
        e = hipGetLastError();
        if (e == hipSuccess && b.nreg > 0 && (dyn == 0 || !pull_takes_compaction<MODE>())) {
            const size_t dync = nwords <= COMPACT_BITMAP_WORDS ? (size_t)nwords * 4 : 0;
            const int gc = compact_grid<MODE>(dync);
            hipLaunchKernelGGL((k_pull_compact<MODE>), dim3(gc), dim3(TPB), dync, s, b);
            e = hipGetLastError();
        }
    }
    if (e != hipSuccess || !(push || b.nreg > 0)) return e;
    int g = push ? grid_for((A.nblk + WAVE - 1) / WAVE, TPB / WAVE, MAX_MAIN_GRID) : 1;
    g = min(g, resident_grid<MODE, PATH_PUSH>(0));
    g = max(g, b.nreg / (TPB / WAVE));
    hipLaunchKernelGGL((k_traverse<MODE, PATH_PUSH>), dim3(g), dim3(TPB), 0, s, b);
    return hipGetLastError();
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
    if (mode == M_F16) hipLaunchKernelGGL(k_ballot<M_F16>, g, b, 0, s, x_dense, A.n, C.xd, C.xmask, C.nxwords, C.counters);
    else hipLaunchKernelGGL(k_ballot<M_F32>, g, b, 0, s, x_dense, A.n, C.xd, C.xmask, C.nxwords, C.counters);
    return hipGetLastError();
}

hipError_t launch_scan(const DevMatrix &A, DevCtx &C, int forced_path, double th3, double th3s, hipStream_t s,
                       double tasks_max)
{
    dim3 g(grid_for(A.nbc, SCAN_TILE, INT_MAX)), b(STPB);
    const int p = C.scan_parity;
    hipLaunchKernelGGL((k_scan<false, 0>), g, b, 0, s, C.xmask, nullptr, nullptr, A.cb_ptr, A.nbc, C.items,
                       C.xbits, C.counters, C.st_scan[p], C.st_scan[1 - p], C.n_st_scan, forced_path, th3, th3s,
                       tasks_max);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) C.scan_parity = 1 - p;
    return e;
}

bool scan_takes_dense(const DevMatrix &A, const void *x_dense)
{
    return A.n % 16 == 0 && ((uintptr_t)x_dense & 15u) == 0 && SCAN_ITEMS % 2 == 0;
}

hipError_t launch_small_x(const DevMatrix &A, const DevCtx &C, int mode, int32_t k, const int32_t *x_idx,
                          const void *x_val, int forced_path, double th3, double th3s, hipStream_t s)
{
    // (the look-back status words of the next k_scan stay zero: none used)
    if (!small_x_fits(A, k)) return hipErrorInvalidValue;
#define SX_ARGS x_idx, x_val, k, A.n, C.xd, C.xmask, A.cb_ptr, A.nbc, C.items, C.xbits, C.counters, \
                forced_path, th3, th3s
    switch (mode) {
    case M_F32: hipLaunchKernelGGL(k_small_x<M_F32>, dim3(1), dim3(SX_TPB), 0, s, SX_ARGS); break;
    case M_F16: hipLaunchKernelGGL(k_small_x<M_F16>, dim3(1), dim3(SX_TPB), 0, s, SX_ARGS); break;
    default: hipLaunchKernelGGL(k_small_x<M_BOOL>, dim3(1), dim3(SX_TPB), 0, s, SX_ARGS); break;
    }
#undef SX_ARGS
    return hipGetLastError();
}

bool small_x_fits(const DevMatrix &A, int32_t k)
{
    return k >= 0 && k <= SMALL_X_MAX && ((int64_t)A.nbc + 31) / 32 <= SMALL_X_WORDS;
}

hipError_t launch_scan_dense(const DevMatrix &A, DevCtx &C, int mode, const void *x_dense, int forced_path,
                             double th3, double th3s, hipStream_t s)
{
    dim3 g(grid_for(A.nbc, SCAN_TILE, INT_MAX)), b(STPB);
    const int p = C.scan_parity;
    if (mode == M_F16)
        hipLaunchKernelGGL((k_scan<true, M_F16>), g, b, 0, s, C.xmask, x_dense, C.xd, A.cb_ptr, A.nbc, C.items,
                           C.xbits, C.counters, C.st_scan[p], C.st_scan[1 - p], C.n_st_scan, forced_path, th3, th3s, -1.0);
    else
        hipLaunchKernelGGL((k_scan<true, M_F32>), g, b, 0, s, C.xmask, x_dense, C.xd, A.cb_ptr, A.nbc, C.items,
                           C.xbits, C.counters, C.st_scan[p], C.st_scan[1 - p], C.n_st_scan, forced_path, th3, th3s, -1.0);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) C.scan_parity = 1 - p;
    return e;
}

static void fill_main_args(const DevMatrix &A, const DevCtx &C, int mode, const void *xd, const uint32_t *omask,
                           int complement, int32_t *parent, MainArgs &a)
{
    a.sl_col = A.sl_col;
    a.hv_col = A.hv_col;
    a.hv_desc = A.hv_desc;
    a.hv_cstart = A.hv_cstart;
    a.hv_crow = A.hv_crow;
    a.nchunk = A.nchunk;
    a.sl_desc = A.sl_desc;
    a.seg_rs = A.seg_rs;
    a.pay = A.pay;
    a.vb = A.dtype == 0 ? 4u : (A.dtype == 1 ? 2u : 0u);
    a.nbc = A.nbc;
    a.csc_row = A.csc_row;
    a.csc_desc = A.csc_desc;
    // without COO blocks every block is in the non-COO list: no segment has work
    a.nseg = A.nheavy < A.nblk ? A.nseg : 0;
    a.xd = xd;
    a.xmask = C.xmask;
    a.xbits = C.xbits;
    a.items = C.items;
    a.counters = C.counters;
    a.omask = omask;
    a.complement = complement;
    a.yacc = C.yacc;
    a.ybits = mode == M_BFS ? C.nextm : C.ybits;
    a.parent = parent;
    a.xstride = 0;
    a.ystride = 0;
    // slot ids are int32
    const bool fits = C.clist && (A.nseg + 4 * MAX_MAIN_GRID) * 16 <= C.clist_cap &&
                      A.nseg * 16 < (int64_t)INT32_MAX;
    a.clist = fits ? C.clist : nullptr;
    a.ccount = C.ccount;
    a.clist_cap = C.clist_cap;
    a.nreg = 0;
    a.cpw = TPB / 16;
    a.cpm = 0;
    a.creg = compact_list_regions();
    a.torder = A.task_order;
    a.ntask = A.ntask;
    a.rowchunks = nullptr;
    a.rdone = nullptr;
    a.ydense = nullptr;
    a.y32 = nullptr;
    a.m = A.m;
}

int64_t compact_list_entries(int64_t nseg) { return (nseg + 4 * MAX_MAIN_GRID) * 16; }
int32_t compact_list_regions() { return 8 * MAX_MAIN_GRID; }

hipError_t launch_main(const DevMatrix &A, const DevCtx &C, int mode, const void *xd,
                       const uint32_t *omask, int complement, int32_t *parent, int forced_path,
                       hipStream_t s)
{
    MainArgs a;
    fill_main_args(A, C, mode, xd, omask, complement, parent, a);
    switch (mode) {
    case M_F32: return launch_paths<M_F32>(A, a, forced_path, s);
    case M_F16: return launch_paths<M_F16>(A, a, forced_path, s);
    case M_BOOL: return launch_paths<M_BOOL>(A, a, forced_path, s);
    default: return launch_paths<M_BFS>(A, a, forced_path, s);
    }
}

bool fused_fits(const DevMatrix &A, int32_t k)
{
    return small_x_fits(A, k) && ((int64_t)A.nbc + 31) / 32 <= LDS_BITMAP_WORDS;
}

// Resident workgroups of the single-launch kernel (one round of residency).
template <int MODE>
static int fused_grid(size_t dyn_lds)
{
    static size_t cached_lds[8];
    static int cached_grid[8];
    static int ncached = 0;
    for (int i = 0; i < ncached; ++i)
        if (cached_lds[i] == dyn_lds) return cached_grid[i];
    int dev = 0, cus = 0, per_cu = 0, grid = 256;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_fused<MODE>, TPB, dyn_lds) == hipSuccess &&
        cus > 0 && per_cu > 0)
        grid = cus * per_cu;
    if (grid > FUSED_MAX_GRID) grid = FUSED_MAX_GRID;
    if (ncached < 8) {
        cached_lds[ncached] = dyn_lds;
        cached_grid[ncached] = grid;
        ++ncached;
    }
    return grid;
}

hipError_t launch_fused(const DevMatrix &A, DevCtx &C, int mode, int32_t k, const int32_t *x_idx,
                        const void *x_val, const uint32_t *omask, int complement, int forced_path, double th3,
                        double th3s, int32_t *y_idx, void *y_val, int32_t *y_nnz, hipStream_t s)
{
    if (!fused_fits(A, k) || !C.sync || mode == M_BFS) return hipErrorInvalidValue;
    MainArgs a;
    fill_main_args(A, C, mode, C.xd, omask, complement, nullptr, a);
    a.clist = nullptr;  // the segment loop at every activity
    FusedArgs f;
    f.x_idx = x_idx;
    f.x_val = x_val;
    f.k = k;
    f.n = A.n;
    f.xd = C.xd;
    f.xmask = C.xmask;
    f.xbits = C.xbits;
    f.items = C.items;
    f.cb_ptr = A.cb_ptr;
    f.forced_path = forced_path;
    f.th3 = th3;
    f.th3s = th3s;
    f.y_idx = y_idx;
    f.y_val = y_val;
    f.y_nnz = y_nnz;
    f.sync = C.sync;
    if (++C.gen == 0) C.gen = 1;
    f.gen = C.gen;
    const int p = C.fin_parity;
    f.status = C.st_fin[p];
    f.next_status = C.st_fin[1 - p];
    f.n_status = C.n_st_fin;
    f.nywords = (A.nbr + 1) / 2;
    f.ntiles = (f.nywords + FF_WORDS - 1) / FF_WORDS;
    if (f.ntiles < 1) f.ntiles = 1;
    const int32_t nwords = (A.nbc + 31) >> 5;
    const size_t dyn = (size_t)(nwords > 0 ? nwords : 1) * 4;
    int grid = 256;
    switch (mode) {
    case M_F32: grid = fused_grid<M_F32>(dyn); break;
    case M_F16: grid = fused_grid<M_F16>(dyn); break;
    default: grid = fused_grid<M_BOOL>(dyn); break;
    }
    f.nfin = std::min(std::min(grid, f.ntiles), FUSED_MAX_FIN);
    if (f.ntiles + 1 > f.n_status) return hipErrorInvalidValue;
    switch (mode) {
    case M_F32: hipLaunchKernelGGL(k_fused<M_F32>, dim3(grid), dim3(TPB), dyn, s, a, f); break;
    case M_F16: hipLaunchKernelGGL(k_fused<M_F16>, dim3(grid), dim3(TPB), dyn, s, a, f); break;
    default: hipLaunchKernelGGL(k_fused<M_BOOL>, dim3(grid), dim3(TPB), dyn, s, a, f); break;
    }
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) C.fin_parity = 1 - p;
    return e;
}

int32_t scan_tiles(int32_t nbc) { return (nbc + SCAN_TILE - 1) / SCAN_TILE; }
int32_t finalize_tiles(int32_t nbr) { return ((nbr + 1) / 2 + FIN_WORDS - 1) / FIN_WORDS; }

hipError_t launch_finalize(const DevMatrix &A, DevCtx &C, int mode, int32_t *y_idx, void *y_val,
                           int32_t *y_nnz, const int32_t *x_idx, int32_t k, hipStream_t s)
{
    int32_t nyw = (A.nbr + 1) / 2;
    dim3 g(grid_for(nyw, FIN_WORDS, INT_MAX)), b(FTPB);
    const int p = C.fin_parity;
    uint64_t *st = C.st_fin[p], *nx = C.st_fin[1 - p];
    const int32_t ns = C.n_st_fin;
    switch (mode) {
    case M_F32: hipLaunchKernelGGL(k_finalize<M_F32>, g, b, 0, s, C.ybits, nyw, C.yacc, A.m, y_idx, y_val, y_nnz, C.counters, st, nx, ns, C.xmask, C.xd, x_idx, k, A.n); break;
    case M_F16: hipLaunchKernelGGL(k_finalize<M_F16>, g, b, 0, s, C.ybits, nyw, C.yacc, A.m, y_idx, y_val, y_nnz, C.counters, st, nx, ns, C.xmask, C.xd, x_idx, k, A.n); break;
    default: hipLaunchKernelGGL(k_finalize<M_BOOL>, g, b, 0, s, C.ybits, nyw, C.yacc, A.m, y_idx, y_val, y_nnz, C.counters, st, nx, ns, C.xmask, C.xd, x_idx, k, A.n); break;
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
        hipLaunchKernelGGL(k_finalize_dense<M_F16>, g, b, 0, s, C.yacc, A.m, y, y32, C.ybits, nyw, C.xmask, C.nxwords, C.xd, A.n, C.counters);
    else
        hipLaunchKernelGGL(k_finalize_dense<M_F32>, g, b, 0, s, C.yacc, A.m, y, y32, C.ybits, nyw, C.xmask, C.nxwords, C.xd, A.n, C.counters);
    return hipGetLastError();
}

bool rows_dx_fits(const DevMatrix &A, const void *x_dense)
{
    // (the caller has excluded pattern matrices)
    return A.nblk > 0 && A.nheavy == A.nblk && scan_takes_dense(A, x_dense) && A.nbc <= ROWS_DX_MAX_NBC;
}

// Chunks per round for k_rows_dx (as rows_cpw), its residency cached per
// dynamic LDS size.
template <int MODE>
static int32_t rows_dx_cpw(int64_t nchunk, size_t dyn)
{
    static size_t cached_lds[8];
    static int cached_res[8];
    static int ncached = 0;
    int res = -1;
    for (int i = 0; i < ncached; ++i)
        if (cached_lds[i] == dyn) res = cached_res[i];
    if (res < 0) {
        int dev = 0, cus = 0, per_cu = 0;
        res = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_rows_dx<MODE>, TPB, dyn) == hipSuccess &&
            cus > 0 && per_cu > 0)
            res = cus * per_cu;
        if (ncached < 8) {
            cached_lds[ncached] = dyn;
            cached_res[ncached] = res;
            ++ncached;
        }
    }
    if (res <= 0) return TPB / 16;
    const int64_t c = (nchunk + res - 1) / res;
    return (int32_t)std::max<int64_t>(1, std::min<int64_t>(c, TPB / 16));
}

hipError_t launch_rows_dx(const DevMatrix &A, const DevCtx &C, int mode, const void *x_dense, void *y,
                          float *y32, hipStream_t s)
{
    MainArgs a;
    fill_main_args(A, C, mode, x_dense, nullptr, 0, nullptr, a);
    a.rowchunks = A.hv_rowchunks;
    a.rdone = C.rdone;
    a.ydense = y;
    a.y32 = y32;
    a.m = A.m;
    const int32_t nwords = (A.nbc + 31) >> 5;
    const size_t dyn = ((size_t)nwords + ((size_t)A.nbc + 1) / 2) * 4;
    if (mode == M_F16) {
        a.cpw = rows_dx_cpw<M_F16>(A.nchunk, dyn);
        hipLaunchKernelGGL(k_rows_dx<M_F16>, dim3(grid_for(A.nchunk, a.cpw, INT_MAX)), dim3(TPB), dyn, s, a);
    } else {
        a.cpw = rows_dx_cpw<M_F32>(A.nchunk, dyn);
        hipLaunchKernelGGL(k_rows_dx<M_F32>, dim3(grid_for(A.nchunk, a.cpw, INT_MAX)), dim3(TPB), dyn, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_ballot_batch(const DevMatrix &A, const DevCtx &C, int mode, const void *x, int32_t nb,
                               int32_t NB, void *xdb, hipStream_t s)
{
    const int64_t xstride = (int64_t)A.nbc * BS;
    const int64_t lanes = (xstride + WAVE - 1) / WAVE * WAVE * NB;
    dim3 g(grid_for(lanes, TPB, INT_MAX)), b(TPB);
    if (mode == M_F16)
        hipLaunchKernelGGL(k_ballot_batch<M_F16>, g, b, 0, s, x, nb, A.n, xstride, NB, xdb, C.xmask, C.nxwords);
    else
        hipLaunchKernelGGL(k_ballot_batch<M_F32>, g, b, 0, s, x, nb, A.n, xstride, NB, xdb, C.xmask, C.nxwords);
    return hipGetLastError();
}

template <int MODE, int NB>
static hipError_t launch_rows_nb(const DevMatrix &A, const MainArgs &a, hipStream_t s)
{
    const int32_t nwords = (A.nbc + 31) >> 5;
    const size_t dyn = nwords <= LDS_BITMAP_WORDS ? (size_t)nwords * 4 : 0;
    MainArgs b = a;
    b.cpw = rows_cpw<MODE, NB>(A.nchunk, dyn);
    hipLaunchKernelGGL((k_rows<MODE, NB>), dim3(grid_for(A.nchunk, b.cpw, INT_MAX)), dim3(TPB), dyn, s, b);
    return hipGetLastError();
}

hipError_t launch_rows_batch(const DevMatrix &A, const DevCtx &C, int mode, int32_t NB, const void *xdb,
                             double *yaccb, hipStream_t s)
{
    MainArgs a;
    fill_main_args(A, C, mode, xdb, nullptr, 0, nullptr, a);
    a.xstride = (int64_t)A.nbc * BS;
    a.yacc = yaccb;
    a.ystride = (int64_t)A.nbr * BS;
    if (mode == M_F16) {
        switch (NB) {
        case 2: return launch_rows_nb<M_F16, 2>(A, a, s);
        case 4: return launch_rows_nb<M_F16, 4>(A, a, s);
        case 8: return launch_rows_nb<M_F16, 8>(A, a, s);
        default: return hipErrorInvalidValue;
        }
    }
    switch (NB) {
    case 2: return launch_rows_nb<M_F32, 2>(A, a, s);
    case 4: return launch_rows_nb<M_F32, 4>(A, a, s);
    case 8: return launch_rows_nb<M_F32, 8>(A, a, s);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_finalize_batch(const DevMatrix &A, const DevCtx &C, int mode, int32_t nb, int32_t NB,
                                 double *yaccb, void *y, float *y32, hipStream_t s)
{
    const int32_t nyw = (A.nbr + 1) / 2;
    const int64_t items = (int64_t)NB * A.m > C.nxwords ? (int64_t)NB * A.m : C.nxwords;
    dim3 g(grid_for(items, TPB, 4096)), b(TPB);
    const int64_t ystride = (int64_t)A.nbr * BS;
    if (mode == M_F16)
        hipLaunchKernelGGL(k_finalize_batch<M_F16>, g, b, 0, s, yaccb, ystride, nb, NB, A.m, y, y32, C.ybits, nyw,
                           C.xmask, C.nxwords, C.counters);
    else
        hipLaunchKernelGGL(k_finalize_batch<M_F32>, g, b, 0, s, yaccb, ystride, nb, NB, A.m, y, y32, C.ybits, nyw,
                           C.xmask, C.nxwords, C.counters);
    return hipGetLastError();
}

hipError_t launch_bfs_init(const DevMatrix &A, const DevCtx &C, int32_t source, int32_t *level,
                           int32_t *parent, hipStream_t s)
{
    int32_t nwords = (A.nbr + 1) / 2;
    dim3 g(grid_for(A.n, TPB, 4096)), b(TPB);
    hipLaunchKernelGGL(k_bfs_init, g, b, 0, s, A.n, source, level, parent, C.visited, C.nextm, C.xmask, nwords,
                       A.row_occ, C.counters);
    return hipGetLastError();
}

hipError_t launch_bfs_update(const DevMatrix &A, const DevCtx &C, int32_t next_level, int32_t *level,
                             hipStream_t s)
{
    int32_t nwords = (A.nbr + 1) / 2;
    // (every mask word holds some row below n: the last one holds block row
    // nbr - 1, whose first row is below m = n)
    dim3 g(grid_for(A.n, TPB, INT_MAX)), b(TPB);
    hipLaunchKernelGGL(k_bfs_update, g, b, 0, s, A.n, nwords, next_level, level, C.visited, C.nextm, C.xmask,
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
