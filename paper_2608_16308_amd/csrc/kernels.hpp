// Host-side launch interface of the gfx950 kernels (implemented in kernels.hip).
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace dbs {

// Device-resident DB matrix (Sec. 3.2.1): dual block views over one payload.
//
// On the device the primary (block-CSR) order is laid out in pull-segment
// slots: segment s owns slots [16 s, 16 s + 16), its blocks in block-CSR
// order followed by padding (block column -1).  A pull lane thus finds its
// block column and descriptor at 16 s + lane without first reading the
// segment.  The block-CSC view holds each block's descriptor (csc_desc)
// next to its block row instead of its primary id, so that push reaches a
// block's record in one step.  The payload records are unchanged.
struct DevMatrix {
    int32_t m = 0, n = 0, nbr = 0, nbc = 0;
    int64_t nblk = 0, nseg = 0;
    int32_t dtype = 0;  // dbs_dtype
    const int32_t *sl_col = nullptr;    // 16 nseg: block column, -1 = padding, sign bit = non-COO (listed)
    const uint64_t *sl_desc = nullptr;  // 16 nseg: descriptor
    const uint32_t *seg_rs = nullptr;   // nseg: block row of the segment
    const int32_t *cb_ptr = nullptr;    // block-CSC view: column pointer (nbc + 1)
    const int32_t *csc_row = nullptr;   // block row per CSC position
    const uint64_t *csc_desc = nullptr; // descriptor per CSC position
    // The non-COO blocks in block-CSR order (pull takes them row-per-lane,
    // see pull_rows), cut into chunks of at most HV_CHUNK consecutive blocks
    // of one block row: chunk c holds list entries hv_cstart[c] ..
    // hv_cstart[c + 1] - 1 of block row hv_crow[c].
    const int32_t *hv_col = nullptr;     // nheavy: block column
    const uint64_t *hv_desc = nullptr;   // nheavy: descriptor
    const int32_t *hv_cstart = nullptr;  // nchunk + 1
    const int32_t *hv_crow = nullptr;    // nchunk
    const int32_t *hv_rowchunks = nullptr;  // nbr: chunks of each block row
    int64_t nheavy = 0, nchunk = 0;
    const uint8_t *pay = nullptr;
    // Segment-loop tasks (PULL_TASK_SEGS consecutive segments each) in
    // descending order of their stored-COO work, so that the waves, dealt
    // the tasks in this order, get even shares (NULL: the tasks in segment
    // order, as for a matrix converted on the device).
    const int32_t *task_order = nullptr;
    int32_t ntask = 0;
    // The rows that hold entries, a 16-bit mask per block row, two per word
    // ((nbr + 1) / 2 words; NULL when not known, as for a matrix converted
    // on the device).  BFS counts the other rows as reached from the start:
    // no edge leads to them, and the pull levels then skip whole block rows
    // sooner.
    const uint32_t *row_occ = nullptr;
};

// Segments per segment-loop task: two wave iterations of 16 segments.
constexpr int32_t PULL_TASK_SEGS = 32;

// Counter slots in the context's device counter array.
enum Counter : int {
    C_NZBLK = 0,     // nonzero vector blocks of this call
    C_TASKS = 1,     // push block tasks (sum of block-CSC lengths of active columns)
    C_PATH = 2,      // 1 push, 2 pull
    C_YNNZ = 3,      // entries written to y
    C_XBAD = 4,      // x indices out of range, counted by the blocker during this call
    C_ERR_LAST = 5,  // error bits of the last completed call
    // (6: unused)
    C_NZACC = 7,     // nonzero vector blocks, summed by the scan tiles (consumed by its last tile)
    C_NTB = 8,       // push work items (nonzero vector blocks with a nonempty block column)
    C_XPOP = 9,      // distinct x indices (mask popcounts), summed by the scan tiles
    C_SYNCERR = 10,  // single launch: a bounded wait for other workgroups ran out
    C_COUNT = 12
};
constexpr int PATH_PUSH = 1, PATH_PULL = 2;
#ifndef HV_CHUNK_BLOCKS
#define HV_CHUNK_BLOCKS 16
#endif
// blocks per chunk of the non-COO list (at most one per lane of a quarter-wave)
constexpr int HV_CHUNK = HV_CHUNK_BLOCKS;
static_assert(HV_CHUNK >= 1 && HV_CHUNK <= 16, "chunk size");

// Tile sizes of the look-back scans (vector blocks per thread of the active
// block scan; 32-row structure words per workgroup of the y compaction).
#ifndef SCAN_ITEMS_PER_THREAD
#define SCAN_ITEMS_PER_THREAD 4
#endif
#ifndef FINALIZE_WORDS
#define FINALIZE_WORDS 128
#endif
int32_t scan_tiles(int32_t nbc);      // workgroups (and status words) of the scan
int32_t finalize_tiles(int32_t nbr);  // workgroups (and status words) of the compaction

// Per-context scratch.  Every buffer is sized for the largest matrix the
// context was created for and is all-zero between calls (each call clears
// exactly what it touched).
struct DevCtx {
    void *xd = nullptr;           // dense x values, 16 * nbc entries (fp32 or fp16)
    uint32_t *xmask = nullptr;    // blk_x_mask, two 16-bit masks per word
    int32_t nxwords = 0;
    uint32_t *xbits = nullptr;    // one activity bit per vector block, written by the scan
    // push work items, one per active vector block with blocks, ascending
    // (nbc + 1): {first task (exclusive scan of block-CSC lengths), vector
    // block, pbase, 0}; task t of item a visits block-CSC position pbase + t;
    // item NT holds the task count
    int4 *items = nullptr;
    double *yacc = nullptr;       // y accumulators (16 * nbr)
    uint32_t *ybits = nullptr;    // y structure, two 16-bit row-block masks per word
    int32_t nywords = 0;
    uint32_t *visited = nullptr;  // BFS visited bitmap (row-block words)
    uint32_t *nextm = nullptr;    // BFS next-frontier bitmap
    int32_t *counters = nullptr;  // C_COUNT int32
    int32_t *rdone = nullptr;     // nbr: chunks of a block row committed so far (dense-output pass)
    // Look-back status words of the two scans, in two copies each: a call
    // uses copy `parity` and clears the other copy for the next call, so no
    // other kernel has to clean up after a scan.
    uint64_t *st_scan[2] = {nullptr, nullptr};  // active-block scan
    int32_t n_st_scan = 0;
    uint64_t *st_fin[2] = {nullptr, nullptr};   // y compaction
    int32_t n_st_fin = 0;
    int scan_parity = 0, fin_parity = 0;
    // Compacted pull (moderate x activity): per-wave regions of active slot
    // ids and their counts; written and read within one call.
    int32_t *clist = nullptr;
    int64_t clist_cap = 0;
    uint32_t *ccount = nullptr;
    // Single launch (short index lists): ready / all-done words (eight
    // copies) and one done word per workgroup (SYNC_WORDS in all), and the
    // number of the last such call (the words hold it once written; 0 is
    // never used).
    uint32_t *sync = nullptr;
    uint32_t gen = 0;
};
constexpr int32_t SYNC_WORDS = 8 * 1024 + 4096;
// Entries and regions of the compacted pull's list for a matrix of nseg
// pull segments.
int64_t compact_list_entries(int64_t nseg);
int32_t compact_list_regions();

enum Mode : int { M_F32 = 0, M_F16 = 1, M_BOOL = 2, M_BFS = 3 };

hipError_t launch_scatter(const DevMatrix &A, const DevCtx &C, int mode, int32_t k,
                          const int32_t *x_idx, const void *x_val, hipStream_t s);
hipError_t launch_ballot(const DevMatrix &A, const DevCtx &C, int mode, const void *x_dense,
                         hipStream_t s);
// th3s > 0: the spread rule as well; tasks_max >= 0: push iff fewer push
// tasks than that, in place of both (BFS levels; see k_scan)
hipError_t launch_scan(const DevMatrix &A, DevCtx &C, int forced_path, double th3, double th3s,
                       hipStream_t s, double tasks_max = -1.0);
// Blocker and scan as one single-workgroup kernel, for up to SMALL_X_MAX
// indices and an activity bitmap of up to SMALL_X_WORDS words (small_x_fits);
// otherwise launch_scatter + launch_scan.
constexpr int32_t SMALL_X_MAX = 2048;
constexpr int32_t SMALL_X_WORDS = 8192;
bool small_x_fits(const DevMatrix &A, int32_t k);
hipError_t launch_small_x(const DevMatrix &A, const DevCtx &C, int mode, int32_t k, const int32_t *x_idx,
                          const void *x_val, int forced_path, double th3, double th3s, hipStream_t s);
// Blocker, selector, traversal and compaction of y in one launch, for an
// index list small_x_fits accepts whose activity bitmap also fits the pull
// kernel's LDS copy (fused_fits); valued and OR-AND modes.
bool fused_fits(const DevMatrix &A, int32_t k);
hipError_t launch_fused(const DevMatrix &A, DevCtx &C, int mode, int32_t k, const int32_t *x_idx,
                        const void *x_val, const uint32_t *omask, int complement, int forced_path, double th3,
                        double th3s, int32_t *y_idx, void *y_val, int32_t *y_nnz, hipStream_t s);
// Dense activation with n a multiple of 16 and a 16-byte aligned x: the
// blocker runs inside the scan (one launch fewer).
bool scan_takes_dense(const DevMatrix &A, const void *x_dense);
hipError_t launch_scan_dense(const DevMatrix &A, DevCtx &C, int mode, const void *x_dense, int forced_path,
                             double th3, double th3s, hipStream_t s);
// Launches the traversal: the pull kernel then the push kernel for an
// automatic path (the one the scan did not choose returns at once; the push
// kernel also walks the compacted pull's list), or only what the forced path
// needs.
hipError_t launch_main(const DevMatrix &A, const DevCtx &C, int mode, const void *xd,
                       const uint32_t *omask, int complement, int32_t *parent, int forced_path,
                       hipStream_t s);
hipError_t launch_finalize(const DevMatrix &A, DevCtx &C, int mode, int32_t *y_idx,
                           void *y_val, int32_t *y_nnz, const int32_t *x_idx, int32_t k,
                           hipStream_t s);
hipError_t launch_finalize_dense(const DevMatrix &A, const DevCtx &C, int mode, void *y,
                                 float *y32, hipStream_t s);
// Dense activation, pull on a matrix without COO blocks: the non-COO pass
// reading the activation itself, with no scan before it and writing the
// dense output y (and y32 when not NULL) itself (k_rows_dx), when
// rows_dx_fits (for a valued matrix: the conditions of scan_takes_dense, no
// COO block, at most ROWS_DX_MAX_NBC vector blocks).
bool rows_dx_fits(const DevMatrix &A, const void *x_dense);
hipError_t launch_rows_dx(const DevMatrix &A, const DevCtx &C, int mode, const void *x_dense, void *y,
                          float *y32, hipStream_t s);
// Batched dense activations (NB in {2, 4, 8} vectors per pass, nb <= NB of
// them real): the padded copies into xdb (NB * 16 nbc entries) and their
// union mask; the pull over a matrix without COO blocks into yaccb (NB * 16
// nbr accumulators); the dense outputs of the nb real vectors.
hipError_t launch_ballot_batch(const DevMatrix &A, const DevCtx &C, int mode, const void *x, int32_t nb,
                               int32_t NB, void *xdb, hipStream_t s);
hipError_t launch_rows_batch(const DevMatrix &A, const DevCtx &C, int mode, int32_t NB, const void *xdb,
                             double *yaccb, hipStream_t s);
hipError_t launch_finalize_batch(const DevMatrix &A, const DevCtx &C, int mode, int32_t nb, int32_t NB,
                                 double *yaccb, void *y, float *y32, hipStream_t s);
hipError_t launch_bfs_init(const DevMatrix &A, const DevCtx &C, int32_t source, int32_t *level,
                           int32_t *parent, hipStream_t s);
hipError_t launch_bfs_update(const DevMatrix &A, const DevCtx &C, int32_t next_level,
                             int32_t *level, hipStream_t s);
hipError_t launch_bfs_finish(const DevMatrix &A, int32_t *parent, hipStream_t s);


}  // namespace dbs
