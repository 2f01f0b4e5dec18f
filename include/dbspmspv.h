/*
 * dbspmspv.h -- C ABI of the MI355X (gfx950) dual-view blocked SpMSpV library.
 *
 * Implements the DB-SpMSpV method: y = A x with A and x both sparse
 * (Sec. 2.1), over a matrix cut once into 16x16 blocks that carries a
 * block-level CSR view and a block-level CSC view over ONE shared block
 * payload (Sec. 3.2.1), with per-call vector blocking (Sec. 3.2.2, 4.1), a
 * global push/pull choice (Sec. 3.3.1), per-block microkernels (Alg. 2-4,
 * Sec. 3.3.3), load-balanced scheduling (Sec. 3.3.2) and hierarchical
 * writeback (Sec. 3.3.3).  BFS (Sec. 4.2, Alg. 5) and sparse decoding
 * (Sec. 4.3) run on the same engine.
 *
 * General conventions
 * -------------------
 *  - Every call returns a dbs_status; no exception crosses the ABI.  On a
 *    non-OK status, dbs_last_error() returns a thread-local message.
 *  - Host-detectable argument errors are reported before anything is
 *    launched.  HIP runtime errors map to DBS_ERR_DEVICE.
 *  - Pointers named d_* are caller-owned DEVICE memory on the current HIP
 *    device; all other pointers are host memory.  The library never frees
 *    caller memory.  dbs_host_matrix, dbs_matrix and dbs_ctx objects are
 *    library-owned and released by their destroy calls (NULL is accepted).
 *  - Indices are 0-based int32.  Vector index lists must be unique and lie
 *    in [0, n); order is free.
 *  - Device calls are asynchronous on the context's stream unless a stats
 *    struct is requested, in which case they synchronize that stream.
 *  - A dbs_matrix is immutable after build and may be shared read-only by
 *    several contexts; one dbs_ctx must not be used by two host threads at
 *    once, and calls on one context run in stream order.
 *  - Output bitmaps/masks hold bit (i & 31) of 32-bit word (i >> 5) for row i.
 */
#ifndef DBSPMSPV_H
#define DBSPMSPV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DBS_OK = 0,
    DBS_ERR_ARG = 1,          /* invalid argument (null, range, duplicate, dtype mismatch) */
    DBS_ERR_ALLOC = 2,        /* host or device allocation failed */
    DBS_ERR_DEVICE = 3,       /* HIP runtime error or no usable gfx950 device */
    DBS_ERR_UNSUPPORTED = 4,  /* size or combination outside what this build supports */
    DBS_ERR_STATE = 5         /* object used in a wrong state */
} dbs_status;

typedef enum { DBS_F32 = 0, DBS_F16 = 1, DBS_PATTERN = 2 } dbs_dtype;
typedef enum { DBS_PLUS_TIMES = 0, DBS_OR_AND = 1 } dbs_semiring;
typedef enum { DBS_PATH_AUTO = 0, DBS_PATH_PUSH = 1, DBS_PATH_PULL = 2 } dbs_path;

/* Global selector threshold (Sec. 3.3.1): AUTO takes push iff
 * N_nzblk < th3 * N_blk.  The paper sets th3 = 0.01 on its GPUs; on MI355X,
 * over R-MAT graphs with uniform and clustered x (bench.py --ablation), the
 * same value gives the smallest summed time of these kernels' automatic
 * choices, so it is the default here too.
 * With the default (a th3 argument <= 0) the selector also takes push when x
 * is spread -- fewer than two of its indices per nonzero vector block -- and
 * N_nzblk < DBS_TH3_SPREAD * N_blk: push then visits blocks that mostly hold
 * one matching column, which measured faster than pull up to about that
 * activity, while clustered x (up to 16 indices per vector block) favours
 * pull from the paper's threshold on.  An explicit th3 > 0 gives the
 * paper's rule alone.
 * BFS levels (dbs_bfs) with the default th3 take push iff the level's push
 * tasks -- the blocks in the block-CSC lists of the frontier's nonzero
 * vector blocks, which the scan sums anyway -- are fewer than
 * DBS_BFS_PUSH_TASKS * nblk.  On R-MAT 22 the frontier's vector blocks stay
 * many (s_b 0.1-0.5) after the largest level, so the paper's rule keeps
 * pull there, while the visited rows leave push 1-10% of the blocks as
 * tasks; pull skips the block rows without unvisited rows, and the two
 * cross at a few percent of the blocks as tasks (whole BFS: the same mean
 * time within 1% for thresholds of 0.02-0.1 of nblk, 14% slower at 0.25).
 * An explicit th3 > 0 gives the paper's rule for BFS too.
 * Dense activations (dbs_spmspv_dense) on a matrix without COO blocks (a
 * decode layer) take pull under the default selector: push would win only
 * below about 1% active vector blocks, while launching its kernel for the
 * device's choice costs every call 2-4 us (of about 25 per call).         */
#define DBS_TH3_DEFAULT 0.01f
#define DBS_TH3_PAPER 0.01f
#define DBS_TH3_SPREAD 0.12f
#define DBS_BFS_PUSH_TASKS 0.1f

/* Low-level block formats (Sec. 3.2.1). */
typedef enum {
    DBS_BLK_COO = 0,    /* packed COO: 4-bit row | 4-bit column per entry    */
    DBS_BLK_DENSE = 1,  /* 256 values row-major, explicit zeros + row masks   */
    DBS_BLK_FCSR = 2,   /* ForceCSR: 16 row masks + row starts, row-major     */
    DBS_BLK_FCSC = 3,   /* ForceCSC: 16 column masks + column starts          */
    DBS_BLK_CSR = 4     /* patched CSR: row view + column starts + row_idx_csc2csr */
} dbs_block_type;
#define DBS_NUM_BLOCK_TYPES 5

/* Build options.  Defaults are the paper's constants: th0 = 32, th1 = 128,
 * th2 = 2.0 (Sec. 3.2.1, taken from CB-SpMV) and a pull segment closes once
 * its accumulated format weight reaches 16 (Sec. 3.3.2).  force_type = -1
 * classifies each block; 0..4 stores every block in that one format (the
 * format ablation of Sec. 5.4).                                             */
typedef struct {
    int32_t th0;        /* nnz < th0            -> COO   */
    int32_t th1;        /* nnz > th1            -> Dense */
    float th2;          /* skew ratio threshold -> ForceCSR / ForceCSC */
    int32_t seg_close;  /* pull segment closes when its weight >= seg_close (1..16 blocks) */
    int32_t force_type; /* -1 auto, else a dbs_block_type */
    int32_t inline_small; /* 1: COO blocks that fit (1 fp32, 2 fp16 or 6 pattern entries)
                             live in the descriptor word, no payload record; 0: never */
} dbs_build_opts;

/* Fills *o with the paper's defaults. */
void dbs_build_opts_default(dbs_build_opts *o);

typedef struct {
    int32_t m, n;               /* matrix shape */
    int64_t nnz;                /* stored entries */
    int32_t dtype;              /* dbs_dtype */
    int32_t nbr, nbc;           /* block rows / block columns, ceil(m/16), ceil(n/16) */
    int64_t nblk;               /* nonzero 16x16 blocks */
    int64_t nseg;               /* pull segments */
    int64_t blocks_by_type[DBS_NUM_BLOCK_TYPES];
    int64_t payload_bytes;      /* low-level block payload */
    int64_t db_bytes;           /* every array of the format (views, metadata, payload, segments) */
    int64_t csr_bytes;          /* plain CSR of the same matrix: (v + 4) nnz + 4 (m + 1) */
    int64_t csr_csc_bytes;      /* CSR plus CSC: csr_bytes + (v + 4) nnz + 4 (n + 1) */
} dbs_matrix_info;

typedef struct dbs_host_matrix dbs_host_matrix;  /* DB format in host memory (CPU only) */
typedef struct dbs_matrix dbs_matrix;            /* DB format resident on the GPU      */
typedef struct dbs_ctx dbs_ctx;                  /* per-stream workspace              */

/* ---------------------------------------------------------------------- */
/* Offline conversion (Sec. 3.1, 3.2.1; done once and reused, Sec. 5.5).  */
/* ---------------------------------------------------------------------- */

/* Converts a host CSR matrix into the DB format in host memory.
 *   m, n       shape (>= 0, < 2^31); nnz = row_ptr[m]
 *   row_ptr    int64[m+1], non-decreasing, row_ptr[0] = 0
 *   col_idx    int32[nnz] in [0, n); any order within a row; no duplicate (i,j)
 *   vals       nnz values of type vt (float for DBS_F32, IEEE binary16 bits
 *              for DBS_F16), ignored (may be NULL) for DBS_PATTERN
 *   opts       NULL for the defaults
 * Errors: DBS_ERR_ARG for malformed CSR or duplicates, DBS_ERR_UNSUPPORTED
 * when the number of nonzero blocks reaches 2^31.  Uses host threads only;
 * never touches a GPU.  The caller keeps ownership of the input arrays.     */
dbs_status dbs_host_build_csr(int32_t m, int32_t n, int64_t nnz, const int64_t *row_ptr,
                              const int32_t *col_idx, const void *vals, dbs_dtype vt,
                              const dbs_build_opts *opts, dbs_host_matrix **out);

dbs_status dbs_host_info(const dbs_host_matrix *h, dbs_matrix_info *out);

/* Read-only views of the host-side format, valid until dbs_host_destroy.
 * Layout (all little-endian):
 *   rb_ptr[nbr+1]   block-CSR row pointer (global_block_csr_row_ptr)
 *   cb_col[nblk]    block column of each block, primary order (global_block_csr_col_idx)
 *   cb_ptr[nbc+1]   block-CSC column pointer (global_block_csc_col_ptr)
 *   csc_row[nblk]   block row per CSC position (global_block_csc_row_idx)
 *   csc2csr[nblk]   primary block id per CSC position (global_block_csc2csr)
 *   desc[nblk]      bits 63..16 payload byte offset, 15..8 nnz-1, 2..0 block type;
 *                   bit 3 set: a COO block held inline, entry e at bits
 *                   16 + e (8 + 8V): coordinate byte, then the V value bytes
 *   payload         one record per block in primary order, V = value bytes
 *                   (4 for F32, 2 for F16, 0 for PATTERN), entries of a block
 *                   ordered by (local row, local column):
 *       COO    V*nnz values, then nnz coordinate bytes (row << 4 | col);
 *              record aligned to max(V, 1)
 *       DENSE  uint16 row_mask[16] (bit c = local column c), then 256 values
 *              row-major with explicit zeros; aligned to 16
 *       FCSR   uint16 row_mask[16], uint8 row_start[16], nnz values row-major
 *       FCSC   uint16 col_mask[16] (bit r = local row r), uint8 col_start[16],
 *              nnz values column-major
 *       CSR    uint16 row_mask[16], uint8 row_start[16], uint8 col_start[16],
 *              nnz bytes row_idx_csc2csr in column-major entry order
 *              (row << 4 | rank of the entry within its row) padded to 16,
 *              then nnz values row-major; the value of an entry is at
 *              row_start[row] + rank
 *   seg[nseg]       bits 31..0 first block, 58..32 block row, 62..59 blocks-1,
 *                   63 = the row block has exactly one segment              */
typedef struct {
    const int32_t *rb_ptr;
    const int32_t *cb_col;
    const int32_t *cb_ptr;
    const int32_t *csc_row;
    const int32_t *csc2csr;
    const uint64_t *desc;
    const uint8_t *payload;
    int64_t payload_bytes;
    const uint64_t *seg;
    int64_t nseg;
} dbs_host_arrays;

dbs_status dbs_host_arrays_get(const dbs_host_matrix *h, dbs_host_arrays *out);
void dbs_host_destroy(dbs_host_matrix *h);

/* The storage accounting used for the CSR and CSR+CSC columns of the
 * memory-overhead comparison (Table 4): CSR = (value_bytes + 4) nnz +
 * 4 (rows + 1); CSR+CSC adds (value_bytes + 4) nnz + 4 (cols + 1).         */
dbs_status dbs_storage_model(int64_t rows, int64_t cols, int64_t nnz, int32_t value_bytes,
                             int64_t *csr_bytes, int64_t *csr_csc_bytes);

/* ---------------------------------------------------------------------- */
/* Device-resident matrix.                                                */
/* ---------------------------------------------------------------------- */

/* Copies a host-side DB matrix to the current device (one upload).
 * DBS_ERR_UNSUPPORTED for more than 2^26 block columns (n > 2^30).          */
dbs_status dbs_matrix_upload(const dbs_host_matrix *h, dbs_matrix **out);

/* dbs_host_build_csr + dbs_matrix_upload + dbs_host_destroy. */
dbs_status dbs_matrix_build_csr(int32_t m, int32_t n, int64_t nnz, const int64_t *row_ptr,
                                const int32_t *col_idx, const void *vals, dbs_dtype vt,
                                const dbs_build_opts *opts, dbs_matrix **out);

/* GPU-side conversion (the offline step of Sec. 3.1, 3.2.1 and 3.3.2 run on
 * the device; for weights that are already in device memory, as decoding
 * loads them, Sec. 4.3).  d_w holds a dense m x n matrix, row-major with a
 * leading dimension of ld >= n elements, float (DBS_F32) or IEEE binary16
 * bits (DBS_F16); an entry is stored iff its value is nonzero (-0 is zero,
 * NaN is stored).  The result equals, array for array and byte for byte,
 * dbs_matrix_build_csr of the CSR of those entries with the same opts.
 * Kernels and copies run on `stream` (a hipStream_t, NULL = the default
 * stream); the call returns after they finish.  Temporary device memory:
 * 20 bytes per 16x16 tile plus O(m/16 + n/16).  d_w stays the caller's.
 * Errors: DBS_ERR_ARG for a bad shape, ld, dtype or opts; DBS_ERR_UNSUPPORTED
 * for n >= 2^26 or the limits of dbs_host_build_csr; DBS_ERR_DEVICE.       */
dbs_status dbs_matrix_build_dense(int32_t m, int32_t n, const void *d_w, int64_t ld, dbs_dtype vt,
                                  const dbs_build_opts *opts, void *stream, dbs_matrix **out);

dbs_status dbs_matrix_info_get(const dbs_matrix *A, dbs_matrix_info *out);
void dbs_matrix_destroy(dbs_matrix *A);

/* Sizes of the device arrays of a matrix (element counts). */
typedef struct {
    int64_t nslots;        /* 16 nseg: pull-segment slots */
    int64_t nseg;          /* segment words */
    int64_t nblk;          /* block-CSC positions */
    int32_t nbc;           /* block columns (block-CSC pointer has nbc + 1) */
    int32_t reserved;
    int64_t nheavy;        /* non-COO list entries */
    int64_t nchunk;        /* non-COO chunks (chunk starts have nchunk + 1) */
    int64_t payload_bytes; /* block payload */
} dbs_matrix_layout;

/* Host buffers for a copy of the device arrays (any member may be NULL to
 * skip that array), each at least as long as dbs_matrix_layout says:
 * slot words (bits 25..0 block column; bit 30 set for a COO block with one
 * entry held inline, bits 29..26 then that entry's local column; -1 for
 * padding and the sign bit set for a block of the non-COO list) and
 * descriptors,
 * segment words (the block row of each segment), the block-CSC
 * pointer, rows and descriptors, the non-COO list's block columns,
 * descriptors, chunk starts and chunk block rows, and the payload.         */
typedef struct {
    int32_t *sl_col;
    uint64_t *sl_desc;
    uint32_t *seg_rs;
    int32_t *cb_ptr;
    int32_t *csc_row;
    uint64_t *csc_desc;
    int32_t *hv_col;
    uint64_t *hv_desc;
    int32_t *hv_cstart;
    int32_t *hv_crow;
    uint8_t *payload;
} dbs_matrix_arrays;

dbs_status dbs_matrix_layout_get(const dbs_matrix *A, dbs_matrix_layout *out);
/* Copies the device arrays into the caller's host buffers (synchronous).    */
dbs_status dbs_matrix_download(const dbs_matrix *A, dbs_matrix_arrays *out);

/* ---------------------------------------------------------------------- */
/* Per-stream context: scratch masks, lists, dense x and y accumulators.  */
/* ---------------------------------------------------------------------- */

/* Creates a context sized for matrices up to sizing's shape (any matrix
 * with m and n not larger may be used with it).  stream is a hipStream_t
 * (NULL = the default stream).  Allocates O(m + n) device memory.          */
dbs_status dbs_ctx_create(const dbs_matrix *sizing, void *stream, dbs_ctx **out);
dbs_status dbs_ctx_set_stream(dbs_ctx *ctx, void *stream);
void dbs_ctx_destroy(dbs_ctx *ctx);

/* Single-launch execution (Sec. 4.1 generates the vector mask and counts
 * the nonzero blocks inside the SpMSpV launch).  enable != 0: a dbs_spmspv
 * call with at most 2048 x indices, on a matrix of at most 131072 block
 * columns, runs as ONE kernel launch -- blocker and selector in one
 * workgroup while the others wait on a ready word, the chosen traversal
 * (pull by the segment loop), then the compaction of y by the first
 * workgroups once every workgroup has set its own done word.  Same results
 * and statistics as the separate launches.  enable = 0 (the default of a
 * new context, and the only mode of dbs_spmspv_noalloc): blocker/scan,
 * traversal and compaction as kernels of their own, which measured faster
 * on the device (the single launch costs the host a third of the enqueue
 * time).  Single-launch calls on different streams may overlap in time.     */
dbs_status dbs_ctx_set_single_launch(dbs_ctx *ctx, int enable);

typedef struct {
    int32_t path;         /* dbs_path actually taken (PUSH or PULL) */
    int32_t n_nzblk;      /* nonzero vector blocks, N_nzblk (Sec. 3.3.1) */
    int32_t n_blk;        /* vector blocks, N_blk = ceil(n/16) */
    int32_t y_nnz;        /* entries written to y */
    int64_t tasks;        /* push: block tasks; pull: segments scanned */
    int32_t error_flags;  /* bit 0: x index out of range (skipped); bit 1: duplicate x index;
                             bit 2: single launch: a bounded wait for other workgroups ran
                             out (y is not valid) */
    int32_t reserved;
} dbs_call_stats;

/* SpMSpV y = A x (Sec. 2.1) under plus-times or Boolean OR-AND, with an
 * optional structural output mask.
 *   x_nnz, d_x_idx     k unique indices in [0, n), int32, any order
 *   d_x_val            k values of A's dtype (float / binary16); ignored for
 *                      DBS_OR_AND (may be NULL).  A listed index is active
 *                      whatever its value.
 *   d_mask             NULL, or ceil(m/32) uint32 words; with complement_mask
 *                      = 0 only rows whose bit is set may appear in y, with
 *                      complement_mask = 1 only rows whose bit is clear.
 *   path               AUTO: push iff N_nzblk < th3 N_blk (Sec. 3.3.1); or forced
 *   th3                <= 0 selects DBS_TH3_DEFAULT with the spread rule
 *                      (see DBS_TH3_SPREAD); > 0 the paper's rule with it
 *   d_y_idx            capacity m: the structural pattern of y ascending
 *                      (every row with a stored A[i][j] at a listed j that the
 *                      mask admits, including entries that sum to 0)
 *   d_y_val            capacity m values of A's dtype (NULL for DBS_OR_AND)
 *   d_y_nnz            one int32: nnz(y)
 *   stats              NULL, or filled after a stream synchronization
 * PATTERN matrices accept only DBS_OR_AND.  Values are accumulated in fp32
 * within a block segment and in fp64 across segments, then rounded once.
 * Out-of-range or duplicate x indices are not detected on the host; they are
 * skipped / flagged on the device and reported through stats.             */
dbs_status dbs_spmspv(dbs_ctx *ctx, const dbs_matrix *A, dbs_semiring sr, int32_t x_nnz,
                      const int32_t *d_x_idx, const void *d_x_val, const uint32_t *d_mask,
                      int complement_mask, dbs_path path, float th3, int32_t *d_y_idx,
                      void *d_y_val, int32_t *d_y_nnz, dbs_call_stats *stats);

/* SpMSpV without device allocation, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops and harnesses
 * that forbid hipMalloc.  Same operation, arguments, results and errors as
 * dbs_spmspv, with no context and no statistics: the scratch buffers of the
 * call (densified x, vector-block masks, push work items, fp64 y
 * accumulators, look-back status words, counters) live in one static device
 * array of DBS_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it
 * runs on until the process ends.  The call allocates nothing (no hipMalloc,
 * hipFree or allocating library routine); the caller passes x and y as for
 * dbs_spmspv.
 *   A        m and n at most DBS_NOALLOC_MAX_DIM, else DBS_ERR_UNSUPPORTED
 *            before anything is launched
 *   stream   a hipStream_t (NULL = the default stream); asynchronous
 * The first call on a device looks up that device's copy of the array,
 * fills it (all-ones bits in the densified x, zeros elsewhere) and waits for
 * the fill on `stream`; make that first call outside a graph capture.  Every
 * call leaves the array as it found it.  All calls on one GPU share that
 * GPU's array: calls that overlap in time on one GPU (on two streams, or
 * from two host threads) race and give undefined results; serialize them.
 * Consecutive calls alternate between two copies of the look-back status
 * words, chosen on the host, so a captured call cannot be replayed.  The
 * pull path takes the segment loop at every activity: the compaction list
 * of moderate activities would need memory proportional to the matrix.     */
#define DBS_NOALLOC_MAX_DIM (1 << 20)
#define DBS_NOALLOC_SCRATCH_BYTES (14u << 20)
dbs_status dbs_spmspv_noalloc(const dbs_matrix *A, dbs_semiring sr, int32_t x_nnz, const int32_t *d_x_idx,
                              const void *d_x_val, const uint32_t *d_mask, int complement_mask,
                              dbs_path path, float th3, int32_t *d_y_idx, void *d_y_val, int32_t *d_y_nnz,
                              void *stream);

/* Sparse decode linear layer (Sec. 4.3): y = A a with a DENSE activation a
 * of length n in A's dtype whose entries are active iff nonzero (+0 and -0
 * are inactive); the vector blocks are built on the GPU by a wave ballot
 * (Sec. 4.1).  d_y_dense receives all m outputs in A's dtype (rows with no
 * active product are 0), rounded to nearest even from the fp64 sum.
 * d_y_f32 (NULL allowed) receives the same sums rounded to fp32.
 * path AUTO with th3 <= 0 on a matrix without COO blocks takes pull (see
 * DBS_TH3_DEFAULT); th3 > 0 applies the paper's rule on the device.
 * F32 and F16 matrices only.                                               */
dbs_status dbs_spmspv_dense(dbs_ctx *ctx, const dbs_matrix *A, const void *d_x_dense,
                            dbs_path path, float th3, void *d_y_dense, float *d_y_f32,
                            dbs_call_stats *stats);

/* Batched sparse decode: Y = A X for nb dense activations at once (several
 * tokens per pass), each as in dbs_spmspv_dense (Sec. 4.3); the paper leaves
 * several vectors per pass (SpMM) to future work (Limitations).
 *   d_x        nb x n activations, row-major, A's dtype (active iff nonzero)
 *   d_y        nb x m outputs, row-major, A's dtype, rounded to nearest even
 *              from the fp64 sums; d_y_f32 (NULL allowed) nb x m fp32 sums
 *   nb         1 .. DBS_MAX_BATCH
 * For a matrix without COO blocks (every block Dense / ForceCSR / ForceCSC /
 * patched CSR, the regime of pruned decode layers) the nb vectors share one
 * pull pass: the blocks active for any vector are visited once and every
 * stored value is loaded once for all of them (the path is pull; N_nzblk in
 * stats counts the union of the vectors' vector blocks).  Otherwise, or for
 * nb = 1, the vectors are taken one dbs_spmspv_dense call each.  The first
 * batched call allocates DBS_MAX_BATCH padded x copies and fp64 accumulator
 * sets for the context's largest shape (kept until dbs_ctx_destroy).        */
#define DBS_MAX_BATCH 8
dbs_status dbs_spmm_dense(dbs_ctx *ctx, const dbs_matrix *A, int32_t nb, const void *d_x, void *d_y,
                          float *d_y_f32, dbs_call_stats *stats);

#define DBS_BFS_MAX_LEVEL_STATS 64
typedef struct {
    int32_t levels;               /* nonempty levels including the source's */
    int32_t reached;              /* vertices with level >= 0 */
    int32_t path[DBS_BFS_MAX_LEVEL_STATS];      /* per level: DBS_PATH_PUSH / PULL */
    int32_t frontier[DBS_BFS_MAX_LEVEL_STATS];  /* per level: frontier size */
} dbs_bfs_stats;

/* BFS from `source` (Sec. 4.2, Alg. 5): each level's frontier is the sparse
 * x of a Boolean SpMSpV masked by the complement of the visited set; push or
 * pull is chosen per level on the device: by the push task count with the
 * default th3 (DBS_BFS_PUSH_TASKS), by the paper's rule for th3 > 0, or
 * forced by policy.
 * Edge u -> v iff A[v][u] is stored; A must be square.  A matrix built
 * from CSR on the host also carries which rows hold entries: BFS counts the
 * others as visited from the start (no edge reaches them), so that pull
 * levels skip their block rows sooner; the results are the same.
 *   d_level[n]   level of each vertex, -1 if unreachable, level[source] = 0
 *   d_parent[n]  smallest-id vertex of the previous level with an edge to v;
 *                parent[source] = source; -1 if unreachable
 * The host reads one small counter per level to detect termination.
 * stats (NULL allowed) is filled on return.                                */
dbs_status dbs_bfs(dbs_ctx *ctx, const dbs_matrix *A, int32_t source, int32_t *d_level,
                   int32_t *d_parent, dbs_path policy, float th3, dbs_bfs_stats *stats);

/* ---------------------------------------------------------------------- */
/* Basic push / pull baselines (Alg. 1, Sec. 2.1-2.2).                    */
/* ---------------------------------------------------------------------- */

/* The two fixed paradigms the method is measured against in the paper's
 * motivation: column-driven push over a plain CSC and row-driven pull over
 * a plain CSR, with no blocking, no selector and no load balancing.  They
 * exist for ablation and comparison only; the blocked method never uses
 * them.  F32 only. */
typedef struct dbs_basic_matrix dbs_basic_matrix;

/* Copies the CSR of A (same conventions as dbs_host_build_csr: row_ptr of
 * m+1 int64, nnz int32 columns in [0, n), nnz float values) to the current
 * device and builds its CSC there-from on the host (rows ascending within a
 * column).  Duplicate (i, j) entries are kept and summed.  Allocates
 * O(m + n + nnz) device memory, including an n-float dense-x scratch that
 * is all zero between calls.                                              */
dbs_status dbs_basic_build(int32_t m, int32_t n, int64_t nnz, const int64_t *row_ptr,
                           const int32_t *col_idx, const float *vals, dbs_basic_matrix **out);
void dbs_basic_destroy(dbs_basic_matrix *B);

/* y = A x into a DENSE fp32 d_y[m] (rows without a product are 0).
 *   path = DBS_PATH_PULL: every row i sums a_ij * x_j over all its stored
 *          entries against the dense x scratch (x scattered into it, then
 *          cleared again after the row pass); fp32 sums, one write per row.
 *   path = DBS_PATH_PUSH: d_y is zeroed, then every listed x_j adds
 *          a_ij * x_j into d_y[i] along column j with fp32 atomics (order,
 *          hence rounding, not deterministic).
 * x: x_nnz unique int32 indices (out-of-range ones are skipped) and fp32
 * values, device memory.  Asynchronous on `stream` (a hipStream_t, NULL =
 * default stream).  Calls that share one dbs_basic_matrix must not overlap
 * in time (the dense-x scratch is shared).                                 */
dbs_status dbs_basic_spmspv(dbs_basic_matrix *B, dbs_path path, int32_t x_nnz, const int32_t *d_x_idx,
                            const float *d_x_val, float *d_y, void *stream);

/* ---------------------------------------------------------------------- */
/* Measurement hooks.                                                     */
/* ---------------------------------------------------------------------- */

/* Kernel classes timed with HIP events on the context's stream. */
typedef enum {
    DBS_K_SCATTER = 0,   /* vector blocker: scatter x or ballot a dense x     */
    DBS_K_SCAN = 1,      /* active vector-block list, task offsets, selector
                            (with the blocker too for up to 2048 x indices)   */
    DBS_K_MAIN = 2,      /* push or pull traversal with block microkernels    */
    DBS_K_FINALIZE = 3,  /* compaction / conversion of y, scratch reset       */
    DBS_K_BFS_UPDATE = 4,/* BFS level, visited and frontier update            */
    DBS_K_OTHER = 5,     /* BFS init / finish                                 */
    DBS_K_FUSED = 6,     /* single launch: blocker, selector, traversal and
                            compaction of y (up to 2048 x indices)            */
    DBS_K_COUNT = 7
} dbs_kernel_class;

typedef struct {
    double ms[DBS_K_COUNT];        /* summed event time per class */
    int64_t launches[DBS_K_COUNT]; /* launches per class */
} dbs_timing;

/* enable != 0 records a HIP event pair around every kernel launched on the
 * context from now on.  dbs_ctx_read_timing synchronizes the stream, returns
 * the sums since the last read, and clears them.                          */
dbs_status dbs_ctx_enable_timing(dbs_ctx *ctx, int enable);
dbs_status dbs_ctx_read_timing(dbs_ctx *ctx, dbs_timing *out);

const char *dbs_last_error(void);
const char *dbs_version(void);

#ifdef __cplusplus
}
#endif
#endif /* DBSPMSPV_H */
