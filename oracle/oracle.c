/*
 * Plain CPU oracle for sparse-matrix x sparse-vector products and BFS.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file: only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header or table with the
 * GPU library; both sides only receive the same seeded inputs.
 *
 * What is computed (DB-SpMSpV paper, Sec. 2.1 "SpMSpV" and Alg. 1, push
 * form): y = A x with A and x both sparse.  The oracle is the plain
 * definition, written as the sequential column gather of Alg. 1 (top) with a
 * dense sparse accumulator:
 *
 *     for every listed (j, x_j):  for every stored A[i][j]:
 *         acc[i] += A[i][j] * x_j       (fp64; fp32 and fp16 products are exact)
 *
 * The output pattern is structural: y_idx = { i : exists listed j with A[i][j]
 * stored } minus the rows excluded by the optional output mask, ascending.
 * Entries that cancel to 0.0 stay in the pattern.
 *
 * BFS (Sec. 4.2 "DB-BFS", Alg. 5 semantics): level-synchronous traversal in
 * which level L+1 is the set of unvisited vertices with an edge from level L.
 * Edge u -> v exists iff A[v][u] is stored (column u lists the successors of
 * u, as in y = A x with x the frontier).  The parent of v is the smallest
 * vertex id u of level L(v)-1 with an edge u -> v; parent[source] = source;
 * unreachable vertices keep level = parent = -1.  Processing each level's
 * frontier in ascending id order makes the first discoverer the minimum.
 *
 * All functions are single-threaded and allocate only what they document.
 */
#define _POSIX_C_SOURCE 199309L
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <time.h>

/* --------------------------------------------------------------------- */
/* CSC from CSR by a stable counting sort: within each column the rows come
 * out ascending because rows are visited in ascending order.  The oracle's
 * own conversion, built once per matrix.                                  */
int oracle_csc_from_csr(int32_t m, int32_t n, int64_t nnz,
                        const int64_t *row_ptr, const int32_t *col_idx,
                        const double *vals, /* may be NULL (pattern) */
                        int64_t *col_ptr,   /* n+1 */
                        int32_t *row_idx,   /* nnz */
                        double *cvals)      /* nnz, NULL iff vals NULL */
{
    if (m < 0 || n < 0 || nnz < 0) return 1;
    if (row_ptr[0] != 0 || row_ptr[m] != nnz) return 2;
    for (int64_t j = 0; j <= n; ++j) col_ptr[j] = 0;
    for (int64_t p = 0; p < nnz; ++p) {
        int32_t j = col_idx[p];
        if (j < 0 || j >= n) return 3;
        col_ptr[j + 1] += 1;
    }
    for (int64_t j = 0; j < n; ++j) col_ptr[j + 1] += col_ptr[j];
    int64_t *next = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    if (!next) return 4;
    for (int64_t j = 0; j < n; ++j) next[j] = col_ptr[j];
    for (int32_t i = 0; i < m; ++i) {
        if (row_ptr[i + 1] < row_ptr[i]) { free(next); return 2; }
        for (int64_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) {
            int64_t q = next[col_idx[p]]++;
            row_idx[q] = i;
            if (vals) cvals[q] = vals[p];
        }
    }
    free(next);
    return 0;
}

static int cmp_i32(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/* Row i survives the output mask: bit (i & 31) of word (i >> 5); the
 * complement flag inverts the test.  NULL mask admits every row.          */
static int row_allowed(const uint32_t *mask, int complement, int32_t i)
{
    if (!mask) return 1;
    int bit = (int)((mask[i >> 5] >> (i & 31)) & 1u);
    return complement ? !bit : bit;
}

/* Plus-times SpMSpV.  Workspace arrays acc[m], sabs[m] (double) and
 * seen[m] (uint8) must be all zero on entry; they are all zero again on
 * return.  touched[m] is scratch.  Outputs (capacity m): y_idx ascending,
 * y_val the fp64 sum, y_abs the sum of |A[i][j] x_j| (the tolerance scale).
 * Listed x indices must be unique (the Python wrapper checks this).
 * Returns nnz(y), or -1 when an index lies outside [0, n).               */
int64_t oracle_spmspv(int32_t m, int32_t n,
                      const int64_t *col_ptr, const int32_t *row_idx,
                      const double *cvals,
                      int32_t k, const int32_t *x_idx, const double *x_val,
                      const uint32_t *mask, int complement,
                      double *acc, double *sabs, uint8_t *seen,
                      int32_t *touched,
                      int32_t *y_idx, double *y_val, double *y_abs)
{
    int64_t nt = 0;
    for (int32_t t = 0; t < k; ++t) {
        int32_t j = x_idx[t];
        if (j < 0 || j >= n) return -1;
        double xj = x_val[t];
        for (int64_t p = col_ptr[j]; p < col_ptr[j + 1]; ++p) {
            int32_t i = row_idx[p];
            if (!row_allowed(mask, complement, i)) continue;
            double prod = cvals[p] * xj;
            acc[i] += prod;
            sabs[i] += prod < 0 ? -prod : prod;
            if (!seen[i]) { seen[i] = 1; touched[nt++] = i; }
        }
    }
    qsort(touched, (size_t)nt, sizeof(int32_t), cmp_i32);
    for (int64_t t = 0; t < nt; ++t) {
        int32_t i = touched[t];
        y_idx[t] = i;
        y_val[t] = acc[i];
        y_abs[t] = sabs[i];
        acc[i] = 0.0; sabs[i] = 0.0; seen[i] = 0;
    }
    (void)m;
    return nt;
}

/* Boolean OR-AND SpMSpV: only the structural pattern of y.  Values of A and
 * x play no part.  seen[m] zero on entry and on return.                   */
int64_t oracle_spmspv_bool(int32_t m, int32_t n,
                           const int64_t *col_ptr, const int32_t *row_idx,
                           int32_t k, const int32_t *x_idx,
                           const uint32_t *mask, int complement,
                           uint8_t *seen, int32_t *y_idx)
{
    int64_t nt = 0;
    for (int32_t t = 0; t < k; ++t) {
        int32_t j = x_idx[t];
        if (j < 0 || j >= n) return -1;
        for (int64_t p = col_ptr[j]; p < col_ptr[j + 1]; ++p) {
            int32_t i = row_idx[p];
            if (!row_allowed(mask, complement, i)) continue;
            if (!seen[i]) { seen[i] = 1; y_idx[nt++] = i; }
        }
    }
    qsort(y_idx, (size_t)nt, sizeof(int32_t), cmp_i32);
    for (int64_t t = 0; t < nt; ++t) seen[y_idx[t]] = 0;
    (void)m;
    return nt;
}

/* Level-synchronous BFS over the CSC columns (column u = successors of u).
 * level[n], parent[n] are outputs.  frontier[n] and next[n] are scratch.
 * Returns the number of nonempty levels (eccentricity of the source + 1), or
 * -1 for a bad source.                                                       */
int32_t oracle_bfs(int32_t n, const int64_t *col_ptr, const int32_t *row_idx,
                   int32_t source, int32_t *level, int32_t *parent,
                   int32_t *frontier, int32_t *next)
{
    if (source < 0 || source >= n) return -1;
    for (int32_t v = 0; v < n; ++v) { level[v] = -1; parent[v] = -1; }
    level[source] = 0;
    parent[source] = source;
    frontier[0] = source;
    int64_t nf = 1;
    int32_t L = 0;
    while (nf > 0) {
        qsort(frontier, (size_t)nf, sizeof(int32_t), cmp_i32);
        int64_t nn = 0;
        for (int64_t t = 0; t < nf; ++t) {
            int32_t u = frontier[t];
            for (int64_t p = col_ptr[u]; p < col_ptr[u + 1]; ++p) {
                int32_t v = row_idx[p];
                if (level[v] == -1) {
                    level[v] = L + 1;
                    parent[v] = u;
                    next[nn++] = v;
                }
            }
        }
        int32_t *tmp = frontier; frontier = next; next = tmp;
        nf = nn;
        L += 1;
    }
    return L;
}

/* Wall-clock timing of `reps` repeated oracle_spmspv calls over a list of
 * vectors (used only for the CPU baseline).  x vectors are concatenated:
 * vector v occupies [x_off[v], x_off[v+1]).  Returns seconds.             */
double oracle_time_spmspv(int32_t m, int32_t n,
                          const int64_t *col_ptr, const int32_t *row_idx,
                          const double *cvals,
                          int32_t nvec, const int64_t *x_off,
                          const int32_t *x_idx, const double *x_val,
                          int32_t reps,
                          double *acc, double *sabs, uint8_t *seen,
                          int32_t *touched,
                          int32_t *y_idx, double *y_val, double *y_abs)
{
    struct timespec t0, t1;
    clock_gettime(CLOCK_MONOTONIC, &t0);
    for (int32_t r = 0; r < reps; ++r)
        for (int32_t v = 0; v < nvec; ++v)
            oracle_spmspv(m, n, col_ptr, row_idx, cvals,
                          (int32_t)(x_off[v + 1] - x_off[v]),
                          x_idx + x_off[v], x_val + x_off[v], NULL, 0,
                          acc, sabs, seen, touched, y_idx, y_val, y_abs);
    clock_gettime(CLOCK_MONOTONIC, &t1);
    return (double)(t1.tv_sec - t0.tv_sec) + 1e-9 * (double)(t1.tv_nsec - t0.tv_nsec);
}

/* Wall-clock timing of one BFS from each listed source.  Returns seconds. */
double oracle_time_bfs(int32_t n, const int64_t *col_ptr, const int32_t *row_idx,
                       int32_t nsrc, const int32_t *sources,
                       int32_t *level, int32_t *parent,
                       int32_t *frontier, int32_t *next)
{
    struct timespec t0, t1;
    clock_gettime(CLOCK_MONOTONIC, &t0);
    for (int32_t s = 0; s < nsrc; ++s)
        oracle_bfs(n, col_ptr, row_idx, sources[s], level, parent, frontier, next);
    clock_gettime(CLOCK_MONOTONIC, &t1);
    return (double)(t1.tv_sec - t0.tv_sec) + 1e-9 * (double)(t1.tv_nsec - t0.tv_nsec);
}
