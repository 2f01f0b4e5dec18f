/*
 * Seeded synthetic-graph generators shared by the tests, the benchmark and
 * the oracle's timing leg.  Holds none of the SpMSpV/BFS arithmetic: it only
 * produces input matrices.
 *
 * Random numbers: SplitMix64 (Steele, Lea and Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014) used as a counter-based
 * generator, value(i) = mix(seed + (i + 1) * golden_gamma).
 *
 * R-MAT (Chakrabarti, Zhan and Faloutsos, SDM 2004): every edge picks one of
 * the four quadrants (a, b, c, d) at each of `scale` recursion levels, most
 * significant bit first.  Quadrant a = (row bit 0, col bit 0), b = (0, 1),
 * c = (1, 0), d = (1, 1).  Each level uses 16 random bits, so probabilities
 * are quantised to 1/65536.  No noise and no vertex permutation.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static inline uint64_t sm64_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static inline uint64_t sm64_at(uint64_t seed, uint64_t i)
{
    return sm64_mix(seed + (i + 1) * 0x9E3779B97F4A7C15ULL);
}

/* LSD radix sort of 64-bit keys on the low `bits` bits, 11 bits a pass.
 * Returns the buffer that holds the result (a or tmp).                    */
#define RADIX_BITS 11
#define RADIX_SIZE (1 << RADIX_BITS)
static uint64_t *radix_sort_u64(uint64_t *a, uint64_t *tmp, int64_t cnt, int bits)
{
    int64_t hist[RADIX_SIZE];
    uint64_t *src = a, *dst = tmp;
    for (int shift = 0; shift < bits; shift += RADIX_BITS) {
        memset(hist, 0, sizeof(hist));
        for (int64_t i = 0; i < cnt; ++i) hist[(src[i] >> shift) & (RADIX_SIZE - 1)]++;
        int64_t s = 0;
        for (int d = 0; d < RADIX_SIZE; ++d) { int64_t c = hist[d]; hist[d] = s; s += c; }
        for (int64_t i = 0; i < cnt; ++i) dst[hist[(src[i] >> shift) & (RADIX_SIZE - 1)]++] = src[i];
        uint64_t *t = src; src = dst; dst = t;
    }
    return src;
}

/* Symmetrised, self-loop-free, de-duplicated R-MAT graph as CSR with sorted
 * columns.  row_ptr has n+1 entries (n = 2^scale); col_idx must hold
 * 2 * edge_factor * n entries.  Returns nnz, or -1 on allocation failure. */
int64_t wl_rmat_csr(int32_t scale, int32_t edge_factor, double a, double b, double c,
                    uint64_t seed, int64_t *row_ptr, int32_t *col_idx)
{
    const int64_t n = (int64_t)1 << scale;
    const int64_t E = (int64_t)edge_factor * n;
    const uint32_t ta = (uint32_t)(a * 65536.0 + 0.5);
    const uint32_t tb = (uint32_t)((a + b) * 65536.0 + 0.5);
    const uint32_t tc = (uint32_t)((a + b + c) * 65536.0 + 0.5);
    const int chunks = (scale + 3) / 4;
    uint64_t *keys = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)(2 * E));
    uint64_t *tmp = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)(2 * E));
    if (!keys || !tmp) { free(keys); free(tmp); return -1; }
    /* Edges are generated independently (counter-based random numbers), so
     * the loop runs in parallel; a self-loop leaves two all-ones sentinels,
     * which sort after every real key and are dropped below.              */
    const uint64_t SENT = ~0ULL;
    #pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < E; ++e) {
        uint64_t src = 0, dst = 0;
        int level = 0;
        for (int q = 0; q < chunks; ++q) {
            uint64_t r = sm64_at(seed, (uint64_t)e * (uint64_t)chunks + (uint64_t)q);
            for (int s = 0; s < 4 && level < scale; ++s, ++level) {
                uint32_t u = (uint32_t)((r >> (16 * s)) & 0xFFFF);
                /* a: (0,0)  b: (0,1)  c: (1,0)  d: (1,1), without branches */
                uint64_t ga = u >= ta, gb = u >= tb, gc = u >= tc;
                uint64_t rb = gb, cb = ga ^ gb ^ gc;
                src = (src << 1) | rb;
                dst = (dst << 1) | cb;
            }
        }
        if (src == dst) {
            keys[2 * e] = SENT;
            keys[2 * e + 1] = SENT;
        } else {
            keys[2 * e] = (src << scale) | dst;
            keys[2 * e + 1] = (dst << scale) | src;
        }
    }
    const int64_t cnt = 2 * E;
    int bits = 2 * scale;
    uint64_t *sorted = radix_sort_u64(keys, tmp, cnt, bits);
    for (int64_t i = 0; i <= n; ++i) row_ptr[i] = 0;
    int64_t nnz = 0;
    uint64_t prev = ~0ULL;
    for (int64_t i = 0; i < cnt; ++i) {
        uint64_t k = sorted[i];
        if (k == SENT) break;
        if (k == prev) continue;
        prev = k;
        int64_t r = (int64_t)(k >> scale);
        col_idx[nnz++] = (int32_t)(k & (uint64_t)(n - 1));
        row_ptr[r + 1]++;
    }
    for (int64_t i = 0; i < n; ++i) row_ptr[i + 1] += row_ptr[i];
    free(keys);
    free(tmp);
    return nnz;
}

/* Connected components of an undirected graph (symmetric CSR) by
 * union-find with path halving.  comp[v] = smallest vertex of v's
 * component.                                                              */
void wl_components(int32_t n, const int64_t *row_ptr, const int32_t *col_idx, int32_t *comp)
{
    for (int32_t v = 0; v < n; ++v) comp[v] = v;
    for (int32_t u = 0; u < n; ++u) {
        for (int64_t p = row_ptr[u]; p < row_ptr[u + 1]; ++p) {
            int32_t v = col_idx[p];
            int32_t ru = u, rv = v;
            while (comp[ru] != ru) { comp[ru] = comp[comp[ru]]; ru = comp[ru]; }
            while (comp[rv] != rv) { comp[rv] = comp[comp[rv]]; rv = comp[rv]; }
            if (ru == rv) continue;
            if (ru < rv) comp[rv] = ru; else comp[ru] = rv;
        }
    }
    for (int32_t v = 0; v < n; ++v) {
        int32_t r = v;
        while (comp[r] != r) r = comp[r];
        comp[v] = r;
    }
}
