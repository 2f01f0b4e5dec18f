// Basic push and pull SpMSpV over plain CSC / CSR (Alg. 1), the two fixed
// paradigms that motivate the method (Sec. 2.1, 2.2): comparison baselines
// for the ablation, not part of the blocked method.
//
//   pull  row-driven over the CSR of A: every row sums a_ij * x_j over all
//         of its stored entries against a dense x (zeros where x is not
//         stored), so inactive columns cost a gather each; y is written for
//         every row.
//   push  column-driven over the CSC of A: every stored x_j walks column j
//         and adds a_ij * x_j into y_i with an fp32 global atomic.
//
// Wave64 mapping: pull gives each row a quarter-wave (16 lanes, four loads
// in flight per lane, a 16-lane shuffle reduction); push gives each x entry
// a whole wave (four loads in flight per lane).  Neither balances long rows
// or columns: that is what the blocked method's segments and flattened
// block tasks add (Sec. 3.3.2).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <new>
#include <vector>

#include "internal.hpp"

namespace {

constexpr int BTPB = 256;
constexpr int BUNROLL = 4;

// Writes (or, with clear, zeroes again) the listed entries of the dense x.
__global__ __launch_bounds__(BTPB) void k_basic_scatter(const int32_t *__restrict__ xi,
                                                        const float *__restrict__ xv, int32_t k,
                                                        int32_t n, float *__restrict__ xd, int clear)
{
    const int32_t t = blockIdx.x * BTPB + threadIdx.x;
    if (t >= k) return;
    const int32_t j = xi[t];
    if (j < 0 || j >= n) return;
    xd[j] = clear ? 0.f : xv[t];
}

__global__ __launch_bounds__(BTPB) void k_basic_pull(const int64_t *__restrict__ row_ptr,
                                                     const int32_t *__restrict__ col,
                                                     const float *__restrict__ val,
                                                     const float *__restrict__ xd, int32_t m,
                                                     float *__restrict__ y)
{
    const int q = threadIdx.x & 15;
    const int64_t rows_per_step = (int64_t)gridDim.x * (BTPB / 16);
    for (int64_t i = (int64_t)blockIdx.x * (BTPB / 16) + (threadIdx.x >> 4); i < m; i += rows_per_step) {
        const int64_t rs = row_ptr[i], re = row_ptr[i + 1];
        float s = 0.f;
        for (int64_t p = rs + q; p < re; p += 16 * BUNROLL) {
            int32_t c[BUNROLL];
            float v[BUNROLL];
#pragma unroll
            for (int u = 0; u < BUNROLL; ++u) {
                const int64_t pp = p + 16 * u;
                c[u] = pp < re ? col[pp] : -1;
                v[u] = pp < re ? val[pp] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < BUNROLL; ++u)
                if (c[u] >= 0) s += v[u] * xd[c[u]];
        }
#pragma unroll
        for (int o = 8; o > 0; o >>= 1) s += __shfl_xor(s, o, 16);
        if (q == 0) y[i] = s;
    }
}

__global__ __launch_bounds__(BTPB) void k_basic_push(const int64_t *__restrict__ col_ptr,
                                                     const int32_t *__restrict__ row,
                                                     const float *__restrict__ val,
                                                     const int32_t *__restrict__ xi,
                                                     const float *__restrict__ xv, int32_t k, int32_t n,
                                                     float *__restrict__ y)
{
    const int lane = threadIdx.x & 63;
    const int64_t waves = (int64_t)gridDim.x * (BTPB / 64);
    for (int64_t t = (int64_t)blockIdx.x * (BTPB / 64) + (threadIdx.x >> 6); t < k; t += waves) {
        const int32_t j = xi[t];
        if (j < 0 || j >= n) continue;
        const float xj = xv[t];
        const int64_t cs = col_ptr[j], ce = col_ptr[j + 1];
        for (int64_t p = cs + lane; p < ce; p += 64 * BUNROLL) {
            int32_t r[BUNROLL];
            float v[BUNROLL];
#pragma unroll
            for (int u = 0; u < BUNROLL; ++u) {
                const int64_t pp = p + 64 * u;
                r[u] = pp < ce ? row[pp] : -1;
                v[u] = pp < ce ? val[pp] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < BUNROLL; ++u)
                if (r[u] >= 0) atomicAdd(&y[r[u]], v[u] * xj);
        }
    }
}

dbs_status basic_hip_fail(hipError_t e, const char *what)
{
    return dbs_fail(DBS_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

#define BASIC_TRY(expr, what)                              \
    do {                                                   \
        hipError_t e_ = (expr);                            \
        if (e_ != hipSuccess) return basic_hip_fail(e_, what); \
    } while (0)

}  // namespace

struct dbs_basic_matrix {
    int32_t m = 0, n = 0;
    int64_t nnz = 0;
    int64_t *row_ptr = nullptr, *col_ptr = nullptr;
    int32_t *col = nullptr, *row = nullptr;
    float *csr_val = nullptr, *csc_val = nullptr;
    float *xd = nullptr;  // dense x scratch, all zero between calls
    int grid_rows = 0, grid_waves = 0;
};

extern "C" {

void dbs_basic_destroy(dbs_basic_matrix *B)
{
    if (!B) return;
    for (void *p : {(void *)B->row_ptr, (void *)B->col_ptr, (void *)B->col, (void *)B->row,
                    (void *)B->csr_val, (void *)B->csc_val, (void *)B->xd})
        if (p) (void)hipFree(p);
    delete B;
}

dbs_status dbs_basic_build(int32_t m, int32_t n, int64_t nnz, const int64_t *row_ptr,
                           const int32_t *col_idx, const float *vals, dbs_basic_matrix **out)
{
    if (!out) return dbs_fail(DBS_ERR_ARG, "dbs_basic_build: out is NULL");
    *out = nullptr;
    if (m < 0 || n < 0 || nnz < 0 || !row_ptr || (nnz > 0 && (!col_idx || !vals)))
        return dbs_fail(DBS_ERR_ARG, "dbs_basic_build: bad sizes or NULL arrays");
    if (row_ptr[0] != 0 || row_ptr[m] != nnz)
        return dbs_fail(DBS_ERR_ARG, "dbs_basic_build: row_ptr must start at 0 and end at nnz");
    for (int32_t i = 0; i < m; ++i)
        if (row_ptr[i + 1] < row_ptr[i]) return dbs_fail(DBS_ERR_ARG, "dbs_basic_build: row_ptr decreases at row %d", i);
    for (int64_t p = 0; p < nnz; ++p)
        if (col_idx[p] < 0 || col_idx[p] >= n)
            return dbs_fail(DBS_ERR_ARG, "dbs_basic_build: column %d out of range at entry %lld", col_idx[p],
                            (long long)p);
    // CSC by a counting sort over columns (rows ascend within a column)
    std::vector<int64_t> cp((size_t)n + 1, 0);
    for (int64_t p = 0; p < nnz; ++p) ++cp[(size_t)col_idx[p] + 1];
    for (int32_t j = 0; j < n; ++j) cp[(size_t)j + 1] += cp[(size_t)j];
    std::vector<int32_t> crow((size_t)nnz);
    std::vector<float> cval((size_t)nnz);
    {
        std::vector<int64_t> fill(cp.begin(), cp.end() - 1);
        for (int32_t i = 0; i < m; ++i)
            for (int64_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) {
                const int64_t d = fill[(size_t)col_idx[p]]++;
                crow[(size_t)d] = i;
                cval[(size_t)d] = vals[p];
            }
    }
    dbs_basic_matrix *B = new (std::nothrow) dbs_basic_matrix;
    if (!B) return dbs_fail(DBS_ERR_ALLOC, "dbs_basic_build: host allocation");
    B->m = m;
    B->n = n;
    B->nnz = nnz;
    auto up = [&](void **dst, const void *src, size_t bytes) -> hipError_t {
        hipError_t e = hipMalloc(dst, std::max<size_t>(bytes, 16));
        if (e != hipSuccess) return e;
        return bytes ? hipMemcpy(*dst, src, bytes, hipMemcpyHostToDevice) : hipSuccess;
    };
    hipError_t e = hipSuccess;
    if (e == hipSuccess) e = up((void **)&B->row_ptr, row_ptr, ((size_t)m + 1) * sizeof(int64_t));
    if (e == hipSuccess) e = up((void **)&B->col, col_idx, (size_t)nnz * sizeof(int32_t));
    if (e == hipSuccess) e = up((void **)&B->csr_val, vals, (size_t)nnz * sizeof(float));
    if (e == hipSuccess) e = up((void **)&B->col_ptr, cp.data(), cp.size() * sizeof(int64_t));
    if (e == hipSuccess) e = up((void **)&B->row, crow.data(), crow.size() * sizeof(int32_t));
    if (e == hipSuccess) e = up((void **)&B->csc_val, cval.data(), cval.size() * sizeof(float));
    if (e == hipSuccess) e = hipMalloc((void **)&B->xd, std::max<size_t>((size_t)n * sizeof(float), 16));
    if (e == hipSuccess) e = hipMemset(B->xd, 0, std::max<size_t>((size_t)n * sizeof(float), 16));
    int per_cu_pull = 0, per_cu_push = 0, dev = 0;
    hipDeviceProp_t prop;
    if (e == hipSuccess) e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipGetDeviceProperties(&prop, dev);
    if (e == hipSuccess)
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu_pull, (const void *)k_basic_pull, BTPB, 0);
    if (e == hipSuccess)
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu_push, (const void *)k_basic_push, BTPB, 0);
    if (e != hipSuccess) {
        dbs_basic_destroy(B);
        return basic_hip_fail(e, "dbs_basic_build");
    }
    B->grid_rows = std::max(1, per_cu_pull) * prop.multiProcessorCount;
    B->grid_waves = std::max(1, per_cu_push) * prop.multiProcessorCount;
    *out = B;
    return DBS_OK;
}

dbs_status dbs_basic_spmspv(dbs_basic_matrix *B, dbs_path path, int32_t x_nnz, const int32_t *d_x_idx,
                            const float *d_x_val, float *d_y, void *stream)
{
    if (!B) return dbs_fail(DBS_ERR_ARG, "dbs_basic_spmspv: matrix is NULL");
    if (path != DBS_PATH_PUSH && path != DBS_PATH_PULL)
        return dbs_fail(DBS_ERR_ARG, "dbs_basic_spmspv: path must be DBS_PATH_PUSH or DBS_PATH_PULL");
    if (x_nnz < 0 || (x_nnz > 0 && (!d_x_idx || !d_x_val)) || (B->m > 0 && !d_y))
        return dbs_fail(DBS_ERR_ARG, "dbs_basic_spmspv: bad x or y");
    hipStream_t s = (hipStream_t)stream;
    if (B->m == 0) return DBS_OK;
    const dim3 b(BTPB);
    if (path == DBS_PATH_PUSH) {
        BASIC_TRY(hipMemsetAsync(d_y, 0, (size_t)B->m * sizeof(float), s), "hipMemsetAsync (y)");
        if (x_nnz > 0) {
            const int64_t need = ((int64_t)x_nnz + BTPB / 64 - 1) / (BTPB / 64);
            const dim3 g((unsigned)std::min<int64_t>(need, B->grid_waves));
            hipLaunchKernelGGL(k_basic_push, g, b, 0, s, B->col_ptr, B->row, B->csc_val, d_x_idx, d_x_val, x_nnz,
                               B->n, d_y);
        }
    } else {
        const dim3 gx((unsigned)std::max<int64_t>(1, ((int64_t)x_nnz + BTPB - 1) / BTPB));
        if (x_nnz > 0)
            hipLaunchKernelGGL(k_basic_scatter, gx, b, 0, s, d_x_idx, d_x_val, x_nnz, B->n, B->xd, 0);
        const int64_t need = ((int64_t)B->m + BTPB / 16 - 1) / (BTPB / 16);
        const dim3 g((unsigned)std::min<int64_t>(need, B->grid_rows));
        hipLaunchKernelGGL(k_basic_pull, g, b, 0, s, B->row_ptr, B->col, B->csr_val, B->xd, B->m, d_y);
        if (x_nnz > 0)
            hipLaunchKernelGGL(k_basic_scatter, gx, b, 0, s, d_x_idx, d_x_val, x_nnz, B->n, B->xd, 1);
    }
    BASIC_TRY(hipGetLastError(), "dbs_basic_spmspv launch");
    return DBS_OK;
}

}  // extern "C"
