// The device-resident matrix object of the C ABI, shared by the upload path
// (api.hip) and the GPU-side conversion (convert.hip).
#pragma once
#include <vector>

#include "internal.hpp"
#include "kernels.hpp"

struct dbs_matrix {
    dbs::DevMatrix d;
    dbs_matrix_info info{};
    std::vector<void *> allocs;  // device allocations owned by the matrix
};
