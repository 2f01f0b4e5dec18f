// Host-side internals shared by the builder and the C-ABI implementation.
#pragma once
#include <cstdarg>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/dbspmspv.h"
#include "db_format.hpp"

// Thread-local message for dbs_last_error().
dbs_status dbs_fail(dbs_status st, const char *fmt, ...);

struct dbs_host_matrix {
    int32_t m = 0, n = 0;
    int64_t nnz = 0;
    dbs_dtype dtype = DBS_F32;
    dbs_build_opts opts{};
    int32_t nbr = 0, nbc = 0;
    int64_t nblk = 0, nseg = 0;
    int64_t by_type[DBS_NUM_BLOCK_TYPES] = {0, 0, 0, 0, 0};
    std::vector<int32_t> rb_ptr;   // nbr + 1
    std::vector<int32_t> cb_col;   // nblk
    std::vector<int32_t> cb_ptr;   // nbc + 1
    std::vector<int32_t> csc_row;  // nblk
    std::vector<int32_t> csc2csr;  // nblk
    std::vector<uint64_t> desc;    // nblk
    std::vector<uint64_t> seg;     // nseg
    // (nbr + 1) / 2 words, a 16-bit mask per block row (two per word): the
    // rows that hold at least one entry
    std::vector<uint32_t> row_occ;
    std::vector<uint8_t> payload;
};

inline uint32_t dtype_bytes(dbs_dtype t) { return t == DBS_F32 ? 4u : (t == DBS_F16 ? 2u : 0u); }

void fill_info(const dbs_host_matrix &h, dbs_matrix_info *out);
