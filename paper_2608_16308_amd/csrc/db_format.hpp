// Layout constants of the dual-view blocked (DB) format, shared by the host
// builder and the gfx950 kernels of this library.
//
// Sec. 3.2.1: the matrix is cut into uniform 16x16 blocks; a block-level CSR
// view and a block-level CSC view index ONE payload stored in primary
// (block-CSR) order.  Per-block metadata is packed into one 64-bit word:
//   bits 63..16  payload byte offset
//   bits 15..8   nnz - 1          (1..256)
//   bits  2..0   block type       (dbs_block_type)
// Pull segments (Sec. 3.3.2) are packed into one 64-bit word:
//   bits 31..0   first block (primary id)
//   bits 58..32  block row
//   bits 62..59  number of blocks - 1 (a segment holds at most 16 blocks)
//   bit  63      the block row has exactly one segment
#pragma once
#include <cstdint>

#ifdef __HIPCC__
#define DBS_HD __host__ __device__ __forceinline__
#else
#define DBS_HD inline
#endif

namespace dbs {

constexpr int BS = 16;            // block edge (Sec. 3.2.1)
constexpr int MAX_SEG_BLOCKS = 16;

enum BlockType : uint32_t { T_COO = 0, T_DENSE = 1, T_FCSR = 2, T_FCSC = 3, T_CSR = 4 };

// Header offsets inside a block record (bytes).
constexpr uint32_t HDR_MASK = 0;     // uint16 mask[16]: row masks, or column masks for FCSC
constexpr uint32_t HDR_START = 32;   // uint8 start[16]: row starts, or column starts for FCSC
constexpr uint32_t HDR_START2 = 48;  // uint8 col_start[16] (patched CSR only)
constexpr uint32_t HDR_RCSC = 64;    // row_idx_csc2csr bytes (patched CSR only)

DBS_HD uint64_t desc_make(uint64_t off, uint32_t nnz, uint32_t type)
{
    return (off << 16) | ((uint64_t)(nnz - 1) << 8) | (uint64_t)type;
}
DBS_HD uint64_t desc_off(uint64_t d) { return d >> 16; }
DBS_HD uint32_t desc_nnz(uint64_t d) { return (uint32_t)((d >> 8) & 0xFFu) + 1u; }
DBS_HD uint32_t desc_type(uint64_t d) { return (uint32_t)(d & 7u); }

// Small COO blocks are stored inside the descriptor instead of the payload
// (bit 3 set): entry e occupies bits [16 + e (8 + 8V), ...) as the
// coordinate byte followed by the V value bytes.  Capacity: 1 entry for
// fp32, 2 for fp16, 6 for pattern matrices.
constexpr uint64_t DESC_INLINE = 8u;
DBS_HD bool desc_inline(uint64_t d) { return (d & DESC_INLINE) != 0; }
DBS_HD uint32_t inline_capacity(uint32_t vbytes) { return 48u / (8u + 8u * vbytes); }
DBS_HD uint32_t inline_shift(uint32_t e, uint32_t vbytes) { return 16u + e * (8u + 8u * vbytes); }

// Device word of a pull-segment slot: the block column, and for a COO block
// with one entry held inline in its descriptor also that entry's local
// column, so that the compaction of the slots can test the exact x entry
// without reading the descriptor:
//   bits 25..0   block column (a matrix has at most 2^26 block columns)
//   bits 29..26  local column of the single inline entry (bit 30 set)
//   bit  30      the block is COO with exactly one entry, held inline
//   bit  31      padding (the whole word is -1) or a block of the non-COO list
constexpr int32_t SLOT_PAD = -1;
constexpr uint32_t SLOT_J_MASK = (1u << 26) - 1u;
constexpr uint32_t SLOT_ONE = 1u << 30;
constexpr uint32_t SLOT_LISTED = 1u << 31;
constexpr int64_t MAX_BLOCK_COLS = (int64_t)1 << 26;
DBS_HD int32_t slot_word(int32_t J, uint64_t d)
{
    if (desc_type(d) != T_COO) return (int32_t)((uint32_t)J | SLOT_LISTED);
    uint32_t w = (uint32_t)J;
    if (desc_inline(d) && desc_nnz(d) == 1) w |= SLOT_ONE | ((uint32_t)((d >> 16) & 15u) << 26);
    return (int32_t)w;
}
DBS_HD int32_t slot_col(int32_t w) { return (int32_t)((uint32_t)w & SLOT_J_MASK); }
DBS_HD uint32_t slot_c(int32_t w) { return ((uint32_t)w >> 26) & 15u; }
DBS_HD bool slot_one(int32_t w) { return w >= 0 && ((uint32_t)w & SLOT_ONE) != 0; }

DBS_HD uint64_t seg_make(uint32_t first, uint32_t brow, uint32_t nb, bool single)
{
    return (uint64_t)first | ((uint64_t)brow << 32) | ((uint64_t)(nb - 1) << 59) |
           ((uint64_t)(single ? 1u : 0u) << 63);
}
DBS_HD uint32_t seg_first(uint64_t s) { return (uint32_t)(s & 0xFFFFFFFFu); }
DBS_HD uint32_t seg_brow(uint64_t s) { return (uint32_t)((s >> 32) & 0x7FFFFFFu); }
DBS_HD uint32_t seg_nb(uint64_t s) { return (uint32_t)((s >> 59) & 0xFu) + 1u; }
DBS_HD bool seg_single(uint64_t s) { return (s >> 63) != 0; }

DBS_HD uint32_t round_up(uint32_t v, uint32_t a) { return (v + a - 1) / a * a; }

// Byte offset of the first value inside a block record.
DBS_HD uint32_t values_at(uint32_t type, uint32_t nnz)
{
    switch (type) {
    case T_COO: return 0;
    case T_DENSE: return HDR_START;            // after the 32-byte row masks
    case T_FCSR:
    case T_FCSC: return HDR_START2;            // after masks + starts
    default: return HDR_RCSC + round_up(nnz, 16);
    }
}

// Total bytes of a block record (before alignment of the next record).
DBS_HD uint32_t record_bytes(uint32_t type, uint32_t nnz, uint32_t vbytes)
{
    switch (type) {
    case T_COO: return vbytes * nnz + nnz;     // values, then coordinates
    case T_DENSE: return HDR_START + 256u * vbytes;
    case T_FCSR:
    case T_FCSC: return HDR_START2 + nnz * vbytes;
    default: return HDR_RCSC + round_up(nnz, 16) + nnz * vbytes;
    }
}

DBS_HD uint32_t record_align(uint32_t type, uint32_t vbytes)
{
    return type == T_COO ? (vbytes > 1 ? vbytes : 1u) : 16u;
}

// Pull segment weights by format (Sec. 3.3.2): Dense 4, ForceCSR / ForceCSC /
// patched CSR 2, COO 1.
DBS_HD uint32_t seg_weight(uint32_t type)
{
    return type == T_DENSE ? 4u : (type == T_COO ? 1u : 2u);
}

}  // namespace dbs
