// Wave64 helpers for the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>

#include <cstdint>

#include "db_format.hpp"

namespace dbs {

constexpr int WAVE = 64;

__device__ __forceinline__ int lane_id() { return (int)__lane_id(); }

__device__ __forceinline__ uint64_t ballot(bool p) { return (uint64_t)__ballot(p ? 1 : 0); }

__device__ __forceinline__ int ctz32(uint32_t v) { return __builtin_ctz(v); }
__device__ __forceinline__ int ctz64(uint64_t v) { return __builtin_ctzll(v); }

__device__ __forceinline__ uint32_t readlane_u32(uint32_t v, int l)
{
    return (uint32_t)__builtin_amdgcn_readlane((int)v, l);
}
__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int l)
{
    uint32_t lo = readlane_u32((uint32_t)v, l), hi = readlane_u32((uint32_t)(v >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}

// Orders this wave's LDS accesses (the LDS slices used here are private to
// one wave, so no workgroup barrier is needed).
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

template <class T>
__device__ __forceinline__ T wave_sum(T v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
    return v;
}

__device__ __forceinline__ uint32_t wave_or(uint32_t v)
{
#pragma unroll
    for (int o = 1; o < WAVE; o <<= 1) v |= __shfl_xor(v, o, WAVE);
    return v;
}

// Cross-lane moves by DPP (data-parallel primitives of the GFX9 vector ALU):
// no LDS round trip and no per-pattern address register, unlike shuffles.
// A lane whose source is outside its row (or the wave) receives `old`.
namespace dppc {
constexpr int ROW_SHR = 0x110;    // + n: lane i of a 16-lane row reads lane i - n of the row
constexpr int ROW_ROR = 0x120;    // + n: rotate right within the row
constexpr int WF_SL1 = 0x130;     // lane i reads lane i + 1 of the wave
constexpr int WF_SR1 = 0x138;     // lane i reads lane i - 1 of the wave
constexpr int ROW_BCAST15 = 0x142;  // lane 15 of each row feeds the next row
constexpr int ROW_BCAST31 = 0x143;  // lane 31 feeds rows 2 and 3
}  // namespace dppc

template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t old, uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROW_MASK, 0xF, false);
}

// Inclusive scans over the 64 lanes (Hillis-Steele inside each row, then the
// two row broadcasts).
__device__ __forceinline__ uint32_t wave_incl_add(uint32_t v)
{
    v += dpp_mov<dppc::ROW_SHR + 1>(0u, v);
    v += dpp_mov<dppc::ROW_SHR + 2>(0u, v);
    v += dpp_mov<dppc::ROW_SHR + 4>(0u, v);
    v += dpp_mov<dppc::ROW_SHR + 8>(0u, v);
    v += dpp_mov<dppc::ROW_BCAST15, 0xA>(0u, v);
    v += dpp_mov<dppc::ROW_BCAST31, 0xC>(0u, v);
    return v;
}
__device__ __forceinline__ uint32_t wave_incl_max(uint32_t v)
{
    v = max(v, dpp_mov<dppc::ROW_SHR + 1>(0u, v));
    v = max(v, dpp_mov<dppc::ROW_SHR + 2>(0u, v));
    v = max(v, dpp_mov<dppc::ROW_SHR + 4>(0u, v));
    v = max(v, dpp_mov<dppc::ROW_SHR + 8>(0u, v));
    v = max(v, dpp_mov<dppc::ROW_BCAST15, 0xA>(0u, v));
    v = max(v, dpp_mov<dppc::ROW_BCAST31, 0xC>(0u, v));
    return v;
}
// The value of lane i - 1 (0 for lane 0).
__device__ __forceinline__ uint32_t wave_shr1(uint32_t v) { return dpp_mov<dppc::WF_SR1>(0u, v); }

// OR of v over the lanes up to this one whose key equals this lane's, for
// keys in contiguous runs (a Hillis-Steele scan that stops at a key change;
// with a key repeated after a gap it may also merge across the gap).
__device__ __forceinline__ uint32_t wave_run_or(uint32_t v, uint32_t key)
{
#define DBS_RUN_STEP(CTRL, RM)                                       \
    {                                                                \
        const uint32_t pv = dpp_mov<CTRL, RM>(0u, v);                \
        const uint32_t pk = dpp_mov<CTRL, RM>(~key, key);            \
        if (pk == key) v |= pv;                                      \
    }
    DBS_RUN_STEP(dppc::ROW_SHR + 1, 0xF)
    DBS_RUN_STEP(dppc::ROW_SHR + 2, 0xF)
    DBS_RUN_STEP(dppc::ROW_SHR + 4, 0xF)
    DBS_RUN_STEP(dppc::ROW_SHR + 8, 0xF)
    DBS_RUN_STEP(dppc::ROW_BCAST15, 0xA)
    DBS_RUN_STEP(dppc::ROW_BCAST31, 0xC)
#undef DBS_RUN_STEP
    return v;
}

__device__ __forceinline__ uint32_t or16_in_quarter(uint32_t v)
{
    // OR over the 16 lanes of this lane's quarter-wave (a DPP row): rotations
    // by 1, 2, 4 and 8 leave the OR of the whole row in every lane.
    v |= dpp_mov<dppc::ROW_ROR + 1>(0u, v);
    v |= dpp_mov<dppc::ROW_ROR + 2>(0u, v);
    v |= dpp_mov<dppc::ROW_ROR + 4>(0u, v);
    v |= dpp_mov<dppc::ROW_ROR + 8>(0u, v);
    return v;
}

// 16-bit vector-block mask J from 32-bit words holding two masks each.
__device__ __forceinline__ uint32_t mask16(const uint32_t *words, int32_t J)
{
    return (words[J >> 1] >> ((J & 1) * 16)) & 0xFFFFu;
}

__device__ __forceinline__ void or_mask16(uint32_t *words, int32_t J, uint32_t bits)
{
    if (bits) atomicOr(&words[J >> 1], bits << ((J & 1) * 16));
}

// Rows of block row R admitted by an optional m-bit output mask.
__device__ __forceinline__ uint32_t allowed16(const uint32_t *mask, int complement, int32_t R)
{
    if (!mask) return 0xFFFFu;
    uint32_t b = (mask[R >> 1] >> ((R & 1) * 16)) & 0xFFFFu;
    return complement ? (~b & 0xFFFFu) : b;
}

// Round-to-nearest-even conversion of a double to IEEE binary16, written
// from the binary16 definition (1 sign, 5 exponent, 10 fraction bits, bias
// 15, subnormals, overflow to infinity).
__device__ __forceinline__ uint16_t f64_to_f16_rne(double x)
{
    uint64_t u = (uint64_t)__double_as_longlong(x);
    uint16_t sign = (uint16_t)((u >> 48) & 0x8000u);
    uint64_t mag = u & 0x7FFFFFFFFFFFFFFFull;
    if (mag >= 0x7FF0000000000000ull) {  // inf or nan
        return (uint16_t)(sign | 0x7C00u | (mag > 0x7FF0000000000000ull ? 0x200u : 0u));
    }
    int e = (int)(mag >> 52) - 1023;        // unbiased exponent
    uint64_t mant = mag & 0xFFFFFFFFFFFFFull;
    if (e > 15) return (uint16_t)(sign | 0x7C00u);
    if (e >= -14) {
        // normal binary16: keep 10 fraction bits of the 52
        uint64_t q = mant >> 42, rem = mant & ((1ull << 42) - 1), half = 1ull << 41;
        uint32_t h = (uint32_t)((e + 15) << 10) | (uint32_t)q;
        if (rem > half || (rem == half && (q & 1))) h += 1;  // may carry into the exponent (ok)
        return (uint16_t)(sign | h);
    }
    // subnormal binary16: value = m * 2^-24, m in [0, 1023]
    if (e < -25) return sign;  // below half of the smallest subnormal
    uint64_t full = mant | (1ull << 52);     // implicit bit
    int shift = 42 + (-14 - e);              // bits to drop
    uint64_t q = full >> shift, rem = full & ((1ull << shift) - 1), half = 1ull << (shift - 1);
    uint32_t h = (uint32_t)q;
    if (rem > half || (rem == half && (q & 1))) h += 1;
    return (uint16_t)(sign | h);
}

__device__ __forceinline__ float h2f(uint16_t h) { return __half2float(__ushort_as_half(h)); }

}  // namespace dbs
