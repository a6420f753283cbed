// kb_device.hpp -- device helpers shared by the library's gfx950 kernels:
// the Philox4x32-10 block function, storage widening, and 64-lane wavefront
// reductions built on DPP row permutations and lane reads.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kb {

// Element type codes (same values as kb_dtype).
enum : int { DT_F32 = 0, DT_F16 = 1, DT_BF16 = 2, DT_U32 = 3 };

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon et al., SC'11): per round the 32x32->64 products
// M0*x0 and M1*x2 are split into (hi, lo); the new state is
// (hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0); the key gains (W0, W1) mod 2^32
// between rounds.  mul_hi and the low product map to one
// v_mad_u64_u32 each.
// ---------------------------------------------------------------------------
struct u32x4 {
    uint32_t x, y, z, w;
};

__device__ __forceinline__ u32x4 philox4x32_10(u32x4 ctr, uint32_t k0, uint32_t k1) {
    constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    constexpr uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        const uint64_t p0 = (uint64_t)M0 * ctr.x;
        const uint64_t p1 = (uint64_t)M1 * ctr.z;
        u32x4 nxt;
        nxt.x = (uint32_t)(p1 >> 32) ^ ctr.y ^ k0;
        nxt.y = (uint32_t)p1;
        nxt.z = (uint32_t)(p0 >> 32) ^ ctr.w ^ k1;
        nxt.w = (uint32_t)p0;
        ctr = nxt;
        k0 += W0;
        k1 += W1;
    }
    return ctr;
}

// ---------------------------------------------------------------------------
// Storage -> binary32 (exact).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float f16_bits_to_f32(uint32_t h16) {
    _Float16 h = __builtin_bit_cast(_Float16, (uint16_t)h16);
    return (float)h;  // v_cvt_f32_f16: exact, f16 subnormals kept
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b16) {
    return __uint_as_float(b16 << 16);
}

// binary32 -> storage, round to nearest even (finite inputs; the generator
// never produces NaN).
__device__ __forceinline__ uint16_t f32_to_f16_bits(float f) {
    _Float16 h = (_Float16)f;  // v_cvt_f16_f32 under the default RNE mode
    return __builtin_bit_cast(uint16_t, h);
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    // NaN: the quiet NaN with the sign kept (rounding the bits would turn a
    // NaN whose payload lies in the dropped half into infinity)
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)(((u >> 16) & 0x8000u) | 0x7FC0u);
    u += 0x7FFFu + ((u >> 16) & 1u);  // ties to even on the dropped half
    return (uint16_t)(u >> 16);
}

// ---------------------------------------------------------------------------
// Wavefront (64-lane) reductions.  Four DPP steps leave every lane of a
// 16-lane row holding the row's result: quad_perm [1,0,3,2] (xor 1),
// quad_perm [2,3,0,1] (xor 2), row_half_mirror (i <-> 7-i) and row_mirror
// (i <-> 15-i).  Each step combines a value with its partner's, and both
// partners compute op(a, b) / op(b, a), which agree for the commutative ops
// used here, so the row result is the same bit pattern on all 16 lanes.
// The four row results are read from lanes 0, 16, 32, 48 and combined in a
// fixed order: the reduction is deterministic.
// ---------------------------------------------------------------------------
constexpr int DPP_QUAD_XOR1 = 0xB1;
constexpr int DPP_QUAD_XOR2 = 0x4E;
constexpr int DPP_ROW_HALF_MIRROR = 0x141;
constexpr int DPP_ROW_MIRROR = 0x140;

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = dpp_u32<CTRL>((uint32_t)u);
    const uint32_t hi = dpp_u32<CTRL>((uint32_t)(u >> 32));
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

template <int CTRL>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t u) {
    const uint32_t lo = dpp_u32<CTRL>((uint32_t)u);
    const uint32_t hi = dpp_u32<CTRL>((uint32_t)(u >> 32));
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint32_t readlane_u32(uint32_t v, int lane) {
    return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}

__device__ __forceinline__ uint64_t readlane_u64(uint64_t u, int lane) {
    const uint32_t lo = readlane_u32((uint32_t)u, lane);
    const uint32_t hi = readlane_u32((uint32_t)(u >> 32), lane);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ double readlane_f64(double v, int lane) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = readlane_u32((uint32_t)u, lane);
    const uint32_t hi = readlane_u32((uint32_t)(u >> 32), lane);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// Max of non-negative binary32 values (never NaN) compared as bit patterns.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    v = max(v, dpp_u32<DPP_QUAD_XOR1>(v));
    v = max(v, dpp_u32<DPP_QUAD_XOR2>(v));
    v = max(v, dpp_u32<DPP_ROW_HALF_MIRROR>(v));
    v = max(v, dpp_u32<DPP_ROW_MIRROR>(v));
    const uint32_t a = max(readlane_u32(v, 0), readlane_u32(v, 16));
    const uint32_t b = max(readlane_u32(v, 32), readlane_u32(v, 48));
    return max(a, b);
}

__device__ __forceinline__ uint32_t wave_or_u32(uint32_t v) {
    v |= dpp_u32<DPP_QUAD_XOR1>(v);
    v |= dpp_u32<DPP_QUAD_XOR2>(v);
    v |= dpp_u32<DPP_ROW_HALF_MIRROR>(v);
    v |= dpp_u32<DPP_ROW_MIRROR>(v);
    return (readlane_u32(v, 0) | readlane_u32(v, 16)) | (readlane_u32(v, 32) | readlane_u32(v, 48));
}

// Sum of per-lane counts; the total of one wave fits 32 bits here.
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
    v += dpp_u32<DPP_QUAD_XOR1>(v);
    v += dpp_u32<DPP_QUAD_XOR2>(v);
    v += dpp_u32<DPP_ROW_HALF_MIRROR>(v);
    v += dpp_u32<DPP_ROW_MIRROR>(v);
    return (readlane_u32(v, 0) + readlane_u32(v, 16)) + (readlane_u32(v, 32) + readlane_u32(v, 48));
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
    v += dpp_u64<DPP_QUAD_XOR1>(v);
    v += dpp_u64<DPP_QUAD_XOR2>(v);
    v += dpp_u64<DPP_ROW_HALF_MIRROR>(v);
    v += dpp_u64<DPP_ROW_MIRROR>(v);
    return (readlane_u64(v, 0) + readlane_u64(v, 16)) + (readlane_u64(v, 32) + readlane_u64(v, 48));
}

__device__ __forceinline__ double wave_sum_f64(double v) {
    v = v + dpp_f64<DPP_QUAD_XOR1>(v);
    v = v + dpp_f64<DPP_QUAD_XOR2>(v);
    v = v + dpp_f64<DPP_ROW_HALF_MIRROR>(v);
    v = v + dpp_f64<DPP_ROW_MIRROR>(v);
    return (readlane_f64(v, 0) + readlane_f64(v, 16)) + (readlane_f64(v, 32) + readlane_f64(v, 48));
}

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
    v = min(v, dpp_u32<DPP_QUAD_XOR1>(v));
    v = min(v, dpp_u32<DPP_QUAD_XOR2>(v));
    v = min(v, dpp_u32<DPP_ROW_HALF_MIRROR>(v));
    v = min(v, dpp_u32<DPP_ROW_MIRROR>(v));
    const uint32_t a = min(readlane_u32(v, 0), readlane_u32(v, 16));
    const uint32_t b = min(readlane_u32(v, 32), readlane_u32(v, 48));
    return min(a, b);
}

__device__ __forceinline__ uint64_t min_u64(uint64_t a, uint64_t b) { return a < b ? a : b; }

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
    v = min_u64(v, dpp_u64<DPP_QUAD_XOR1>(v));
    v = min_u64(v, dpp_u64<DPP_QUAD_XOR2>(v));
    v = min_u64(v, dpp_u64<DPP_ROW_HALF_MIRROR>(v));
    v = min_u64(v, dpp_u64<DPP_ROW_MIRROR>(v));
    return min_u64(min_u64(readlane_u64(v, 0), readlane_u64(v, 16)),
                   min_u64(readlane_u64(v, 32), readlane_u64(v, 48)));
}

// Reductions within one 16-lane DPP row: the four steps above leave every
// lane of a row holding the row's result (no cross-row reads), so a
// work-group can reduce up to 16 independent values, one per row.
__device__ __forceinline__ uint32_t row_max_u32(uint32_t v) {
    v = max(v, dpp_u32<DPP_QUAD_XOR1>(v));
    v = max(v, dpp_u32<DPP_QUAD_XOR2>(v));
    v = max(v, dpp_u32<DPP_ROW_HALF_MIRROR>(v));
    return max(v, dpp_u32<DPP_ROW_MIRROR>(v));
}

__device__ __forceinline__ uint32_t row_or_u32(uint32_t v) {
    v |= dpp_u32<DPP_QUAD_XOR1>(v);
    v |= dpp_u32<DPP_QUAD_XOR2>(v);
    v |= dpp_u32<DPP_ROW_HALF_MIRROR>(v);
    return v | dpp_u32<DPP_ROW_MIRROR>(v);
}

__device__ __forceinline__ uint64_t row_sum_u64(uint64_t v) {
    v += dpp_u64<DPP_QUAD_XOR1>(v);
    v += dpp_u64<DPP_QUAD_XOR2>(v);
    v += dpp_u64<DPP_ROW_HALF_MIRROR>(v);
    return v + dpp_u64<DPP_ROW_MIRROR>(v);
}

__device__ __forceinline__ uint64_t row_min_u64(uint64_t v) {
    v = min_u64(v, dpp_u64<DPP_QUAD_XOR1>(v));
    v = min_u64(v, dpp_u64<DPP_QUAD_XOR2>(v));
    v = min_u64(v, dpp_u64<DPP_ROW_HALF_MIRROR>(v));
    return min_u64(v, dpp_u64<DPP_ROW_MIRROR>(v));
}

__device__ __forceinline__ double row_sum_f64(double v) {
    v = v + dpp_f64<DPP_QUAD_XOR1>(v);
    v = v + dpp_f64<DPP_QUAD_XOR2>(v);
    v = v + dpp_f64<DPP_ROW_HALF_MIRROR>(v);
    return v + dpp_f64<DPP_ROW_MIRROR>(v);
}

}  // namespace kb
