// MFMA building blocks for the bf16 attention kernels (gfx950, wave64).
//
// v_mfma_f32_16x16x32_bf16 operand layouts (lane l, i the element within the lane):
//   A (16 x 32, row-major M x K):  A[m = l % 16][k = 8 (l / 16) + i],  i < 8
//   B (32 x 16, K x N):            B[k = 8 (l / 16) + i][n = l % 16],  i < 8
//   C (16 x 16, fp32):             C[m = 4 (l / 16) + i][n = l % 16],  i < 4
// Every operand is K-contiguous within a lane, so a product over keys needs its key-side
// operand stored key-contiguous (V^T in LDS).  The C layout of a 32-key pair of M-blocks
// (keys 4g..4g+3 and 16+4g..16+4g+3 in lane group g = l / 16) is used directly as a
// K-operand with the matching key permutation on the other operand.
#pragma once

#include "common.h"

namespace hsa {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));   // 16 raw bytes

__device__ __forceinline__ f32x4_t mfma16(const bf16x8_t& a, const bf16x8_t& b, const f32x4_t& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x4_t zero4() { return f32x4_t{0.f, 0.f, 0.f, 0.f}; }

// round-to-nearest-even fp32 -> bf16 (finite inputs)
__device__ __forceinline__ __bf16 f2bf(float x) { return (__bf16)x; }

__device__ __forceinline__ bf16x8_t ld_bf16x8(const void* p) {
    return *reinterpret_cast<const bf16x8_t*>(p);
}
__device__ __forceinline__ bf16x4_t ld_bf16x4(const void* p) {
    return *reinterpret_cast<const bf16x4_t*>(p);
}
__device__ __forceinline__ bf16x8_t cat(const bf16x4_t& a, const bf16x4_t& b) {
    return bf16x8_t{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// Reductions over the four lanes l, l^16, l^32, l^48 that hold one column of a C layout,
// with the gfx950 lane-swap instructions (no LDS traffic): a swap of v with itself returns
// (v[l], v[partner]) in some order, so the pair sum / max is order-free.
__device__ __forceinline__ float pair16_sum(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float pair32_sum(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float pair16_max(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair32_max(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float col_sum(float v) { return pair32_sum(pair16_sum(v)); }
__device__ __forceinline__ float col_max(float v) { return pair32_max(pair16_max(v)); }

// 2^x on the hardware exponential (inputs here are <= 0; results below 2^-126 flush to 0,
// which is exact enough for softmax probabilities)
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Transposed LDS tiles T[d][n] (n keys or rows per d-row, n a power of two >= 32) store
// entry (d, s) at position tpos(d, s, n): a rotation by 8 (d / 16).  Staging threads that
// cover 16 consecutive column blocks of a few rows then write 64 distinct banks, and every
// 4-aligned group of 4 entries stays contiguous (8-byte reads), rotated as a unit.
__device__ __forceinline__ int tpos(int d, int s, int n) { return (s + 8 * (d >> 4)) & (n - 1); }

// A value pair (a, b) of the C layout as a bf16 hi/lo operand pair: hi + lo carries ~16
// mantissa bits, for products whose fp32 result cancels or accumulates many terms.
__device__ __forceinline__ void split8(const f32x4_t& a, const f32x4_t& b, bf16x8_t& hi,
                                       bf16x8_t& lo) {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const float x0 = j < 2 ? a[2 * j] : b[2 * j - 4];
        const float x1 = j < 2 ? a[2 * j + 1] : b[2 * j - 3];
        // one conversion of the pair; its two halves read back as floats
        const bf16x2_t hp = bf16x2_t{f2bf(x0), f2bf(x1)};
        uint32_t u;
        __builtin_memcpy(&u, &hp, 4);
        hi[2 * j] = hp[0];
        hi[2 * j + 1] = hp[1];
        lo[2 * j] = f2bf(x0 - __uint_as_float(u << 16));
        lo[2 * j + 1] = f2bf(x1 - __uint_as_float(u & 0xFFFF0000u));
    }
}

// Per-(token, slot) partial outputs are stored as blocks of 8 values in 16 bytes (block
// floating point): one power-of-two scale per block and a 16-bit signed integer per value.
// With E the biased exponent of the block's largest magnitude (at least 14), every value is
// below 2^(E - 126) in magnitude; x 2^(126 - E) is converted to a normalised 16-bit integer
// (q = x 2^(126 - E) 32767, rounded, by v_cvt_pknorm_i16_f32), and the low bit of field i is
// replaced by bit i of E.  The decoded value is field 2^(E - 126) / 32767: the conversion
// and the replaced bit are off by at most 2 units of 2^(E - 126) / 32767, i.e. at most 2^-13
// of the block's largest magnitude (bf16 storage: up to 2^-8 of each value's own), in the
// bytes of bf16.
__device__ __forceinline__ u32x4_t bfp_pack8(const f32x4_t& a, const f32x4_t& b) {
    float m = fmaxf(fmaxf(fabsf(a[0]), fabsf(a[1])), fabsf(a[2]));
    m = fmaxf(fmaxf(m, fabsf(a[3])), fabsf(b[0]));
    m = fmaxf(fmaxf(m, fabsf(b[1])), fabsf(b[2]));
    m = fmaxf(m, fabsf(b[3]));
    const uint32_t e = max((__float_as_uint(m) >> 23) & 0xFFu, 14u);
    const float s = __uint_as_float((253u - e) << 23);          // 2^(126 - e)
    const auto p0 = __builtin_amdgcn_cvt_pknorm_i16(a[0] * s, a[1] * s);
    const auto p1 = __builtin_amdgcn_cvt_pknorm_i16(a[2] * s, a[3] * s);
    const auto p2 = __builtin_amdgcn_cvt_pknorm_i16(b[0] * s, b[1] * s);
    const auto p3 = __builtin_amdgcn_cvt_pknorm_i16(b[2] * s, b[3] * s);
    uint32_t w[4];
    __builtin_memcpy(&w[0], &p0, 4);
    __builtin_memcpy(&w[1], &p1, 4);
    __builtin_memcpy(&w[2], &p2, 4);
    __builtin_memcpy(&w[3], &p3, 4);
    // bit 2j of E to field 2j (bit 0 of word j), bit 2j + 1 to field 2j + 1 (bit 16)
    const uint32_t t = e | (e << 15);
#pragma unroll
    for (int j = 0; j < 4; ++j) w[j] = (w[j] & 0xFFFEFFFEu) | ((t >> (2 * j)) & 0x00010001u);
    return u32x4_t{w[0], w[1], w[2], w[3]};
}

// Adds the 8 values of a block to acc[0..7] (field i to acc[i]); with use false, adds zeros
// whatever the 16 bytes hold (the scale is selected away, never multiplied by zero).
__device__ __forceinline__ void bfp_accum8(const u32x4_t& v, float acc[8], bool use = true) {
    const uint32_t x = (v[0] & 0x00010001u) | ((v[1] & 0x00010001u) << 2) |
                       ((v[2] & 0x00010001u) << 4) | ((v[3] & 0x00010001u) << 6);
    const uint32_t e = (x | (x >> 15)) & 0xFFu;
    const float sc1 = __uint_as_float((e + 1u) << 23) * (1.0f / 32767.0f);  // 2^(e - 126) / 32767
    const float sc = use ? sc1 : 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        acc[2 * j] = fmaf((float)(int16_t)(v[j] & 0xFFFFu), sc, acc[2 * j]);
        acc[2 * j + 1] = fmaf((float)((int32_t)v[j] >> 16), sc, acc[2 * j + 1]);
    }
}

// Waits until every global load of this wave has landed.  Called once after the loads of
// operands that stay in registers for a whole loop (Q^T, K / V blocks): the compiler cannot
// tell at the loop header that those loads are complete, and otherwise makes the loop's
// MFMAs wait for the in-order load counter to drain, i.e. for the next chunk's prefetch.
// (s_waitcnt immediate: vmcnt 0, expcnt and lgkmcnt at their no-wait maxima.)
__device__ __forceinline__ void wait_global_loads() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// A compile-time integer as a value (selects a constant stage of a ring in unrolled loops).
template <int N>
struct IntC {
    static constexpr int value = N;
};

// Logical workgroup id with an XCD-aware order: hardware dispatches consecutive ids to the
// 8 XCDs round-robin, so consecutive logical ids (same (b, g), neighbouring tiles, sharing
// chunks through L2) are mapped to the same XCD.  Returns -1 for padding ids.
__device__ __forceinline__ int xcd_logical_id(int nlogical) {
    const int id = blockIdx.x;
    const int per = (nlogical + 7) >> 3;
    const int lid = (id & 7) * per + (id >> 3);
    return lid < nlogical ? lid : -1;
}

}  // namespace hsa
