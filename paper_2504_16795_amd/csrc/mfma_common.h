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
__device__ __forceinline__ bf16x8_t pack8(const f32x4_t& a, const f32x4_t& b, float s) {
    return bf16x8_t{f2bf(a[0] * s), f2bf(a[1] * s), f2bf(a[2] * s), f2bf(a[3] * s),
                    f2bf(b[0] * s), f2bf(b[1] * s), f2bf(b[2] * s), f2bf(b[3] * s)};
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
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float v = (i < 4) ? a[i] : b[i - 4];
        hi[i] = f2bf(v);
        lo[i] = f2bf(v - (float)hi[i]);
    }
}

// Per-(token, slot) partial outputs are stored as blocks of 8 values in 16 bytes (block
// floating point): one power-of-two scale per block and a 13-bit signed integer per value.
// With E the biased exponent of the block's largest magnitude (at least 14), the value x
// is stored as q = round(x 2^(139 - E)), |q| < 2^13, in the 16-bit field (q << 1) | bit i of
// E (field i carries bit i of E).  The error is at most 2^-13 of the block's largest
// magnitude (bf16 storage: up to 2^-8 of each value's own), in the bytes of bf16.
__device__ __forceinline__ u32x4_t bfp_pack8(const f32x4_t& a, const f32x4_t& b) {
    const float m = fmaxf(fmaxf(fmaxf(fabsf(a[0]), fabsf(a[1])), fmaxf(fabsf(a[2]), fabsf(a[3]))),
                          fmaxf(fmaxf(fabsf(b[0]), fabsf(b[1])), fmaxf(fabsf(b[2]), fabsf(b[3]))));
    const uint32_t e = max((__float_as_uint(m) >> 23) & 0xFFu, 14u);
    const float sc = __uint_as_float((266u - e) << 23);        // 2^(139 - e)
    uint32_t f[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float x = i < 4 ? a[i] : b[i - 4];
        // round to the nearest integer: |x sc| < 2^13, so x sc + 1.5 2^23 keeps it in the
        // low mantissa bits
        const int q = __float_as_int(fmaf(x, sc, 12582912.f)) - 0x4B400000;
        f[i] = (((uint32_t)q << 1) | ((e >> i) & 1u)) & 0xFFFFu;
    }
    return u32x4_t{f[0] | (f[1] << 16), f[2] | (f[3] << 16), f[4] | (f[5] << 16),
                   f[6] | (f[7] << 16)};
}

__device__ __forceinline__ void bfp_unpack8(const u32x4_t& v, float x[8]) {
    uint32_t e = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) e |= ((v[j] & 1u) << (2 * j)) | (((v[j] >> 16) & 1u) << (2 * j + 1));
    const float inv = __uint_as_float((e - 12u) << 23);         // 2^(e - 139)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        x[2 * j] = (float)(((int32_t)(v[j] << 16)) >> 17) * inv;
        x[2 * j + 1] = (float)(((int32_t)v[j]) >> 17) * inv;
    }
}

// Waits until every global load of this wave has landed.  Called once after the loads of
// operands that stay in registers for a whole loop (Q^T, K / V blocks): the compiler cannot
// tell at the loop header that those loads are complete, and otherwise makes the loop's
// MFMAs wait for the in-order load counter to drain, i.e. for the next chunk's prefetch.
// (s_waitcnt immediate: vmcnt 0, expcnt and lgkmcnt at their no-wait maxima.)
__device__ __forceinline__ void wait_global_loads() { __builtin_amdgcn_s_waitcnt(0x0F70); }

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
