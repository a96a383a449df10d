// LDS staging of key / value chunks for the MFMA kernels (gfx950).
//
// A chunk is S rows of d = 128 bf16 (one row per key), 256 bytes per row, stored unpadded
// with its 16-byte units swizzled: unit j of row r sits at unit position j ^ f(r), with
// f(r) = 2 (r & 7) + ((r >> 3) & 1), a permutation of the low 4 bits of r.
//   - row reads (16 bytes per lane; one unit of each of 16 consecutive rows per 16-lane
//     pass) land on 16 distinct positions: f is injective on r mod 16;
//   - transposed reads (8 bytes per lane; per 32-lane pass, two neighbouring units of 8
//     consecutive rows 8a .. 8a + 7) land on 16 distinct positions: f(r) >> 1 = r & 7
//     differs between those rows and f's low bit is the same for all of them.
// Both cover all 64 banks without conflicts.
// Chunks are copied straight from global memory into LDS with global_load_lds_dwordx4
// (16 bytes per lane, no registers): lane l of a copy instruction writes bytes
// [16 l, 16 l + 16) of the instruction's 1 KB LDS block, so each lane fetches the global
// unit that belongs at its position.
//
// ds_read_b64_tr_b16 reads 4 bf16 per lane and transposes them inside each 16-lane group:
// lane i receives element (i & 3) of the 4 loaded by lane 4 m + (i >> 2), for m = 0..3.
// If lane 4 m + q loads row kb + m at columns d0 + 4 q .. +3, lane i ends up with column
// d0 + i of rows kb .. kb + 3: the key-contiguous operand fragment an MFMA needs from a
// row-major (key-major) tile.
#pragma once

#include "mfma_common.h"

namespace hsa {

typedef short i16x4_t __attribute__((ext_vector_type(4)));

constexpr int kChunkD = 128;          // bf16 elements per row

__device__ __forceinline__ int swz(int r) { return ((r & 7) << 1) | ((r >> 3) & 1); }
__device__ __forceinline__ int unit_pos(int r, int j) { return j ^ swz(r); }

// One LDS stage of a chunk: K and V rows, each swizzled.  V sits at a fixed offset from K,
// so reads of both use one address register per lane and immediate offsets.
template <int S>
struct ChunkStage {
    __bf16 k[S * kChunkD];
    __bf16 v[S * kChunkD];
};

// One global_load_lds_dwordx4: lane l copies 16 bytes from gsrc to LDS byte address
// lds_base + 16 l (lds_base wave-uniform, passed in M0).  Issued as inline assembly: the
// compiler's wait insertion would otherwise make every later transposed LDS read wait for
// all copies in flight, including the ones into stages not being read.  Completion is
// tracked by the callers with explicit vmcnt waits; no compiler-visible global load may be
// outstanding across these copies (the kernels drain theirs before the copy loop).
__device__ __forceinline__ void lds_copy16(const void* gsrc, uint32_t lds_base) {
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(gsrc), "{m0}"(lds_base)
                 : "memory");
}

__device__ __forceinline__ uint32_t lds_address(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// Copies rows [0, S) of a chunk (row r at src + r * rowstride) into dst (S * 128 bf16,
// swizzled).  NW waves share the work: wave w issues the 1 KB blocks w, w + NW, ...
// (rows 4 blk .. 4 blk + 3).  Each wave issues S / 4 / NW copy instructions.
template <int S, int NW>
__device__ __forceinline__ void chunk_to_lds(const __bf16* __restrict__ src, size_t rowstride,
                                             __bf16* dst, int wave, int lane) {
    static_assert((S / 4) % NW == 0, "blocks must split evenly over the waves");
#pragma unroll
    for (int i = 0; i < S / 4 / NW; ++i) {
        const int blk = wave + i * NW;
        const int r = blk * 4 + (lane >> 4);
        const int j = unit_pos(r, lane & 15);
        lds_copy16(src + (size_t)r * rowstride + j * 8,
                   __builtin_amdgcn_readfirstlane(lds_address(dst + blk * 512)));
    }
}

// Workgroup barrier that leaves this wave's copies in flight (__syncthreads would wait for
// all of them).  The caller's explicit waits make its own copies and LDS writes complete
// first; the empty assembly statements keep the compiler from moving memory accesses
// across the barrier.
__device__ __forceinline__ void barrier_keep_copies() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Waits until at most n of this wave's global loads (copies included) are in flight.
template <int N>
__device__ __forceinline__ void wait_loads_le() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

__device__ __forceinline__ bf16x4_t ld_tr16(const __bf16* p) {
    const i16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) i16x4_t*)(p));
    return __builtin_bit_cast(bf16x4_t, v);
}

// Per-lane element offsets of the row reads of a chunk: the 16 x 32 A fragment of key
// block mb, d step ks (lane: key 16 mb + (lane & 15), d 32 ks + 8 (lane >> 4) .. +7) is at
// koff[ks] + mb * 2048.
__device__ __forceinline__ void row_read_offsets(int lane, int koff[4]) {
    const int row = lane & 15, grp = lane >> 4;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) koff[ks] = row * kChunkD + unit_pos(row, 4 * ks + grp) * 8;
}

// Per-lane element offsets of the transposed reads of a chunk: for column block db
// (d = 16 db + (lane & 15)) the lane's 4 keys kb .. kb + 3, kb = 4 (lane >> 4) + 16 hf +
// 32 ks2, are at toff[db] + (16 hf + 32 ks2) * 128.  The lane loads row kb + (p >> 2),
// columns 16 db + 4 (p & 3) .. +3 (p = lane & 15), which the transpose hands to the lanes
// of its 16-lane group.
__device__ __forceinline__ void tr_read_offsets(int lane, int toff[8]) {
    const int p = lane & 15, grp = lane >> 4;
    const int r = 4 * grp + (p >> 2);                // row within the 16-row half block
#pragma unroll
    for (int db = 0; db < 8; ++db)
        toff[db] = r * kChunkD + unit_pos(r, 2 * db + ((p & 3) >> 1)) * 8 + 4 * (p & 1);
}

}  // namespace hsa
