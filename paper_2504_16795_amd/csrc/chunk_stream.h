// The even split of chunk-major work used by the fused forward and backward passes (bf16,
// h = 8, d = 128, S = 64) and by the generic key pass, and helpers they share.
//
// Work is counted in groups of 4 consecutive tokens of a chunk's selecting tokens (in the
// fused passes 32 rows = 4 tokens x 8 heads of a KV group).  A chunk's tokens come from the selection bitmap (bit t
// of row (b, g, c) set when token t selected chunk c) in increasing order.  The groups of all
// rows are laid end to end (slices, then chunks) and split into kStreamWGs equal ranges, one
// per workgroup: stream_rowcount counts each row's tokens, stream_plan lays out the group
// prefix gstart[] and the range length T.  A workgroup walks the rows its range touches; it
// covers a row whole, or shares it with its neighbours (then it is the first or the last row
// of the range, partial slot 0 or 1).
#pragma once

#include "chunk_lds.h"

namespace hsa {
namespace {

constexpr int CS = 64;              // chunk size of the fused passes
constexpr int NW = 4;               // waves per workgroup, 16 keys each
constexpr int NT = NW * 64;
constexpr int FLIST = 1024;         // tokens listed at once (a multiple of 4)
constexpr int kStreamWGs = 512;     // workgroups of the split: two per CU

__host__ __device__ inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// dZ^T tile: 64 keys x 32 rows of bf16, 64 bytes per key in 8-byte units of 4 rows; unit u
// of key j sits at position u ^ zsw(j).  Both the C-layout writes (unit 4 rb + lane group of
// 16 consecutive keys per instruction) and the transposed reads (4 units of 8 consecutive
// keys per 32-lane pass) then fall on distinct banks.
__device__ __forceinline__ int zsw(int j) { return (((j >> 2) & 1) << 2) | (((j >> 3) & 1) << 1); }
__device__ __forceinline__ int zpos(int j, int u) { return j * 32 + 4 * (u ^ zsw(j)); }

// Reductions of N rows at once over the 16 lanes of each row (the lanes holding one row of a
// C layout): each step is applied to every row before the next, so no step waits on the
// one before it.  Maxima on the order-preserving integer image of the floats (finite
// inputs), one integer max with a DPP operand per step; sums with a DPP operand per step.
template <int N>
__device__ __forceinline__ void rows16_max(float (&x)[N]) {
    int v[N];
#pragma unroll
    for (int i = 0; i < N; ++i) {
        v[i] = __float_as_int(x[i]);
        v[i] ^= (v[i] >> 31) & 0x7fffffff;
    }
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = max(v[i], dpp_mov<kDppXor1>(v[i]));
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = max(v[i], dpp_mov<kDppXor2>(v[i]));
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = max(v[i], dpp_mov<kDppHalfMirror>(v[i]));
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = max(v[i], dpp_mov<kDppMirror>(v[i]));
#pragma unroll
    for (int i = 0; i < N; ++i) x[i] = __int_as_float(v[i] ^ ((v[i] >> 31) & 0x7fffffff));
}
// Softmax exponentials of N row values per lane (rows of 16 lanes, the wave's keys along the
// row): e = 2^(x - m) with m a reference per row, and m.  Any finite reference gives the same
// softmax once the combine rescales by 2^(m - max); the reference is the row's value at its
// first lane (one DPP broadcast) unless some exponential of the wave would exceed 2^64, in
// which case (a logit spread of more than 64 in log2 units around that key) the rows take
// their maxima.  Either way no exponential overflows and the row's largest is at least 1.
template <int N>
__device__ __forceinline__ void rows16_exp(const float (&x)[N], float (&e)[N], float (&m)[N]) {
    float emax = 0.f;
#pragma unroll
    for (int i = 0; i < N; ++i) {
        // row_newbcast:0: lane 16 r of each row of 16 lanes to the whole row
        m[i] = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x[i]), 0x150, 0xF, 0xF, true));
        e[i] = fast_exp2(x[i] - m[i]);
        emax = fmaxf(emax, e[i]);
    }
    if (__builtin_amdgcn_ballot_w64(!(emax <= 0x1p64f))) {
#pragma unroll
        for (int i = 0; i < N; ++i) m[i] = x[i];
        rows16_max(m);
#pragma unroll
        for (int i = 0; i < N; ++i) e[i] = fast_exp2(x[i] - m[i]);
    }
}

template <int N>
__device__ __forceinline__ void rows16_sum(float (&x)[N]) {
#pragma unroll
    for (int i = 0; i < N; ++i) x[i] += dpp_mov<kDppXor1>(x[i]);
#pragma unroll
    for (int i = 0; i < N; ++i) x[i] += dpp_mov<kDppXor2>(x[i]);
#pragma unroll
    for (int i = 0; i < N; ++i) x[i] += dpp_mov<kDppHalfMirror>(x[i]);
#pragma unroll
    for (int i = 0; i < N; ++i) x[i] += dpp_mov<kDppMirror>(x[i]);
}

// maximum over the 16 lanes of a row, on the order-preserving integer image of the floats
// (finite inputs): each step is one integer max with a DPP operand
__device__ __forceinline__ float row16_max(float x) {
    int v = __float_as_int(x);
    v ^= (v >> 31) & 0x7fffffff;
    v = max(v, dpp_mov<kDppXor1>(v));
    v = max(v, dpp_mov<kDppXor2>(v));
    v = max(v, dpp_mov<kDppHalfMirror>(v));
    v = max(v, dpp_mov<kDppMirror>(v));
    return __int_as_float(v ^ ((v >> 31) & 0x7fffffff));
}

// LDS writes of this wave complete (before a barrier that publishes them)
__device__ __forceinline__ void lds_wait() {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

// Tokens at positions [p0, p1) of a chunk's ascending token list (the set bits of bitmap
// words wbeg .. nwords - 1 of its row) into list[0 .. p1 - p0).  Whole workgroup (NTT
// threads); the words are counted NTT at a time with a workgroup prefix sum, stopping once
// p1 is reached.
template <int NTT = NT>
__device__ __forceinline__ void collect_tokens(const uint32_t* __restrict__ bmrow, int wbeg,
                                               int nwords, int p0, int p1, int* list,
                                               int* wtot, int tid) {
    const int lane = tid & 63, wave = tid >> 6;
    int base = 0;
    for (int wb = wbeg; wb < nwords; wb += NTT) {
        const int wi = wb + tid;
        const uint32_t word = wi < nwords ? bmrow[wi] : 0u;
        const int cnt = __popc(word);
        int incl = cnt;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int v = __shfl_up(incl, o, 64);
            if (lane >= o) incl += v;
        }
        if (lane == 63) wtot[wave] = incl;
        __syncthreads();
        int before = 0, tot = 0;
#pragma unroll
        for (int w2 = 0; w2 < NTT / 64; ++w2) {
            const int v = wtot[w2];
            before += (w2 < wave) ? v : 0;
            tot += v;
        }
        int pos = base + before + incl - cnt;
        if (pos < p1 && pos + cnt > p0) {
            uint32_t x = word;
            while (x) {
                if (pos >= p0 && pos < p1) list[pos - p0] = wi * 32 + (__ffs(x) - 1);
                ++pos;
                x &= x - 1;
            }
        }
        base += tot;
        __syncthreads();                // wtot is rewritten by the next block
        if (base >= p1) break;
    }
}

// The row (b, g, chunk) holding global group gpos: the last r with gstart[r] <= gpos
// (gstart is non-decreasing, gstart[0] = 0 <= gpos < gstart[R]).
__device__ __forceinline__ int find_row(const int* __restrict__ gstart, int R, int gpos) {
    int lo = 0, hi = R;                 // gstart[lo] <= gpos < gstart[hi]
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (gstart[mid] <= gpos) lo = mid;
        else hi = mid;
    }
    return lo;
}

// tokens per bitmap row (one wave per row)
__global__ __launch_bounds__(256) void stream_rowcount(const uint32_t* __restrict__ bm, int R,
                                                    int nwords, int C, int S,
                                                    int* __restrict__ cnt) {
    const int lane = threadIdx.x & 63;
    const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= R) return;
    const int c = r % C;
    const uint32_t* row = bm + (size_t)r * nwords;
    int n = 0;
    for (int wi = ((c + 1) * S >> 5) + lane; wi < nwords; wi += 64) n += __popc(row[wi]);
    n = (int)group_sum<64>((float)n);   // exact: counts stay far below 2^24
    if (lane == 0) cnt[r] = n;
}

// group prefix over the rows (one workgroup): gstart[r] = sum_{r' < r} ceil(cnt[r'] / 4);
// plan = {total groups, groups per workgroup}
__global__ __launch_bounds__(1024) void stream_plan(const int* __restrict__ cnt, int R, int nwg,
                                                 int* __restrict__ gstart, int* __restrict__ plan) {
    __shared__ int wt[16];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int carry = 0;
    for (int r0 = 0; r0 < R; r0 += 1024) {
        const int r = r0 + tid;
        const int ng = r < R ? (cnt[r] + 3) >> 2 : 0;
        int incl = ng;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int v = __shfl_up(incl, o, 64);
            if (lane >= o) incl += v;
        }
        if (lane == 63) wt[wave] = incl;
        __syncthreads();
        int before = 0, tot = 0;
        for (int w2 = 0; w2 < 16; ++w2) {
            before += (w2 < wave) ? wt[w2] : 0;
            tot += wt[w2];
        }
        if (r < R) gstart[r] = carry + before + incl - ng;
        carry += tot;
        __syncthreads();
    }
    if (tid == 0) {
        gstart[R] = carry;
        plan[0] = carry;
        plan[1] = carry > 0 ? (carry + nwg - 1) / nwg : 1;
    }
}

// Offset (in a chunk tile of chunk_lds.h) of the transposed read that hands lane i of each
// 16-lane group column d0 + 8 (i >> 2) + 4 dt + (i & 3) of rows kb .. kb + 3, kb = 4 (lane >>
// 4) (the caller adds 16 hf + 32 ks2 rows): lane p loads row kb + (p >> 2) at columns d0 +
// 8 (p & 3) + 4 dt .. +3.  With these as the A operand of a product whose rows are columns
// of d, the C layout of tiles dt = 0, 1 gives each lane 8 consecutive columns, stored as one
// 16-byte write.  Read once per chunk, so its 2-way bank conflicts do not matter.
__device__ __forceinline__ int tr_perm_offset(int lane, int d0, int dt) {
    const int p = lane & 15, r = 4 * (lane >> 4) + (p >> 2);
    return r * kChunkD + unit_pos(r, (d0 >> 3) + (p & 3)) * 8 + 4 * dt;
}

// The segment of row r covered by groups [g0, g1): groups [j0, j1) of the row; whole when
// that is all of them; pslot 0 when r is the first row of the range, else 1 (only the last
// row of a range can then be partial).
struct Segment {
    int j0, j1, pslot;
    bool whole;
};
__device__ __forceinline__ Segment segment_of(int rs, int re, int g0, int g1) {
    Segment s;
    s.j0 = max(g0, rs) - rs;
    s.j1 = min(g1, re) - rs;
    s.whole = (s.j0 == 0 && s.j1 == re - rs);
    s.pslot = (rs <= g0) ? 0 : 1;
    return s;
}

}  // namespace
}  // namespace hsa
