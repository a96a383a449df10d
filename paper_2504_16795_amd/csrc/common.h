// Shared definitions of the HSA kernels for gfx950 (CDNA4, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hsa.h"

namespace hsa {

// Problem description passed by value to every kernel.
struct Dims {
    int B, L, H, G, h, d, S, k;
    int C;          // complete chunks, floor(L / S)
    int Call;       // chunks including a trailing partial one, ceil(L / S)
    float alpha;    // selection-score scale
    float beta;     // intra-chunk attention scale
    int stick;      // chunk weights: 0 softmax of the selected scores, 1 stick-breaking
    int off1;       // attention inside a chunk: 0 softmax, 1 softmax off by one (an extra
                    // logit 0 with no value: the row maximum covers it, and the normaliser
                    // gains exp(0 - max))
    // backward of the attention alone (the selection scores come from inputs of their
    // own): dw = d loss / d w per (b, t, g, slot) goes to dwo (added to it with dwacc),
    // and no score term reaches Q or K.  nullptr: the full backward.
    float* dwo;
    int dwacc;
};

// Kernel-family override of an op (hsa_attn_set_path; HSA_PATH_AUTO unless a caller set
// one): one relaxed atomic load, so a launcher may read it on every call.
int path_override(int op);

// bfloat16 storage type of the generic kernels (bit pattern only).
struct bf16 {
    uint16_t v;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return __uint_as_float(((uint32_t)x.v) << 16); }

// Round to nearest even; inputs are finite by contract (NaN is kept quiet anyway).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u >> 16) | ((u & 0xFFFF) ? 0x40 : 0));
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return bf16{f32_to_bf16_bits(x)}; }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}

// Cross-lane reductions without LDS traffic: DPP moves inside 16-lane rows (quad
// permutations, half-row and row mirrors), then the gfx950 lane swaps across rows.  After
// each step every lane of a group holds the group's value, and each combine takes the
// same two operands in both lanes of a pair, so all lanes end with the same result.
constexpr int kDppXor1 = 0xB1;          // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;          // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;   // lane i <- lane 7 - i within each 8 lanes
constexpr int kDppMirror = 0x140;       // lane i <- lane 15 - i within each 16 lanes

template <int CTRL>
__device__ __forceinline__ int dpp_mov(int v) {
    // every control used here reads a lane of the same row, so no lane is out of bounds
    return __builtin_amdgcn_mov_dpp(v, CTRL, 0xF, 0xF, true);
}
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
    return __int_as_float(dpp_mov<CTRL>(__float_as_int(v)));
}
// (own, partner) across 16-lane rows (l <-> l ^ 16) and across halves (l <-> l ^ 32)
template <bool HALVES>
__device__ __forceinline__ void lane_swap(float& a, float& b, float v) {
    const auto r = HALVES ? __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false)
                          : __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    a = __uint_as_float(r[0]);
    b = __uint_as_float(r[1]);
}
template <bool HALVES>
__device__ __forceinline__ void lane_swap(int& a, int& b, int v) {
    const auto r = HALVES ? __builtin_amdgcn_permlane32_swap((uint32_t)v, (uint32_t)v, false, false)
                          : __builtin_amdgcn_permlane16_swap((uint32_t)v, (uint32_t)v, false, false);
    a = (int)r[0];
    b = (int)r[1];
}

// sum over aligned groups of N consecutive lanes (N in {8, 16, 32, 64})
template <int N>
__device__ __forceinline__ float group_sum(float v) {
    v += dpp_mov<kDppXor1>(v);
    v += dpp_mov<kDppXor2>(v);
    v += dpp_mov<kDppHalfMirror>(v);
    if constexpr (N >= 16) v += dpp_mov<kDppMirror>(v);
    if constexpr (N >= 32) {
        float a, b;
        lane_swap<false>(a, b, v);
        v = a + b;
    }
    if constexpr (N >= 64) {
        float a, b;
        lane_swap<true>(a, b, v);
        v = a + b;
    }
    return v;
}

__device__ __forceinline__ float wave_max_dpp(float v) {
    v = fmaxf(v, dpp_mov<kDppXor1>(v));
    v = fmaxf(v, dpp_mov<kDppXor2>(v));
    v = fmaxf(v, dpp_mov<kDppHalfMirror>(v));
    v = fmaxf(v, dpp_mov<kDppMirror>(v));
    float a, b;
    lane_swap<false>(a, b, v);
    v = fmaxf(a, b);
    lane_swap<true>(a, b, v);
    return fmaxf(a, b);
}

// wave-wide best (s, c) pair: larger s, ties to the smaller c
__device__ __forceinline__ void pick_better(float& s, int& c, float s2, int c2) {
    if (s2 > s || (s2 == s && c2 < c)) {
        s = s2;
        c = c2;
    }
}
__device__ __forceinline__ void wave_argmax_dpp(float& s, int& c) {
    pick_better(s, c, dpp_mov<kDppXor1>(s), dpp_mov<kDppXor1>(c));
    pick_better(s, c, dpp_mov<kDppXor2>(s), dpp_mov<kDppXor2>(c));
    pick_better(s, c, dpp_mov<kDppHalfMirror>(s), dpp_mov<kDppHalfMirror>(c));
    pick_better(s, c, dpp_mov<kDppMirror>(s), dpp_mov<kDppMirror>(c));
    float s0, s1;
    int c0, c1;
    lane_swap<false>(s0, s1, s);
    lane_swap<false>(c0, c1, c);
    s = s0;
    c = c0;
    pick_better(s, c, s1, c1);
    lane_swap<true>(s0, s1, s);
    lane_swap<true>(c0, c1, c);
    s = s0;
    c = c0;
    pick_better(s, c, s1, c1);
}

// (score, chunk) as one unsigned 64-bit key ordered like (score desc, chunk asc): the float
// bits mapped to an order-preserving unsigned value above the complemented chunk id.  Key 0
// is below every key of a real candidate (even one scoring -inf).
__device__ __forceinline__ uint64_t order_key(float s, int c) {
    const uint32_t u = __float_as_uint(s + 0.0f);     // -0 and +0 rank alike

    const uint32_t o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ((uint64_t)o << 32) | (uint32_t)(~(uint32_t)c);
}
__device__ __forceinline__ int key_chunk(uint64_t key) { return (int)~(uint32_t)key; }
__device__ __forceinline__ float key_score(uint64_t key) {
    const uint32_t o = (uint32_t)(key >> 32);
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}
__device__ __forceinline__ uint64_t max_u64(uint64_t a, uint64_t b) { return b > a ? b : a; }

// Wave-wide maximum of an unsigned 32-bit value (DPP inside rows, then the lane swaps).
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
    x = max(x, (uint32_t)dpp_mov<kDppXor1>((int)x));
    x = max(x, (uint32_t)dpp_mov<kDppXor2>((int)x));
    x = max(x, (uint32_t)dpp_mov<kDppHalfMirror>((int)x));
    x = max(x, (uint32_t)dpp_mov<kDppMirror>((int)x));
    int a, b;
    lane_swap<false>(a, b, (int)x);
    x = max((uint32_t)a, (uint32_t)b);
    lane_swap<true>(a, b, (int)x);
    return max((uint32_t)a, (uint32_t)b);
}

// The maximum of wave_max_key, found on the upper word first (one 32-bit wave maximum) and
// on the lower word only when several lanes share that upper word.  Every lane of the wave
// must be active.
__device__ __forceinline__ uint64_t wave_max_key_hi(uint64_t x) {
    const uint32_t hi = (uint32_t)(x >> 32);
    const uint32_t bh = wave_max_u32(hi);
    const uint64_t tied = __builtin_amdgcn_ballot_w64(hi == bh);
    uint32_t bl;
    if (__builtin_popcountll(tied) == 1)
        bl = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, __builtin_ctzll(tied));
    else
        bl = wave_max_u32(hi == bh ? (uint32_t)x : 0u);
    return ((uint64_t)bh << 32) | bl;
}

// Wave-wide maximum of a 64-bit key, branch-free (DPP moves inside rows, then the lane
// swaps across rows); every lane ends with the maximum.
__device__ __forceinline__ uint64_t wave_max_key(uint64_t x) {
    auto step = [&](auto mov) __attribute__((always_inline)) {
        const uint32_t lo = (uint32_t)mov((int)(uint32_t)x);
        const uint32_t hi = (uint32_t)mov((int)(uint32_t)(x >> 32));
        x = max_u64(x, ((uint64_t)hi << 32) | lo);
    };
    step([](int v) { return dpp_mov<kDppXor1>(v); });
    step([](int v) { return dpp_mov<kDppXor2>(v); });
    step([](int v) { return dpp_mov<kDppHalfMirror>(v); });
    step([](int v) { return dpp_mov<kDppMirror>(v); });
    int a0, a1, b0, b1;
    lane_swap<false>(a0, a1, (int)(uint32_t)x);
    lane_swap<false>(b0, b1, (int)(uint32_t)(x >> 32));
    x = max_u64(((uint64_t)(uint32_t)b0 << 32) | (uint32_t)a0,
                ((uint64_t)(uint32_t)b1 << 32) | (uint32_t)a1);
    lane_swap<true>(a0, a1, (int)(uint32_t)x);
    lane_swap<true>(b0, b1, (int)(uint32_t)(x >> 32));
    x = max_u64(((uint64_t)(uint32_t)b0 << 32) | (uint32_t)a0,
                ((uint64_t)(uint32_t)b1 << 32) | (uint32_t)a1);
    return x;
}

__host__ __device__ __forceinline__ int cdiv(int a, int b) { return (a + b - 1) / b; }

// Chunk weights of the n best entries of a selection list (scores ls[j] in descending score
// order, chunks lc[j], j < n) and each entry's slot in descending chunk order (rank[j]).
// Softmax over the n scores (Sec. 3.1.1, the ablation without stick-breaking), or, with
// stick, stick-breaking in slot order: b_j = sigmoid(s_j), w_j = b_j times the product of
// (1 - b_i) over the entries i in earlier slots (higher chunks).
template <int KC>
__device__ __forceinline__ void list_weights(const float (&ls)[KC], const int (&lc)[KC], int n,
                                             bool stick, float (&wt)[KC], int (&rank)[KC]) {
#pragma unroll
    for (int j = 0; j < KC; ++j) {
        int r = 0;
#pragma unroll
        for (int i = 0; i < KC; ++i) r += (i < n && lc[i] > lc[j]) ? 1 : 0;
        rank[j] = r;
    }
    if (stick) {
        float om[KC];                            // 1 - b = sigmoid(-s)
#pragma unroll
        for (int j = 0; j < KC; ++j) om[j] = (j < n) ? 1.f / (1.f + expf(ls[j])) : 1.f;
#pragma unroll
        for (int j = 0; j < KC; ++j) {
            float left = 1.f;
#pragma unroll
            for (int i = 0; i < KC; ++i) left *= (i < n && lc[i] > lc[j]) ? om[i] : 1.f;
            wt[j] = (j < n) ? left / (1.f + expf(-ls[j])) : 0.f;
        }
    } else {
        float z = 0.f;
#pragma unroll
        for (int j = 0; j < KC; ++j) {
            wt[j] = (j < n) ? expf(ls[j] - ls[0]) : 0.f;
            z += wt[j];
        }
        const float iz = 1.f / z;
#pragma unroll
        for (int j = 0; j < KC; ++j) wt[j] *= iz;
    }
}

// Stick-breaking gradient w.r.t. the score of slot s (Sec. 3.1.1 weights, see list_weights)
// from the slots' weights w(i) and dw(i) = dL/dw_i, over the slots with ok(i): b_s is
// recovered from the weights as w_s / (1 - sum_{m<s} w_m), and
// ds_s = (1 - b_s) w_s dw_s - b_s sum_{m>s} w_m dw_m (b_s directly, and through the factor
// (1 - b_s) of every later slot).
template <class W, class DW, class OK>
__device__ __forceinline__ float stick_ds(int s, int k, W w, DW dw, OK ok) {
    if (!ok(s)) return 0.f;
    float before = 0.f, tail = 0.f;
    for (int m = 0; m < k; ++m) {
        if (!ok(m)) continue;
        if (m < s) before += w(m);
        if (m > s) tail = fmaf(w(m), dw(m), tail);
    }
    const float u = 1.f - before;
    const float bs = u > 0.f ? w(s) / u : 0.f;
    return (1.f - bs) * w(s) * dw(s) - bs * tail;
}

// The same with one entry per lane (lane r holds the r-th best, (ls, lc), present when has;
// the first n lanes hold entries): the lane's weight and slot.
__device__ __forceinline__ void lane_weights(float ls, int lc, bool has, int n, bool stick,
                                             float& wt, int& rank) {
    rank = 0;
    for (int j = 0; j < n; ++j) rank += (__shfl(lc, j, 64) > lc) ? 1 : 0;
    if (stick) {
        const float om = has ? 1.f / (1.f + expf(ls)) : 1.f;
        float left = 1.f;
        for (int j = 0; j < n; ++j) {
            const float oj = __shfl(om, j, 64);
            left *= (__shfl(lc, j, 64) > lc) ? oj : 1.f;
        }
        wt = has ? left / (1.f + expf(-ls)) : 0.f;
    } else {
        const float m = __shfl(ls, 0, 64);
        const float ex = has ? expf(ls - m) : 0.f;
        wt = ex / wave_sum(ex);
    }
}

// RAII bracket of one kernel launch for the optional per-kernel timing (timing.hip).
class KernelTimer {
  public:
    KernelTimer(const char* name, hipStream_t st);
    ~KernelTimer();
    KernelTimer(const KernelTimer&) = delete;
    KernelTimer& operator=(const KernelTimer&) = delete;

  private:
    const char* name_;
    hipStream_t st_;
    hipEvent_t a_ = nullptr, b_ = nullptr;
};

#define HSA_TIMED(name, st) ::hsa::KernelTimer hsa_kernel_timer_(name, st)

}  // namespace hsa

// Host launchers implemented in the kernel translation units (called by hsa_api.hip).
namespace hsa {
hipError_t launch_landmarks(const Dims& dm, bool in_bf16, const void* K, void* Kbar,
                            bool out_bf16, int c0, int c1, hipStream_t st);
hipError_t launch_select(const Dims& dm, bool in_bf16, const void* Q, const float* Kbar,
                         int32_t* idx, float* w, hipStream_t st);
hipError_t launch_forward(const Dims& dm, bool in_bf16, const void* Q, const void* K,
                          const void* V, const int32_t* idx, const float* w, void* O,
                          void* ws, hipStream_t st);
size_t forward_workspace(const Dims& dm, bool in_bf16);
size_t backward_workspace(const Dims& dm);
hipError_t launch_backward(const Dims& dm, bool in_bf16, const void* Q, const void* K,
                           const void* V, const float* Kbar, const int32_t* idx,
                           const float* w, const void* dO, void* dQ, void* dK, void* dV,
                           void* ws, hipStream_t st);
size_t select_backward_workspace(const Dims& dm);
bool select_backward_supported(const Dims& dm);
hipError_t launch_select_backward(const Dims& dm, bool in_bf16, const void* Q,
                                  const float* Kbar, const int32_t* idx, const float* w,
                                  const float* dw, void* dQ, float* dKbar, void* ws,
                                  hipStream_t st);
size_t decode_workspace(const Dims& dm);
size_t decode_host_workspace(const Dims& dm, bool in_bf16);
hipError_t launch_decode_host(const Dims& dm, bool in_bf16, const void* q, const void* Kh,
                              const void* Vh, const void* Kbar, bool kbar_bf16,
                              const int32_t* cache_len, void* o, int32_t* idx, float* w,
                              void* ws, hipStream_t st);
hipError_t launch_decode(const Dims& dm, bool in_bf16, const void* q, const void* Kc,
                         const void* Vc, const void* Kbar, bool kbar_bf16,
                         const int32_t* cache_len, void* o, int32_t* idx, float* w,
                         void* ws, hipStream_t st);
}  // namespace hsa
