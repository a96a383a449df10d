// Forward of hierarchical sparse attention (Sec. 3.1.1 "Hierarchical Attention").
//
// Generic path (any supported h, d, S; fp32 or bf16): one workgroup per (b, t, g), as in
// the paper's per-token program: the group's h query rows live in LDS, each selected chunk
// is staged in LDS, each wave takes a head, lanes take keys, the softmax over the S keys
// is a wave reduction, and the weighted chunk output is accumulated in registers.
// Without an online softmax: every chunk is normalised on its own and scaled by w_i.
//
// The bf16 MFMA paths for the main shapes live in forward_mfma.hip (tile-major) and
// forward_fused.hip (chunk-major, for sequences with many chunks); launch_forward selects
// them when they apply.
#include <type_traits>

#include "common.h"

namespace hsa {

bool forward_mfma_supported(const Dims& dm, bool in_bf16);
bool forward_chunk_used(const Dims& dm, bool in_bf16);
size_t forward_chunk_workspace(const Dims& dm, bool in_bf16);
hipError_t launch_forward_chunk(const Dims& dm, const void* Q, const void* K, const void* V,
                                const int32_t* idx, const float* w, void* O, void* ws,
                                hipStream_t st);
hipError_t launch_forward_mfma(const Dims& dm, const void* Q, const void* K, const void* V,
                               const int32_t* idx, const float* w, void* O, void* ws,
                               hipStream_t st);

namespace {

constexpr int kThreads = 256;
constexpr int HMAX = 16;
constexpr int KMAX = 32;

template <typename T, int D, int CS>
__global__ __launch_bounds__(kThreads) void forward_generic(Dims dm, const T* __restrict__ Q,
                                                            const T* __restrict__ K,
                                                            const T* __restrict__ V,
                                                            const int32_t* __restrict__ idx,
                                                            const float* __restrict__ w,
                                                            T* __restrict__ O) {
    constexpr int KP = D + (sizeof(T) == 4 ? 1 : 2);
    constexpr int NACC = HMAX * D / kThreads;
    __shared__ T Ks[CS * KP];
    __shared__ T Vs[CS * D];
    __shared__ float qf[HMAX * D];
    __shared__ float p[HMAX * CS];
    __shared__ int sc[KMAX];
    __shared__ float sw[KMAX];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int t = blockIdx.x;
    const int bg = blockIdx.y, b = bg / dm.G, g = bg % dm.G;
    const int h = dm.h, S = dm.S, k = dm.k;
    const size_t qoff = (((size_t)b * dm.L + t) * dm.H + (size_t)g * h) * D;

    // the token's slots (an empty or out-of-range one as -1), its query rows
    const size_t sel = (((size_t)b * dm.L + t) * dm.G + g) * k;
    if (tid < k) {
        const int c = idx[sel + tid];
        sc[tid] = (c < 0 || c >= t / S) ? -1 : c;
        sw[tid] = w[sel + tid];
    }
    for (int i = tid; i < h * D; i += kThreads) qf[i] = to_f32(Q[qoff + i]);
    float acc[NACC];
#pragma unroll
    for (int r = 0; r < NACC; ++r) acc[r] = 0.f;
    __syncthreads();

    // each slot's K / V rows are loaded into registers while the slot before is computed
    // (for chunks of up to 4096 elements; larger ones would cost the workgroups per CU)
    constexpr int NS = CS * D / kThreads;
    constexpr bool PREF = CS * D <= 4096;
    T kr[NS], vr[NS];
    auto load_chunk = [&](int c) __attribute__((always_inline)) {
#pragma unroll
        for (int r = 0; r < NS; ++r) {
            const int i = tid + r * kThreads, s = i / D, e = i % D;
            const size_t gi = (((size_t)b * dm.L + (size_t)c * S + s) * dm.G + g) * D + e;
            kr[r] = K[gi];
            vr[r] = V[gi];
        }
    };
    auto next_slot = [&](int from) __attribute__((always_inline)) {
        int s2 = from;
        while (s2 < k && sc[s2] < 0) ++s2;
        return s2;
    };
    int slot = next_slot(0);
    if constexpr (PREF) {
        if (slot < k) load_chunk(sc[slot]);
    }
    while (slot < k) {
        const float wi = sw[slot];
        __syncthreads();                  // the previous slot's tiles and weights are read
        if constexpr (PREF) {
#pragma unroll
            for (int r = 0; r < NS; ++r) {
                const int i = tid + r * kThreads, s = i / D, e = i % D;
                Ks[s * KP + e] = kr[r];
                Vs[s * D + e] = vr[r];
            }
        } else {
            const int c = sc[slot];
            for (int i = tid; i < S * D; i += kThreads) {
                const int s = i / D, e = i % D;
                const size_t gi = (((size_t)b * dm.L + (size_t)c * S + s) * dm.G + g) * D + e;
                Ks[s * KP + e] = K[gi];
                Vs[s * D + e] = V[gi];
            }
        }
        const int nslot = next_slot(slot + 1);
        if constexpr (PREF) {
            if (nslot < k) load_chunk(sc[nslot]);
        }
        slot = nslot;
        __syncthreads();
        for (int j = wave; j < h; j += kThreads / 64) {
            float z[2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int s = lane + 64 * u;
                if (s < S) {
                    // four partial sums, so the products do not wait on one another
                    float a4[4] = {0.f, 0.f, 0.f, 0.f};
                    for (int e = 0; e < D; e += 4) {
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            a4[q] = fmaf(qf[j * D + e + q], to_f32(Ks[s * KP + e + q]), a4[q]);
                    }
                    z[u] = dm.beta * ((a4[0] + a4[1]) + (a4[2] + a4[3]));
                } else {
                    z[u] = -INFINITY;
                }
            }
            float m = wave_max(fmaxf(z[0], z[1]));
            if (dm.off1) m = fmaxf(m, 0.f);
            const float e0 = expf(z[0] - m), e1 = expf(z[1] - m);
            const float scale = wi / (wave_sum(e0 + e1) + (dm.off1 ? expf(-m) : 0.f));
            if (lane < S) p[j * CS + lane] = e0 * scale;
            if (lane + 64 < S) p[j * CS + lane + 64] = e1 * scale;
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < NACC; ++r) {
            const int i = tid + r * kThreads;
            if (i < h * D) {
                const int j = i / D, e = i % D;
                float a4[4] = {0.f, 0.f, 0.f, 0.f};   // S is a multiple of 4
                for (int s = 0; s < S; s += 4) {
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        a4[q] = fmaf(p[j * CS + s + q], to_f32(Vs[(s + q) * D + e]), a4[q]);
                }
                acc[r] += (a4[0] + a4[1]) + (a4[2] + a4[3]);
            }
        }
    }
#pragma unroll
    for (int r = 0; r < NACC; ++r) {
        const int i = tid + r * kThreads;
        if (i < h * D) O[qoff + i] = from_f32<T>(acc[r]);
    }
}

template <typename T>
hipError_t launch_t(const Dims& dm, const void* Q, const void* K, const void* V,
                    const int32_t* idx, const float* w, void* O, hipStream_t st) {
    dim3 grid(dm.L, dm.B * dm.G);
    // LDS sized for the chunk (so short chunks leave room for more workgroups per CU)
    auto fwd = [&](auto dc, auto sc) {
        constexpr int DD = decltype(dc)::value, SS = decltype(sc)::value;
        HSA_TIMED("forward_generic", st);
        hipLaunchKernelGGL((forward_generic<T, DD, SS>), grid, dim3(kThreads), 0, st, dm,
                           (const T*)Q, (const T*)K, (const T*)V, idx, w, (T*)O);
    };
    auto fwd_s = [&](auto dc) {
        switch (dm.S) {
            case 16: fwd(dc, std::integral_constant<int, 16>{}); break;
            case 32: fwd(dc, std::integral_constant<int, 32>{}); break;
            case 64: fwd(dc, std::integral_constant<int, 64>{}); break;
            default:
                // float32 with S = 128 and d = 128 is rejected by the argument checks
                if constexpr (!(sizeof(T) == 4 && decltype(dc)::value == 128))
                    fwd(dc, std::integral_constant<int, 128>{});
                break;
        }
    };
    if (dm.d == 128) fwd_s(std::integral_constant<int, 128>{});
    else fwd_s(std::integral_constant<int, 64>{});
    return hipGetLastError();
}

}  // namespace

hipError_t launch_forward(const Dims& dm, bool in_bf16, const void* Q, const void* K,
                          const void* V, const int32_t* idx, const float* w, void* O, void* ws,
                          hipStream_t st) {
    if (dm.B == 0 || dm.L == 0) return hipSuccess;
    if (forward_chunk_used(dm, in_bf16))
        return launch_forward_chunk(dm, Q, K, V, idx, w, O, ws, st);
    if (forward_mfma_supported(dm, in_bf16))
        return launch_forward_mfma(dm, Q, K, V, idx, w, O, ws, st);
    return in_bf16 ? launch_t<bf16>(dm, Q, K, V, idx, w, O, st)
                   : launch_t<float>(dm, Q, K, V, idx, w, O, st);
}

size_t forward_workspace(const Dims& dm, bool in_bf16) {
    return forward_chunk_workspace(dm, in_bf16);
}

hipError_t launch_forward_generic(const Dims& dm, bool in_bf16, const void* Q, const void* K,
                                  const void* V, const int32_t* idx, const float* w, void* O,
                                  hipStream_t st) {
    if (dm.B == 0 || dm.L == 0) return hipSuccess;
    return in_bf16 ? launch_t<bf16>(dm, Q, K, V, idx, w, O, st)
                   : launch_t<float>(dm, Q, K, V, idx, w, O, st);
}

}  // namespace hsa
