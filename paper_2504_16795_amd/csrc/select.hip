// Chunk selection + chunk weights (Sec. 3.1: the top-k chunks by the landmark score
// s_c = alpha * (sum_j q_j) . Kbar_c over the chunks before the token's own, and their
// softmax weights).
//
// One wave per tile of 64 consecutive tokens of one (b, g); lane = token.  Each lane keeps
// its group query q~ = sum_j q_j (fp32, d registers) and a running top-KC list (scores and
// chunk indices, registers, descending).  Candidates are visited in increasing chunk
// order; the landmark row Kbar_c is read at the same address by every lane.  A candidate enters a list only when its score is strictly greater than the
// list's last entry and moves up past every entry it beats strictly: on equal scores the
// lower chunk index stays first.  The k best get softmax weights and are written in
// descending chunk order, padded with -1 / 0.
#include "common.h"

namespace hsa {
namespace {

constexpr int kTile = 64;     // tokens per wave

// q~ = sum over the h heads of the group, for token t (d fp32 values in qb)
template <int D>
__device__ __forceinline__ void group_query(const bf16* __restrict__ qp, int h, float (&qb)[D]) {
#pragma unroll
    for (int e = 0; e < D; ++e) qb[e] = 0.f;
    for (int j = 0; j < h; ++j) {
        const uint4* p = reinterpret_cast<const uint4*>(qp + (size_t)j * D);
#pragma unroll
        for (int v = 0; v < D / 8; ++v) {
            const uint4 u = p[v];
            const uint32_t wds[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                qb[8 * v + 2 * i] += __uint_as_float(wds[i] << 16);
                qb[8 * v + 2 * i + 1] += __uint_as_float(wds[i] & 0xFFFF0000u);
            }
        }
    }
}

template <int D>
__device__ __forceinline__ void group_query(const float* __restrict__ qp, int h, float (&qb)[D]) {
#pragma unroll
    for (int e = 0; e < D; ++e) qb[e] = 0.f;
    for (int j = 0; j < h; ++j) {
        const float4* p = reinterpret_cast<const float4*>(qp + (size_t)j * D);
#pragma unroll
        for (int v = 0; v < D / 8; ++v) {
            const float4 u0 = p[2 * v], u1 = p[2 * v + 1];
            qb[8 * v] += u0.x;
            qb[8 * v + 1] += u0.y;
            qb[8 * v + 2] += u0.z;
            qb[8 * v + 3] += u0.w;
            qb[8 * v + 4] += u1.x;
            qb[8 * v + 5] += u1.y;
            qb[8 * v + 6] += u1.z;
            qb[8 * v + 7] += u1.w;
        }
    }
}

template <typename T, int D, int KC>
__global__ __launch_bounds__(kTile) void select_kernel(Dims dm, const T* __restrict__ Q,
                                                       const float* __restrict__ Kbar,
                                                       int32_t* __restrict__ idx,
                                                       float* __restrict__ w, int ntiles) {
    const int lane = threadIdx.x;
    // latest tiles (most candidates) first
    const int nbg = dm.B * dm.G;
    const int tile = ntiles - 1 - (int)blockIdx.x / nbg;
    const int bg = (int)blockIdx.x % nbg, b = bg / dm.G, g = bg % dm.G;
    const int t0 = tile * kTile;
    const int t = t0 + lane;
    const bool valid = t < dm.L;
    const int ncand = valid ? t / dm.S : 0;
    const int nwave = (min(t0 + kTile, dm.L) - 1) / dm.S;     // candidates of the last token
    const int k = dm.k;

    float qb[D];
    if (valid) {
        group_query<D>(Q + (((size_t)b * dm.L + t) * dm.H + (size_t)g * dm.h) * D, dm.h, qb);
    } else {
#pragma unroll
        for (int e = 0; e < D; ++e) qb[e] = 0.f;
    }
    float ls[KC];
    int lc[KC];
#pragma unroll
    for (int j = 0; j < KC; ++j) {
        ls[j] = -INFINITY;
        lc[j] = -1;
    }

    const float* kb = Kbar + ((size_t)b * dm.C * dm.G + g) * D;   // row c at kb + c G D
    const size_t cstride = (size_t)dm.G * D;
    for (int c = 0; c < nwave; ++c) {
        const float* kr = kb + (size_t)c * cstride;              // same for every lane
        float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
        for (int e = 0; e < D; e += 4) {
            a0 = fmaf(qb[e], kr[e], a0);
            a1 = fmaf(qb[e + 1], kr[e + 1], a1);
            a2 = fmaf(qb[e + 2], kr[e + 2], a2);
            a3 = fmaf(qb[e + 3], kr[e + 3], a3);
        }
        float s = (c < ncand) ? dm.alpha * ((a0 + a1) + (a2 + a3)) : -INFINITY;
        if (__ballot(s > ls[KC - 1]) == 0) continue;
        int ci = c;
#pragma unroll
        for (int j = 0; j < KC; ++j) {          // insertion: strictly greater moves up
            const bool gt = s > ls[j];
            const float ts = gt ? s : ls[j];
            const int tc = gt ? ci : lc[j];
            s = gt ? ls[j] : s;
            ci = gt ? lc[j] : ci;
            ls[j] = ts;
            lc[j] = tc;
        }
    }
    if (!valid) return;

    // softmax over the k best, written in descending chunk order
    const int n = min(k, ncand);
    const size_t o = (((size_t)b * dm.L + t) * dm.G + g) * k;
    float ex[KC];
    float z = 0.f;
#pragma unroll
    for (int j = 0; j < KC; ++j) {
        ex[j] = (j < n) ? expf(ls[j] - ls[0]) : 0.f;
        z += ex[j];
    }
    const float iz = 1.f / z;
#pragma unroll
    for (int j = 0; j < KC; ++j) {
        if (j < n) {
            int rank = 0;
#pragma unroll
            for (int i = 0; i < KC; ++i) rank += (i < n && lc[i] > lc[j]) ? 1 : 0;
            idx[o + rank] = lc[j];
            w[o + rank] = ex[j] * iz;
        } else if (j < k) {
            idx[o + j] = -1;
            w[o + j] = 0.f;
        }
    }
}

template <typename T, int D>
hipError_t launch_d(const Dims& dm, const void* Q, const float* Kbar, int32_t* idx, float* w,
                    hipStream_t st) {
    const int ntiles = cdiv(dm.L, kTile);
    const dim3 grid(ntiles * dm.B * dm.G);
    HSA_TIMED("select_kernel", st);
    if (dm.k <= 8)
        hipLaunchKernelGGL((select_kernel<T, D, 8>), grid, dim3(kTile), 0, st, dm, (const T*)Q,
                           Kbar, idx, w, ntiles);
    else if (dm.k <= 16)
        hipLaunchKernelGGL((select_kernel<T, D, 16>), grid, dim3(kTile), 0, st, dm, (const T*)Q,
                           Kbar, idx, w, ntiles);
    else
        hipLaunchKernelGGL((select_kernel<T, D, 32>), grid, dim3(kTile), 0, st, dm, (const T*)Q,
                           Kbar, idx, w, ntiles);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_t(const Dims& dm, const void* Q, const float* Kbar, int32_t* idx, float* w,
                    hipStream_t st) {
    return dm.d == 128 ? launch_d<T, 128>(dm, Q, Kbar, idx, w, st)
                       : launch_d<T, 64>(dm, Q, Kbar, idx, w, st);
}

}  // namespace

hipError_t launch_select(const Dims& dm, bool in_bf16, const void* Q, const float* Kbar,
                         int32_t* idx, float* w, hipStream_t st) {
    if (dm.B == 0 || dm.L == 0) return hipSuccess;
    return in_bf16 ? launch_t<bf16>(dm, Q, Kbar, idx, w, st)
                   : launch_t<float>(dm, Q, Kbar, idx, w, st);
}

}  // namespace hsa
