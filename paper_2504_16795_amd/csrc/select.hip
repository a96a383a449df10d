// Chunk selection + chunk weights (Sec. 3.1 chunk-selection equation; softmax weights).
//
// Workgroup = (b, g, tile of TQ <= 64 tokens inside one query chunk): all tokens of a
// tile share the candidate set c < floor(t0 / S).  The tile's group queries
// q~ = sum_j q_j are kept in LDS (fp32); landmarks stream through LDS in blocks of 64;
// a 4x4 register tile per thread computes 64x64 fp32 scores per block.  Each wave then
// merges the 64 new scores of its tokens into a running top-k list with a wave-wide
// partial sort: only lanes above the current k-th score (ballot) are inserted, each
// insertion is a ballot-rank plus a one-lane shift of the sorted list.  Candidates arrive
// in increasing chunk order, so "ties to the lower index" is "strictly greater wins".
// The final list gets softmax weights and is written in descending chunk order.
#include "common.h"

namespace hsa {
namespace {

constexpr int kThreads = 256;
constexpr int TQ = 64;      // tokens per tile (max)
constexpr int NB = 64;      // landmarks per block
constexpr int KMAX = 32;

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void select_kernel(Dims dm, const T* __restrict__ Q,
                                                          const float* __restrict__ Kbar,
                                                          int32_t* __restrict__ idx,
                                                          float* __restrict__ w, int tq) {
    constexpr int DP = D + 1;
    __shared__ float qs[TQ * DP];
    __shared__ float kb[NB * DP];
    __shared__ float sc[TQ * (NB + 1)];
    __shared__ float lst_s[TQ * KMAX];
    __shared__ int lst_c[TQ * KMAX];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bg = blockIdx.y, b = bg / dm.G, g = bg % dm.G;
    const int t0 = blockIdx.x * tq;
    const int ntok = min(tq, dm.L - t0);
    const int ncand = t0 / dm.S;
    const int k = dm.k, h = dm.h;

    // group queries of the tile
    for (int i = tid; i < TQ * D; i += kThreads) {
        const int tau = i / D, e = i % D;
        float s = 0.f;
        if (tau < ntok) {
            const T* qp = Q + (((size_t)b * dm.L + t0 + tau) * dm.H + (size_t)g * h) * D + e;
            for (int j = 0; j < h; ++j) s += to_f32(qp[(size_t)j * D]);
        }
        qs[tau * DP + e] = s;
    }
    for (int i = tid; i < TQ * KMAX; i += kThreads) {
        lst_s[i] = -INFINITY;
        lst_c[i] = 0x7FFFFFFF;
    }
    int count = 0;   // entries in every running list of this tile (identical for all tokens)

    const int ty = tid >> 4, tx = tid & 15;
    for (int cb = 0; cb < ncand; cb += NB) {
        const int nb = min(NB, ncand - cb);
        __syncthreads();
        for (int i = tid; i < nb * D; i += kThreads) {
            const int cl = i / D, e = i % D;
            kb[cl * DP + e] = Kbar[(((size_t)b * dm.C + cb + cl) * dm.G + g) * D + e];
        }
        __syncthreads();
        float acc[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int m = 0; m < 4; ++m) acc[i][m] = 0.f;
        for (int e = 0; e < D; ++e) {
            float qv[4], kv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) qv[i] = qs[(ty * 4 + i) * DP + e];
#pragma unroll
            for (int m = 0; m < 4; ++m) kv[m] = kb[(tx + 16 * m) * DP + e];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int m = 0; m < 4; ++m) acc[i][m] = fmaf(qv[i], kv[m], acc[i][m]);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int cl = tx + 16 * m;
                sc[(ty * 4 + i) * (NB + 1) + cl] = (cl < nb) ? dm.alpha * acc[i][m] : -INFINITY;
            }
        __syncthreads();

        // merge: wave `wave` owns tokens [wave*16, wave*16+16)
        for (int tt = 0; tt < 16; ++tt) {
            const int tau = wave * 16 + tt;
            if (tau >= ntok) break;
            const float s = sc[tau * (NB + 1) + lane];   // -inf for lanes >= nb
            float ls = (lane < k) ? lst_s[tau * KMAX + lane] : -INFINITY;
            int lc = (lane < k) ? lst_c[tau * KMAX + lane] : 0x7FFFFFFF;
            int cnt = count;
            float thr = (cnt == k) ? __shfl(ls, k - 1, 64) : -INFINITY;
            uint64_t mask = __ballot(s > thr);
            while (mask) {
                const int src = __ffsll((unsigned long long)mask) - 1;
                const float sn = __shfl(s, src, 64);
                const int cn = cb + src;
                const bool ahead = (lane < k) && (ls > sn || (ls == sn && lc < cn));
                const int pos = __popcll(__ballot(ahead));
                const float ls_up = __shfl_up(ls, 1, 64);
                const int lc_up = __shfl_up(lc, 1, 64);
                if (lane < k) {
                    if (lane > pos) {
                        ls = ls_up;
                        lc = lc_up;
                    } else if (lane == pos) {
                        ls = sn;
                        lc = cn;
                    }
                }
                cnt = min(cnt + 1, k);
                thr = (cnt == k) ? __shfl(ls, k - 1, 64) : -INFINITY;
                mask &= ~(1ull << src);
                mask &= __ballot(s > thr);
            }
            if (lane < k) {
                lst_s[tau * KMAX + lane] = ls;
                lst_c[tau * KMAX + lane] = lc;
            }
        }
        count = min(count + nb, k);
    }
    __syncthreads();

    // finalize: softmax weights, descending chunk order, padding
    const int n = min(k, ncand);
    for (int tt = 0; tt < 16; ++tt) {
        const int tau = wave * 16 + tt;
        if (tau >= ntok) break;
        const int t = t0 + tau;
        const float ls = (lane < n) ? lst_s[tau * KMAX + lane] : -INFINITY;
        const int lc = (lane < n) ? lst_c[tau * KMAX + lane] : -1;
        const float m = __shfl(ls, 0, 64);
        const float ex = (lane < n) ? expf(ls - m) : 0.f;
        const float z = wave_sum(ex);
        int rank = 0;
        for (int j = 0; j < n; ++j) rank += (__shfl(lc, j, 64) > lc) ? 1 : 0;
        const size_t o = (((size_t)b * dm.L + t) * dm.G + g) * k;
        if (lane < n) {
            idx[o + rank] = lc;
            w[o + rank] = ex / z;
        } else if (lane < k) {
            idx[o + lane] = -1;
            w[o + lane] = 0.f;
        }
    }
}

template <typename T>
hipError_t launch_t(const Dims& dm, const void* Q, const float* Kbar, int32_t* idx, float* w,
                    hipStream_t st) {
    const int tq = dm.S < TQ ? dm.S : TQ;
    dim3 grid(cdiv(dm.L, tq), dm.B * dm.G);
    if (dm.d == 128) {
        HSA_TIMED("select_kernel", st);
        hipLaunchKernelGGL((select_kernel<T, 128>), grid, dim3(kThreads), 0, st, dm,
                           (const T*)Q, Kbar, idx, w, tq);
    } else {
        HSA_TIMED("select_kernel", st);
        hipLaunchKernelGGL((select_kernel<T, 64>), grid, dim3(kThreads), 0, st, dm,
                           (const T*)Q, Kbar, idx, w, tq);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_select(const Dims& dm, bool in_bf16, const void* Q, const float* Kbar,
                         int32_t* idx, float* w, hipStream_t st) {
    if (dm.B == 0 || dm.L == 0) return hipSuccess;
    return in_bf16 ? launch_t<bf16>(dm, Q, Kbar, idx, w, st)
                   : launch_t<float>(dm, Q, Kbar, idx, w, st);
}

}  // namespace hsa
