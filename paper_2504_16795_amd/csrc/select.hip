// Chunk selection + chunk weights (Sec. 3.1: the top-k chunks by the landmark score
// s_c = alpha * (sum_j q_j) . Kbar_c over the chunks before the token's own, and their
// softmax or stick-breaking weights).
//
// Lane = token; each lane keeps its group query q~ = sum_j q_j (fp32, d registers) and a
// running top-KC list (scores and chunk indices, registers, descending).  The landmark rows
// of the candidates are copied into LDS (direct copies, the next block in flight) and read
// with broadcast LDS loads, in increasing chunk order.  Two schedules of the 4 waves of a
// workgroup:
//   - few candidates (short sequences): the waves hold 4 consecutive 64-token tiles and
//     share blocks of 64 landmark rows;
//   - many candidates: the waves hold the same tile and split its candidates (wave w takes
//     the 16-row blocks w, w + 4, ...); the four lists are merged at the end.
// A candidate enters a list only when its score is strictly greater than the list's last
// entry and moves up past every entry it beats strictly: on equal scores the lower chunk
// index stays first (the merge compares (score, chunk) the same way).  The k best get
// softmax weights and are written in descending chunk order, padded with -1 / 0.
#include "common.h"

namespace hsa {
namespace {

constexpr int kTile = 64;     // tokens per wave
constexpr int NW = 4;         // waves per workgroup, all on the same 64 tokens
constexpr int kThreads = NW * kTile;
constexpr int NB = 16;        // candidate rows per LDS block
constexpr int NST = 2;        // LDS blocks per wave
constexpr int TNB = 64;       // candidate rows per LDS block when the 4 waves share blocks
constexpr int kSplitFrom = 256;   // more complete chunks than this: split the candidates

// One global_load_lds_dwordx4 (lane l copies 16 bytes to lds_base + 16 l; lds_base
// wave-uniform in M0), as inline assembly so that the compiler's waits do not make the
// LDS reads wait for copies of the other block.  Completion is awaited with vmcnt(0);
// no compiler-visible global load is in flight across the copies.
__device__ __forceinline__ void sel_copy16(const void* gsrc, uint32_t lds_base) {
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(gsrc), "{m0}"(lds_base)
                 : "memory");
}
__device__ __forceinline__ uint32_t sel_lds_address(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
__device__ __forceinline__ void sel_wait_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }
__device__ __forceinline__ void wait_global_loads_sel() { __builtin_amdgcn_s_waitcnt(0x0F70); }
__device__ __forceinline__ void sel_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

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
__global__ __launch_bounds__(kThreads) void select_tiles_kernel(Dims dm, const T* __restrict__ Q,
                                                          const float* __restrict__ Kbar,
                                                          int32_t* __restrict__ idx,
                                                          float* __restrict__ w, int ngroups) {
    __shared__ float kb_s[NST][TNB * D];        // landmark rows of the staged candidate blocks
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // latest token groups (most candidates) first
    const int nbg = dm.B * dm.G;
    const int grp = ngroups - 1 - (int)blockIdx.x / nbg;
    const int bg = (int)blockIdx.x % nbg, b = bg / dm.G, g = bg % dm.G;
    const int t0 = grp * kThreads + wave * kTile;        // this wave's 64 tokens
    const int t = t0 + lane;
    const bool valid = t < dm.L;
    const int ncand = valid ? t / dm.S : 0;
    const int nwave = t0 < dm.L ? (min(t0 + kTile, dm.L) - 1) / dm.S : 0;
    const int tlast = min(grp * kThreads + kThreads, dm.L) - 1;
    const int nwg = (tlast >= grp * kThreads) ? tlast / dm.S : 0;   // candidates of the group
    const int k = dm.k;

    float qb[D];
    if (valid) {
        group_query<D>(Q + (((size_t)b * dm.L + t) * dm.H + (size_t)g * dm.h) * D, dm.h, qb);
    } else {
#pragma unroll
        for (int e = 0; e < D; ++e) qb[e] = 0.f;
    }
    wait_global_loads_sel();
    float ls[KC];
    int lc[KC];
#pragma unroll
    for (int j = 0; j < KC; ++j) {
        ls[j] = -INFINITY;
        lc[j] = -1;
    }

    // candidate blocks of TNB rows (row c of group g: D fp32 at Kbar + ((b C + c) G + g) D),
    // copied into LDS by the NW waves: 2 rows per 1 KB copy instruction
    const float* kb = Kbar + ((size_t)b * dm.C * dm.G + g) * D;
    const size_t cstride = (size_t)dm.G * D;
    const int nblk = cdiv(nwg, TNB);
    auto issue = [&](int blk) __attribute__((always_inline)) {
        float* dst = kb_s[blk % NST];
        constexpr int RPI = 1024 / (D * 4);                // rows per copy instruction
#pragma unroll
        for (int i = 0; i < TNB / RPI / NW; ++i) {
            const int ci = (wave + i * NW);                // copy instruction of the block
            const int r = ci * RPI + lane / (64 / RPI);    // row within the block
            const int c = min(blk * TNB + r, nwg - 1);      // past the end: repeat a valid row
            sel_copy16(kb + (size_t)c * cstride + (lane % (64 / RPI)) * 4,
                       __builtin_amdgcn_readfirstlane(sel_lds_address(dst + ci * 256)));
        }
    };
    if (nblk > 0) issue(0);
    for (int blk = 0; blk < nblk; ++blk) {
        sel_wait_all();
        sel_barrier();                                     // block landed; other stage free
        if (blk + 1 < nblk) issue(blk + 1);
        const float* rows = kb_s[blk % NST];
        const int cend = min(nwave, blk * TNB + TNB);
        for (int c = blk * TNB; c < cend; ++c) {
            const float4* kr = reinterpret_cast<const float4*>(rows + (c - blk * TNB) * D);
            float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
            for (int e = 0; e < D / 4; ++e) {
                const float4 kv = kr[e];
                a0 = fmaf(qb[4 * e], kv.x, a0);
                a1 = fmaf(qb[4 * e + 1], kv.y, a1);
                a2 = fmaf(qb[4 * e + 2], kv.z, a2);
                a3 = fmaf(qb[4 * e + 3], kv.w, a3);
            }
            float s = (c < ncand) ? dm.alpha * ((a0 + a1) + (a2 + a3)) : -INFINITY;
            if (__ballot(s > ls[KC - 1]) == 0) continue;
            int ci = c;
#pragma unroll
            for (int j = 0; j < KC; ++j) {      // insertion: strictly greater moves up
                const bool gt = s > ls[j];
                const float ts = gt ? s : ls[j];
                const int tc = gt ? ci : lc[j];
                s = gt ? ls[j] : s;
                ci = gt ? lc[j] : ci;
                ls[j] = ts;
                lc[j] = tc;
            }
        }
    }
    if (!valid) return;

    // weights of the k best, written in descending chunk order
    const int n = min(k, ncand);
    const size_t o = (((size_t)b * dm.L + t) * dm.G + g) * k;
    float wt[KC];
    int rank[KC];
    list_weights<KC>(ls, lc, n, dm.stick != 0, wt, rank);
#pragma unroll
    for (int j = 0; j < KC; ++j) {
        if (j < n) {
            idx[o + rank[j]] = lc[j];
            w[o + rank[j]] = wt[j];
        } else if (j < k) {
            idx[o + j] = -1;
            w[o + j] = 0.f;
        }
    }
}

template <typename T, int D, int KC>
__global__ __launch_bounds__(kThreads) void select_split_kernel(Dims dm, const T* __restrict__ Q,
                                                          const float* __restrict__ Kbar,
                                                          int32_t* __restrict__ idx,
                                                          float* __restrict__ w, int ntiles) {
    // per wave: NST blocks of NB landmark rows; reused for the list merge at the end
    constexpr int KBF = NW * NST * NB * D, MERGEF = 2 * NW * KC * 64;
    __shared__ float lds_f[KBF > MERGEF ? KBF : MERGEF];
    auto kb_s = reinterpret_cast<float (*)[NST][NB * D]>(lds_f);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // latest tiles (most candidates) first
    const int nbg = dm.B * dm.G;
    const int tile = ntiles - 1 - (int)blockIdx.x / nbg;
    const int bg = (int)blockIdx.x % nbg, b = bg / dm.G, g = bg % dm.G;
    const int t0 = tile * kTile;
    const int t = t0 + lane;
    const bool valid = t < dm.L;
    const int ncand = valid ? t / dm.S : 0;
    const int ntile = (min(t0 + kTile, dm.L) - 1) / dm.S;   // candidates of the last token
    const int k = dm.k;

    float qb[D];
    if (valid) {
        group_query<D>(Q + (((size_t)b * dm.L + t) * dm.H + (size_t)g * dm.h) * D, dm.h, qb);
    } else {
#pragma unroll
        for (int e = 0; e < D; ++e) qb[e] = 0.f;
    }
    wait_global_loads_sel();
    float ls[KC];
    int lc[KC];
#pragma unroll
    for (int j = 0; j < KC; ++j) {
        ls[j] = -INFINITY;
        lc[j] = -1;
    }

    // wave w takes the candidate blocks w, w + NW, ... (NB rows each; row c of group g is
    // D fp32 at Kbar + ((b C + c) G + g) D), copied into its own LDS blocks
    const float* kb = Kbar + ((size_t)b * dm.C * dm.G + g) * D;
    const size_t cstride = (size_t)dm.G * D;
    const int nblk = cdiv(ntile, NB);
    auto issue = [&](int blk) __attribute__((always_inline)) {
        float* dst = kb_s[wave][(blk / NW) % NST];
        constexpr int RPI = 1024 / (D * 4);                // rows per copy instruction
#pragma unroll
        for (int ci = 0; ci < NB / RPI; ++ci) {
            const int r = ci * RPI + lane / (64 / RPI);
            const int c = min(blk * NB + r, ntile - 1);   // past the end: repeat a valid row
            sel_copy16(kb + (size_t)c * cstride + (lane % (64 / RPI)) * 4,
                       __builtin_amdgcn_readfirstlane(sel_lds_address(dst + ci * 256)));
        }
    };
    if (wave < nblk) issue(wave);
    for (int blk = wave; blk < nblk; blk += NW) {
        sel_wait_all();                                    // this wave's block has landed
        if (blk + NW < nblk) issue(blk + NW);
        const float* rows = kb_s[wave][(blk / NW) % NST];
        const int cend = min(ntile, blk * NB + NB);
        for (int c = blk * NB; c < cend; ++c) {
            const float4* kr = reinterpret_cast<const float4*>(rows + (c - blk * NB) * D);
            float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
            for (int e = 0; e < D / 4; ++e) {
                const float4 kv = kr[e];
                a0 = fmaf(qb[4 * e], kv.x, a0);
                a1 = fmaf(qb[4 * e + 1], kv.y, a1);
                a2 = fmaf(qb[4 * e + 2], kv.z, a2);
                a3 = fmaf(qb[4 * e + 3], kv.w, a3);
            }
            float s = (c < ncand) ? dm.alpha * ((a0 + a1) + (a2 + a3)) : -INFINITY;
            if (__ballot(s > ls[KC - 1]) == 0) continue;
            int ci = c;
#pragma unroll
            for (int j = 0; j < KC; ++j) {      // insertion: strictly greater moves up
                const bool gt = s > ls[j];
                const float ts = gt ? s : ls[j];
                const int tc = gt ? ci : lc[j];
                s = gt ? ls[j] : s;
                ci = gt ? lc[j] : ci;
                ls[j] = ts;
                lc[j] = tc;
            }
        }
    }
    // merge the waves' lists into wave 0's: each list is ordered by (score desc, chunk asc);
    // the merge compares the same way, so ties keep the lower chunk first
    __syncthreads();
    float* ms = lds_f;                                      // [NW][KC][64] scores, then chunks
    int* mc = reinterpret_cast<int*>(ms + NW * KC * 64);
    if (wave > 0) {
#pragma unroll
        for (int j = 0; j < KC; ++j) {
            ms[(wave * KC + j) * 64 + lane] = ls[j];
            mc[(wave * KC + j) * 64 + lane] = lc[j];
        }
    }
    __syncthreads();
    if (wave != 0 || !valid) return;
    for (int ow = 1; ow < NW; ++ow) {
        for (int jj = 0; jj < KC; ++jj) {
            float s = ms[(ow * KC + jj) * 64 + lane];
            int ci = mc[(ow * KC + jj) * 64 + lane];
            if (__ballot(s > ls[KC - 1] || (s == ls[KC - 1] && ci < lc[KC - 1] && s > -INFINITY)) == 0)
                break;                                     // the rest of this list is no better
#pragma unroll
            for (int j = 0; j < KC; ++j) {
                const bool gt = s > ls[j] || (s == ls[j] && ci < lc[j] && s > -INFINITY);
                const float ts = gt ? s : ls[j];
                const int tc = gt ? ci : lc[j];
                s = gt ? ls[j] : s;
                ci = gt ? lc[j] : ci;
                ls[j] = ts;
                lc[j] = tc;
            }
        }
    }

    // weights of the k best, written in descending chunk order
    const int n = min(k, ncand);
    const size_t o = (((size_t)b * dm.L + t) * dm.G + g) * k;
    float wt[KC];
    int rank[KC];
    list_weights<KC>(ls, lc, n, dm.stick != 0, wt, rank);
#pragma unroll
    for (int j = 0; j < KC; ++j) {
        if (j < n) {
            idx[o + rank[j]] = lc[j];
            w[o + rank[j]] = wt[j];
        } else if (j < k) {
            idx[o + j] = -1;
            w[o + j] = 0.f;
        }
    }
}

template <typename T, int D, int KC>
void launch_kc(const Dims& dm, const void* Q, const float* Kbar, int32_t* idx, float* w,
               hipStream_t st) {
    if (dm.C <= kSplitFrom) {
        // few candidates: four consecutive tiles share each landmark block
        const int ngroups = cdiv(dm.L, kThreads);
        hipLaunchKernelGGL((select_tiles_kernel<T, D, KC>), dim3(ngroups * dm.B * dm.G),
                           dim3(kThreads), 0, st, dm, (const T*)Q, Kbar, idx, w, ngroups);
    } else {
        // many candidates: the four waves of a tile split them
        const int ntiles = cdiv(dm.L, kTile);
        hipLaunchKernelGGL((select_split_kernel<T, D, KC>), dim3(ntiles * dm.B * dm.G),
                           dim3(kThreads), 0, st, dm, (const T*)Q, Kbar, idx, w, ntiles);
    }
}

template <typename T, int D>
hipError_t launch_d(const Dims& dm, const void* Q, const float* Kbar, int32_t* idx, float* w,
                    hipStream_t st) {
    HSA_TIMED("select_kernel", st);
    if (dm.k <= 8) launch_kc<T, D, 8>(dm, Q, Kbar, idx, w, st);
    else if (dm.k <= 16) launch_kc<T, D, 16>(dm, Q, Kbar, idx, w, st);
    else launch_kc<T, D, 32>(dm, Q, Kbar, idx, w, st);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_t(const Dims& dm, const void* Q, const float* Kbar, int32_t* idx, float* w,
                    hipStream_t st) {
    return dm.d == 128 ? launch_d<T, 128>(dm, Q, Kbar, idx, w, st)
                       : launch_d<T, 64>(dm, Q, Kbar, idx, w, st);
}

}  // namespace

bool select_mfma_supported(const Dims& dm, bool in_bf16);
hipError_t launch_select_mfma(const Dims& dm, const void* Q, const float* Kbar, int32_t* idx,
                              float* w, hipStream_t st);

hipError_t launch_select(const Dims& dm, bool in_bf16, const void* Q, const float* Kbar,
                         int32_t* idx, float* w, hipStream_t st) {
    if (dm.B == 0 || dm.L == 0) return hipSuccess;
    if (select_mfma_supported(dm, in_bf16)) return launch_select_mfma(dm, Q, Kbar, idx, w, st);
    return in_bf16 ? launch_t<bf16>(dm, Q, Kbar, idx, w, st)
                   : launch_t<float>(dm, Q, Kbar, idx, w, st);
}

}  // namespace hsa
