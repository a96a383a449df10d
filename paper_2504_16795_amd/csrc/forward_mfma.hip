// bf16 MFMA forward of hierarchical sparse attention (Sec. 3.1.1), for h = 8 query heads
// per KV head, d = 128, S in {64, 128}.
//
// Workgroup = (b, g, tile of 2 NW tokens inside one query chunk), NW waves (16 for S = 64,
// 8 for S = 128); wave w owns tokens 2w, 2w+1 as one row block of 16 rows (2 tokens x 8
// heads).
//  1. Each token's valid selections are sorted by descending chunk; the tile's union is
//     marked in an LDS bitmap over the candidates and listed in descending chunk order, so
//     every lane follows its token's slot list with a register pointer.
//  2. Each union chunk is staged once in LDS (double-buffered): K row-major [S][d], V
//     transposed [d][S]; the next chunk's global loads are in flight meanwhile.
//  3. A wave whose tokens selected the chunk (wave-uniform test) runs
//        Z^T [S x 16] = K_c [S x d] . Q^T [d x 16]        (S/16 * 4 MFMAs)
//        P^T = softmax over keys, scaled by w_{t,c} (0 for the row block's other token)
//        O^T [d x 16] += V_c^T [d x S] . P^T [S x 16]     (8 * S/32 MFMAs)
//     The C layout of Z^T feeds P^T straight into the B operand of the second product with
//     a key permutation applied to the V^T reads.  Q^T lives in registers for the whole
//     kernel and O^T accumulates in registers (fp32), so each chunk is read from L2/HBM
//     once per tile instead of once per (token, slot), and no online softmax is needed.
#include <cstdlib>

#include "tile_sel.h"

namespace hsa {
namespace {

constexpr int D = 128;
constexpr int HG = 8;            // query heads per KV head
constexpr int KMAX = 32;
constexpr int KP = D + 8;        // padded K row (bf16 elements)
constexpr int UWORDS = 1024;     // union bitmap words: up to 32768 candidate chunks

// Waves per workgroup (a tile holds 2 NW tokens, 2 per wave) and the waves per SIMD the
// register budget is sized for.  At S = 64 the 32-token tile shares each staged chunk
// among more tokens; S = 128 needs the register room of 8 waves.
template <int S>
struct FCfg;
template <>
struct FCfg<64> {
    static constexpr int NW = 16, WPE = 4;
};
template <>
struct FCfg<128> {
    static constexpr int NW = 8, WPE = 2;
};

template <int S>
struct Smem {
    static constexpr int NW = FCfg<S>::NW, TQ = 2 * NW;
    static constexpr int VP = S + 8;              // padded V^T row (keys)
    __bf16 Ks[2][S * KP];                         // double-buffered chunk stage
    __bf16 Vt[2][D * VP];
    int32_t oidx[TQ * KMAX];                      // selection tables (see tile_sel.h)
    float ow[TQ * KMAX];
    int32_t sidx[TQ * KMAX];
    float sw[TQ * KMAX];
    int32_t ulist[TQ * KMAX];
    uint8_t sslot[TQ * KMAX];
    int wsum[NW];
};

// Staging of one chunk: K vectors (key v / 16, columns 8 (v % 16) .. +7) go row-major to
// LDS; V vector pairs (keys 2 (p / 16), 2 (p / 16) + 1, same columns) go transposed as
// packed key pairs.
template <int S>
struct Stage {
    static constexpr int kThreads = FCfg<S>::NW * 64;
    static constexpr int NK = S * D / 8 / kThreads;                      // K vectors / thread
    static constexpr int NV = (S * D / 16 + kThreads - 1) / kThreads;    // V pairs / thread
    u32x4_t k[NK];
    u32x4_t v[2 * NV];
};

template <int S>
__device__ __forceinline__ void load_chunk(Stage<S>& st, const __bf16* __restrict__ K,
                                           const __bf16* __restrict__ V, size_t base,
                                           size_t rowstride, int tid) {
#pragma unroll
    for (int i = 0; i < Stage<S>::NK; ++i) {
        const int v = tid + i * Stage<S>::kThreads;
        st.k[i] = *reinterpret_cast<const u32x4_t*>(K + base + (size_t)(v >> 4) * rowstride +
                                                    (v & 15) * 8);
    }
#pragma unroll
    for (int i = 0; i < Stage<S>::NV; ++i) {
        const int p = tid + i * Stage<S>::kThreads;
        if (p < S * 8) {
            const size_t o = base + (size_t)((p >> 4) * 2) * rowstride + (p & 15) * 8;
            st.v[2 * i] = *reinterpret_cast<const u32x4_t*>(V + o);
            st.v[2 * i + 1] = *reinterpret_cast<const u32x4_t*>(V + o + rowstride);
        }
    }
}

template <int S>
__device__ __forceinline__ void store_chunk(const Stage<S>& st, __bf16* Ks, __bf16* Vt,
                                            int tid) {
    constexpr int VP = S + 8;
#pragma unroll
    for (int i = 0; i < Stage<S>::NK; ++i) {
        const int v = tid + i * Stage<S>::kThreads;
        *reinterpret_cast<u32x4_t*>(&Ks[(v >> 4) * KP + (v & 15) * 8]) = st.k[i];
    }
#pragma unroll
    for (int i = 0; i < Stage<S>::NV; ++i) {
        const int p = tid + i * Stage<S>::kThreads;
        if (p < S * 8) {
            const int r = (p >> 4) * 2, col = (p & 15) * 8;
            const u32x4_t a = st.v[2 * i], c2 = st.v[2 * i + 1];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int d0 = col + 2 * j, d1 = d0 + 1;
                *reinterpret_cast<uint32_t*>(&Vt[d0 * VP + tpos(d0, r, S)]) =
                    (a[j] & 0xFFFFu) | (c2[j] << 16);
                *reinterpret_cast<uint32_t*>(&Vt[d1 * VP + tpos(d1, r, S)]) =
                    (a[j] >> 16) | (c2[j] & 0xFFFF0000u);
            }
        }
    }
}

template <int S>
__global__ __launch_bounds__(FCfg<S>::NW * 64, FCfg<S>::WPE) void forward_mfma(
    Dims dm, const __bf16* __restrict__ Q, const __bf16* __restrict__ K,
    const __bf16* __restrict__ V, const int32_t* __restrict__ idx, const float* __restrict__ w,
    __bf16* __restrict__ O, int ntiles) {
    constexpr int VP = Smem<S>::VP;
    constexpr int NW = Smem<S>::NW, TQ = Smem<S>::TQ, kThreads = NW * 64;
    constexpr int MB = S / 16;            // key blocks of Z^T
    constexpr int KS2 = S / 32;           // key steps of P V
    __shared__ Smem<S> sm;

    const int lid = xcd_logical_id(ntiles * dm.B * dm.G);
    if (lid < 0) return;
    const int tile = lid % ntiles, bg = lid / ntiles;
    const int b = bg / dm.G, g = bg % dm.G;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int k = dm.k;
    const int t0 = tile * TQ;
    const int ncand = t0 / S;
    const int row = lane & 15, grp = lane >> 4;

    // ---- Q^T operand of the wave's row block (registers, whole kernel) -------------------
    const int tau = wave * 2 + (row >> 3);
    const int t_row = t0 + tau;
    bf16x8_t qB[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
        if (t_row < dm.L) {
            const size_t qo = (((size_t)b * dm.L + t_row) * dm.H + (size_t)g * HG + (row & 7)) * D +
                              32 * ks + 8 * grp;
            qB[ks] = ld_bf16x8(Q + qo);
        } else {
            qB[ks] = bf16x8_t{};
        }
    }
    // ---- selections of the tile, sorted per token, and their union ----------------------
    // (the union bitmap lives in stage 1, which is first written after the union is listed)
    static_assert(sizeof(sm.Ks[1]) >= UWORDS * 4, "bitmap does not fit the stage");
    const TileSel ts{sm.oidx, sm.ow, sm.sidx, sm.sslot, sm.sw,
                     reinterpret_cast<uint32_t*>(sm.Ks[1]), sm.ulist, sm.wsum};
    const int nu = tile_selection<kThreads, TQ>(
        ts, idx, w, (((size_t)b * dm.L + t0) * dm.G + g) * k, (size_t)dm.G * k, k,
        min(TQ, dm.L - t0), ncand);
    wait_global_loads();
    f32x4_t acc[8];
#pragma unroll
    for (int db = 0; db < 8; ++db) acc[db] = zero4();
    // this lane's token: next selected chunk and its weight
    int sp = 0;
    int cur_c = sm.sidx[tau * k];
    float cur_w = sm.sw[tau * k];

    const size_t rowstride = (size_t)dm.G * D;
    const size_t bgbase = (size_t)b * dm.L * rowstride + (size_t)g * D;
    Stage<S> st;
    // Pipeline: chunk u is computed from stage u % 2 while chunk u + 1 (already in registers)
    // is written to the other stage and chunk u + 2 is being fetched; one barrier per chunk.
    if (nu > 0) {
        load_chunk<S>(st, K, V, bgbase + (size_t)sm.ulist[0] * S * rowstride, rowstride, tid);
        store_chunk<S>(st, sm.Ks[0], sm.Vt[0], tid);
    }
    if (nu > 1)
        load_chunk<S>(st, K, V, bgbase + (size_t)sm.ulist[1] * S * rowstride, rowstride, tid);
    __syncthreads();
    const float sl2 = dm.beta * 1.44269504088896341f;   // beta * log2(e)
    for (int u = 0; u < nu; ++u) {
        const int c = sm.ulist[u];
        const bool mine = (cur_c == c);
        if (__ballot(mine) != 0) {
            const __bf16* Ks = sm.Ks[u & 1];
            const __bf16* Vt = sm.Vt[u & 1];
            const float wl = mine ? cur_w : 0.f;
            // Z^T = K_c Q^T
            f32x4_t z[MB];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) z[mb] = zero4();
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) {
                    const bf16x8_t a = ld_bf16x8(&Ks[(16 * mb + row) * KP + 32 * ks + 8 * grp]);
                    z[mb] = mfma16(a, qB[ks], z[mb]);
                }
            // softmax over the S keys of each row (column `row` of Z^T)
            float m = -INFINITY;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int i = 0; i < 4; ++i) m = fmaxf(m, z[mb][i]);
            m = col_max(m);
            float ssum = 0.f;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    z[mb][i] = fast_exp2((z[mb][i] - m) * sl2);
                    ssum += z[mb][i];
                }
            ssum = col_sum(ssum);
            const float scale = wl / ssum;
            // O^T += V^T P^T
#pragma unroll
            for (int ks2 = 0; ks2 < KS2; ++ks2) {
                const bf16x8_t pb = pack8(z[2 * ks2], z[2 * ks2 + 1], scale);
#pragma unroll
                for (int db = 0; db < 8; ++db) {
                    const int d = 16 * db + row;
                    const __bf16* vr = &Vt[d * VP];
                    const bf16x8_t a = cat(ld_bf16x4(vr + tpos(d, 32 * ks2 + 4 * grp, S)),
                                           ld_bf16x4(vr + tpos(d, 32 * ks2 + 16 + 4 * grp, S)));
                    acc[db] = mfma16(a, pb, acc[db]);
                }
            }
            if (mine) {
                ++sp;
                cur_c = sp < k ? sm.sidx[tau * k + sp] : -1;
                cur_w = sp < k ? sm.sw[tau * k + sp] : 0.f;
            }
        }
        if (u + 1 < nu) store_chunk<S>(st, sm.Ks[(u + 1) & 1], sm.Vt[(u + 1) & 1], tid);
        __syncthreads();
        if (u + 2 < nu)
            load_chunk<S>(st, K, V, bgbase + (size_t)sm.ulist[u + 2] * S * rowstride, rowstride,
                          tid);
    }

    // ---- output: O^T C layout -> O[b, t, g*8 + j, d] ----------------------------------
    if (t_row < dm.L) {
        __bf16* op = O + (((size_t)b * dm.L + t_row) * dm.H + (size_t)g * HG + (row & 7)) * D;
#pragma unroll
        for (int db = 0; db < 8; ++db) {
            const bf16x4_t o4{f2bf(acc[db][0]), f2bf(acc[db][1]), f2bf(acc[db][2]),
                              f2bf(acc[db][3])};
            *reinterpret_cast<bf16x4_t*>(op + 16 * db + 4 * grp) = o4;
        }
    }
}

}  // namespace

bool forward_mfma_supported(const Dims& dm, bool in_bf16) {
    return in_bf16 && dm.h == HG && dm.d == D && (dm.S == 64 || dm.S == 128) && dm.k <= KMAX &&
           dm.C <= UWORDS * 32 && !getenv("HSA_FORCE_GENERIC");
}

hipError_t launch_forward_mfma(const Dims& dm, const void* Q, const void* K, const void* V,
                               const int32_t* idx, const float* w, void* O, void*,
                               hipStream_t st) {
    if (dm.S == 64) {
        constexpr int NW = FCfg<64>::NW;
        const int ntiles = cdiv(dm.L, 2 * NW);
        const int grid = 8 * cdiv(ntiles * dm.B * dm.G, 8);
        HSA_TIMED("forward_mfma", st);
        hipLaunchKernelGGL((forward_mfma<64>), dim3(grid), dim3(NW * 64), 0, st, dm,
                           (const __bf16*)Q, (const __bf16*)K, (const __bf16*)V, idx, w,
                           (__bf16*)O, ntiles);
    } else {
        constexpr int NW = FCfg<128>::NW;
        const int ntiles = cdiv(dm.L, 2 * NW);
        const int grid = 8 * cdiv(ntiles * dm.B * dm.G, 8);
        HSA_TIMED("forward_mfma", st);
        hipLaunchKernelGGL((forward_mfma<128>), dim3(grid), dim3(NW * 64), 0, st, dm,
                           (const __bf16*)Q, (const __bf16*)K, (const __bf16*)V, idx, w,
                           (__bf16*)O, ntiles);
    }
    return hipGetLastError();
}

}  // namespace hsa
