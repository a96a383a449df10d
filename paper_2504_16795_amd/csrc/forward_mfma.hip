// bf16 MFMA forward of hierarchical sparse attention (Sec. 3.1.1), for h = 8 query heads
// per KV head, d = 128, S in {64, 128}.
//
// Workgroup = (b, g, tile of 32 tokens inside one query chunk), 8 waves; wave w owns tokens
// 4w..4w+3 as two row blocks of 16 rows (2 tokens x 8 heads).
//  1. The tile's selections are deduplicated into a union list of chunks.
//  2. Each union chunk is staged once in LDS: K row-major [S][d], V transposed [d][S]
//     (the next chunk's global loads are in flight while the current one is computed).
//  3. Per row block whose tokens selected the chunk (a wave-uniform test), the wave runs
//        Z^T [S x 16] = K_c [S x d] . Q^T [d x 16]        (S/16 * 4 MFMAs)
//        P^T = softmax over keys, scaled by w_{t,c} (0 for rows that did not select c)
//        O^T [d x 16] += V_c^T [d x S] . P^T [S x 16]     (8 * S/32 MFMAs)
//     The C layout of Z^T feeds P^T straight into the B operand of the second product with
//     a key permutation applied to the V^T reads.  Q^T lives in registers for the whole
//     kernel and O^T accumulates in registers (fp32), so each chunk is read from L2/HBM
//     once per tile instead of once per (token, slot), and no online softmax is needed.
#include <cstdlib>

#include "mfma_common.h"

namespace hsa {
namespace {

constexpr int D = 128;
constexpr int HG = 8;            // query heads per KV head
constexpr int NW = 8;            // waves per workgroup
constexpr int kThreads = NW * 64;
constexpr int TQ = 32;           // tokens per tile
constexpr int KMAX = 32;
constexpr int KP = D + 8;        // padded K row (bf16 elements)

template <int S>
struct Smem {
    static constexpr int VP = S + 8;                  // padded V^T row (keys)
    __bf16 Ks[2][S * KP];             // double-buffered chunk stage
    __bf16 Vt[2][D * VP];
    int32_t sidx[TQ * KMAX];
    float sw[TQ * KMAX];
    int32_t ulist[TQ * KMAX];
    uint8_t flag[TQ * KMAX];
    int nu;
};

// Staging of one chunk: global -> registers (load_chunk) and registers -> LDS (store_chunk).
// K: vector v (16 bytes) = key v / 16, columns 8 (v % 16) .. +7, stored row-major.
// V: vector pair p = keys 2 (p / 16) and 2 (p / 16) + 1, columns 8 (p % 16) .. +7, stored
//    transposed as 8 packed key pairs.
template <int S>
__device__ __forceinline__ void load_chunk(u32x4_t (&kreg)[S * D / 8 / kThreads],
                                           u32x4_t (&vreg)[S * D / 8 / kThreads],
                                           const __bf16* __restrict__ K,
                                           const __bf16* __restrict__ V, size_t base,
                                           size_t rowstride, int tid) {
    constexpr int NPF = S * D / 8 / kThreads;
#pragma unroll
    for (int i = 0; i < NPF; ++i) {
        const int v = tid + i * kThreads;
        const int r = v >> 4, col = (v & 15) * 8;
        kreg[i] = *reinterpret_cast<const u32x4_t*>(K + base + (size_t)r * rowstride + col);
    }
#pragma unroll
    for (int i = 0; i < NPF / 2; ++i) {
        const int p = tid + i * kThreads;
        const int r = (p >> 4) * 2, col = (p & 15) * 8;
        vreg[2 * i] = *reinterpret_cast<const u32x4_t*>(V + base + (size_t)r * rowstride + col);
        vreg[2 * i + 1] =
            *reinterpret_cast<const u32x4_t*>(V + base + (size_t)(r + 1) * rowstride + col);
    }
}

template <int S>
__device__ __forceinline__ void store_chunk(const u32x4_t (&kreg)[S * D / 8 / kThreads],
                                            const u32x4_t (&vreg)[S * D / 8 / kThreads],
                                            __bf16* Ks, __bf16* Vt, int tid) {
    constexpr int NPF = S * D / 8 / kThreads;
    constexpr int VP = S + 8;
#pragma unroll
    for (int i = 0; i < NPF; ++i) {
        const int v = tid + i * kThreads;
        const int r = v >> 4, col = (v & 15) * 8;
        *reinterpret_cast<u32x4_t*>(&Ks[r * KP + col]) = kreg[i];
    }
#pragma unroll
    for (int i = 0; i < NPF / 2; ++i) {
        const int p = tid + i * kThreads;
        const int r = (p >> 4) * 2, col = (p & 15) * 8;
        const u32x4_t a = vreg[2 * i], c2 = vreg[2 * i + 1];
        // column col + 2j from the low halves, col + 2j + 1 from the high halves
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

template <int S>
__global__ __launch_bounds__(kThreads, 1) void forward_mfma(
    Dims dm, const __bf16* __restrict__ Q, const __bf16* __restrict__ K,
    const __bf16* __restrict__ V, const int32_t* __restrict__ idx, const float* __restrict__ w,
    __bf16* __restrict__ O, int ntiles) {
    constexpr int VP = Smem<S>::VP;
    constexpr int MB = S / 16;            // key blocks of Z^T
    constexpr int KS2 = S / 32;           // key steps of P V
    constexpr int NPF = S * D / 8 / kThreads;   // 16-byte K vectors per thread per chunk
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

    // ---- selections of the tile and their union -------------------------------------
    const int ne = TQ * k;
    for (int e = tid; e < ne; e += kThreads) {
        const int tau = e / k, t = t0 + tau;
        int c = -1;
        float wt = 0.f;
        if (t < dm.L) {
            const size_t o = (((size_t)b * dm.L + t) * dm.G + g) * k + e % k;
            c = idx[o];
            wt = w[o];
            if (c < 0 || c >= ncand) {
                c = -1;
                wt = 0.f;
            }
        }
        sm.sidx[e] = c;
        sm.sw[e] = wt;
    }
    __syncthreads();
    for (int e = tid; e < ne; e += kThreads) {
        const int c = sm.sidx[e];
        bool first = c >= 0;
        for (int e2 = 0; e2 < e && first; ++e2) first = sm.sidx[e2] != c;
        sm.flag[e] = first ? 1 : 0;
    }
    __syncthreads();
    if (wave == 0) {
        const int per = (ne + 63) / 64;
        const int e0 = lane * per, e1 = min(ne, e0 + per);
        int cnt = 0;
        for (int e = e0; e < e1; ++e) cnt += sm.flag[e];
        int incl = cnt;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int v = __shfl_up(incl, o, 64);
            if (lane >= o) incl += v;
        }
        int pos = incl - cnt;
        for (int e = e0; e < e1; ++e)
            if (sm.flag[e]) sm.ulist[pos++] = sm.sidx[e];
        if (lane == 63) sm.nu = incl;
    }

    // ---- Q^T operands of the wave's two row blocks (registers, whole kernel) ------------
    bf16x8_t qB[2][4];
    f32x4_t acc[2][8];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
        const int tau = wave * 4 + rb * 2 + (row >> 3);
        const int t = t0 + tau;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            if (t < dm.L) {
                const size_t qo = (((size_t)b * dm.L + t) * dm.H + (size_t)g * HG + (row & 7)) * D +
                                  32 * ks + 8 * grp;
                qB[rb][ks] = ld_bf16x8(Q + qo);
            } else {
                qB[rb][ks] = bf16x8_t{};
            }
        }
#pragma unroll
        for (int db = 0; db < 8; ++db) acc[rb][db] = zero4();
    }
    __syncthreads();
    const int nu = sm.nu;

    // ---- staging of one chunk: global -> registers -> LDS -----------------------------
    // K: vector v (16 bytes) = row v / 16, columns 8 (v % 16) .. +7.
    // V: vector pair p = (keys 2 (p / 16), 2 (p / 16) + 1; columns 8 (p % 16) .. +7),
    //    written to V^T as 8 packed key pairs.
    const size_t rowstride = (size_t)dm.G * D;          // elements between token rows
    const size_t bgbase = (size_t)b * dm.L * rowstride + (size_t)g * D;
    u32x4_t kreg[NPF], vreg[NPF];

    const float sl2 = dm.beta * 1.44269504088896341f;   // beta * log2(e)
    // Pipeline: chunk u is computed from stage u % 2 while chunk u + 1 (already in registers)
    // is written to the other stage and chunk u + 2 is being fetched; one barrier per chunk.
    auto chunk_base = [&](int u) { return bgbase + (size_t)sm.ulist[u] * S * rowstride; };
    if (nu > 0) {
        load_chunk<S>(kreg, vreg, K, V, chunk_base(0), rowstride, tid);
        store_chunk<S>(kreg, vreg, sm.Ks[0], sm.Vt[0], tid);
    }
    if (nu > 1) load_chunk<S>(kreg, vreg, K, V, chunk_base(1), rowstride, tid);
    __syncthreads();
    for (int u = 0; u < nu; ++u) {
        const int c = sm.ulist[u];
        const __bf16* Ks = sm.Ks[u & 1];
        const __bf16* Vt = sm.Vt[u & 1];
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
            const int tau = wave * 4 + rb * 2 + (row >> 3);
            float wl = 0.f;
            for (int s = 0; s < k; ++s)
                if (sm.sidx[tau * k + s] == c) wl = sm.sw[tau * k + s];
            if (__ballot(wl != 0.f) == 0) continue;

            // Z^T = K_c Q^T
            f32x4_t z[MB];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) z[mb] = zero4();
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) {
                    const bf16x8_t a = ld_bf16x8(&Ks[(16 * mb + row) * KP + 32 * ks + 8 * grp]);
                    z[mb] = mfma16(a, qB[rb][ks], z[mb]);
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
                    acc[rb][db] = mfma16(a, pb, acc[rb][db]);
                }
            }
        }
        if (u + 1 < nu) store_chunk<S>(kreg, vreg, sm.Ks[(u + 1) & 1], sm.Vt[(u + 1) & 1], tid);
        __syncthreads();
        if (u + 2 < nu) load_chunk<S>(kreg, vreg, K, V, chunk_base(u + 2), rowstride, tid);
    }

    // ---- output: O^T C layout -> O[b, t, g*8 + j, d] ----------------------------------
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
        const int tau = wave * 4 + rb * 2 + (row >> 3);
        const int t = t0 + tau;
        if (t >= dm.L) continue;
        __bf16* op = O + (((size_t)b * dm.L + t) * dm.H + (size_t)g * HG + (row & 7)) * D;
#pragma unroll
        for (int db = 0; db < 8; ++db) {
            const bf16x4_t o4{f2bf(acc[rb][db][0]), f2bf(acc[rb][db][1]), f2bf(acc[rb][db][2]),
                              f2bf(acc[rb][db][3])};
            *reinterpret_cast<bf16x4_t*>(op + 16 * db + 4 * grp) = o4;
        }
    }
}

}  // namespace

bool forward_mfma_supported(const Dims& dm, bool in_bf16) {
    return in_bf16 && dm.h == HG && dm.d == D && (dm.S == 64 || dm.S == 128) && dm.k <= KMAX &&
           !getenv("HSA_FORCE_GENERIC");
}

hipError_t launch_forward_mfma(const Dims& dm, const void* Q, const void* K, const void* V,
                               const int32_t* idx, const float* w, void* O, void*,
                               hipStream_t st) {
    const int ntiles = cdiv(dm.L, TQ);
    const int nlog = ntiles * dm.B * dm.G;
    const int grid = 8 * cdiv(nlog, 8);
    if (dm.S == 64) {
        HSA_TIMED("forward_mfma", st);
        hipLaunchKernelGGL((forward_mfma<64>), dim3(grid), dim3(kThreads), 0, st, dm,
                           (const __bf16*)Q, (const __bf16*)K, (const __bf16*)V, idx, w,
                           (__bf16*)O, ntiles);
    } else {
        HSA_TIMED("forward_mfma", st);
        hipLaunchKernelGGL((forward_mfma<128>), dim3(grid), dim3(kThreads), 0, st, dm,
                           (const __bf16*)Q, (const __bf16*)K, (const __bf16*)V, idx, w,
                           (__bf16*)O, ntiles);
    }
    return hipGetLastError();
}

}  // namespace hsa
