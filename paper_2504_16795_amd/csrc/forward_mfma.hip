// bf16 MFMA forward of hierarchical sparse attention (Sec. 3.1.1), for h = 8 query heads
// per KV head, d = 128, S in {64, 128}.
//
// Workgroup = (b, g, tile of 2 NW RB tokens inside one query chunk), NW waves; wave w owns RB
// row blocks of 16 rows (2 tokens x 8 heads each).
//  1. Each token's valid selections are sorted by descending chunk and the tile's union is
//     listed in the same order (tile_sel.h), so every lane follows its token's slot list
//     with a register pointer.
//  2. Each union chunk is copied once from global memory into LDS (chunk_lds.h: direct
//     global-to-LDS copies, no registers), into a ring of NST stages: NST - 1 chunks are
//     in flight while one is computed, with one barrier per chunk.
//  3. For each of its row blocks whose tokens selected the chunk (wave-uniform test), a wave
//     runs
//        Z^T [S x 16] = K_c [S x d] . Q^T [d x 16]        (S/16 * 4 MFMAs)
//        P^T = softmax over keys, scaled by w_{t,c} (0 for the row block's other token),
//              as a bf16 pair hi + lo
//        O^T [d x 16] += V_c^T [d x S] . P^T [S x 16]     (2 * 8 * S/32 MFMAs)
//     The C layout of Z^T feeds P^T straight into the B operand of the second product with
//     a key permutation applied to the V^T fragments, which come from transposed LDS
//     reads of the row-major V tile.  Q^T lives in registers for the whole kernel and O^T
//     accumulates in registers (fp32), so each chunk is read from L2/HBM once per tile
//     instead of once per (token, slot), and no online softmax is needed.
#include "chunk_lds.h"
#include "tile_sel.h"

namespace hsa {
namespace {

constexpr int D = 128;
constexpr int HG = 8;            // query heads per KV head
constexpr int KMAX = 32;
constexpr int UWORDS = 1024;     // union bitmap words: up to 32768 candidate chunks

// Waves per workgroup, row blocks (of 2 tokens) per wave, the waves per SIMD the register
// budget is sized for, and the chunk stages in LDS.  A tile holds 2 NW RB tokens; a staged
// chunk serves every row block of the tile that selected it.  At S = 64 two workgroups of 8
// waves with one row block each share a CU: while one waits at its per-chunk barrier or for
// a copy, the other computes.  (Tiles of 32 tokens, 8 waves with 2 row blocks each, stage
// each chunk for twice the work but fill a CU alone: 0.61 against 0.54 ms at 4K tokens, 4.2
// against 2.5 ms at 64K.)
template <int S>
struct FCfg;
template <>
struct FCfg<64> {
    static constexpr int NW = 8, RB = 1, WPE = 4, NST = 2;
};
template <>
struct FCfg<128> {
    static constexpr int NW = 8, RB = 1, WPE = 2, NST = 2;
};

// KT: table entries per token (at least k)
template <int S, int KT>
struct Smem {
    static constexpr int NW = FCfg<S>::NW, TQ = 2 * NW * FCfg<S>::RB, NST = FCfg<S>::NST;
    ChunkStage<S> st[NST];                        // K, V rows, swizzled (chunk_lds.h)
    int32_t oidx[TQ * KT];                        // selection tables (see tile_sel.h)
    float ow[TQ * KT];
    int32_t sidx[TQ * KT];
    float sw[TQ * KT];
    int32_t ulist[TQ * KT];
    uint8_t sslot[TQ * KT];
    int wsum[NW];
    uint32_t ubits[NST > 2 ? 1 : UWORDS];         // with 3 stages the bitmap uses stage 2
};

template <int S, int KT>
__global__ __launch_bounds__(FCfg<S>::NW * 64, FCfg<S>::WPE) void forward_mfma(
    Dims dm, const __bf16* __restrict__ Q, const __bf16* __restrict__ K,
    const __bf16* __restrict__ V, const int32_t* __restrict__ idx, const float* __restrict__ w,
    __bf16* __restrict__ O, int ntiles) {
    using SM = Smem<S, KT>;
    constexpr int NW = SM::NW, TQ = SM::TQ, NST = SM::NST, kThreads = NW * 64;
    constexpr int RB = FCfg<S>::RB;
    constexpr int MB = S / 16;            // key blocks of Z^T
    constexpr int KS2 = S / 32;           // key steps of P V
    constexpr int IPC = 2 * (S / 4) / NW; // copy instructions per chunk and wave
    __shared__ SM sm;

    const int lid = xcd_logical_id(ntiles * dm.B * dm.G);
    if (lid < 0) return;
    const int tile = lid % ntiles, bg = lid / ntiles;
    const int b = bg / dm.G, g = bg % dm.G;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int k = dm.k;
    const int t0 = tile * TQ;
    const int ncand = t0 / S;
    const int row = lane & 15, grp = lane >> 4;

    // ---- Q^T operands of the wave's row blocks (registers, whole kernel) -----------------
    // row block r of wave w holds tokens 2 (w RB + r) and 2 (w RB + r) + 1
    bf16x8_t qB[RB][4];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
        const int t_row = t0 + (wave * RB + r) * 2 + (row >> 3);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            if (t_row < dm.L) {
                const size_t qo =
                    (((size_t)b * dm.L + t_row) * dm.H + (size_t)g * HG + (row & 7)) * D +
                    32 * ks + 8 * grp;
                qB[r][ks] = ld_bf16x8(Q + qo);
            } else {
                qB[r][ks] = bf16x8_t{};
            }
        }
    }
    // ---- selections of the tile, sorted per token, and their union ----------------------
    uint32_t* ubits;
    if constexpr (NST > 2) {
        static_assert(sizeof(sm.st[NST - 1]) >= UWORDS * 4, "bitmap does not fit the stage");
        ubits = reinterpret_cast<uint32_t*>(sm.st[NST - 1].k);   // first written in the loop
    } else {
        ubits = sm.ubits;
    }
    const TileSel ts{sm.oidx, sm.ow, sm.sidx, sm.sslot, sm.sw, ubits, sm.ulist, sm.wsum};
    const int nu = tile_selection<kThreads, TQ>(
        ts, idx, w, (((size_t)b * dm.L + t0) * dm.G + g) * k, (size_t)dm.G * k, k,
        min(TQ, dm.L - t0), ncand);
    wait_global_loads();
    f32x4_t acc[RB][8];
#pragma unroll
    for (int r = 0; r < RB; ++r)
#pragma unroll
        for (int db = 0; db < 8; ++db) acc[r][db] = zero4();
    // each row block: this lane's token's next selected chunk and its weight
    int sp[RB], cur_c[RB];
    float cur_w[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
        const int tau = (wave * RB + r) * 2 + (row >> 3);
        sp[r] = 0;
        cur_c[r] = sm.sidx[tau * k];
        cur_w[r] = sm.sw[tau * k];
    }

    const size_t rowstride = (size_t)dm.G * D;
    const size_t bgbase = (size_t)b * dm.L * rowstride + (size_t)g * D;
    auto issue = [&](int u) __attribute__((always_inline)) {
        const size_t base = bgbase + (size_t)sm.ulist[u] * S * rowstride;
        chunk_to_lds<S, NW>(K + base, rowstride, sm.st[u % NST].k, wave, lane);
        chunk_to_lds<S, NW>(V + base, rowstride, sm.st[u % NST].v, wave, lane);
    };
    int koff[4], toff[8];
    row_read_offsets(lane, koff);
    tr_read_offsets(lane, toff);
    const float sl2 = dm.beta * 1.44269504088896341f;   // beta * log2(e)
    // softmax off by one: the row maximum also covers the extra logit 0
    const bool off1 = dm.off1 != 0;
    const float mfloor = off1 ? 0.f : -INFINITY;

#pragma unroll
    for (int u = 0; u < NST - 1; ++u)
        if (u < nu) issue(u);
    for (int u = 0; u < nu; ++u) {
        // chunk u has landed once at most the copies of the chunks issued after it remain
        if constexpr (NST == 3) {
            if (u + 1 < nu) wait_loads_le<IPC>();
            else wait_loads_le<0>();
        } else {
            wait_loads_le<0>();
        }
        barrier_keep_copies();    // ... for every wave; and stage (u - 1) % NST is free
        if (u + NST - 1 < nu) issue(u + NST - 1);

        const int c = sm.ulist[u];
        const ChunkStage<S>& cs = sm.st[u % NST];
#pragma unroll
        for (int r = 0; r < RB; ++r) {
            const bool mine = (cur_c[r] == c);
            if (__ballot(mine) == 0) continue;
            const float wl = mine ? cur_w[r] : 0.f;
            // Z^T = K_c Q^T
            f32x4_t z[MB];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) z[mb] = zero4();
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
                    z[mb] = mfma16(ld_bf16x8(cs.k + koff[ks] + mb * 2048), qB[r][ks], z[mb]);
            // softmax over the S keys of each row (column `row` of Z^T)
            float m = -INFINITY;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int i = 0; i < 4; ++i) m = fmaxf(m, z[mb][i]);
            const float msl = fmaxf(col_max(m), mfloor) * sl2;
            float ssum = 0.f;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    z[mb][i] = fast_exp2(fmaf(z[mb][i], sl2, -msl));
                    ssum += z[mb][i];
                }
            ssum = col_sum(ssum) + (off1 ? fast_exp2(-msl) : 0.f);
            const float scale = wl * __builtin_amdgcn_rcpf(ssum);
            // O^T += V^T P^T
#pragma unroll
            for (int ks2 = 0; ks2 < KS2; ++ks2) {
                // w P as a bf16 pair hi + lo (about 16 bits): one bf16 rounding of each
                // weighted probability would leave an error of up to 2^-9 of it in O
                f32x4_t pa, pc;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    pa[i] = z[2 * ks2][i] * scale;
                    pc[i] = z[2 * ks2 + 1][i] * scale;
                }
                bf16x8_t ph, pl;
                split8(pa, pc, ph, pl);
                // in halves of 4 column blocks: the hi products, then the lo ones, so that no
                // product waits for the one just before it
#pragma unroll
                for (int d0 = 0; d0 < 8; d0 += 4) {
                    bf16x8_t vt[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const __bf16* p = cs.v + toff[d0 + j] + 32 * ks2 * D;
                        vt[j] = cat(ld_tr16(p), ld_tr16(p + 16 * D));
                    }
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[r][d0 + j] = mfma16(vt[j], ph, acc[r][d0 + j]);
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[r][d0 + j] = mfma16(vt[j], pl, acc[r][d0 + j]);
                }
            }
            if (mine) {
                const int tau = (wave * RB + r) * 2 + (row >> 3);
                ++sp[r];
                cur_c[r] = sp[r] < k ? sm.sidx[tau * k + sp[r]] : -1;
                cur_w[r] = sp[r] < k ? sm.sw[tau * k + sp[r]] : 0.f;
            }
        }
    }

    // ---- output: O^T C layout -> O[b, t, g*8 + j, d] ----------------------------------
#pragma unroll
    for (int r = 0; r < RB; ++r) {
        const int t_row = t0 + (wave * RB + r) * 2 + (row >> 3);
        if (t_row < dm.L) {
            __bf16* op =
                O + (((size_t)b * dm.L + t_row) * dm.H + (size_t)g * HG + (row & 7)) * D;
#pragma unroll
            for (int db = 0; db < 8; ++db) {
                const bf16x4_t o4{f2bf(acc[r][db][0]), f2bf(acc[r][db][1]), f2bf(acc[r][db][2]),
                                  f2bf(acc[r][db][3])};
                *reinterpret_cast<bf16x4_t*>(op + 16 * db + 4 * grp) = o4;
            }
        }
    }
}

template <int S, int KT>
void launch_fwd(const Dims& dm, const void* Q, const void* K, const void* V,
                const int32_t* idx, const float* w, void* O, hipStream_t st) {
    constexpr int TQ = Smem<S, KT>::TQ;
    const int ntiles = cdiv(dm.L, TQ);
    const int grid = 8 * cdiv(ntiles * dm.B * dm.G, 8);
    HSA_TIMED("forward_mfma", st);
    hipLaunchKernelGGL((forward_mfma<S, KT>), dim3(grid), dim3(FCfg<S>::NW * 64), 0, st, dm,
                       (const __bf16*)Q, (const __bf16*)K, (const __bf16*)V, idx, w,
                       (__bf16*)O, ntiles);
}

template <int S>
void launch_fwd_k(const Dims& dm, const void* Q, const void* K, const void* V,
                  const int32_t* idx, const float* w, void* O, hipStream_t st) {
    if (dm.k <= 8) launch_fwd<S, 8>(dm, Q, K, V, idx, w, O, st);
    else if (dm.k <= 16) launch_fwd<S, 16>(dm, Q, K, V, idx, w, O, st);
    else launch_fwd<S, KMAX>(dm, Q, K, V, idx, w, O, st);
}

}  // namespace

bool forward_mfma_supported(const Dims& dm, bool in_bf16) {
    return in_bf16 && dm.h == HG && dm.d == D && (dm.S == 64 || dm.S == 128) && dm.k <= KMAX &&
           dm.C <= UWORDS * 32 && path_override(HSA_OP_FORWARD) != HSA_PATH_GENERIC;
}

hipError_t launch_forward_mfma(const Dims& dm, const void* Q, const void* K, const void* V,
                               const int32_t* idx, const float* w, void* O, void*,
                               hipStream_t st) {
    if (dm.S == 64) launch_fwd_k<64>(dm, Q, K, V, idx, w, O, st);
    else launch_fwd_k<128>(dm, Q, K, V, idx, w, O, st);
    return hipGetLastError();
}

}  // namespace hsa
