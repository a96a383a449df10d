// bf16 MFMA backward of hierarchical sparse attention (Sec. 3.1.2, two-phase backward),
// for h = 8 query heads per KV head, d = 128, S in {64, 128}.
//
// Query pass (bwd_q_mfma): the forward's tiling (a tile of 2 NW tokens inside one query
// chunk, wave w owning tokens 2w, 2w+1 as one row block of 16 rows; the tile's union of
// chunks listed in descending order and copied once into a ring of LDS stages, each lane
// following its token's descending slot list with a pointer).  Per chunk selected by the
// row block:
//     Z^T  = K_c Q^T,  dP^T = V_c dO^T                     (keys x rows, MFMA)
//     P    = softmax over keys;  D_row = sum_keys P dP      (= dO_row . O_{row,c})
//     dZ^T = w P (dP - D)
//     dQ^T += K_c^T dZ^T                                    (MFMA, K^T fragments from
//                                                             transposed reads of the K
//                                                             tile; dZ as a bf16 hi/lo pair)
//     dw_{t,c} = sum over the token's 8 heads of D_row
// then ds_i = w_i (dw_i - sum_m w_m dw_m) and dQ = beta dQ + alpha sum_i ds_i Kbar_{c_i}.
// For the key pass it stores, per (token, slot, head), the log-sum-exp of the scaled logits
// and D, plus ds per (token, slot).
//
// Key pass: chunk-major, reading those statistics (see bwd_kv_mfma below).
#include "chunk_stream.h"
#include "tile_sel.h"

namespace hsa {

size_t backward_generic_workspace(const Dims& dm);
hipError_t launch_selection_bitmap(const Dims& dm, const int32_t* idx, uint32_t* bm,
                                   hipStream_t st);

namespace {

constexpr int D = 128;
constexpr int HG = 8;
constexpr int KMAX = 32;
constexpr int UWORDS = 1024;     // union bitmap words: up to 32768 candidate chunks


// workspace layout shared by both passes (ds and the bitmap first, as in the generic path)
// (the key pass's even split: tokens per (b, g, chunk) row, the group prefix, the plan, and
// two fp32 partial dK / dV tiles per workgroup for the rows it shares)
constexpr int kKvWGs = 512;      // workgroups of the key pass: two per CU

struct WsLayout {
    size_t ds, bitmap, lse, dd, cnt, gstart, plan, pk, pv, end;
};
__host__ __device__ inline WsLayout ws_layout(const Dims& dm) {
    WsLayout l;
    const size_t nsel = (size_t)dm.B * dm.L * dm.G * dm.k;
    const size_t nwords = (size_t)((dm.L + 31) / 32);
    const size_t R = (size_t)dm.B * dm.G * dm.C;
    l.ds = 0;
    l.bitmap = align256(nsel * 4);
    l.lse = l.bitmap + align256(R * nwords * 4);
    l.dd = l.lse + align256(nsel * dm.h * 4);
    l.cnt = l.dd + align256(nsel * dm.h * 4);
    l.gstart = l.cnt + align256(R * 4);
    l.plan = l.gstart + align256((R + 1) * 4);
    l.pk = l.plan + 256;
    l.pv = l.pk + (size_t)kKvWGs * 2 * dm.S * D * 4;
    l.end = l.pv + (size_t)kKvWGs * 2 * dm.S * D * 4;
    return l;
}

// Query-pass shape: waves per workgroup (one row block each) and chunk stages in LDS.  At
// S = 64 two workgroups of 4 waves share a CU (76 KB of LDS each), so one computes while
// the other waits at its per-chunk barrier.
template <int S>
struct QCfg;
template <>
struct QCfg<64> {
    static constexpr int NW = 4, NST = 2;
};
template <>
struct QCfg<128> {
    static constexpr int NW = 8, NST = 2;
};

template <int S>
struct SmemQ {
    static constexpr int NW = QCfg<S>::NW, NST = QCfg<S>::NST, TQ = 2 * NW;
    ChunkStage<S> st[NST];        // K, V rows, swizzled (chunk_lds.h)
    int32_t oidx[TQ * KMAX];      // selection tables (see tile_sel.h)
    float ow[TQ * KMAX];
    int32_t sidx[TQ * KMAX];
    float sw[TQ * KMAX];
    int32_t ulist[TQ * KMAX];
    uint32_t ubits[UWORDS];
    float dw[TQ * KMAX];          // per slot: dw of the token
    uint8_t sslot[TQ * KMAX];
    int wsum[NW];
};

template <int S>
__global__ __launch_bounds__(QCfg<S>::NW * 64, 2) void bwd_q_mfma(
    Dims dm, const __bf16* __restrict__ Q, const __bf16* __restrict__ K,
    const __bf16* __restrict__ V, const float* __restrict__ Kbar,
    const int32_t* __restrict__ idx, const float* __restrict__ w,
    const __bf16* __restrict__ dO, __bf16* __restrict__ dQ, float* __restrict__ ds_out,
    float* __restrict__ lse_out, float* __restrict__ d_out, int ntiles) {
    using SM = SmemQ<S>;
    constexpr int NW = SM::NW, NT = NW * 64, TQ = SM::TQ, NST = SM::NST;
    constexpr int MB = S / 16;
    constexpr int KS2 = S / 32;
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

    // ---- Q^T and dO^T operands of the wave's row block ---------------------------------
    const int tau = wave * 2 + (row >> 3);
    const int t_row = t0 + tau;
    bf16x8_t qB[4], gB[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
        if (t_row < dm.L) {
            const size_t o = (((size_t)b * dm.L + t_row) * dm.H + (size_t)g * HG + (row & 7)) * D +
                             32 * ks + 8 * grp;
            qB[ks] = ld_bf16x8(Q + o);
            gB[ks] = ld_bf16x8(dO + o);
        } else {
            qB[ks] = bf16x8_t{};
            gB[ks] = bf16x8_t{};
        }
    }
    // ---- selections of the tile, sorted per token, and their union ----------------------
    const TileSel ts{sm.oidx, sm.ow, sm.sidx, sm.sslot, sm.sw, sm.ubits, sm.ulist, sm.wsum};
    const int nu = tile_selection<NT, TQ>(ts, idx, w, (((size_t)b * dm.L + t0) * dm.G + g) * k,
                                          (size_t)dm.G * k, k, min(TQ, dm.L - t0), ncand);
    for (int e = tid; e < TQ * k; e += NT) sm.dw[e] = 0.f;
    wait_global_loads();
    f32x4_t acc[8];
#pragma unroll
    for (int db = 0; db < 8; ++db) acc[db] = zero4();
    // this lane's token: next selected chunk, its first slot and its weight
    int sp = 0;
    int cur_c = sm.sidx[tau * k];
    int cur_s = sm.sslot[tau * k];
    float cur_w = sm.sw[tau * k];

    const size_t rowstride = (size_t)dm.G * D;
    const size_t bgbase = (size_t)b * dm.L * rowstride + (size_t)g * D;
    const float beta = dm.beta;
    const float sl2 = beta * 1.44269504088896341f;
    const bool off1 = dm.off1 != 0;
    const float mfloor = off1 ? 0.f : -INFINITY;
    auto issue = [&](int u) __attribute__((always_inline)) {
        const size_t base = bgbase + (size_t)sm.ulist[u] * S * rowstride;
        chunk_to_lds<S, NW>(K + base, rowstride, sm.st[u % NST].k, wave, lane);
        chunk_to_lds<S, NW>(V + base, rowstride, sm.st[u % NST].v, wave, lane);
    };
    int koff[4], toff[8];
    row_read_offsets(lane, koff);
    tr_read_offsets(lane, toff);

    // ring of NST stages: NST - 1 chunks in flight while one is computed
#pragma unroll
    for (int u = 0; u < NST - 1; ++u)
        if (u < nu) issue(u);
    for (int u = 0; u < nu; ++u) {
        if constexpr (NST == 3) {
            if (u + 1 < nu) wait_loads_le<IPC>();
            else wait_loads_le<0>();
        } else {
            wait_loads_le<0>();
        }
        barrier_keep_copies();    // chunk u landed for every wave; stage (u - 1) % NST free
        if (u + NST - 1 < nu) issue(u + NST - 1);

        const int c = sm.ulist[u];
        const bool mine = (cur_c == c);
        if (__ballot(mine) != 0) {
            const ChunkStage<S>& cs = sm.st[u % NST];
            const float wl = mine ? cur_w : 0.f;
            // K rows at kp[ks] + mb * 2048, V rows at the same offsets in cs.v
            constexpr int VOFF = S * D;
            f32x4_t z[MB], dp[MB];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) z[mb] = dp[mb] = zero4();
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) {
                    z[mb] = mfma16(ld_bf16x8(cs.k + koff[ks] + mb * 2048), qB[ks], z[mb]);
                    dp[mb] = mfma16(ld_bf16x8(cs.k + koff[ks] + VOFF + mb * 2048), gB[ks], dp[mb]);
                }
            float m = -INFINITY;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int i = 0; i < 4; ++i) m = fmaxf(m, z[mb][i]);
            m = fmaxf(col_max(m), mfloor);      // off by one: the extra logit 0 included
            const float msl = m * sl2;
            // unnormalised probabilities Pu = exp(beta (z - m)), their sum and sum Pu dP
            float ssum = 0.f, dsu = 0.f;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    z[mb][i] = fast_exp2(fmaf(z[mb][i], sl2, -msl));
                    ssum += z[mb][i];
                    dsu = fmaf(z[mb][i], dp[mb][i], dsu);
                }
            ssum = col_sum(ssum) + (off1 ? fast_exp2(-msl) : 0.f);
            const float inv = __builtin_amdgcn_rcpf(ssum);
            const float dsum = col_sum(dsu) * inv;                    // D of this row
            // dZ = w P (dP - D), fed as the B operand of dQ^T += K^T dZ^T.  sum_s dZ_s = 0,
            // so dQ is a cancelling sum: dZ enters as a bf16 pair (hi + lo, ~16 mantissa
            // bits) to keep its rounding from being amplified by the key magnitudes.
            const float wp = wl * inv;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int i = 0; i < 4; ++i) z[mb][i] = (wp * z[mb][i]) * (dp[mb][i] - dsum);
#pragma unroll
            for (int ks2 = 0; ks2 < KS2; ++ks2) {
                bf16x8_t zh, zl;
                split8(z[2 * ks2], z[2 * ks2 + 1], zh, zl);
                // in halves of 4 column blocks: the hi products, then the lo ones, so that no
                // product waits for the one just before it
#pragma unroll
                for (int d0 = 0; d0 < 8; d0 += 4) {
                    bf16x8_t a[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const __bf16* p = cs.k + toff[d0 + j] + 32 * ks2 * D;
                        a[j] = cat(ld_tr16(p), ld_tr16(p + 16 * D));
                    }
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[d0 + j] = mfma16(a[j], zh, acc[d0 + j]);
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[d0 + j] = mfma16(a[j], zl, acc[d0 + j]);
                }
            }
            // statistics of this (token, slot, head) and dw of the token
            float dtok = dsum;
            dtok += __shfl_xor(dtok, 1, 64);
            dtok += __shfl_xor(dtok, 2, 64);
            dtok += __shfl_xor(dtok, 4, 64);
            if (mine) {
                const size_t so = (((size_t)b * dm.L + t_row) * dm.G + g) * k + cur_s;
                if (grp == 0) {
                    lse_out[so * HG + (row & 7)] = m * beta + __logf(ssum);
                    d_out[so * HG + (row & 7)] = dsum;
                }
                if (grp == 0 && (row & 7) == 0) sm.dw[tau * k + cur_s] = dtok;
                ++sp;
                cur_c = sp < k ? sm.sidx[tau * k + sp] : -1;
                cur_s = sp < k ? sm.sslot[tau * k + sp] : 0;
                cur_w = sp < k ? sm.sw[tau * k + sp] : 0.f;
            }
        }
    }
    __syncthreads();

    // ---- chunk-weight Jacobian, score term, write dQ and ds --------------------------------
    if (t_row >= dm.L) return;
    float wdw = 0.f;
    for (int s = 0; s < k; ++s) wdw = fmaf(sm.ow[tau * k + s], sm.dw[tau * k + s], wdw);
    f32x4_t out[8];
#pragma unroll
    for (int db = 0; db < 8; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) out[db][i] = beta * acc[db][i];
    // score term: empty slots add 0 (their loads use chunk 0, which exists when any slot of
    // the tile is valid); loads of several slots are in flight at once
    const bool stick = dm.stick != 0;
    auto slot_ds = [&](int s) __attribute__((always_inline)) {
        if (sm.oidx[tau * k + s] < 0) return 0.f;
        if (!stick) return sm.ow[tau * k + s] * (sm.dw[tau * k + s] - wdw);
        return stick_ds(s, k, [&](int m) { return sm.ow[tau * k + m]; },
                        [&](int m) { return sm.dw[tau * k + m]; },
                        [&](int m) { return sm.oidx[tau * k + m] >= 0; });
    };
    const bool attn_only = dm.dwo != nullptr;
    for (int s = 0; s < k; ++s) {
        const size_t so = (((size_t)b * dm.L + t_row) * dm.G + g) * k + s;
        if (attn_only) {
            // attention alone: dw per slot, ds = 0 (no landmark term in the key pass)
            if (grp == 0 && (row & 7) == 0) {
                const float v = sm.oidx[tau * k + s] >= 0 ? sm.dw[tau * k + s] : 0.f;
                dm.dwo[so] = dm.dwacc ? dm.dwo[so] + v : v;
                ds_out[so] = 0.f;
            }
            continue;
        }
        const float dsv = slot_ds(s);
        if (grp == 0 && (row & 7) == 0) ds_out[so] = dsv;
    }
    if (ncand > 0 && !attn_only) {
#pragma unroll 4
        for (int s = 0; s < k; ++s) {
            const int c = sm.oidx[tau * k + s];
            const float dsv = slot_ds(s);
            const float* kb = Kbar + (((size_t)b * dm.C + max(c, 0)) * dm.G + g) * D;
            const float coef = dm.alpha * dsv;
#pragma unroll
            for (int db = 0; db < 8; ++db) {
                const float4 kv = *reinterpret_cast<const float4*>(kb + 16 * db + 4 * grp);
                out[db][0] = fmaf(coef, kv.x, out[db][0]);
                out[db][1] = fmaf(coef, kv.y, out[db][1]);
                out[db][2] = fmaf(coef, kv.z, out[db][2]);
                out[db][3] = fmaf(coef, kv.w, out[db][3]);
            }
        }
    }
    __bf16* op = dQ + (((size_t)b * dm.L + t_row) * dm.H + (size_t)g * HG + (row & 7)) * D;
#pragma unroll
    for (int db = 0; db < 8; ++db) {
        const bf16x4_t o4{f2bf(out[db][0]), f2bf(out[db][1]), f2bf(out[db][2]),
                          f2bf(out[db][3])};
        *reinterpret_cast<bf16x4_t*>(op + 16 * db + 4 * grp) = o4;
    }
}

// ----------------------------------------------------------------------------------------
// Key pass (bwd_kv_mfma): chunk-major over an even split of the work.  The selecting tokens
// of each (b, g, chunk) row come from the selection bitmap in increasing order, in groups of
// four (32 rows = 4 tokens x 8 heads); the groups of all rows are laid end to end and split
// into kKvWGs equal ranges (stream_rowcount / stream_plan), so a chunk selected by thousands
// of tokens is shared by several workgroups instead of setting the kernel time.  Wave w owns
// keys 16w..16w+15 of the current chunk and keeps K_sub, V_sub as B operands in registers
// and dK_sub, dV_sub [16 x 128] as fp32 accumulators.  Per group:
//     Z  [32 x 16] = Q_rows K_sub^T,   dP = dO_rows V_sub^T          (MFMA)
//     P  = exp(beta Z - lse_row),  dZ = w P (dP - D_row)            (stored by the query pass)
//     dV_sub += (w P)^T dO_rows,  dK_sub += dZ^T Q_rows              (MFMA, K = 32 rows;
//                                                 w P and dZ as bf16 hi/lo pairs)
// A group's Q and dO rows (and their lse / D) are copied straight into a ring of LDS stages
// (chunk_lds.h), two groups in flight while one is computed.  Z and dP read the rows; the
// last two products read them transposed, in the row order of the C layout of Z, which
// then serves as their A operand directly.  The landmark term dKbar_c / S =
// (alpha / S) sum ds q~ is folded into dZ.  A workgroup that covers a row whole writes its
// dK, dV; for a shared row (the first or last of its range) it writes fp32 partials, which
// bwd_kv_finish adds in workgroup order.  No atomics; fixed token order.
constexpr int LISTCAP = 2048;    // tokens listed at once (a multiple of 4)
constexpr int KV_NST = 3;

struct KvStage {
    __bf16 q[32 * D];             // Q rows of the group (row 8 token + head), swizzled
    __bf16 g[32 * D];             // dO rows
    float meta[256];              // [0, 32): lse per row, [32, 64): D per row, rest scratch
};

struct SmemKV {
    KvStage st[KV_NST];
    int list[LISTCAP];
    float lw[LISTCAP], lds[LISTCAP];
    uint8_t lslot[LISTCAP];
    int wtot[16];
};

template <int S>
__global__ __launch_bounds__(S * 4, 2) void bwd_kv_mfma(
    Dims dm, const __bf16* __restrict__ Q, const __bf16* __restrict__ K,
    const __bf16* __restrict__ V, const int32_t* __restrict__ idx, const float* __restrict__ w,
    const __bf16* __restrict__ dO, const float* __restrict__ ds, const float* __restrict__ lse,
    const float* __restrict__ dd, const uint32_t* __restrict__ bm, int nwords,
    const int* __restrict__ gstart, const int* __restrict__ cntr, const int* __restrict__ plan,
    float* __restrict__ pk, float* __restrict__ pv, __bf16* __restrict__ dK,
    __bf16* __restrict__ dV) {
    constexpr int NWK = S / 16;             // waves
    constexpr int NTK = NWK * 64;
    constexpr int BPW = 8 / NWK;            // 1 KB row blocks of Q (and of dO) per wave
    __shared__ SmemKV sm;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int row = lane & 15, grp = lane >> 4;
    // consecutive ranges (the chunks of one slice) run on one XCD, so a token's Q / dO rows,
    // read once per chunk it selected, are shared through that XCD's L2
    const int lid = xcd_logical_id(kKvWGs);
    if (lid < 0) return;
    const int R = dm.B * dm.G * dm.C;
    const int total = plan[0], T = plan[1];
    const int g0 = lid * T, g1 = min(g0 + T, total);
    if (g0 >= g1) return;
    const int k = dm.k;
    const size_t rowstride = (size_t)dm.G * D;
    const float beta = dm.beta;
    const float l2e = 1.44269504088896341f;
    const float lmk = dm.alpha / (beta * (float)S);
    int koff[4], toff[8];
    row_read_offsets(lane, koff);
    tr_read_offsets(lane, toff);

    for (int r = find_row(gstart, R, g0); r < R; ++r) {
        const int rs = gstart[r], re = gstart[r + 1];
        if (rs >= g1) break;
        if (re == rs) continue;
        const Segment sg = segment_of(rs, re, g0, g1);
        const int c = r % dm.C;
        const int bg = r / dm.C, b = bg / dm.G, g = bg % dm.G;
        const size_t cbase = ((size_t)b * dm.L + (size_t)c * S) * rowstride + (size_t)g * D;
        const int ntok = cntr[r];

        __syncthreads();                  // the previous row's stages and lists are read
        // B operands of the wave's 16 keys: K_sub^T[d][key], V_sub^T[d][key]
        bf16x8_t kB[4], vB[4];
        const int key = 16 * wave + row;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            kB[ks] = ld_bf16x8(K + cbase + (size_t)key * rowstride + 32 * ks + 8 * grp);
            vB[ks] = ld_bf16x8(V + cbase + (size_t)key * rowstride + 32 * ks + 8 * grp);
        }
        wait_global_loads();
        f32x4_t aK[8], aV[8];
#pragma unroll
        for (int db = 0; db < 8; ++db) aK[db] = aV[db] = zero4();

        // copies of group gi (tokens 4 gi .. 4 gi + 3 of the list; a missing token repeats
        // the group's first one, with weight and ds 0): wave w copies the Q and dO row blocks
        // w BPW .. w BPW + BPW - 1 (4 rows = half a token each); the last wave also copies
        // the lse and D of the 32 rows
        auto issue = [&](int gi, int nl, KvStage& st) __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < BPW; ++i) {
                const int blk = wave * BPW + i;
                const int rr = blk * 4 + (lane >> 4);
                int li = gi * 4 + (rr >> 3);
                if (li >= nl) li = gi * 4;
                const size_t o = (((size_t)b * dm.L + sm.list[li]) * dm.H + (size_t)g * HG + (rr & 7)) * D +
                                 unit_pos(rr, lane & 15) * 8;
                lds_copy16(Q + o, __builtin_amdgcn_readfirstlane(lds_address(st.q + blk * 512)));
                lds_copy16(dO + o, __builtin_amdgcn_readfirstlane(lds_address(st.g + blk * 512)));
            }
            if (wave == NWK - 1) {
                // lanes 16 m + 2 j + h (j < 4 tokens, h halves of the 8 heads): m = 0 lse,
                // m = 1 D, m >= 2 repeat (scratch)
                int li = gi * 4 + ((lane & 7) >> 1);
                if (li >= nl) li = gi * 4;
                const size_t so =
                    ((((size_t)b * dm.L + sm.list[li]) * dm.G + g) * k + sm.lslot[li]) * HG +
                    4 * (lane & 1);
                lds_copy16(((lane >> 3) & 1 ? dd : lse) + so,
                           __builtin_amdgcn_readfirstlane(lds_address(st.meta)));
            }
        };

        const uint32_t* bmrow = bm + (size_t)r * nwords;
        const int wbeg = ((c + 1) * S) >> 5;
        const int tend = min(4 * sg.j1, ntok);
        for (int p0 = 4 * sg.j0; p0 < tend; p0 += LISTCAP) {
            const int p1 = min(p0 + LISTCAP, tend);
            const int nl = p1 - p0;
            __syncthreads();              // the list of the previous batch is read
            collect_tokens<NTK>(bmrow, wbeg, nwords, p0, p1, sm.list, sm.wtot, tid);
            // per listed token: the slot holding c (a token's valid entries are distinct, so
            // one matches; consecutive (token, slot) entries per thread keep the idx loads
            // independent and coalesced), then its weight and ds there
            for (int e = tid; e < nl * k; e += NTK) {
                const int li = e / k, s2 = e - li * k;
                const size_t so = (((size_t)b * dm.L + sm.list[li]) * dm.G + g) * k;
                if (idx[so + s2] == c) sm.lslot[li] = (uint8_t)s2;
            }
            __syncthreads();
            for (int li = tid; li < nl; li += NTK) {
                const size_t so =
                    (((size_t)b * dm.L + sm.list[li]) * dm.G + g) * k + sm.lslot[li];
                sm.lw[li] = w[so];
                sm.lds[li] = ds[so];
            }
            __syncthreads();
            const int ngroups = (nl + 3) / 4;
#pragma unroll
            for (int u = 0; u < KV_NST - 1; ++u)
                if (u < ngroups) issue(u, nl, sm.st[u]);
            // one group's step; its stage index SI = gi % KV_NST is a constant (the loop
            // below is unrolled by KV_NST), so stage addresses are lane bases plus immediates
            auto group = [&](int gi, auto si) __attribute__((always_inline)) {
                constexpr int SI = decltype(si)::value;
                // group gi has landed once at most the next group's copies remain
                if (gi + 1 < ngroups) {
                    if (wave == NWK - 1) wait_loads_le<2 * BPW + 1>();
                    else wait_loads_le<2 * BPW>();
                } else {
                    wait_loads_le<0>();
                }
                barrier_keep_copies();        // ... for every wave; stage (gi - 1) % NST free
                if (gi + KV_NST - 1 < ngroups) issue(gi + KV_NST - 1, nl, sm.st[(SI + KV_NST - 1) % KV_NST]);
                const KvStage& st = sm.st[SI];

                // ---- Z, dP for the wave's 16 keys ---------------------------------------
                f32x4_t z[2], dp[2];
                z[0] = z[1] = dp[0] = dp[1] = zero4();
#pragma unroll
                for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                    for (int rb = 0; rb < 2; ++rb) {
                        z[rb] = mfma16(ld_bf16x8(st.q + koff[ks] + rb * 2048), kB[ks], z[rb]);
                        dp[rb] = mfma16(ld_bf16x8(st.g + koff[ks] + rb * 2048), vB[ks], dp[rb]);
                    }
                // rows of this lane: 16 rb + 4 grp + i (token 2 rb + grp / 2).  The landmark
                // term dKbar_c / S = (alpha / S) sum_rows ds_tok q_row reaches every key of the
                // chunk, so it is folded into dZ as alpha ds_tok / (beta S) before the dZ^T Q
                // product.
                f32x4_t pw[2], dz[2];
#pragma unroll
                for (int rb = 0; rb < 2; ++rb) {
                    const int li = gi * 4 + 2 * rb + (grp >> 1);
                    const float wt = li < nl ? sm.lw[li] : 0.f;
                    const float lm = li < nl ? sm.lds[li] * lmk : 0.f;
                    const f32x4_t lv = *reinterpret_cast<const f32x4_t*>(&st.meta[16 * rb + 4 * grp]);
                    const f32x4_t dv =
                        *reinterpret_cast<const f32x4_t*>(&st.meta[32 + 16 * rb + 4 * grp]);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float p = fast_exp2((beta * z[rb][i] - lv[i]) * l2e);
                        pw[rb][i] = wt * p;
                        dz[rb][i] = wt * p * (dp[rb][i] - dv[i]) + lm;
                    }
                }
                // both products accumulate over every row that selected the chunk (thousands
                // for a popular chunk): w P and dZ enter as bf16 hi/lo pairs
                bf16x8_t pvh, pvl, dzh, dzl;
                split8(pw[0], pw[1], pvh, pvl);
                split8(dz[0], dz[1], dzh, dzl);
                // per column block the hi products of dV and dK, then their lo ones, so that
                // no product waits for the one just before it
#pragma unroll
                for (int db = 0; db < 8; ++db) {
                    const bf16x8_t gb =
                        cat(ld_tr16(st.g + toff[db]), ld_tr16(st.g + toff[db] + 16 * D));
                    const bf16x8_t qb =
                        cat(ld_tr16(st.q + toff[db]), ld_tr16(st.q + toff[db] + 16 * D));
                    aV[db] = mfma16(pvh, gb, aV[db]);
                    aK[db] = mfma16(dzh, qb, aK[db]);
                    aV[db] = mfma16(pvl, gb, aV[db]);
                    aK[db] = mfma16(dzl, qb, aK[db]);
                }
            };
            static_assert(KV_NST == 3, "the group loop is unrolled by the ring depth");
            for (int gb = 0; gb < ngroups; gb += KV_NST) {
                group(gb, IntC<0>{});
                if (gb + 1 < ngroups) group(gb + 1, IntC<1>{});
                if (gb + 2 < ngroups) group(gb + 2, IntC<2>{});
            }
        }
        // the chunk's sums: final when this workgroup covered all its groups
        float* ok = pk + ((size_t)lid * 2 + sg.pslot) * S * D;
        float* ov = pv + ((size_t)lid * 2 + sg.pslot) * S * D;
#pragma unroll
        for (int db = 0; db < 8; ++db) {
            const int d = 16 * db + row;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int kr = 16 * wave + 4 * grp + i;
                if (sg.whole) {
                    const size_t o = cbase + (size_t)kr * rowstride + d;
                    dK[o] = f2bf(beta * aK[db][i]);
                    dV[o] = f2bf(aV[db][i]);
                } else {
                    ok[kr * D + d] = beta * aK[db][i];
                    ov[kr * D + d] = aV[db][i];
                }
            }
        }
    }
}

// Per chunk (b, g, c): the sum of the partials of the workgroups that shared it, in
// workgroup order; zeros for chunks nobody selected and for the trailing partial chunk.  A
// chunk one workgroup covered is final already.
template <int S>
__global__ __launch_bounds__(256) void bwd_kv_finish(
    Dims dm, const int* __restrict__ gstart, const int* __restrict__ cntr,
    const int* __restrict__ plan, const float* __restrict__ pk, const float* __restrict__ pv,
    __bf16* __restrict__ dK, __bf16* __restrict__ dV) {
    const int tid = threadIdx.x;
    const int c = blockIdx.x % dm.Call;
    const int bg = blockIdx.x / dm.Call, b = bg / dm.G, g = bg % dm.G;
    const size_t rowstride = (size_t)dm.G * D;
    const size_t cbase = ((size_t)b * dm.L + (size_t)c * S) * rowstride + (size_t)g * D;
    const int r = bg * dm.C + c;
    if (c >= dm.C || cntr[r] == 0) {            // trailing partial chunk, or never selected
        const int rows = min(S, dm.L - c * S);
        const bf16x4_t z4{__bf16(0.f), __bf16(0.f), __bf16(0.f), __bf16(0.f)};
        for (int e = tid; e < rows * 32; e += 256) {
            const size_t o = cbase + (size_t)(e >> 5) * rowstride + 4 * (e & 31);
            *reinterpret_cast<bf16x4_t*>(dK + o) = z4;
            *reinterpret_cast<bf16x4_t*>(dV + o) = z4;
        }
        return;
    }
    const int T = plan[1];
    const int rs = gstart[r], re = gstart[r + 1];
    const int wf = rs / T, wl = (re - 1) / T;
    if (wf == wl) return;                       // written by its workgroup
    for (int e = tid; e < S * 32; e += 256) {
        float4 sk{0.f, 0.f, 0.f, 0.f}, sv{0.f, 0.f, 0.f, 0.f};
        for (int wg = wf; wg <= wl; ++wg) {
            // the row is the first of the ranges after wf's, and of wf's when it starts there
            const int sl = (wg > wf || rs == wf * T) ? 0 : 1;
            const size_t po = ((size_t)wg * 2 + sl) * S * D + 4 * (size_t)e;
            const float4 a = *reinterpret_cast<const float4*>(pk + po);
            const float4 v = *reinterpret_cast<const float4*>(pv + po);
            sk.x += a.x; sk.y += a.y; sk.z += a.z; sk.w += a.w;
            sv.x += v.x; sv.y += v.y; sv.z += v.z; sv.w += v.w;
        }
        const size_t o = cbase + (size_t)(e >> 5) * rowstride + 4 * (e & 31);
        *reinterpret_cast<bf16x4_t*>(dK + o) = bf16x4_t{f2bf(sk.x), f2bf(sk.y), f2bf(sk.z), f2bf(sk.w)};
        *reinterpret_cast<bf16x4_t*>(dV + o) = bf16x4_t{f2bf(sv.x), f2bf(sv.y), f2bf(sv.z), f2bf(sv.w)};
    }
}

}  // namespace

bool backward_mfma_supported(const Dims& dm, bool in_bf16) {
    return in_bf16 && dm.h == HG && dm.d == D && (dm.S == 64 || dm.S == 128) && dm.k <= KMAX &&
           dm.C <= UWORDS * 32 && path_override(HSA_OP_BACKWARD) != HSA_PATH_GENERIC;
}

size_t backward_mfma_workspace(const Dims& dm) {
    if (dm.h != HG || dm.d != D) return 0;
    return ws_layout(dm).end;
}

hipError_t launch_backward_mfma(const Dims& dm, const void* Q, const void* K, const void* V,
                                const float* Kbar, const int32_t* idx, const float* w,
                                const void* dO, void* dQ, void* dK, void* dV, void* ws,
                                hipStream_t st) {
    const WsLayout l = ws_layout(dm);
    char* wsb = (char*)ws;
    float* ds = (float*)(wsb + l.ds);
    float* lse = (float*)(wsb + l.lse);
    float* dd = (float*)(wsb + l.dd);
    if (dm.S == 64) {
        constexpr int NW = QCfg<64>::NW;
        const int ntiles = cdiv(dm.L, 2 * NW);
        const int grid = 8 * cdiv(ntiles * dm.B * dm.G, 8);
        HSA_TIMED("bwd_q_mfma", st);
        hipLaunchKernelGGL((bwd_q_mfma<64>), dim3(grid), dim3(NW * 64), 0, st, dm,
                           (const __bf16*)Q, (const __bf16*)K, (const __bf16*)V, Kbar, idx, w,
                           (const __bf16*)dO, (__bf16*)dQ, ds, lse, dd, ntiles);
    } else {
        constexpr int NW = QCfg<128>::NW;
        const int ntiles = cdiv(dm.L, 2 * NW);
        const int grid = 8 * cdiv(ntiles * dm.B * dm.G, 8);
        HSA_TIMED("bwd_q_mfma", st);
        hipLaunchKernelGGL((bwd_q_mfma<128>), dim3(grid), dim3(NW * 64), 0, st, dm,
                           (const __bf16*)Q, (const __bf16*)K, (const __bf16*)V, Kbar, idx, w,
                           (const __bf16*)dO, (__bf16*)dQ, ds, lse, dd, ntiles);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // selection bitmap (shared with the generic path), then the key pass
    e = launch_selection_bitmap(dm, idx, (uint32_t*)(wsb + l.bitmap), st);
    if (e != hipSuccess) return e;
    const int nwords = cdiv(dm.L, 32);
    const int R = dm.B * dm.G * dm.C;
    int* cnt = (int*)(wsb + l.cnt);
    int* gstart = (int*)(wsb + l.gstart);
    int* plan = (int*)(wsb + l.plan);
    float* pk = (float*)(wsb + l.pk);
    float* pv = (float*)(wsb + l.pv);
    {
        HSA_TIMED("bwd_plan", st);
        if (R > 0)                       // no complete chunk: the plan is empty
            hipLaunchKernelGGL(stream_rowcount, dim3(cdiv(R, 4)), dim3(256), 0, st,
                               (const uint32_t*)(wsb + l.bitmap), R, nwords, dm.C, dm.S, cnt);
        hipLaunchKernelGGL(stream_plan, dim3(1), dim3(1024), 0, st, (const int*)cnt, R, kKvWGs,
                           gstart, plan);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (dm.S == 64) {
        HSA_TIMED("bwd_kv_mfma", st);
        hipLaunchKernelGGL((bwd_kv_mfma<64>), dim3(kKvWGs), dim3(256), 0, st, dm,
                           (const __bf16*)Q, (const __bf16*)K, (const __bf16*)V, idx, w,
                           (const __bf16*)dO, ds, lse, dd, (const uint32_t*)(wsb + l.bitmap),
                           nwords, (const int*)gstart, (const int*)cnt, (const int*)plan, pk, pv,
                           (__bf16*)dK, (__bf16*)dV);
    } else {
        HSA_TIMED("bwd_kv_mfma", st);
        hipLaunchKernelGGL((bwd_kv_mfma<128>), dim3(kKvWGs), dim3(512), 0, st, dm,
                           (const __bf16*)Q, (const __bf16*)K, (const __bf16*)V, idx, w,
                           (const __bf16*)dO, ds, lse, dd, (const uint32_t*)(wsb + l.bitmap),
                           nwords, (const int*)gstart, (const int*)cnt, (const int*)plan, pk, pv,
                           (__bf16*)dK, (__bf16*)dV);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 gf(dm.Call * dm.B * dm.G);
    HSA_TIMED("bwd_kv_finish", st);
    if (dm.S == 64)
        hipLaunchKernelGGL((bwd_kv_finish<64>), gf, dim3(256), 0, st, dm, (const int*)gstart,
                           (const int*)cnt, (const int*)plan, (const float*)pk, (const float*)pv,
                           (__bf16*)dK, (__bf16*)dV);
    else
        hipLaunchKernelGGL((bwd_kv_finish<128>), gf, dim3(256), 0, st, dm, (const int*)gstart,
                           (const int*)cnt, (const int*)plan, (const float*)pk, (const float*)pv,
                           (__bf16*)dK, (__bf16*)dV);
    return hipGetLastError();
}

}  // namespace hsa
