// Backward of hierarchical sparse attention in one chunk-major pass over the selected
// (token, chunk) pairs (Sec. 3.1.2: gradients of the chunk attention, of the chunk weights
// and, through them, of the landmark scores), for bf16 inputs with h = 8 query heads per KV
// head, d = 128 and S = 64.
//
// Work is counted in groups of 4 consecutive tokens of a chunk's selecting tokens (32 rows =
// 4 tokens x 8 heads).  A chunk's tokens come from the selection bitmap in increasing order.
// The groups of all (b, g, chunk) rows are laid end to end (row-major: slices, then chunks)
// and split into kStreamWGs equal ranges, one per workgroup, so a popular chunk (selected by
// thousands of tokens) is shared by several workgroups instead of setting the kernel time.
// A workgroup writes the key-side results of the chunks it covers entirely; for the first
// and last chunk of its range, when shared, it writes fp32 partial sums that bwd_finish adds
// in workgroup order.
//
// bwd_fused_mfma: 4 waves; wave w owns keys 16 w .. 16 w + 15 of the current chunk (K_sub,
// V_sub operands in registers, dK_sub, dV_sub [16 x 128] fp32 accumulators).  Per group:
//     Z [32 x 16] = Q_rows K_sub^T,  dP = dO_rows V_sub^T                 (MFMA)
//     each wave reduces its 16 keys per row (max m_w of the scaled logits, sum of
//     exp(z - m_w), sum of exp(z - m_w) dP); the four waves' values are exchanged through
//     LDS and combined into P = softmax over the chunk's 64 keys and D = sum_keys P dP
//     (= dO_row . O_{row,c})
//     dZ = W P (dP - D), W the token's weight for c (summed over slots repeating c)
//     dV_sub += (W P)^T dO_rows,  dK_sub += dZ^T Q_rows                   (MFMA, hi/lo)
//     dZ^T [64 keys x 32 rows] is staged in LDS; wave w forms the partial
//     dQ^T [d 32 w .. 32 w + 31 x 32 rows] = K_c^T dZ^T                     (MFMA, hi/lo)
//     and stores it (bf16) at the (token, slot, head) of the token's first slot holding c;
//     dw_{t,c} = sum over the token's heads of D is stored beside it.
// The partial dQ of a group is formed at the start of the next group's step, so a group
// needs two workgroup barriers (its stage landed / the previous dZ^T complete, and the
// statistics exchange).
//
// bwd_dq_reduce (token-major, one wave per (b, t, g)): ds_i = w_i (dw_i - sum_m w_m dw_m),
// dQ = beta * (sum of the token's partials) + alpha * sum_i ds_i Kbar_{c_i}, and the token's
// summed query q~ = sum_j q_j (stored as bf16) for the landmark term of dK.
//
// bwd_lmk_stream (same ranges): dKbar_c = alpha * sum_t ds_{t,c} q~_t, per chunk or partial,
// from the (token, slot) of each pair recorded by the fused pass.
// bwd_finish (per chunk): dK = beta dK_raw + dKbar_c / S (Kbar_c is the mean of the chunk's
// keys), dV; zeros for the trailing partial chunk.
//
// No atomics; every sum runs in a fixed order.
#include "chunk_stream.h"

namespace hsa {

hipError_t launch_selection_bitmap(const Dims& dm, const int32_t* idx, uint32_t* bm,
                                   hipStream_t st);

namespace {

constexpr int D = 128;
constexpr int HG = 8;
constexpr int KMAX = 32;
constexpr int FNST = 3;             // LDS stages of the group ring
constexpr int BPW = 8 / NW;         // 1 KB row blocks of Q (and of dO) copied per wave and group
constexpr int kStoresPerStep = 3;   // global stores per lane of one dq step (2 partial, 1 dw)

// target of the dw stores of padding rows (a group's missing tokens), so that every wave
// issues the same number of stores per group: 64 float pairs (their partial dQ rows go to the
// spare block after the partials)
constexpr size_t kTrashBytes = 64 * 8;

struct FusedWs {
    size_t bitmap, cnt, gstart, plan, pairsel, part, dkraw, dw, ds, qsum, pk, pv, pkb, dkbar, kmean,
        trash, end;
};
__host__ __device__ inline FusedWs fused_ws(const Dims& dm) {
    FusedWs l;
    const size_t nsel = (size_t)dm.B * dm.L * dm.G * dm.k;
    const size_t nrow = (size_t)dm.B * dm.L * dm.G;
    const size_t nwords = (size_t)((dm.L + 31) / 32);
    const size_t R = (size_t)dm.B * dm.G * dm.C;
    l.bitmap = 0;
    l.cnt = align256(R * nwords * 4);
    l.gstart = l.cnt + align256(R * 4);
    l.plan = l.gstart + align256((R + 1) * 4);
    // a pair's record in stream order, ((b L + t) G + g) * 32 + first slot holding the chunk:
    // 4 per group, at most one group per 4 selections plus one partial group per row
    l.pairsel = l.plan + 256;
    l.part = l.pairsel + align256((nsel + 4 * R) * 4);
    l.dkraw = l.part + align256((nsel + 1) * HG * D * 2);     // + the spare block
    l.dw = l.dkraw + align256(nrow * D * 4);
    // dw per (token, slot); off by one, per (token, slot, head) the pair {dw, sum_keys dZ}
    l.ds = l.dw + align256(nsel * 4 * (dm.off1 ? 2 * HG : 1));
    l.qsum = l.ds + align256(nsel * 4);
    l.pk = l.qsum + align256(nrow * D * 2);
    l.pv = l.pk + (size_t)kStreamWGs * 2 * CS * D * 4;
    l.pkb = l.pv + (size_t)kStreamWGs * 2 * CS * D * 4;
    l.dkbar = l.pkb + (size_t)kStreamWGs * 2 * D * 4;
    // the layer's own key means, for the off-by-one term of dQ when the backward is of the
    // attention alone (no landmarks are given then)
    l.kmean = l.dkbar + align256(R * D * 4);
    l.trash = l.kmean + align256(R * D * 4);
    l.end = l.trash + kTrashBytes;
    return l;
}

struct FStage {
    __bf16 q[32 * D];               // Q rows of a group (row 8 token + head), swizzled
    __bf16 g[32 * D];               // dO rows
};

struct SmemF {
    FStage st[FNST];                // stage 0 holds the chunk's K rows while K^T is read
    __bf16 dzt[2][CS * 32];         // dZ^T of a group, hi and lo parts: [key][row], see zpos
    float stat[NW][3][32];          // per wave and row: m_w, sum exp, sum exp * dP
    float fac[NW][3][32];           // per wave and row: P scale of the wave's keys, D, and
                                    // (off by one) the mean over the keys of dZ / W
    int list[FLIST];                // token; then its first Q / dO row, (b L + t) H + g h
    int lsel[FLIST];                // (token, first slot holding c): ((b L + t) G + g) k + s
    float lw[FLIST];                // the token's total weight for c
    int wtot[NW];
};

__global__ __launch_bounds__(NT, 2) void bwd_fused_mfma(
    Dims dm, const __bf16* __restrict__ Q, const __bf16* __restrict__ K,
    const __bf16* __restrict__ V, const int32_t* __restrict__ idx, const float* __restrict__ w,
    const __bf16* __restrict__ dO, const uint32_t* __restrict__ bm, int nwords,
    const int* __restrict__ gstart, const int* __restrict__ cntr, const int* __restrict__ plan,
    int* __restrict__ pairsel, uint16_t* __restrict__ part, float* __restrict__ dwc,
    float* __restrict__ dkraw,
    float* __restrict__ pk, float* __restrict__ pv, char* __restrict__ trash,
    __bf16* __restrict__ dV) {
    __shared__ SmemF sm;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int row = lane & 15, grp = lane >> 4;
    // consecutive ranges (the chunks of one slice) run on one XCD, so a token's Q / dO rows,
    // read once per chunk it selected, are shared through that XCD's L2
    const int lid = xcd_logical_id(kStreamWGs);
    if (lid < 0) return;
    const int R = dm.B * dm.G * dm.C;
    const int total = plan[0], T = plan[1];
    const int g0 = lid * T, g1 = min(g0 + T, total);
    if (g0 >= g1) return;
    const int k = dm.k;
    const size_t rowstride = (size_t)dm.G * D;
    const float beta = dm.beta;
    const float sl2 = beta * 1.44269504088896341f;
    const bool off1 = dm.off1 != 0;
    const float mfloor = off1 ? 0.f : -INFINITY;

    // LDS offsets of the chunk-swizzled tiles (see chunk_lds.h), from per-lane bases:
    //   row reads, d step ks:        kb0 + 32 (ks ^ ks_x)       (+ 2048 per 16-row block)
    //   transposed reads, block db:  tb0 + 16 (db ^ tr_x)       (+ 16 rows: + 16 D)
    const int swr = swz(row);
    const int kb0 = row * D + 8 * (grp ^ (swr & 3)), ks_x = swr >> 2;
    const int trr = 4 * grp + (row >> 2);
    const int tb0 = trr * D + 8 * (((row & 3) >> 1) ^ ((trr >> 3) & 1)) + 4 * (row & 1);
    const int tr_x = trr & 7;
    auto koff = [&](int ks) __attribute__((always_inline)) { return kb0 + 32 * (ks ^ ks_x); };
    auto toff = [&](int db) __attribute__((always_inline)) { return tb0 + 16 * (db ^ tr_x); };
    // transposed-read offsets of the dZ^T tile in the key order of the K^T fragments: lane
    // (grp, p) loads key kb + (p >> 2), rows 16 rt + 4 (p & 3) .. +3, kb = 32 ks2 + 16 hf +
    // 4 grp, at zpos(kb + (p >> 2), 4 rt + (p & 3)) = zb[rt] + 1024 ks2 + 512 hf (zsw of
    // those keys depends on grp only)
    int zb[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) zb[rt] = zpos(4 * grp + (row >> 2), 4 * rt + (row & 3));
    // a lane's partial-store address is pbase + 2 KB * block, block = the (token, slot) or,
    // for rows of missing tokens, tblk: the spare block after the partials
    char* const pbase = reinterpret_cast<char*>(part) + 2 * ((row & 7) * D + 32 * wave + 8 * grp);
    const uint32_t tblk = (uint32_t)((size_t)dm.B * dm.L * dm.G * dm.k);
    float* const tdw = reinterpret_cast<float*>(trash);

    for (int r = find_row(gstart, R, g0); r < R; ++r) {
        const int rs = gstart[r], re = gstart[r + 1];
        if (rs >= g1) break;
        if (re == rs) continue;
        const Segment sg = segment_of(rs, re, g0, g1);
        const int j0 = sg.j0, j1 = sg.j1, pslot = sg.pslot;
        const bool whole = sg.whole;
        const int c = r % dm.C;
        const int bg = r / dm.C, b = bg / dm.G, g = bg % dm.G;
        const size_t cbase = ((size_t)b * dm.L + (size_t)c * CS) * rowstride + (size_t)g * D;
        const int ntok = cntr[r];

        // ---- the chunk's operands: K_sub^T, V_sub^T (B operands of Z, dP) and K^T (A
        // operand of dQ^T: row m of tile dt is column 32 wave + 8 (m >> 2) + 4 dt + (m & 3) of
        // d, so a lane's C values of both tiles are 8 consecutive columns; keys of lane group
        // grp in step ks2: 32 ks2 + 4 grp + (0..3) and 32 ks2 + 16 + 4 grp + (0..3))
        __syncthreads();                          // the previous chunk's stages are read
        bf16x8_t kB[4], vB[4];
        const int key = 16 * wave + row;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            kB[ks] = ld_bf16x8(K + cbase + (size_t)key * rowstride + 32 * ks + 8 * grp);
            vB[ks] = ld_bf16x8(V + cbase + (size_t)key * rowstride + 32 * ks + 8 * grp);
        }
        chunk_to_lds<CS, NW>(K + cbase, rowstride, sm.st[0].q, wave, lane);
        wait_loads_le<0>();
        __syncthreads();
        bf16x8_t kT[2][2];
#pragma unroll
        for (int dt = 0; dt < 2; ++dt)
#pragma unroll
            for (int ks2 = 0; ks2 < 2; ++ks2) {
                const __bf16* p = sm.st[0].q + tr_perm_offset(lane, 32 * wave, dt) + 32 * ks2 * D;
                kT[dt][ks2] = cat(ld_tr16(p), ld_tr16(p + 16 * D));
            }
        f32x4_t aK[8], aV[8];
#pragma unroll
        for (int db = 0; db < 8; ++db) aK[db] = aV[db] = zero4();

        auto issue = [&](int gi, int nl, FStage& st) __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < BPW; ++i) {
                const int blk = wave * BPW + i;
                const int rr = blk * 4 + (lane >> 4);
                int li = gi * 4 + (rr >> 3);
                if (li >= nl) li = gi * 4;   // a missing token repeats the group's first (W = 0)
                const size_t o = ((size_t)(uint32_t)(sm.list[li] + (rr & 7)) << 7) +
                                 unit_pos(rr, lane & 15) * 8;
                lds_copy16(Q + o, __builtin_amdgcn_readfirstlane(lds_address(st.q + blk * 512)));
                lds_copy16(dO + o, __builtin_amdgcn_readfirstlane(lds_address(st.g + blk * 512)));
            }
        };

        // partial dQ^T of group gj from the staged dZ^T (all waves' keys), stored per (token,
        // slot, head): rows 16 rt + (lane & 15), d = 32 wave + 8 grp + (0..7); then
        // the group's dw (wave 0, carried from its combine step), off by one with the row's
        // sum of dZ over the keys (sig, times W here).  Exactly kStoresPerStep stores per
        // lane: rows of missing tokens go to the spare block and the trash area.
        auto dq_step = [&](int gj, int nl, float dtok, float sig) __attribute__((always_inline)) {
            f32x4_t qa[2][2];
#pragma unroll
            for (int dt = 0; dt < 2; ++dt) qa[dt][0] = qa[dt][1] = zero4();
            // both row tiles' operands of a step loaded first: four independent accumulators
            // between two products on one
#pragma unroll
            for (int ks2 = 0; ks2 < 2; ++ks2)
#pragma unroll
                for (int hl = 0; hl < 2; ++hl) {
                    bf16x8_t bz[2];
#pragma unroll
                    for (int rt = 0; rt < 2; ++rt) {
                        const __bf16* zp = sm.dzt[hl] + zb[rt] + 1024 * ks2;
                        bz[rt] = cat(ld_tr16(zp), ld_tr16(zp + 512));
                    }
#pragma unroll
                    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
                        for (int dt = 0; dt < 2; ++dt)
                            qa[dt][rt] = mfma16(kT[dt][ks2], bz[rt], qa[dt][rt]);
                }
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) {
                const int li = gj * 4 + 2 * rt + (row >> 3);
                const int so = li < nl ? sm.lsel[li] : -1;
                const uint32_t blk = so >= 0 ? (uint32_t)so : tblk;
                *reinterpret_cast<u32x4_t*>(pbase + ((size_t)blk << 11)) =
                    bfp_pack8(qa[0][rt], qa[1][rt]);
            }
            if (off1) {
                // lane (token, head) of wave 0: {dw, W sum_keys dZ} of that head's row
                const int li = gj * 4 + ((lane & 31) >> 3);
                const int so = (wave == 0 && lane < 32 && li < nl) ? sm.lsel[li] : -1;
                float2* dst = so >= 0 ? reinterpret_cast<float2*>(dwc) + (size_t)(uint32_t)so * HG +
                                            (lane & 7)
                                      : reinterpret_cast<float2*>(tdw) + lane;
                *dst = float2{dtok, so >= 0 ? sm.lw[li] * sig : 0.f};
            } else {
                const int li = gj * 4 + ((lane & 31) >> 3);
                const int so = (wave == 0 && lane < 32 && (lane & 7) == 0 && li < nl)
                                   ? sm.lsel[li] : -1;
                float* dst = so >= 0 ? dwc + (uint32_t)so : tdw + lane;
                *dst = dtok;
            }
        };

        const uint32_t* bmrow = bm + (size_t)r * nwords;
        const int wbeg = ((c + 1) * CS) >> 5;
        const int tend = min(4 * j1, ntok);
        for (int p0 = 4 * j0; p0 < tend; p0 += FLIST) {
            const int p1 = min(p0 + FLIST, tend);
            const int nl = p1 - p0;
            __syncthreads();                      // the list of the previous batch is read
            collect_tokens(bmrow, wbeg, nwords, p0, p1, sm.list, sm.wtot, tid);
            // per listed token: its first slot holding c (a set bit means there is one) and
            // its total weight for c.  All idx and w loads of a token are issued before use.
            for (int li = tid; li < nl; li += NT) {
                const int t = sm.list[li];
                const size_t so = (((size_t)b * dm.L + t) * dm.G + g) * k;
                int first = KMAX;
                float wsum = 0.f;
                for (int s0 = 0; s0 < k; s0 += 8) {
                    int cc[8];
                    float ww[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const bool in = s0 + j < k;
                        cc[j] = in ? idx[so + s0 + j] : -1;
                        ww[j] = in ? w[so + s0 + j] : 0.f;
                    }
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        if (cc[j] == c) {
                            first = min(first, s0 + j);
                            wsum += ww[j];
                        }
                }
                // -1: no slot holding c (not expected: the bitmap bit says there is one)
                sm.lsel[li] = first < k ? (int)(so + first) : -1;
                // the pair's record for the landmark term: its q~ row times 32 plus its slot
                pairsel[4 * (size_t)rs + p0 + li] =
                    first < k ? (int)((((size_t)b * dm.L + t) * dm.G + g) * 32 + first) : -1;
                sm.lw[li] = first < k ? wsum : 0.f;
                sm.list[li] = (int)(((size_t)b * dm.L + t) * dm.H + (size_t)g * HG);
            }
            __syncthreads();
            const int ngroups = (nl + 3) / 4;
#pragma unroll
            for (int u = 0; u < FNST - 1; ++u)
                if (u < ngroups) issue(u, nl, sm.st[u]);
            float dtok_pend = 0.f, sig_pend = 0.f;
            // one group's step; its stage index SI = gi % FNST is a constant (the loop below
            // is unrolled by FNST), so the stage's LDS addresses are lane bases plus immediates
            auto group = [&](int gi, auto si) __attribute__((always_inline)) {
                constexpr int SI = decltype(si)::value;
                // Group gi has landed once only the memory operations issued after its copies
                // remain: the previous iteration's dq stores (when it ran one) and the next
                // group's copies (when there is a next group).  Loads and stores complete in
                // issue order.
                const bool more = gi + 1 < ngroups, stored = gi >= 2;
                if (more && stored) wait_loads_le<2 * BPW + kStoresPerStep>();
                else if (more) wait_loads_le<2 * BPW>();
                else if (stored) wait_loads_le<kStoresPerStep>();
                else wait_loads_le<0>();
                lds_wait();
                barrier_keep_copies();   // stage gi landed, dZ^T of gi - 1 complete, stage gi - 1 free
                if (gi > 0) dq_step(gi - 1, nl, dtok_pend, sig_pend);
                if (gi + FNST - 1 < ngroups) issue(gi + FNST - 1, nl, sm.st[(SI + FNST - 1) % FNST]);
                const FStage& st = sm.st[SI];

                // ---- Z, dP for the wave's 16 keys (rows 16 rb + 4 grp + i, key 16 wave + row) --
                f32x4_t z[2], dp[2];
                z[0] = z[1] = dp[0] = dp[1] = zero4();
    #pragma unroll
                for (int ks = 0; ks < 4; ++ks)
    #pragma unroll
                    for (int rb = 0; rb < 2; ++rb) {
                        z[rb] = mfma16(ld_bf16x8(st.q + koff(ks) + rb * 2048), kB[ks], z[rb]);
                        dp[rb] = mfma16(ld_bf16x8(st.g + koff(ks) + rb * 2048), vB[ks], dp[rb]);
                    }
                // ---- the wave's row statistics over its 16 keys, to LDS ------------------------
                f32x4_t e[2];
                float zl8[8], e8[8], m8[8];
    #pragma unroll
                for (int i = 0; i < 8; ++i) zl8[i] = z[i >> 2][i & 3] * sl2;
                rows16_exp(zl8, e8, m8);
    #pragma unroll
                for (int rb = 0; rb < 2; ++rb) {
                    f32x4_t sm_m, sm_l, sm_n;
    #pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float ev = e8[4 * rb + i];
                        e[rb][i] = ev;
                        sm_m[i] = m8[4 * rb + i];
                        sm_l[i] = group_sum<16>(ev);
                        sm_n[i] = group_sum<16>(ev * dp[rb][i]);
                        // complete in every lane before the branch below (otherwise the last
                        // DPP step is sunk into it and can no longer fuse with its add)
                        asm volatile("" : "+v"(sm_l[i]), "+v"(sm_n[i]));
                    }
                    if (row == 0) {
                        *reinterpret_cast<f32x4_t*>(&sm.stat[wave][0][16 * rb + 4 * grp]) = sm_m;
                        *reinterpret_cast<f32x4_t*>(&sm.stat[wave][1][16 * rb + 4 * grp]) = sm_l;
                        *reinterpret_cast<f32x4_t*>(&sm.stat[wave][2][16 * rb + 4 * grp]) = sm_n;
                    }
                }
                lds_wait();
                barrier_keep_copies();   // every wave's statistics of group gi written
                // ---- combine: lane r (and r + 32) handles row r = lane & 31 --------------------
                const int r32 = lane & 31;
                float mv[NW], lv[NW], nv[NW];
    #pragma unroll
                for (int w2 = 0; w2 < NW; ++w2) {
                    mv[w2] = sm.stat[w2][0][r32];
                    lv[w2] = sm.stat[w2][1][r32];
                    nv[w2] = sm.stat[w2][2][r32];
                }
                // off by one, the extra logit 0 joins the maximum and the sum (its value,
                // and so its share of D, is zero)
                const float M = fmaxf(fmaxf(fmaxf(mv[0], mv[1]), fmaxf(mv[2], mv[3])), mfloor);
                float lsum = off1 ? fast_exp2(-M) : 0.f, nsum = 0.f, aown = 0.f;
    #pragma unroll
                for (int w2 = 0; w2 < NW; ++w2) {
                    const float a = fast_exp2(mv[w2] - M);
                    lsum = fmaf(a, lv[w2], lsum);
                    nsum = fmaf(a, nv[w2], nsum);
                    aown = (w2 == wave) ? a : aown;
                }
                const float inv = __builtin_amdgcn_rcpf(lsum);
                const float Drow = nsum * inv;
                // off by one, a row's dZ sums over the keys to W D P0 (P0: the extra logit's
                // probability) instead of 0
                const float dzsum = off1 ? Drow * fast_exp2(-M) * inv : 0.f;
                if (lane < 32) {
                    sm.fac[wave][0][r32] = aown * inv;
                    sm.fac[wave][1][r32] = Drow;
                    sm.fac[wave][2][r32] = dzsum * (1.f / CS);
                }
                // dw of each token of the group: sum of D over its 8 heads (rows 8 tau .. 8 tau + 7),
                // stored with the group's partial dQ
                dtok_pend = group_sum<8>(Drow);
                sig_pend = dzsum;
                // back in the C layout (the wave's own LDS writes, read in order)
                f32x4_t fv[2], dv[2], pw[2], dz[2];
    #pragma unroll
                for (int rb = 0; rb < 2; ++rb) {
                    fv[rb] = *reinterpret_cast<const f32x4_t*>(&sm.fac[wave][0][16 * rb + 4 * grp]);
                    dv[rb] = *reinterpret_cast<const f32x4_t*>(&sm.fac[wave][1][16 * rb + 4 * grp]);
                }
    #pragma unroll
                for (int rb = 0; rb < 2; ++rb) {
                    const int li = gi * 4 + 2 * rb + (grp >> 1);
                    const float wt = li < nl ? sm.lw[li] : 0.f;
    #pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float p = e[rb][i] * fv[rb][i];
                        pw[rb][i] = wt * p;
                        dz[rb][i] = wt * p * (dp[rb][i] - dv[rb][i]);
                    }
                }
                // every product below accumulates over many rows (dV, dK) or cancels (dQ, since
                // sum_keys dZ = 0): W P and dZ enter as bf16 hi/lo pairs.  Off by one, dZ^T for
                // dQ is centred over the keys (its mean W D P0 / S taken out, so the partial
                // keeps cancelling; dQ completion adds W D P0 Kbar_c back in fp32), while dK
                // takes dZ itself.
                bf16x8_t pvh, pvl, dzh, dzl;
                split8(pw[0], pw[1], pvh, pvl);
                auto centre = [&](float sgn) __attribute__((always_inline)) {
    #pragma unroll
                    for (int rb = 0; rb < 2; ++rb) {
                        const int li = gi * 4 + 2 * rb + (grp >> 1);
                        const float wt = li < nl ? sgn * sm.lw[li] : 0.f;
                        const f32x4_t cv =
                            *reinterpret_cast<const f32x4_t*>(&sm.fac[wave][2][16 * rb + 4 * grp]);
    #pragma unroll
                        for (int i = 0; i < 4; ++i) dz[rb][i] = fmaf(wt, cv[i], dz[rb][i]);
                    }
                };
                if (off1) centre(-1.f);
                split8(dz[0], dz[1], dzh, dzl);
                {
                    // dZ^T to LDS: key 16 wave + row, rows 16 rb + 4 grp .. +3 = unit 4 rb + grp
                    const int j = 16 * wave + row;
                    *reinterpret_cast<bf16x4_t*>(sm.dzt[0] + zpos(j, grp)) =
                        bf16x4_t{dzh[0], dzh[1], dzh[2], dzh[3]};
                    *reinterpret_cast<bf16x4_t*>(sm.dzt[0] + zpos(j, 4 + grp)) =
                        bf16x4_t{dzh[4], dzh[5], dzh[6], dzh[7]};
                    *reinterpret_cast<bf16x4_t*>(sm.dzt[1] + zpos(j, grp)) =
                        bf16x4_t{dzl[0], dzl[1], dzl[2], dzl[3]};
                    *reinterpret_cast<bf16x4_t*>(sm.dzt[1] + zpos(j, 4 + grp)) =
                        bf16x4_t{dzl[4], dzl[5], dzl[6], dzl[7]};
                }
                if (off1) {
                    centre(1.f);
                    split8(dz[0], dz[1], dzh, dzl);
                }
    #pragma unroll
                for (int db = 0; db < 8; ++db) {
                    const int to = toff(db);
                    const bf16x8_t gb = cat(ld_tr16(st.g + to), ld_tr16(st.g + to + 16 * D));
                    aV[db] = mfma16(pvh, gb, aV[db]);
                    aV[db] = mfma16(pvl, gb, aV[db]);
                    const bf16x8_t qb = cat(ld_tr16(st.q + to), ld_tr16(st.q + to + 16 * D));
                    aK[db] = mfma16(dzh, qb, aK[db]);
                    aK[db] = mfma16(dzl, qb, aK[db]);
                }
            };
            static_assert(FNST == 3, "the group loop is unrolled by the ring depth");
            for (int gb = 0; gb < ngroups; gb += FNST) {
                group(gb, IntC<0>{});
                if (gb + 1 < ngroups) group(gb + 1, IntC<1>{});
                if (gb + 2 < ngroups) group(gb + 2, IntC<2>{});
            }
            lds_wait();
            barrier_keep_copies();   // dZ^T of the batch's last group complete
            dq_step(ngroups - 1, nl, dtok_pend, sig_pend);
        }
        // the chunk's key-side sums: final when this workgroup covered all its groups
        float* ok = whole ? dkraw : pk + ((size_t)lid * 2 + pslot) * CS * D;
        float* ov = pv + ((size_t)lid * 2 + pslot) * CS * D;
#pragma unroll
        for (int db = 0; db < 8; ++db) {
            const int d = 16 * db + row;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int kr = 16 * wave + 4 * grp + i;
                if (whole) {
                    const size_t o = cbase + (size_t)kr * rowstride + d;
                    ok[o] = beta * aK[db][i];
                    dV[o] = f2bf(aV[db][i]);
                } else {
                    ok[kr * D + d] = beta * aK[db][i];
                    ov[kr * D + d] = aV[db][i];
                }
            }
        }
    }
}

// Token-major completion of dQ (one wave per (b, t, g); lane: head lane >> 3, columns
// 16 (lane & 7) .. +15).  A slot counts when 0 <= c < floor(t / S); a slot repeating an
// earlier slot's chunk shares that slot's partial (already weighted by the sum of their
// weights) and its dw.  OFF1: the softmax off by one (the partials leave out a per-head
// Kbar_c term, added here); a separate instantiation, so that the plain softmax's kernel
// holds no per-slot key means in registers.
template <bool OFF1>
__global__ __launch_bounds__(256) void bwd_dq_reduce(
    Dims dm, const __bf16* __restrict__ Q, const float* __restrict__ Kbar,
    const int32_t* __restrict__ idx, const float* __restrict__ w,
    const uint16_t* __restrict__ part, const float* __restrict__ dwc, __bf16* __restrict__ dQ,
    float* __restrict__ ds, __bf16* __restrict__ qsum) {
    const int lane = threadIdx.x & 63;
    const size_t item = (size_t)blockIdx.x * 4 + (threadIdx.x >> 6);    // ((b L) + t) G + g
    if (item >= (size_t)dm.B * dm.L * dm.G) return;
    const int g = (int)(item % dm.G);
    const size_t bt = item / dm.G;
    const int t = (int)(bt % dm.L);
    const int b = (int)(bt / dm.L);
    const int k = dm.k;
    const size_t so = item * k;
    const int ncand = t / dm.S;
    const int head = lane >> 3, c0 = 16 * (lane & 7);

    // this lane's view of the token's query rows, for q~ (issued first)
    const __bf16* qrow = Q + ((bt * dm.H) + (size_t)g * HG + head) * D + c0;
    const bf16x8_t q0 = ld_bf16x8(qrow), q1 = ld_bf16x8(qrow + 8);

    int cl = -1;
    float wl = 0.f, dwl = 0.f;
    if (lane < k) {
        cl = idx[so + lane];
        wl = w[so + lane];
        dwl = OFF1 ? dwc[(so + lane) * (2 * HG)] : dwc[so + lane];
    }
    const bool valid = lane < k && cl >= 0 && cl < ncand;
    int canon = lane;                       // first slot holding the same chunk
    for (int s = 0; s < k; ++s) {
        const int cs = __builtin_amdgcn_readlane(cl, s);
        if (s < canon && cs == cl) canon = s;
    }
    const float dws = __shfl(dwl, canon, 64);
    const float wd = valid ? wl * dws : 0.f;
    const bool attn_only = dm.dwo != nullptr;
    float dsl;
    if (attn_only) {
        // attention alone: every slot holding a chunk gets the chunk's dw; no score term
        if (lane < k) {
            float* o = dm.dwo + so + lane;
            const float v = valid ? dws : 0.f;
            *o = dm.dwacc ? *o + v : v;
        }
        dsl = 0.f;
    } else if (dm.stick) {
        // stick-breaking: b = w / (1 - weight of the earlier valid slots), and
        // ds = (1 - b) w dw - b (sum of w dw over the later valid slots)
        float before = 0.f, tail = 0.f;
        const float wv = valid ? wl : 0.f;
        for (int s = 0; s < k; ++s) {
            const float ws = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wv), s));
            const float wds = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wd), s));
            if (s < lane) before += ws;
            if (s > lane) tail += wds;
        }
        const float u = 1.f - before;
        const float bs = u > 0.f ? wl / u : 0.f;
        dsl = valid ? (1.f - bs) * wd - bs * tail : 0.f;
    } else {
        const float wdw = group_sum<64>(wd);
        dsl = valid ? wl * (dws - wdw) : 0.f;
    }
    // ds summed over the slots holding the same chunk, at the first of them (the landmark
    // term of dK reads it there), in slot order
    float dsm = 0.f;
    for (int s = 0; s < k; ++s) {
        const int cs = __builtin_amdgcn_readlane(canon, s);
        const int vs = __builtin_amdgcn_readlane((int)valid, s);
        const float d2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(dsl), s));
        if (vs && cs == lane) dsm += d2;
    }
    if (lane < k) ds[so + lane] = dsm;
    const int own = (valid && canon == lane) ? 1 : 0;

    float acc[16], lmk[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = lmk[i] = 0.f;
    const size_t kbbase = (size_t)b * dm.C * dm.G + g;
    // All loads of J slots are issued before their first use, with no branch between them
    // (a slot past k reads slot k - 1's data, a slot that does not own its chunk reads its
    // own stale partial); what is not used is dropped by a select on the partial's scale.
    // Slot values are wave-uniform (lane reads), so the remaining branches are scalar.
    if constexpr (!OFF1) {
        // the landmark term sum_i ds_i Kbar_{c_i} is the same for every head: lane (head j)
        // takes the slots j, j + 8, ..., and the 8 lanes of a column block sum their parts
        // (its loads follow the first partial loads)
        const bool need_kb = ncand > 0 && !attn_only;
        auto landmark = [&]() __attribute__((always_inline)) {
            for (int m = 0; m * HG < k; ++m) {
                const int s = head + HG * m;
                const int cs = __shfl(cl, min(s, k - 1), 64);
                const float coef = s < k ? __shfl(dsl, min(s, k - 1), 64) : 0.f;
                const int cc = (cs >= 0 && cs < ncand) ? cs : 0;
                const float* kb = Kbar + (kbbase + (size_t)cc * dm.G) * D + c0;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const float4 x = *reinterpret_cast<const float4*>(kb + 4 * v);
                    lmk[4 * v + 0] = fmaf(coef, x.x, lmk[4 * v + 0]);
                    lmk[4 * v + 1] = fmaf(coef, x.y, lmk[4 * v + 1]);
                    lmk[4 * v + 2] = fmaf(coef, x.z, lmk[4 * v + 2]);
                    lmk[4 * v + 3] = fmaf(coef, x.w, lmk[4 * v + 3]);
                }
            }
        };
        constexpr int J = 4;
        for (int s0 = 0; s0 < k; s0 += J) {
            u32x4_t pv[J][2];
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const int s = min(s0 + j, k - 1);
                const uint16_t* pp = part + ((so + s) * HG + head) * D + c0;
                pv[j][0] = *reinterpret_cast<const u32x4_t*>(pp);
                pv[j][1] = *reinterpret_cast<const u32x4_t*>(pp + 8);
            }
            if (s0 == 0 && need_kb) landmark();
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const int s = s0 + j;
                const bool use = s < k && __builtin_amdgcn_readlane(own, min(s, k - 1)) != 0;
                bfp_accum8(pv[j][0], acc, use);
                bfp_accum8(pv[j][1], acc + 8, use);
            }
        }
        if (need_kb) {
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float v = lmk[i] + dpp_mov<0x128>(lmk[i]);   // row_ror:8 = lane ^ 8
                lmk[i] = pair32_sum(pair16_sum(v));
            }
        }
    } else {
        // off by one: per slot the key mean serves the landmark term and the head's
        // W sum_keys dZ term, whose Kbar_c part the partial left out (given the attention
        // alone, the launcher passes the layer's key means)
        const bool need_kb = ncand > 0;
        for (int s0 = 0; s0 < k; s0 += 4) {
            u32x4_t pv[4][2];
            float4 kv[4][4];
            float sgv[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                sgv[j] = dwc[((so + min(s0 + j, k - 1)) * HG + head) * 2 + 1];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int s = min(s0 + j, k - 1);
                const uint16_t* pp = part + ((so + s) * HG + head) * D + c0;
                pv[j][0] = *reinterpret_cast<const u32x4_t*>(pp);
                pv[j][1] = *reinterpret_cast<const u32x4_t*>(pp + 8);
            }
            if (need_kb) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int cs = __builtin_amdgcn_readlane(cl, min(s0 + j, k - 1));
                    const int cc = (cs >= 0 && cs < ncand) ? cs : 0;
                    const float* kb = Kbar + (kbbase + (size_t)cc * dm.G) * D + c0;
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        kv[j][v] = *reinterpret_cast<const float4*>(kb + 4 * v);
                }
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int s = s0 + j;
                const bool use = s < k && __builtin_amdgcn_readlane(own, min(s, k - 1)) != 0;
                bfp_accum8(pv[j][0], acc, use);
                bfp_accum8(pv[j][1], acc + 8, use);
                if (!need_kb) continue;
                const float coef =
                    s < k ? __int_as_float(__builtin_amdgcn_readlane(__float_as_int(dsl), s))
                          : 0.f;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    lmk[4 * v + 0] = fmaf(coef, kv[j][v].x, lmk[4 * v + 0]);
                    lmk[4 * v + 1] = fmaf(coef, kv[j][v].y, lmk[4 * v + 1]);
                    lmk[4 * v + 2] = fmaf(coef, kv[j][v].z, lmk[4 * v + 2]);
                    lmk[4 * v + 3] = fmaf(coef, kv[j][v].w, lmk[4 * v + 3]);
                }
                const float sg = use ? sgv[j] : 0.f;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    acc[4 * v + 0] = fmaf(sg, kv[j][v].x, acc[4 * v + 0]);
                    acc[4 * v + 1] = fmaf(sg, kv[j][v].y, acc[4 * v + 1]);
                    acc[4 * v + 2] = fmaf(sg, kv[j][v].z, acc[4 * v + 2]);
                    acc[4 * v + 3] = fmaf(sg, kv[j][v].w, acc[4 * v + 3]);
                }
            }
        }
    }
    bf16x8_t o0, o1;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        o0[i] = f2bf(fmaf(dm.beta, acc[i], dm.alpha * lmk[i]));
        o1[i] = f2bf(fmaf(dm.beta, acc[8 + i], dm.alpha * lmk[8 + i]));
    }
    __bf16* op = dQ + ((bt * dm.H) + (size_t)g * HG + head) * D + c0;
    *reinterpret_cast<bf16x8_t*>(op) = o0;
    *reinterpret_cast<bf16x8_t*>(op + 8) = o1;

    if (attn_only) return;              // q~ only serves the landmark term
    // q~ = sum over the group's heads (lanes with the same column block): rows of 16 lanes
    // pair heads 2m, 2m + 1 (lane ^ 8), then across rows (lane ^ 16, lane ^ 32)
    float qs[16];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        qs[i] = (float)q0[i];
        qs[8 + i] = (float)q1[i];
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        float v = qs[i] + dpp_mov<0x128>(qs[i]);      // row_ror:8 = lane ^ 8 within 16
        v = pair16_sum(v);
        qs[i] = pair32_sum(v);
    }
    if (lane < 8) {                               // stored as bf16 (the landmark term's input)
        __bf16* qd = qsum + item * D + c0;
        bf16x8_t a, b2;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            a[i] = f2bf(qs[i]);
            b2[i] = f2bf(qs[8 + i]);
        }
        *reinterpret_cast<bf16x8_t*>(qd) = a;
        *reinterpret_cast<bf16x8_t*>(qd + 8) = b2;
    }
}


// Landmark term of dK over the same ranges as bwd_fused_mfma: per pair (in stream order, as
// the fused pass recorded it) the token's ds summed over its slots holding the chunk, times
// the token's q~; dKbar_c = alpha * sum over pairs, in 8 interleaved pair streams (lane group
// j = tid / 32 takes every 8th pair, lane 4 columns) summed in a fixed order; per chunk when
// the range covers all its groups, else as the range's partial.
__global__ __launch_bounds__(NT) void bwd_lmk_stream(
    Dims dm, const int* __restrict__ pairsel, const float* __restrict__ dsm,
    const __bf16* __restrict__ qsum, const int* __restrict__ gstart, const int* __restrict__ cntr,
    const int* __restrict__ plan, float* __restrict__ dkbar, float* __restrict__ pkb) {
    constexpr int U = 4;                      // pairs per lane group in flight
    constexpr int SEG = 2048;                 // pair records staged in LDS at once
    __shared__ float4 red[8][32];
    __shared__ int sels[SEG];
    const int tid = threadIdx.x;
    const int lid = xcd_logical_id(kStreamWGs);
    if (lid < 0) return;
    const int R = dm.B * dm.G * dm.C;
    const int total = plan[0], T = plan[1];
    const int g0 = lid * T, g1 = min(g0 + T, total);
    if (g0 >= g1) return;
    const int k = dm.k;
    const int j8 = tid >> 5, c4 = tid & 31;
    for (int r = find_row(gstart, R, g0); r < R; ++r) {
        const int rs = gstart[r], re = gstart[r + 1];
        if (rs >= g1) break;
        if (re == rs) continue;
        const Segment sg = segment_of(rs, re, g0, g1);
        const int j0 = sg.j0, j1 = sg.j1, pslot = sg.pslot;
        const bool whole = sg.whole;
        const int* ps = pairsel + 4 * (size_t)rs;
        const int pend = min(4 * j1, cntr[r]);
        float4 acc{0.f, 0.f, 0.f, 0.f};
        for (int q0 = 4 * j0; q0 < pend; q0 += SEG) {
            // the segment's pair records, one coalesced load, then U pairs per lane group in
            // flight; positions past the chunk's last token add 0
            const int qn = min(SEG, pend - q0);
            __syncthreads();                      // sels of the previous segment are read
            for (int i = tid; i < qn; i += NT) sels[i] = ps[q0 + i];
            __syncthreads();
            for (int p = j8; p < qn; p += 8 * U) {
                float cf[U];
                float4 q[U];
                // positions past the segment's end load the segment's last record (a real
                // row, so no address is shared by every workgroup) and add 0
                bool live[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int pu = p + 8 * u;
                    const int sel = sels[min(pu, qn - 1)];
                    live[u] = pu < qn && sel >= 0;
                    const int su = max(sel, 0);
                    const int qr = su >> 5;                      // the token's q~ row
                    cf[u] = dsm[(size_t)qr * k + (su & 31)];
                    const bf16x4_t qv = ld_bf16x4(qsum + (size_t)qr * D + 4 * c4);
                    q[u] = float4{(float)qv[0], (float)qv[1], (float)qv[2], (float)qv[3]};
                }
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const float c = live[u] ? cf[u] : 0.f;
                    acc.x = fmaf(c, q[u].x, acc.x);
                    acc.y = fmaf(c, q[u].y, acc.y);
                    acc.z = fmaf(c, q[u].z, acc.z);
                    acc.w = fmaf(c, q[u].w, acc.w);
                }
            }
        }
        red[j8][c4] = acc;
        __syncthreads();
        if (tid < 32) {
            float4 s = red[0][tid];
#pragma unroll
            for (int j = 1; j < 8; ++j) {
                s.x += red[j][tid].x;
                s.y += red[j][tid].y;
                s.z += red[j][tid].z;
                s.w += red[j][tid].w;
            }
            const float a = dm.alpha;
            float* out = whole ? dkbar + (size_t)r * D : pkb + ((size_t)lid * 2 + pslot) * D;
            *reinterpret_cast<float4*>(out + 4 * tid) = float4{s.x * a, s.y * a, s.z * a, s.w * a};
        }
        __syncthreads();                          // red is rewritten for the next chunk
    }
}

// Per chunk (b, g, c): dV and dK = beta dK_raw + dKbar_c / S from the chunk's own sums (one
// workgroup covered it) or from the partials of the workgroups that shared it, added in
// workgroup order; zeros for chunks nobody selected and for the trailing partial chunk.
__global__ __launch_bounds__(NT) void bwd_finish(
    Dims dm, const int* __restrict__ gstart, const int* __restrict__ cntr,
    const int* __restrict__ plan, const float* __restrict__ dkraw, const float* __restrict__ pk,
    const float* __restrict__ pv, const float* __restrict__ dkbar, const float* __restrict__ pkb,
    __bf16* __restrict__ dK, __bf16* __restrict__ dV) {
    __shared__ float4 lm[32];
    const int tid = threadIdx.x;
    const int c = blockIdx.x % dm.Call;
    const int bg = blockIdx.x / dm.Call, b = bg / dm.G, g = bg % dm.G;
    const size_t rowstride = (size_t)dm.G * D;
    const size_t cbase = ((size_t)b * dm.L + (size_t)c * CS) * rowstride + (size_t)g * D;
    const bf16x4_t z4{__bf16(0.f), __bf16(0.f), __bf16(0.f), __bf16(0.f)};
    const int r = bg * dm.C + c;
    if (c >= dm.C || cntr[r] == 0) {            // trailing partial chunk, or never selected
        const int rows = min(CS, dm.L - c * CS);
        for (int e = tid; e < rows * 32; e += NT) {
            const size_t o = cbase + (size_t)(e >> 5) * rowstride + 4 * (e & 31);
            *reinterpret_cast<bf16x4_t*>(dK + o) = z4;
            *reinterpret_cast<bf16x4_t*>(dV + o) = z4;
        }
        return;
    }
    const int T = plan[1];
    const int rs = gstart[r], re = gstart[r + 1];
    const int wf = rs / T, wl = (re - 1) / T;
    const float invS = 1.f / (float)CS;
    constexpr int PER = CS * 32 / NT;          // float4 columns per thread
    float4 sk[PER];
    if (wf == wl) {                             // one workgroup covered the chunk: its dK_raw
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int e = tid + u * NT;
            sk[u] = *reinterpret_cast<const float4*>(dkraw + cbase + (size_t)(e >> 5) * rowstride +
                                                     4 * (e & 31));
        }
    }
    if (tid < 32) {
        float4 s{0.f, 0.f, 0.f, 0.f};
        if (dm.dwo != nullptr) {
            // attention alone: no landmark term
        } else if (wf == wl) {
            s = *reinterpret_cast<const float4*>(dkbar + (size_t)r * D + 4 * tid);
        } else {
            for (int wg = wf; wg <= wl; ++wg) {
                const int sl = (wg > wf || rs == wf * T) ? 0 : 1;
                const float4 v = *reinterpret_cast<const float4*>(pkb + ((size_t)wg * 2 + sl) * D + 4 * tid);
                s.x += v.x;
                s.y += v.y;
                s.z += v.z;
                s.w += v.w;
            }
        }
        lm[tid] = float4{s.x * invS, s.y * invS, s.z * invS, s.w * invS};
    }
    __syncthreads();
    if (wf == wl) {
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int e = tid + u * NT;
            const float4 l4 = lm[e & 31];
            *reinterpret_cast<bf16x4_t*>(dK + cbase + (size_t)(e >> 5) * rowstride + 4 * (e & 31)) =
                bf16x4_t{f2bf(sk[u].x + l4.x), f2bf(sk[u].y + l4.y), f2bf(sk[u].z + l4.z),
                         f2bf(sk[u].w + l4.w)};
        }
        return;
    }
    float4 sv[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) sk[u] = sv[u] = float4{0.f, 0.f, 0.f, 0.f};
    for (int wg = wf; wg <= wl; ++wg) {
        const int sl = (wg > wf || rs == wf * T) ? 0 : 1;
        const size_t pb = ((size_t)wg * 2 + sl) * CS * D;
        float4 a[PER], v[PER];
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int e = tid + u * NT;
            a[u] = *reinterpret_cast<const float4*>(pk + pb + 4 * e);
            v[u] = *reinterpret_cast<const float4*>(pv + pb + 4 * e);
        }
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            sk[u].x += a[u].x; sk[u].y += a[u].y; sk[u].z += a[u].z; sk[u].w += a[u].w;
            sv[u].x += v[u].x; sv[u].y += v[u].y; sv[u].z += v[u].z; sv[u].w += v[u].w;
        }
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        const int e = tid + u * NT;
        const size_t o = cbase + (size_t)(e >> 5) * rowstride + 4 * (e & 31);
        const float4 l4 = lm[e & 31];
        *reinterpret_cast<bf16x4_t*>(dV + o) =
            bf16x4_t{f2bf(sv[u].x), f2bf(sv[u].y), f2bf(sv[u].z), f2bf(sv[u].w)};
        *reinterpret_cast<bf16x4_t*>(dK + o) =
            bf16x4_t{f2bf(sk[u].x + l4.x), f2bf(sk[u].y + l4.y), f2bf(sk[u].z + l4.z),
                     f2bf(sk[u].w + l4.w)};
    }
}

}  // namespace

// Row and (token, slot) indices of this path are 32-bit: B L G < 2^26.  The default for its
// shapes (4K tokens: 1.52 ms against 1.68 for the two-pass kernels; 64K: 3.62 against 5.62);
// HSA_PATH_TWO_PASS selects the two-pass kernels instead.
bool backward_fused_supported(const Dims& dm, bool in_bf16) {
    const int path = path_override(HSA_OP_BACKWARD);
    return in_bf16 && dm.h == HG && dm.d == D && dm.S == CS && dm.k <= KMAX &&
           (size_t)dm.B * dm.L * dm.G < ((size_t)1 << 26) &&
           (path == HSA_PATH_FUSED || path == HSA_PATH_AUTO);
}

size_t backward_fused_workspace(const Dims& dm) {
    if (dm.h != HG || dm.d != D || dm.S != CS) return 0;
    return fused_ws(dm).end;
}

hipError_t launch_backward_fused(const Dims& dm, const void* Q, const void* K, const void* V,
                                 const float* Kbar, const int32_t* idx, const float* w,
                                 const void* dO, void* dQ, void* dK, void* dV, void* ws,
                                 hipStream_t st) {
    const FusedWs l = fused_ws(dm);
    char* wsb = (char*)ws;
    uint32_t* bmp = (uint32_t*)(wsb + l.bitmap);
    int* cnt = (int*)(wsb + l.cnt);
    int* gstart = (int*)(wsb + l.gstart);
    int* plan = (int*)(wsb + l.plan);
    int* pairsel = (int*)(wsb + l.pairsel);
    uint16_t* part = (uint16_t*)(wsb + l.part);
    float* dkraw = (float*)(wsb + l.dkraw);
    float* dwc = (float*)(wsb + l.dw);
    float* dsb = (float*)(wsb + l.ds);
    __bf16* qs = (__bf16*)(wsb + l.qsum);
    float* pk = (float*)(wsb + l.pk);
    float* pv = (float*)(wsb + l.pv);
    float* pkb = (float*)(wsb + l.pkb);
    float* dkbar = (float*)(wsb + l.dkbar);
    const int R = dm.B * dm.G * dm.C;
    const int nwords = cdiv(dm.L, 32);
    hipError_t e = launch_selection_bitmap(dm, idx, bmp, st);
    if (e != hipSuccess) return e;
    if (dm.dwo != nullptr && dm.off1 && dm.C > 0) {
        float* km = (float*)(wsb + l.kmean);
        e = launch_landmarks(dm, true, K, km, false, 0, dm.C, st);
        if (e != hipSuccess) return e;
        Kbar = km;
    }
    if (R > 0) {
        {
            HSA_TIMED("bwd_plan", st);
            hipLaunchKernelGGL(stream_rowcount, dim3(cdiv(R, 4)), dim3(256), 0, st,
                               (const uint32_t*)bmp, R, nwords, dm.C, dm.S, cnt);
            hipLaunchKernelGGL(stream_plan, dim3(1), dim3(1024), 0, st, (const int*)cnt, R,
                               kStreamWGs, gstart, plan);
        }
        HSA_TIMED("bwd_fused_mfma", st);
        hipLaunchKernelGGL(bwd_fused_mfma, dim3(kStreamWGs), dim3(NT), 0, st, dm,
                           (const __bf16*)Q, (const __bf16*)K, (const __bf16*)V, idx, w,
                           (const __bf16*)dO, (const uint32_t*)bmp, nwords, (const int*)gstart,
                           (const int*)cnt, (const int*)plan, pairsel, part, dwc, dkraw, pk, pv,
                           wsb + l.trash, (__bf16*)dV);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    {
        const size_t items = (size_t)dm.B * dm.L * dm.G;
        HSA_TIMED("bwd_dq_reduce", st);
        hipLaunchKernelGGL(dm.off1 ? bwd_dq_reduce<true> : bwd_dq_reduce<false>,
                           dim3((unsigned)((items + 3) / 4)), dim3(256), 0, st, dm,
                           (const __bf16*)Q, Kbar, idx, w, (const uint16_t*)part, (const float*)dwc,
                           (__bf16*)dQ, dsb, qs);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (R > 0 && dm.dwo == nullptr) {
        HSA_TIMED("bwd_lmk_stream", st);
        hipLaunchKernelGGL(bwd_lmk_stream, dim3(kStreamWGs), dim3(NT), 0, st, dm,
                           (const int*)pairsel, (const float*)dsb, (const __bf16*)qs,
                           (const int*)gstart, (const int*)cnt, (const int*)plan, dkbar, pkb);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    {
        HSA_TIMED("bwd_finish", st);
        hipLaunchKernelGGL(bwd_finish, dim3(dm.B * dm.G * dm.Call), dim3(NT), 0, st, dm,
                           (const int*)gstart, (const int*)cnt, (const int*)plan,
                           (const float*)dkraw, (const float*)pk, (const float*)pv,
                           (const float*)dkbar, (const float*)pkb, (__bf16*)dK, (__bf16*)dV);
    }
    return hipGetLastError();
}

}  // namespace hsa
