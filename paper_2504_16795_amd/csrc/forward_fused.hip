// Chunk-major forward of hierarchical sparse attention (Sec. 3.1.1 hierarchical attention
// equation: O_t = sum_i w_i softmax(beta q K_{c_i}^T) V_{c_i}), for bf16 inputs with h = 8
// query heads per KV head, d = 128 and S = 64, over the even split of chunk_stream.h.
//
// fwd_chunk_mfma: 4 waves; wave w owns keys 16 w .. 16 w + 15 of the current chunk (K_sub
// in registers) and columns 32 w .. 32 w + 31 of d for the output product (V^T fragments of
// all 64 keys, read transposed from the chunk staged in LDS).  Per group of 4 tokens (32
// rows):
//     Z [32 x 16] = Q_rows K_sub^T                                          (MFMA)
//     each wave reduces its 16 keys per row (max m_w of the scaled logits, sum of
//     exp(z - m_w)); the four waves' values are exchanged through LDS and combined into
//     P = softmax over the chunk's 64 keys
//     (W P)^T [64 keys x 32 rows] is staged in LDS as a bf16 pair hi + lo, W the token's
//     weight for c
//     (summed over slots repeating c); wave w forms
//     O_c^T [d 32 w .. 32 w + 31 x 32 rows] = V_c^T (W P)^T                 (MFMA)
//     and stores it (bf16) at the (token, slot, head) of the token's first slot holding c.
// fwd_reduce (token-major, one wave per (b, t, g)): O = sum of the token's partials.
//
// Against the tile-major forward (forward_mfma.hip) this reads each chunk's K / V once per
// range instead of once per query tile, and uses every matrix row, at the cost of a 2 KB
// partial per (token, slot) written and read back: it pays when tokens of a tile rarely share
// chunks (long contexts).  No atomics; every sum runs in a fixed order.
#include "chunk_stream.h"

namespace hsa {

hipError_t launch_selection_bitmap(const Dims& dm, const int32_t* idx, uint32_t* bm,
                                   hipStream_t st);

namespace {

constexpr int D = 128;
constexpr int HG = 8;
constexpr int KMAX = 32;
constexpr int ONST = 3;             // LDS stages of the group ring (Q rows only)
constexpr int OBPW = 8 / NW;        // 1 KB row blocks of Q copied per wave and group
constexpr int kOStores = 2;         // global stores per lane of one output step (16 B each)
constexpr int kFwdWGs = 768;        // workgroups of the split: three per CU (46 KB of LDS each)

struct FwdWs {
    size_t bitmap, cnt, gstart, plan, part, end;
};
__host__ __device__ inline FwdWs fwd_ws(const Dims& dm) {
    FwdWs l;
    const size_t nsel = (size_t)dm.B * dm.L * dm.G * dm.k;
    const size_t nwords = (size_t)((dm.L + 31) / 32);
    const size_t R = (size_t)dm.B * dm.G * dm.C;
    l.bitmap = 0;
    l.cnt = align256(R * nwords * 4);
    l.gstart = l.cnt + align256(R * 4);
    l.plan = l.gstart + align256((R + 1) * 4);
    l.part = l.plan + 256;
    l.end = l.part + align256((nsel + 1) * HG * D * 2);       // + the spare block
    return l;
}

struct SmemO {
    __bf16 st[ONST][32 * D];        // Q rows of a group, swizzled; stages 0, 1 hold the
                                    // chunk's V rows while V^T is read
    __bf16 pt[2][CS * 32];          // (W P)^T of a group as a bf16 pair hi, lo: [key][row],
                                    // see zpos
    float stat[NW][2][32];          // per wave and row: m_w, sum exp
    float fac[NW][32];              // per wave and row: P scale of the wave's keys
    int list[FLIST];                // token; then its first Q row, (b L + t) H + g h
    int lsel[FLIST];                // (token, first slot holding c): ((b L + t) G + g) k + s
    float lw[FLIST];                // the token's total weight for c
    int wtot[NW];
};
static_assert(ONST * 32 * D >= CS * D, "the V rows of a chunk fit in the first stages");

__global__ __launch_bounds__(NT, 3) void fwd_chunk_mfma(
    Dims dm, const __bf16* __restrict__ Q, const __bf16* __restrict__ K,
    const __bf16* __restrict__ V, const int32_t* __restrict__ idx, const float* __restrict__ w,
    const uint32_t* __restrict__ bm, int nwords, const int* __restrict__ gstart,
    const int* __restrict__ cntr, const int* __restrict__ plan, uint16_t* __restrict__ part) {
    __shared__ SmemO sm;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int row = lane & 15, grp = lane >> 4;
    const int lid = xcd_logical_id(kFwdWGs);
    if (lid < 0) return;
    const int R = dm.B * dm.G * dm.C;
    const int total = plan[0], T = plan[1];
    const int g0 = lid * T, g1 = min(g0 + T, total);
    if (g0 >= g1) return;
    const int k = dm.k;
    const size_t rowstride = (size_t)dm.G * D;
    const float sl2 = dm.beta * 1.44269504088896341f;
    const bool off1 = dm.off1 != 0;
    const float mfloor = off1 ? 0.f : -INFINITY;

    // LDS offsets of the row reads of a chunk-swizzled tile (chunk_lds.h), d step ks:
    // kb0 + 32 (ks ^ ks_x) (+ 2048 per 16-row block)
    const int swr = swz(row);
    const int kb0 = row * D + 8 * (grp ^ (swr & 3)), ks_x = swr >> 2;
    auto koff = [&](int ks) __attribute__((always_inline)) { return kb0 + 32 * (ks ^ ks_x); };
    int zb[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) zb[rt] = zpos(4 * grp + (row >> 2), 4 * rt + (row & 3));
    // a lane's partial-store address is pbase + 2 KB * block, block = the (token, slot) or,
    // for rows of missing tokens, tblk: the spare block after the partials
    char* const pbase = reinterpret_cast<char*>(part) + 2 * ((row & 7) * D + 32 * wave + 8 * grp);
    const uint32_t tblk = (uint32_t)((size_t)dm.B * dm.L * dm.G * dm.k);

    for (int r = find_row(gstart, R, g0); r < R; ++r) {
        const int rs = gstart[r], re = gstart[r + 1];
        if (rs >= g1) break;
        if (re == rs) continue;
        const Segment sg = segment_of(rs, re, g0, g1);
        const int c = r % dm.C;
        const int bg = r / dm.C, b = bg / dm.G, g = bg % dm.G;
        const size_t cbase = ((size_t)b * dm.L + (size_t)c * CS) * rowstride + (size_t)g * D;
        const int ntok = cntr[r];

        // ---- the chunk's operands: K_sub^T (B operand of Z) and V^T (A operand of O^T: row
        // m of tile dt is column 32 wave + 8 (m >> 2) + 4 dt + (m & 3) of d, so a lane's C values
        // of both tiles are 8 consecutive columns; keys of lane group grp in step ks2:
        // 32 ks2 + 4 grp + (0..3) and 32 ks2 + 16 + 4 grp + (0..3))
        __syncthreads();                          // the previous chunk's stages are read
        bf16x8_t kB[4];
        const int key = 16 * wave + row;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
            kB[ks] = ld_bf16x8(K + cbase + (size_t)key * rowstride + 32 * ks + 8 * grp);
        chunk_to_lds<CS, NW>(V + cbase, rowstride, sm.st[0], wave, lane);
        wait_loads_le<0>();
        __syncthreads();
        bf16x8_t vT[2][2];
#pragma unroll
        for (int dt = 0; dt < 2; ++dt)
#pragma unroll
            for (int ks2 = 0; ks2 < 2; ++ks2) {
                const __bf16* p = sm.st[0] + tr_perm_offset(lane, 32 * wave, dt) + 32 * ks2 * D;
                vT[dt][ks2] = cat(ld_tr16(p), ld_tr16(p + 16 * D));
            }

        auto issue = [&](int gi, int nl, __bf16* st) __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < OBPW; ++i) {
                const int blk = wave * OBPW + i;
                const int rr = blk * 4 + (lane >> 4);
                int li = gi * 4 + (rr >> 3);
                if (li >= nl) li = gi * 4;   // a missing token repeats the group's first (W = 0)
                const size_t o = ((size_t)(uint32_t)(sm.list[li] + (rr & 7)) << 7) +
                                 unit_pos(rr, lane & 15) * 8;
                lds_copy16(Q + o, __builtin_amdgcn_readfirstlane(lds_address(st + blk * 512)));
            }
        };

        // output partial of group gj from the staged (W P)^T (all waves' keys): rows
        // 16 rt + (lane & 15), d = 32 wave + 8 grp + (0..7) (tile dt holds 4 dt + (0..3));
        // exactly kOStores stores per lane (rows of missing tokens go to the spare block)
        auto o_step = [&](int gj, int nl) __attribute__((always_inline)) {
            f32x4_t oa[2][2];
#pragma unroll
            for (int dt = 0; dt < 2; ++dt) oa[dt][0] = oa[dt][1] = zero4();
#pragma unroll
            for (int rt = 0; rt < 2; ++rt)
#pragma unroll
                for (int ks2 = 0; ks2 < 2; ++ks2)
#pragma unroll
                    for (int hl = 0; hl < 2; ++hl) {
                        const __bf16* zp = sm.pt[hl] + zb[rt] + 1024 * ks2;
                        const bf16x8_t bp = cat(ld_tr16(zp), ld_tr16(zp + 512));
#pragma unroll
                        for (int dt = 0; dt < 2; ++dt)
                            oa[dt][rt] = mfma16(vT[dt][ks2], bp, oa[dt][rt]);
                    }
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) {
                const int li = gj * 4 + 2 * rt + (row >> 3);
                const int so = li < nl ? sm.lsel[li] : -1;
                const uint32_t blk = so >= 0 ? (uint32_t)so : tblk;
                *reinterpret_cast<u32x4_t*>(pbase + ((size_t)blk << 11)) =
                    bfp_pack8(oa[0][rt], oa[1][rt]);
            }
        };

        const uint32_t* bmrow = bm + (size_t)r * nwords;
        const int wbeg = ((c + 1) * CS) >> 5;
        const int tend = min(4 * sg.j1, ntok);
        for (int p0 = 4 * sg.j0; p0 < tend; p0 += FLIST) {
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
                sm.lw[li] = first < k ? wsum : 0.f;
                sm.list[li] = (int)(((size_t)b * dm.L + t) * dm.H + (size_t)g * HG);
            }
            __syncthreads();
            const int ngroups = (nl + 3) / 4;
#pragma unroll
            for (int u = 0; u < ONST - 1; ++u)
                if (u < ngroups) issue(u, nl, sm.st[u]);
            // one group's step; its stage index SI = gi % ONST is a constant (the loop below
            // is unrolled by ONST), so the stage's LDS addresses are lane bases plus immediates
            auto group = [&](int gi, auto si) __attribute__((always_inline)) {
                constexpr int SI = decltype(si)::value;
                // Group gi has landed once only the memory operations issued after its copies
                // remain: the previous iteration's output stores (when it ran one) and the
                // next group's copies (when there is a next group).  Loads and stores complete
                // in issue order.
                const bool more = gi + 1 < ngroups, stored = gi >= 2;
                if (more && stored) wait_loads_le<OBPW + kOStores>();
                else if (more) wait_loads_le<OBPW>();
                else if (stored) wait_loads_le<kOStores>();
                else wait_loads_le<0>();
                lds_wait();
                barrier_keep_copies();   // stage gi landed, (W P)^T of gi - 1 complete
                if (gi > 0) o_step(gi - 1, nl);
                if (gi + ONST - 1 < ngroups) issue(gi + ONST - 1, nl, sm.st[(SI + ONST - 1) % ONST]);
                const __bf16* st = sm.st[SI];

                // ---- Z for the wave's 16 keys (rows 16 rb + 4 grp + i, key 16 wave + row) --
                f32x4_t z[2];
                z[0] = z[1] = zero4();
#pragma unroll
                for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                    for (int rb = 0; rb < 2; ++rb)
                        z[rb] = mfma16(ld_bf16x8(st + koff(ks) + rb * 2048), kB[ks], z[rb]);
                // ---- the wave's row statistics over its 16 keys, to LDS -----------------
                // (rows 16 rb + 4 grp + i at index 4 rb + i)
                float zl[8], mx[8], ls[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) zl[i] = z[i >> 2][i & 3] * sl2;
                rows16_exp(zl, ls, mx);
#pragma unroll
                for (int i = 0; i < 8; ++i) zl[i] = ls[i];
                rows16_sum(ls);
                // complete in every lane before the branch below (otherwise the last DPP step
                // is sunk into it and can no longer fuse with its add)
#pragma unroll
                for (int i = 0; i < 8; ++i) asm volatile("" : "+v"(ls[i]));
                f32x4_t e[2];
#pragma unroll
                for (int rb = 0; rb < 2; ++rb) {
                    e[rb] = f32x4_t{zl[4 * rb], zl[4 * rb + 1], zl[4 * rb + 2], zl[4 * rb + 3]};
                    if (row == 0) {
                        *reinterpret_cast<f32x4_t*>(&sm.stat[wave][0][16 * rb + 4 * grp]) =
                            f32x4_t{mx[4 * rb], mx[4 * rb + 1], mx[4 * rb + 2], mx[4 * rb + 3]};
                        *reinterpret_cast<f32x4_t*>(&sm.stat[wave][1][16 * rb + 4 * grp]) =
                            f32x4_t{ls[4 * rb], ls[4 * rb + 1], ls[4 * rb + 2], ls[4 * rb + 3]};
                    }
                }
                lds_wait();
                barrier_keep_copies();   // every wave's statistics of group gi written
                // ---- combine: lane r (and r + 32) handles row r = lane & 31 ------------------
                {
                    const int r32 = lane & 31;
                    float mv[NW], lv[NW];
#pragma unroll
                    for (int w2 = 0; w2 < NW; ++w2) {
                        mv[w2] = sm.stat[w2][0][r32];
                        lv[w2] = sm.stat[w2][1][r32];
                    }
                    // off by one, the extra logit 0 joins the maximum and the sum
                    const float M = fmaxf(fmaxf(fmaxf(mv[0], mv[1]), fmaxf(mv[2], mv[3])), mfloor);
                    float lsum = off1 ? fast_exp2(-M) : 0.f, aown = 0.f;
#pragma unroll
                    for (int w2 = 0; w2 < NW; ++w2) {
                        const float a = fast_exp2(mv[w2] - M);
                        lsum = fmaf(a, lv[w2], lsum);
                        aown = (w2 == wave) ? a : aown;
                    }
                    if (lane < 32) sm.fac[wave][r32] = aown * __builtin_amdgcn_rcpf(lsum);
                }
                // back in the C layout (the wave's own LDS writes, read in order); W P to LDS as
                // (W P)^T: key 16 wave + row, rows 16 rb + 4 grp .. +3 = unit 4 rb + grp
                const int j = 16 * wave + row;
#pragma unroll
                for (int rb = 0; rb < 2; ++rb) {
                    const f32x4_t fv = *reinterpret_cast<const f32x4_t*>(&sm.fac[wave][16 * rb + 4 * grp]);
                    const int li = gi * 4 + 2 * rb + (grp >> 1);
                    const float wt = li < nl ? sm.lw[li] : 0.f;
                    // as a bf16 pair hi + lo (about 16 bits): one bf16 rounding of each
                    // weighted probability would leave an error of up to 2^-9 of it in O
                    f32x4_t x, x0;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        x[i] = wt * e[rb][i] * fv[i];
                        x0[i] = 0.f;
                    }
                    bf16x8_t h8, l8;
                    split8(x, x0, h8, l8);
                    *reinterpret_cast<bf16x4_t*>(sm.pt[0] + zpos(j, 4 * rb + grp)) =
                        bf16x4_t{h8[0], h8[1], h8[2], h8[3]};
                    *reinterpret_cast<bf16x4_t*>(sm.pt[1] + zpos(j, 4 * rb + grp)) =
                        bf16x4_t{l8[0], l8[1], l8[2], l8[3]};
                }
            };
            static_assert(ONST == 3, "the group loop is unrolled by the ring depth");
            for (int gb = 0; gb < ngroups; gb += ONST) {
                group(gb, IntC<0>{});
                if (gb + 1 < ngroups) group(gb + 1, IntC<1>{});
                if (gb + 2 < ngroups) group(gb + 2, IntC<2>{});
            }
            lds_wait();
            barrier_keep_copies();   // (W P)^T of the batch's last group complete
            o_step(ngroups - 1, nl);
        }
    }
}

// O of one (b, t, g) (one wave; lane: head lane >> 3, columns 16 (lane & 7) .. +15): the sum
// of the partials at the token's slots that hold a chunk first (0 <= c < floor(t / S); a slot
// repeating an earlier slot's chunk adds nothing: that partial carries both weights).
__global__ __launch_bounds__(256) void fwd_reduce(Dims dm, const int32_t* __restrict__ idx,
                                                  const uint16_t* __restrict__ part,
                                                  __bf16* __restrict__ O) {
    const int lane = threadIdx.x & 63;
    const size_t item = (size_t)blockIdx.x * 4 + (threadIdx.x >> 6);    // ((b L) + t) G + g
    if (item >= (size_t)dm.B * dm.L * dm.G) return;
    const int g = (int)(item % dm.G);
    const size_t bt = item / dm.G;
    const int t = (int)(bt % dm.L);
    const int k = dm.k;
    const size_t so = item * k;
    const int ncand = t / dm.S;
    const int head = lane >> 3, c0 = 16 * (lane & 7);
    const int cl = lane < k ? idx[so + lane] : -1;
    const bool valid = lane < k && cl >= 0 && cl < ncand;
    int canon = lane;
    for (int s = 0; s < k; ++s) {
        const int cs = __builtin_amdgcn_readlane(cl, s);
        if (s < canon && cs == cl) canon = s;
    }
    const int own = (valid && canon == lane) ? 1 : 0;
    float acc[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = 0.f;
    // All loads of 4 slots are issued before their first use, with no branch between them
    // (a slot past k reads slot k - 1's data, a slot that does not own its chunk reads its
    // own stale partial); what is not used is dropped by a select on the partial's scale.
    for (int s0 = 0; s0 < k; s0 += 4) {
        u32x4_t pv[4][2];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint16_t* pp = part + ((so + min(s0 + j, k - 1)) * HG + head) * D + c0;
            pv[j][0] = *reinterpret_cast<const u32x4_t*>(pp);
            pv[j][1] = *reinterpret_cast<const u32x4_t*>(pp + 8);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int s = s0 + j;
            const bool use = s < k && __builtin_amdgcn_readlane(own, min(s, k - 1)) != 0;
            bfp_accum8(pv[j][0], acc, use);
            bfp_accum8(pv[j][1], acc + 8, use);
        }
    }
    bf16x8_t o0, o1;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        o0[i] = f2bf(acc[i]);
        o1[i] = f2bf(acc[8 + i]);
    }
    __bf16* op = O + ((bt * dm.H) + (size_t)g * HG + head) * D + c0;
    *reinterpret_cast<bf16x8_t*>(op) = o0;
    *reinterpret_cast<bf16x8_t*>(op + 8) = o1;
}

}  // namespace

// The chunk-major forward serves bf16, h = 8, d = 128, S = 64 by default from 256 chunks on
// (64K tokens: 1.75 ms against 2.51 for the tile-major kernel, whose tiles then rarely share
// a chunk; at 4K tokens 0.81 against 0.54); HSA_PATH_CHUNK_MAJOR or HSA_PATH_TILE_MAJOR
// forces the choice.
bool forward_chunk_used(const Dims& dm, bool in_bf16) {
    const int path = path_override(HSA_OP_FORWARD);
    if (!(in_bf16 && dm.h == HG && dm.d == D && dm.S == CS && dm.k <= KMAX) ||
        (size_t)dm.B * dm.L * dm.G >= ((size_t)1 << 26) || path == HSA_PATH_GENERIC)
        return false;                             // (row and (token, slot) indices are 32-bit)
    if (path == HSA_PATH_CHUNK_MAJOR) return true;
    if (path == HSA_PATH_TILE_MAJOR) return false;
    return dm.C >= 256;
}

size_t forward_chunk_workspace(const Dims& dm, bool in_bf16) {
    return forward_chunk_used(dm, in_bf16) ? fwd_ws(dm).end : 0;
}

hipError_t launch_forward_chunk(const Dims& dm, const void* Q, const void* K, const void* V,
                                const int32_t* idx, const float* w, void* O, void* ws,
                                hipStream_t st) {
    const FwdWs l = fwd_ws(dm);
    char* wsb = (char*)ws;
    uint32_t* bmp = (uint32_t*)(wsb + l.bitmap);
    int* cnt = (int*)(wsb + l.cnt);
    int* gstart = (int*)(wsb + l.gstart);
    int* plan = (int*)(wsb + l.plan);
    uint16_t* part = (uint16_t*)(wsb + l.part);
    const int R = dm.B * dm.G * dm.C;
    const int nwords = cdiv(dm.L, 32);
    hipError_t e = launch_selection_bitmap(dm, idx, bmp, st);
    if (e != hipSuccess) return e;
    if (R > 0) {
        {
            HSA_TIMED("fwd_plan", st);
            hipLaunchKernelGGL(stream_rowcount, dim3(cdiv(R, 4)), dim3(256), 0, st,
                               (const uint32_t*)bmp, R, nwords, dm.C, dm.S, cnt);
            hipLaunchKernelGGL(stream_plan, dim3(1), dim3(1024), 0, st, (const int*)cnt, R,
                               kFwdWGs, gstart, plan);
        }
        HSA_TIMED("fwd_chunk_mfma", st);
        hipLaunchKernelGGL(fwd_chunk_mfma, dim3(kFwdWGs), dim3(NT), 0, st, dm,
                           (const __bf16*)Q, (const __bf16*)K, (const __bf16*)V, idx, w,
                           (const uint32_t*)bmp, nwords, (const int*)gstart, (const int*)cnt,
                           (const int*)plan, part);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    {
        const size_t items = (size_t)dm.B * dm.L * dm.G;
        HSA_TIMED("fwd_reduce", st);
        hipLaunchKernelGGL(fwd_reduce, dim3((unsigned)((items + 3) / 4)), dim3(256), 0, st, dm,
                           idx, (const uint16_t*)part, (__bf16*)O);
    }
    return hipGetLastError();
}

}  // namespace hsa
