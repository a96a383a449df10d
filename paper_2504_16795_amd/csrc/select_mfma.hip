// Chunk selection + chunk weights on matrix cores (Sec. 3.1: the top-k chunks by the
// landmark score s_c = alpha * (sum_j q_j) . Kbar_c over the chunks before the token's own,
// and their softmax weights), for bf16 queries with d = 128, or, for a selection over inputs
// of its own (one query row per group, h = 1), d = 128 ND up to 1024: the products then run
// over ND slices of 128 columns of each candidate block, and the query, exact in bf16, has
// no lo part (two products per slice instead of three).
//
// Workgroup = (b, g, tile of 64 consecutive tokens), 4 waves of 16 tokens.  The scores of a
// block of 64 candidate chunks for the tile are the product
//     S^T [64 chunks x 64 tokens] = Kbar_blk [64 x d] . q~^T [d x 64]
// on v_mfma_f32_16x16x32_bf16, each operand a bf16 pair hi + lo (the fp32 value rounded to
// bf16 and its remainder rounded to bf16, 16 mantissa bits together) and the product taken
// as hi.hi + hi.lo + lo.hi, so the scores carry about 16 bits (the dropped lo.lo term is
// below 2^-16 of each product).  The fp32 landmark rows of a block are loaded with
// coalesced 16-byte loads (the next block in flight during the current block's products),
// split into bf16 hi / lo once per workgroup and staged in LDS (double buffer, or one stage
// when every tile's candidates fit one block; the row swizzle of chunk_lds.h, conflict-free
// row reads).
//
// In the C layout each lane holds 4 candidates of one token per 16-chunk block and keeps a
// running top-KC list of its candidates (registers, descending; a candidate moves up past
// the entries it beats strictly, and a lane sees its chunks in increasing order, so equal
// scores keep the lower chunk first).  The 4 lanes of a token merge their lists at the
// end by a bitonic merge on 64-bit order keys (score desc, chunk asc as one integer).  The
// k best get softmax (or stick-breaking) weights and are written in descending chunk order,
// padded -1 / 0.
#include "chunk_lds.h"

namespace hsa {
namespace {

constexpr int D = 128;            // columns of a staged slice
constexpr int kMT = 64;            // tokens per workgroup
constexpr int kNW = 4;             // waves, 16 tokens each
constexpr int kNT = kNW * 64;
constexpr int kCB = 64;            // candidate chunks per staged block

struct SelStage {
    __bf16 hi[kCB * D];            // landmark rows rounded to bf16, swizzled
    __bf16 lo[kCB * D];            // their remainders rounded to bf16, swizzled
};

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, m, 64);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), m, 64);
    return ((uint64_t)hi << 32) | lo;
}

// ND: slices of 128 columns (d = 128 ND); QLO: the query is a sum over h > 1 heads (fp32,
// so it enters as a bf16 hi / lo pair); otherwise it is one bf16 row, exact.  NSTG: LDS
// stages; with a single stage (every tile's candidates fit one block of 64 chunks and one
// column slice) a workgroup takes 32 KB of LDS and at most 128 VGPRs, so four workgroups
// share a CU and their load and compute phases overlap.
template <int KC, int ND, bool QLO, int NSTG>
__global__ __launch_bounds__(kNT, NSTG == 1 ? 4 : 2) void select_mfma(Dims dm, const __bf16* __restrict__ Q,
                                                      const float* __restrict__ Kbar,
                                                      int32_t* __restrict__ idx,
                                                      float* __restrict__ w, int ntiles) {
    static_assert(ND == 1 || !QLO, "a head sum needs d = 128");
    constexpr int DD = D * ND;         // the query / landmark row length
    static_assert(NSTG == 1 || NSTG == 2, "one stage or a double buffer");
    __shared__ SelStage st[NSTG];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int row = lane & 15, grp = lane >> 4;
    const int nbg = dm.B * dm.G;
    const int tile = ntiles - 1 - (int)blockIdx.x / nbg;       // latest tiles first
    const int bg = (int)blockIdx.x % nbg, b = bg / dm.G, g = bg % dm.G;
    const int t0 = tile * kMT;
    const int nwg = (min(t0 + kMT, dm.L) - 1) / dm.S;         // candidates of the last token
    const int t = t0 + 16 * wave + row;                         // this lane's token
    const bool valid = t < dm.L;
    const int ncand = valid ? t / dm.S : 0;
    const int k = dm.k;

    // staging of stage si (candidate block si / ND, columns 128 (si % ND) ..): wave w
    // converts rows 16 w .. 16 w + 15; lane l covers row 16 w + 2 i + l / 32 (i < 8),
    // floats 4 (l % 32) .. +3 of the slice
    const size_t cstride = (size_t)dm.G * DD;
    const float* kb = Kbar + ((size_t)b * dm.C * dm.G + g) * DD + 4 * (lane & 31);
    float4 reg[8];
    auto load_block = [&](int si) __attribute__((always_inline)) {
        const int blk = si / ND, db = si % ND;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int c = min(blk * kCB + 16 * wave + 2 * i + (lane >> 5), nwg - 1);
            reg[i] = *reinterpret_cast<const float4*>(kb + (size_t)c * cstride + D * db);
        }
    };
    auto store_block = [&](int s) __attribute__((always_inline)) {
        const int f = lane & 31;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int r = 16 * wave + 2 * i + (lane >> 5);
            const float v[4] = {reg[i].x, reg[i].y, reg[i].z, reg[i].w};
            bf16x4_t h4, l4;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                h4[e] = f2bf(v[e]);
                l4[e] = f2bf(v[e] - (float)h4[e]);
            }
            const int off = r * D + unit_pos(r, f >> 1) * 8 + (f & 1) * 4;
            *reinterpret_cast<bf16x4_t*>(st[s].hi + off) = h4;
            *reinterpret_cast<bf16x4_t*>(st[s].lo + off) = l4;
        }
    };

    const int nblk = cdiv(nwg, kCB);
    const int nst = nblk * ND;         // stages: (candidate block, column slice)
    // the first block's landmark loads go out before the query loads (independent of
    // them), so both latencies overlap; with a single stage they follow the query sum
    // (the registers they need are then free)
    if (NSTG == 2 && nblk > 0) load_block(0);

    // B operand: q~ of the wave's 16 tokens as bf16 hi / lo; the lane holds d = 128 db +
    // 32 ks + 8 grp + i of token `row` (a token past the end reads the last one; unused)
    bf16x8_t qh[ND][4], ql[QLO ? 4 : 1];
    if constexpr (!QLO) {
        const __bf16* qp = Q + (((size_t)b * dm.L + min(t, dm.L - 1)) * dm.H + g) * DD + 8 * grp;
#pragma unroll
        for (int db = 0; db < ND; ++db)
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) qh[db][ks] = ld_bf16x8(qp + D * db + 32 * ks);
    } else {
        float qs[4][8];
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
            for (int i = 0; i < 8; ++i) qs[ks][i] = 0.f;
        const __bf16* qp = Q + (((size_t)b * dm.L + min(t, dm.L - 1)) * dm.H + (size_t)g * dm.h) * D +
                           8 * grp;
        // HB heads at a time: all their loads are issued (head index clamped, branch-free)
        // before the first sum, so the wave waits for one round trip per HB heads rather
        // than one per head (HB = 4 within the single-stage register budget)
        constexpr int HB = NSTG == 1 ? 4 : 8;
        for (int j0 = 0; j0 < dm.h; j0 += HB) {
            bf16x8_t v[HB][4];
#pragma unroll
            for (int jj = 0; jj < HB; ++jj)
#pragma unroll
                for (int ks = 0; ks < 4; ++ks)
                    v[jj][ks] = ld_bf16x8(qp + (size_t)min(j0 + jj, dm.h - 1) * D + 32 * ks);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int jj = 0; jj < HB; ++jj) {
                const bool use = j0 + jj < dm.h;     // a select, so no load is sunk
#pragma unroll
                for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                    for (int i = 0; i < 8; ++i) qs[ks][i] += use ? (float)v[jj][ks][i] : 0.f;
            }
        }
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const __bf16 h = f2bf(qs[ks][i]);
                qh[0][ks][i] = h;
                ql[ks][i] = f2bf(qs[ks][i] - (float)h);
            }
    }

    float ls[KC];
    int lc[KC];
#pragma unroll
    for (int j = 0; j < KC; ++j) {
        ls[j] = -INFINITY;
        lc[j] = -1;
    }
    int koff[4];
    row_read_offsets(lane, koff);
    const float alpha = dm.alpha;
    if (NSTG == 1 && nblk > 0) load_block(0);
    if (nblk > 0) store_block(0);
    constexpr int MB = kCB / 16;
    for (int blk = 0; blk < nblk; ++blk) {
        // the 4 row blocks' products interleaved (independent accumulators) over the
        // block's column slices, then the candidates
        f32x4_t acc[MB];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[mb] = zero4();
#pragma unroll
        for (int db = 0; db < ND; ++db) {
            const int si = blk * ND + db;
            __syncthreads();           // stage si staged; the other stage's readers are done
            if (NSTG == 2 && si + 1 < nst) load_block(si + 1);
            const SelStage& sb = st[si & (NSTG - 1)];
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                bf16x8_t ah[MB], al[MB];
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) {
                    ah[mb] = ld_bf16x8(sb.hi + koff[ks] + mb * 2048);
                    al[mb] = ld_bf16x8(sb.lo + koff[ks] + mb * 2048);
                }
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) acc[mb] = mfma16(ah[mb], qh[db][ks], acc[mb]);
                if constexpr (QLO) {
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb) acc[mb] = mfma16(ah[mb], ql[ks], acc[mb]);
                }
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) acc[mb] = mfma16(al[mb], qh[db][ks], acc[mb]);
            }
            if (NSTG == 2 && si + 1 < nst) store_block((si + 1) & (NSTG - 1));
        }
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int c = blk * kCB + 16 * mb + 4 * grp + i;
                float s = (c < ncand) ? alpha * acc[mb][i] : -INFINITY;
                if (__ballot(s > ls[KC - 1]) == 0) continue;
                int ci = c;
#pragma unroll
                for (int j = 0; j < KC; ++j) {   // insertion: strictly greater moves up
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
    }

    // merge the lists of a token's 4 lanes (l, l ^ 16, l ^ 32, l ^ 48): the top KC of two
    // descending lists is the elementwise maximum of one and the other reversed (a bitonic
    // sequence), sorted by a bitonic half-cleaner network
    uint64_t key[KC];
#pragma unroll
    for (int j = 0; j < KC; ++j) key[j] = lc[j] >= 0 ? order_key(ls[j], lc[j]) : 0;
#pragma unroll
    for (int xm = 16; xm <= 32; xm <<= 1) {
        uint64_t other[KC];
#pragma unroll
        for (int j = 0; j < KC; ++j) other[j] = shfl_xor_u64(key[j], xm);
#pragma unroll
        for (int j = 0; j < KC; ++j) key[j] = max_u64(key[j], other[KC - 1 - j]);
#pragma unroll
        for (int half = KC / 2; half >= 1; half >>= 1)
#pragma unroll
            for (int j = 0; j < KC; ++j)
                if ((j & half) == 0) {
                    const uint64_t a = key[j], c = key[j + half];
                    key[j] = max_u64(a, c);
                    key[j + half] = a > c ? c : a;
                }
    }
    if (!valid || grp != 0) return;

    // weights of the k best, written in descending chunk order
    const int n = min(k, ncand);
#pragma unroll
    for (int j = 0; j < KC; ++j) {
        ls[j] = key[j] ? key_score(key[j]) : -INFINITY;
        lc[j] = key[j] ? key_chunk(key[j]) : -1;
    }
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

template <int KC, int ND, bool QLO>
void launch_nd(const Dims& dm, const void* Q, const float* Kbar, int32_t* idx, float* w,
               hipStream_t st) {
    const int ntiles = cdiv(dm.L, kMT);
    const dim3 grid(ntiles * dm.B * dm.G);
    // one stage when the last token's candidates fit one block (and one column slice)
    if constexpr (ND == 1 && KC == 8) {
        if (dm.L > 0 && (dm.L - 1) / dm.S <= kCB) {
            hipLaunchKernelGGL((select_mfma<KC, ND, QLO, 1>), grid, dim3(kNT), 0, st, dm,
                               (const __bf16*)Q, Kbar, idx, w, ntiles);
            return;
        }
    }
    hipLaunchKernelGGL((select_mfma<KC, ND, QLO, 2>), grid, dim3(kNT), 0, st, dm,
                       (const __bf16*)Q, Kbar, idx, w, ntiles);
}

template <int KC>
void launch_kc_mfma(const Dims& dm, const void* Q, const float* Kbar, int32_t* idx, float* w,
                    hipStream_t st) {
    switch (dm.d) {
        case 256: launch_nd<KC, 2, false>(dm, Q, Kbar, idx, w, st); break;
        case 512: launch_nd<KC, 4, false>(dm, Q, Kbar, idx, w, st); break;
        case 1024: launch_nd<KC, 8, false>(dm, Q, Kbar, idx, w, st); break;
        default:
            if (dm.h > 1) launch_nd<KC, 1, true>(dm, Q, Kbar, idx, w, st);
            else launch_nd<KC, 1, false>(dm, Q, Kbar, idx, w, st);
    }
}

}  // namespace

bool select_mfma_supported(const Dims& dm, bool in_bf16) {
    if (dm.d > D) return in_bf16 && dm.h == 1 && dm.k <= 32;    // only path for wide rows
    return in_bf16 && dm.d == D && dm.k <= 32 && path_override(HSA_OP_SELECT) != HSA_PATH_GENERIC;
}

hipError_t launch_select_mfma(const Dims& dm, const void* Q, const float* Kbar, int32_t* idx,
                              float* w, hipStream_t st) {
    HSA_TIMED("select_kernel", st);
    if (dm.k <= 8) launch_kc_mfma<8>(dm, Q, Kbar, idx, w, st);
    else if (dm.k <= 16) launch_kc_mfma<16>(dm, Q, Kbar, idx, w, st);
    else launch_kc_mfma<32>(dm, Q, Kbar, idx, w, st);
    return hipGetLastError();
}

}  // namespace hsa
