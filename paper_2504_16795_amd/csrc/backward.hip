// Backward of hierarchical sparse attention (Sec. 3.1.2, two-phase backward).
//
// Phase 1 (query-major, one workgroup per (b, t, g)): recompute P and O for every slot,
// D_j = dO_j . O_{j,i}, dw_i = sum_j D_j, dz = w_i P (dP - D_j), dq_j += beta dz K; then
// the softmax-weight Jacobian ds_i = w_i (dw_i - sum_m w_m dw_m) and the score term
// dq_j += alpha sum_i ds_i Kbar_{c_i}.  ds is kept in the workspace for phase 2.
//
// Selection matrix: the paper's M[t, c] ("token t selected chunk c") is built as a bitmap
// per (b, g, chunk) over tokens with bitwise-OR atomics (order-independent, exact).
//
// Phase 2 (chunk-major, one workgroup per (b, g, chunk)): walks the chunk's bitmap row in
// increasing token order, recomputes P, dP, D for the selecting tokens and accumulates
// dV = sum w P^T dO, dK = beta sum dz^T q and dKbar = alpha sum ds q~ in registers, then
// writes dK = dK + dKbar / S and dV.  No float atomics: every dK/dV row is owned by one
// workgroup and summed in a fixed order, so results are bitwise reproducible.
//
// The MFMA path for the main bf16 shapes lives in backward_mfma.hip.
#include <type_traits>

#include "common.h"
#include "chunk_stream.h"

namespace hsa {

bool backward_mfma_supported(const Dims& dm, bool in_bf16);
size_t backward_mfma_workspace(const Dims& dm);
bool backward_fused_supported(const Dims& dm, bool in_bf16);
size_t backward_fused_workspace(const Dims& dm);
hipError_t launch_backward_fused(const Dims& dm, const void* Q, const void* K, const void* V,
                                 const float* Kbar, const int32_t* idx, const float* w,
                                 const void* dO, void* dQ, void* dK, void* dV, void* ws,
                                 hipStream_t st);
hipError_t launch_backward_mfma(const Dims& dm, const void* Q, const void* K, const void* V,
                                const float* Kbar, const int32_t* idx, const float* w,
                                const void* dO, void* dQ, void* dK, void* dV, void* ws,
                                hipStream_t st);

namespace {

constexpr int kThreads = 256;
constexpr int HMAX = 16;
constexpr int KMAX = 32;
// the generic key pass: workgroups of the even split of (chunk, 4-token group) work, and the
// tokens of a chunk listed at once
constexpr int kGenWGs = 512;
constexpr int kGenList = 256;


template <typename T, int D, int CS>
__global__ __launch_bounds__(kThreads) void bwd_q_generic(
    Dims dm, const T* __restrict__ Q, const T* __restrict__ K, const T* __restrict__ V,
    const float* __restrict__ Kbar, const int32_t* __restrict__ idx, const float* __restrict__ w,
    const T* __restrict__ dO, T* __restrict__ dQ, float* __restrict__ ds_out) {
    constexpr int KP = D + (sizeof(T) == 4 ? 1 : 2);
    constexpr int NACC = HMAX * D / kThreads;
    __shared__ T Ks[CS * KP];
    __shared__ T Vs[CS * KP];
    __shared__ float qf[HMAX * D];
    __shared__ float gf[HMAX * D];
    __shared__ float dz[HMAX * CS];
    __shared__ float Dl[HMAX];
    __shared__ float dwl[KMAX];
    __shared__ int sc[KMAX];
    __shared__ float sw[KMAX];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int t = blockIdx.x;
    const int bg = blockIdx.y, b = bg / dm.G, g = bg % dm.G;
    const int h = dm.h, S = dm.S, k = dm.k;
    const int ncand = t / S;
    const size_t qoff = (((size_t)b * dm.L + t) * dm.H + (size_t)g * h) * D;
    const size_t sel = (((size_t)b * dm.L + t) * dm.G + g) * k;

    for (int i = tid; i < h * D; i += kThreads) {
        qf[i] = to_f32(Q[qoff + i]);
        gf[i] = to_f32(dO[qoff + i]);
    }
    if (tid < KMAX) dwl[tid] = 0.f;
    // the token's slots (an empty or out-of-range one as -1)
    if (tid < k) {
        const int c = idx[sel + tid];
        sc[tid] = (c < 0 || c >= ncand) ? -1 : c;
        sw[tid] = w[sel + tid];
    }
    float acc[NACC];
#pragma unroll
    for (int r = 0; r < NACC; ++r) acc[r] = 0.f;
    __syncthreads();

    // each slot's K / V rows are loaded into registers while the slot before is computed
    // (for chunks of up to 4096 elements; larger ones would cost the workgroups per CU)
    constexpr int NS = CS * D / kThreads;
    constexpr bool PREF = CS * D <= 4096;
    T kr[PREF ? NS : 1], vr[PREF ? NS : 1];
    auto load_chunk = [&](int c) __attribute__((always_inline)) {
#pragma unroll
        for (int r = 0; r < NS; ++r) {
            const int i = tid + r * kThreads, s = i / D, e = i % D;
            const size_t gi = (((size_t)b * dm.L + (size_t)c * S + s) * dm.G + g) * D + e;
            kr[r] = K[gi];
            vr[r] = V[gi];
        }
    };
    auto next_slot = [&](int from) __attribute__((always_inline)) {
        int s2 = from;
        while (s2 < k && sc[s2] < 0) ++s2;
        return s2;
    };
    int slot = next_slot(0);
    if constexpr (PREF) {
        if (slot < k) load_chunk(sc[slot]);
    }
    while (slot < k) {
        const int cur = slot;
        const float wi = sw[cur];
        __syncthreads();                  // the previous slot's tiles and sums are read
        if constexpr (PREF) {
#pragma unroll
            for (int r = 0; r < NS; ++r) {
                const int i = tid + r * kThreads, s = i / D, e = i % D;
                Ks[s * KP + e] = kr[r];
                Vs[s * KP + e] = vr[r];
            }
        } else {
            const int c = sc[cur];
            for (int i = tid; i < S * D; i += kThreads) {
                const int s = i / D, e = i % D;
                const size_t gi = (((size_t)b * dm.L + (size_t)c * S + s) * dm.G + g) * D + e;
                Ks[s * KP + e] = K[gi];
                Vs[s * KP + e] = V[gi];
            }
        }
        slot = next_slot(cur + 1);
        if constexpr (PREF) {
            if (slot < k) load_chunk(sc[slot]);
        }
        __syncthreads();
        for (int j = wave; j < h; j += kThreads / 64) {
            float z[2], dp[2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int s = lane + 64 * u;
                float a = 0.f, bb = 0.f;
                if (s < S) {
                    // four partial sums each, so the products do not wait on one another
                    float a4[4] = {0.f, 0.f, 0.f, 0.f}, b4[4] = {0.f, 0.f, 0.f, 0.f};
                    for (int e = 0; e < D; e += 4) {
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            a4[q] = fmaf(qf[j * D + e + q], to_f32(Ks[s * KP + e + q]), a4[q]);
                            b4[q] = fmaf(gf[j * D + e + q], to_f32(Vs[s * KP + e + q]), b4[q]);
                        }
                    }
                    a = (a4[0] + a4[1]) + (a4[2] + a4[3]);
                    bb = (b4[0] + b4[1]) + (b4[2] + b4[3]);
                    z[u] = dm.beta * a;
                } else {
                    z[u] = -INFINITY;
                }
                dp[u] = bb;
            }
            float m = wave_max(fmaxf(z[0], z[1]));
            if (dm.off1) m = fmaxf(m, 0.f);
            float p0 = expf(z[0] - m), p1 = expf(z[1] - m);
            const float inv = 1.f / (wave_sum(p0 + p1) + (dm.off1 ? expf(-m) : 0.f));
            p0 *= inv;
            p1 *= inv;
            const float Dj = wave_sum(p0 * dp[0] + p1 * dp[1]);
            if (lane < S) dz[j * CS + lane] = wi * p0 * (dp[0] - Dj);
            if (lane + 64 < S) dz[j * CS + lane + 64] = wi * p1 * (dp[1] - Dj);
            if (lane == 0) Dl[j] = Dj;
        }
        __syncthreads();
        if (tid == 0) {
            float s = 0.f;
            for (int j = 0; j < h; ++j) s += Dl[j];
            dwl[cur] = s;
        }
#pragma unroll
        for (int r = 0; r < NACC; ++r) {
            const int i = tid + r * kThreads;
            if (i < h * D) {
                const int j = i / D, e = i % D;
                float a4[4] = {0.f, 0.f, 0.f, 0.f};   // S is a multiple of 4
                for (int s = 0; s < S; s += 4) {
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        a4[q] = fmaf(dz[j * CS + s + q], to_f32(Ks[(s + q) * KP + e]), a4[q]);
                }
                acc[r] = fmaf(dm.beta, (a4[0] + a4[1]) + (a4[2] + a4[3]), acc[r]);
            }
        }
    }
    __syncthreads();
    if (dm.dwo != nullptr) {
        // attention alone: dw per slot (0 in empty slots); ds = 0, so the key pass adds no
        // landmark term
        if (tid < k) {
            const int c = idx[sel + tid];
            const float v = (c >= 0 && c < ncand) ? dwl[tid] : 0.f;
            float* o = dm.dwo + sel + tid;
            *o = dm.dwacc ? *o + v : v;
            ds_out[sel + tid] = 0.f;
        }
#pragma unroll
        for (int r = 0; r < NACC; ++r) {
            const int i = tid + r * kThreads;
            if (i < h * D) dQ[qoff + i] = from_f32<T>(acc[r]);
        }
        return;
    }
    // chunk-weight Jacobian (softmax or stick-breaking) and the score term
    float wdw = 0.f;
    for (int i = 0; i < k; ++i) {
        const int c = idx[sel + i];
        if (c >= 0 && c < ncand) wdw += w[sel + i] * dwl[i];
    }
    auto okf = [&](int i) { const int c2 = idx[sel + i]; return c2 >= 0 && c2 < ncand; };
    for (int i = 0; i < k; ++i) {
        const int c = idx[sel + i];
        const bool ok = (c >= 0 && c < ncand);
        const float dsi = !ok ? 0.f
                        : dm.stick ? stick_ds(i, k, [&](int m) { return w[sel + m]; },
                                              [&](int m) { return dwl[m]; }, okf)
                                   : w[sel + i] * (dwl[i] - wdw);
        if (tid == 0) ds_out[sel + i] = dsi;
        if (!ok) continue;
        const float* kb = Kbar + (((size_t)b * dm.C + c) * dm.G + g) * D;
#pragma unroll
        for (int r = 0; r < NACC; ++r) {
            const int ii = tid + r * kThreads;
            if (ii < h * D) acc[r] = fmaf(dm.alpha * dsi, kb[ii % D], acc[r]);
        }
    }
#pragma unroll
    for (int r = 0; r < NACC; ++r) {
        const int i = tid + r * kThreads;
        if (i < h * D) dQ[qoff + i] = from_f32<T>(acc[r]);
    }
}

// The selection bitmap (the M matrix of the key-side program as bits): bit t of word
// (b, g, c, t / 32) is set when a slot of token t holds chunk c, 0 <= c < floor(t / S), and
// every other bit is clear.  One workgroup per (256-token block, b g, range of kBmRange
// chunks) builds its 8-word slice of every row of the range in LDS (one LDS atomic OR per
// valid (token, slot), order-independent and exact) and writes the whole slice, zeros
// included, so no separate clearing pass and no global atomics are needed.  Chunks at or
// past floor((t0 + 255) / S) cannot hold a bit of the block and are written as zeros
// without touching LDS.
constexpr int kBmRange = 1024;

__global__ __launch_bounds__(256) void bitmap_build(Dims dm, const int32_t* __restrict__ idx,
                                                    uint32_t* __restrict__ bm, int nwords) {
    __shared__ uint32_t sl[kBmRange * 8];
    const int tid = threadIdx.x;
    const int t0 = blockIdx.x * 256;
    const int bg = blockIdx.y;
    const int b = bg / dm.G, g = bg % dm.G;
    const int c0 = blockIdx.z * kBmRange;
    const int c1 = min(dm.C, c0 + kBmRange);
    const int tend = min(dm.L, t0 + 256);
    const int nact = max(0, min(c1, (tend - 1) / dm.S) - c0);   // rows that can hold bits
    for (int i = tid; i < nact * 8; i += 256) sl[i] = 0u;
    __syncthreads();
    const int t = t0 + tid;
    if (t < dm.L) {
        const int32_t* row = idx + (((size_t)b * dm.L + t) * dm.G + g) * dm.k;
        const int lim = min(t / dm.S, c1);
        const uint32_t bit = 1u << (tid & 31);
#pragma unroll 8
        for (int s = 0; s < dm.k; ++s) {
            const int c = row[s];
            if (c >= c0 && c < lim) atomicOr(&sl[(c - c0) * 8 + (tid >> 5)], bit);
        }
    }
    __syncthreads();
    const int w0 = t0 >> 5;
    const int nw = min(8, nwords - w0);
    uint32_t* out = bm + (size_t)bg * dm.C * nwords + w0;
    for (int i = tid; i < (c1 - c0) * 8; i += 256) {
        const int cr = i >> 3, j = i & 7;
        if (j < nw) out[(size_t)(c0 + cr) * nwords + j] = cr < nact ? sl[i] : 0u;
    }
}

template <typename T, int D, int CS>
__global__ __launch_bounds__(kThreads) void bwd_kv_generic(
    Dims dm, const T* __restrict__ Q, const T* __restrict__ K, const T* __restrict__ V,
    const int32_t* __restrict__ idx, const float* __restrict__ w, const T* __restrict__ dO,
    const float* __restrict__ ds, const uint32_t* __restrict__ bm, int nwords,
    const int* __restrict__ gstart, const int* __restrict__ cntr, const int* __restrict__ plan,
    T* __restrict__ dK, T* __restrict__ dV, float* __restrict__ part) {
    constexpr int KP = D + (sizeof(T) == 4 ? 1 : 2);
    constexpr int NE = CS * D / kThreads;
    __shared__ T Ks[CS * KP];
    __shared__ T Vs[CS * KP];
    __shared__ float qf[HMAX * D];
    __shared__ float gf[HMAX * D];
    __shared__ float pw[HMAX * CS];
    __shared__ float dz[HMAX * CS];
    __shared__ float dkb[D];
    __shared__ int tlist[kGenList];          // a run of the chunk's tokens
    __shared__ int wtot[kThreads / 64];
    __shared__ float twt[HMAX], tds[HMAX];   // a batch's weights and ds for this chunk

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h = dm.h, k = dm.k;
    const int R = dm.B * dm.G * dm.C;
    const int lid = blockIdx.x;
    const int total = plan[0], Tg = plan[1];
    const int g0 = lid * Tg, g1 = min(g0 + Tg, total);
    if (g0 >= g1) return;
    const float invS = 1.f / (float)CS;

    // the rows (b, g, chunk) that this workgroup's range of 4-token groups touches
    for (int r = find_row(gstart, R, g0); r < R; ++r) {
        const int rs = gstart[r], re = gstart[r + 1];
        if (rs >= g1) break;
        if (re == rs) continue;
        const Segment sg = segment_of(rs, re, g0, g1);
        const int c = r % dm.C;
        const int bg = r / dm.C, b = bg / dm.G, g = bg % dm.G;
        const size_t rowbase = ((size_t)b * dm.L + (size_t)c * CS) * dm.G + g;   // row cS

        __syncthreads();                     // the previous row's tiles and sums are read
        for (int i = tid; i < CS * D; i += kThreads) {
            const int s = i / D, e = i % D;
            const size_t gi = (rowbase + (size_t)s * dm.G) * D + e;
            Ks[s * KP + e] = K[gi];
            Vs[s * KP + e] = V[gi];
        }
        float aK[NE], aV[NE];
#pragma unroll
        for (int r2 = 0; r2 < NE; ++r2) aK[r2] = aV[r2] = 0.f;
        float dkbar = 0.f;   // thread tid < D owns element tid of dKbar

        // Tokens are taken TB = floor(HMAX / h) at a time: the batch's (token, head) rows fill
        // the HMAX-row LDS arrays, so a batch costs the barriers and memory round trips of one
        // token.
        const int TB = HMAX / h;
        auto batch = [&](const int* tl, int n) __attribute__((always_inline)) {
            const int nrows = n * h;
            __syncthreads();                  // the previous batch's rows are read
            for (int i = tid; i < nrows * D; i += kThreads) {
                const int tk = i / (h * D), r = i - tk * (h * D);
                const size_t qoff = (((size_t)b * dm.L + tl[tk]) * dm.H + (size_t)g * h) * D;
                qf[i] = to_f32(Q[qoff + r]);
                gf[i] = to_f32(dO[qoff + r]);
            }
            if (tid < n) {                    // the token's slot holding c: its w and ds
                const size_t sel = (((size_t)b * dm.L + tl[tid]) * dm.G + g) * k;
                int slot = 0;
                for (int i = 0; i < k; ++i)
                    if (idx[sel + i] == c) slot = i;
                twt[tid] = w[sel + slot];
                tds[tid] = ds[sel + slot];
            }
            __syncthreads();
            for (int j = wave; j < nrows; j += kThreads / 64) {
                const float wt = twt[j / h];
                float z[2], dp[2];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    const int s = lane + 64 * u;
                    float a = 0.f, bb = 0.f;
                    if (s < CS) {
                        // four partial sums each, so the products do not wait on one another
                        float a4[4] = {0.f, 0.f, 0.f, 0.f}, b4[4] = {0.f, 0.f, 0.f, 0.f};
                        #pragma unroll 4
                        for (int e = 0; e < D; e += 4) {
#pragma unroll
                            for (int q = 0; q < 4; ++q) {
                                a4[q] = fmaf(qf[j * D + e + q], to_f32(Ks[s * KP + e + q]), a4[q]);
                                b4[q] = fmaf(gf[j * D + e + q], to_f32(Vs[s * KP + e + q]), b4[q]);
                            }
                        }
                        a = (a4[0] + a4[1]) + (a4[2] + a4[3]);
                        bb = (b4[0] + b4[1]) + (b4[2] + b4[3]);
                        z[u] = dm.beta * a;
                    } else {
                        z[u] = -INFINITY;
                    }
                    dp[u] = bb;
                }
                float m = wave_max(fmaxf(z[0], z[1]));
                if (dm.off1) m = fmaxf(m, 0.f);
                float p0 = expf(z[0] - m), p1 = expf(z[1] - m);
                const float inv = 1.f / (wave_sum(p0 + p1) + (dm.off1 ? expf(-m) : 0.f));
                p0 *= inv;
                p1 *= inv;
                const float Dj = wave_sum(p0 * dp[0] + p1 * dp[1]);
                // dZ carries beta, so the sums below go straight into the chunk's accumulators
                const float bwt = dm.beta * wt;
                if (lane < CS) {
                    pw[j * CS + lane] = wt * p0;
                    dz[j * CS + lane] = bwt * p0 * (dp[0] - Dj);
                }
                if (lane + 64 < CS) {
                    pw[j * CS + lane + 64] = wt * p1;
                    dz[j * CS + lane + 64] = bwt * p1 * (dp[1] - Dj);
                }
            }
            if (tid < D) {
                for (int tk = 0; tk < n; ++tk) {
                    float qs = 0.f;
                    for (int j = 0; j < h; ++j) qs += qf[(tk * h + j) * D + tid];
                    dkbar = fmaf(dm.alpha * tds[tk], qs, dkbar);
                }
            }
            __syncthreads();
            // a thread's elements share their column when kThreads is a multiple of D: the
            // batch's q and dO values of that column are read once per row
            if constexpr (kThreads % D == 0) {
                const int e = tid % D;
                for (int j = 0; j < nrows; ++j) {
                    const float gv = gf[j * D + e], qv = qf[j * D + e];
#pragma unroll
                    for (int r = 0; r < NE; ++r) {
                        const int s = (tid + r * kThreads) / D;
                        aV[r] = fmaf(pw[j * CS + s], gv, aV[r]);
                        aK[r] = fmaf(dz[j * CS + s], qv, aK[r]);
                    }
                }
            } else {
#pragma unroll
                for (int r = 0; r < NE; ++r) {
                    const int i = tid + r * kThreads;
                    const int s = i / D, e = i % D;
                    for (int j = 0; j < nrows; ++j) {
                        aV[r] = fmaf(pw[j * CS + s], gf[j * D + e], aV[r]);
                        aK[r] = fmaf(dz[j * CS + s], qf[j * D + e], aK[r]);
                    }
                }
            }
        };

        // the segment's tokens [4 j0, min(4 j1, count)) of the chunk's ascending token list, a
        // run of kGenList at a time, in batches of TB
        const uint32_t* bmrow = bm + (size_t)r * nwords;
        const int p0 = 4 * sg.j0, p1 = min(4 * sg.j1, cntr[r]);
        for (int q0 = p0; q0 < p1; q0 += kGenList) {
            const int q1 = min(q0 + kGenList, p1);
            __syncthreads();                 // the previous run's list is read
            collect_tokens<kThreads>(bmrow, ((c + 1) * CS) >> 5, nwords, q0, q1, tlist, wtot, tid);
            __syncthreads();
            for (int i0 = 0; i0 < q1 - q0; i0 += TB) batch(tlist + i0, min(TB, q1 - q0 - i0));
        }
        __syncthreads();
        if (tid < D) dkb[tid] = dkbar;
        __syncthreads();
        // a row covered whole is final; a shared one leaves fp32 partials in the workgroup's
        // slot (first row of its range 0, last 1), added in workgroup order by kv_generic_finish
        float* pk = part + ((size_t)lid * 2 + sg.pslot) * (2 * CS * D);
#pragma unroll
        for (int r2 = 0; r2 < NE; ++r2) {
            const int i = tid + r2 * kThreads;
            const int s = i / D, e = i % D;
            if (sg.whole) {
                const size_t gi = (rowbase + (size_t)s * dm.G) * D + e;
                dK[gi] = from_f32<T>(aK[r2] + dkb[e] * invS);
                dV[gi] = from_f32<T>(aV[r2]);
            } else {
                pk[i] = aK[r2] + dkb[e] * invS;
                pk[CS * D + i] = aV[r2];
            }
        }
    }
}

// dK, dV of every chunk row the key pass did not write: zeros for a trailing partial chunk or
// one no token selected, and for a chunk shared by several workgroups the sum of their
// partials in workgroup order (a chunk selected by most tokens is shared by a hundred and
// more: its elements are spread over gridDim.y workgroups, and the loads of 16 partials are
// in flight together)
template <typename T, int D, int CS>
__global__ __launch_bounds__(kThreads) void kv_generic_finish(
    Dims dm, const int* __restrict__ gstart, const int* __restrict__ cntr,
    const int* __restrict__ plan, const float* __restrict__ part, T* __restrict__ dK,
    T* __restrict__ dV) {
    const int c = blockIdx.x % dm.Call;
    const int bg = blockIdx.x / dm.Call, b = bg / dm.G, g = bg % dm.G;
    const size_t rowbase = ((size_t)b * dm.L + (size_t)c * CS) * dm.G + g;
    const int r = bg * dm.C + c;
    const int i0 = blockIdx.y * kThreads + threadIdx.x, istep = gridDim.y * kThreads;
    if (c >= dm.C || cntr[r] == 0) {
        const int rows = min(CS, dm.L - c * CS);
        for (int i = i0; i < rows * D; i += istep) {
            const size_t gi = (rowbase + (size_t)(i / D) * dm.G) * D + i % D;
            dK[gi] = from_f32<T>(0.f);
            dV[gi] = from_f32<T>(0.f);
        }
        return;
    }
    const int Tg = plan[1];
    const int rs = gstart[r], re = gstart[r + 1];
    const int wf = rs / Tg, wl = (re - 1) / Tg;
    if (wf == wl) return;                // written by its workgroup
    for (int i = i0; i < CS * D; i += istep) {
        float sk = 0.f, sv = 0.f;
        for (int w0 = wf; w0 <= wl; w0 += 16) {
            float vk[16], vv[16];
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int wg = min(w0 + j, wl);
                // the row is the first of each later workgroup's range, and of wf's when
                // wf's range starts there
                const int sl = (wg > wf || rs == wf * Tg) ? 0 : 1;
                const float* pk = part + ((size_t)wg * 2 + sl) * (2 * CS * D);
                vk[j] = pk[i];
                vv[j] = pk[CS * D + i];
            }
#pragma unroll
            for (int j = 0; j < 16; ++j)
                if (w0 + j <= wl) {
                    sk += vk[j];
                    sv += vv[j];
                }
        }
        const size_t gi = (rowbase + (size_t)(i / D) * dm.G) * D + i % D;
        dK[gi] = from_f32<T>(sk);
        dV[gi] = from_f32<T>(sv);
    }
}

// The generic key pass runs on the even split of (chunk, 4-token group) work over kGenWGs
// workgroups (stream_rowcount, stream_plan), so a chunk selected by most tokens is shared
// by several workgroups instead of setting the kernel time (tiny fp32 workload: key pass and
// finish 110 -> 69 us with the plan, against 32 fixed splits per chunk).
template <typename T, int D, int CS>
void launch_kv(const Dims& dm, const void* Q, const void* K, const void* V, const int32_t* idx,
               const float* w, const void* dO, const float* ds, const uint32_t* bm, int nwords,
               void* dK, void* dV, int* plan_ws, float* part, hipStream_t st) {
    const int R = dm.B * dm.G * dm.C;
    int* cnt = plan_ws;
    int* gstart = cnt + R;
    int* plan = gstart + R + 1;
    if (R > 0) {
        {
            HSA_TIMED("bwd_plan", st);
            hipLaunchKernelGGL(stream_rowcount, dim3(cdiv(R, 4)), dim3(256), 0, st, bm, R,
                               nwords, dm.C, dm.S, cnt);
            hipLaunchKernelGGL(stream_plan, dim3(1), dim3(1024), 0, st, (const int*)cnt, R,
                               kGenWGs, gstart, plan);
        }
        HSA_TIMED("bwd_kv_generic", st);
        hipLaunchKernelGGL((bwd_kv_generic<T, D, CS>), dim3(kGenWGs), dim3(kThreads), 0, st, dm,
                           (const T*)Q, (const T*)K, (const T*)V, idx, w, (const T*)dO, ds, bm,
                           nwords, (const int*)gstart, (const int*)cnt, (const int*)plan,
                           (T*)dK, (T*)dV, part);
    }
    HSA_TIMED("bwd_kv_finish", st);
    hipLaunchKernelGGL((kv_generic_finish<T, D, CS>), dim3(dm.Call * dm.B * dm.G, 16),
                       dim3(kThreads), 0, st, dm, (const int*)gstart, (const int*)cnt,
                       (const int*)plan, (const float*)part, (T*)dK, (T*)dV);
}

template <typename T, int D>
void launch_kv_s(const Dims& dm, const void* Q, const void* K, const void* V,
                 const int32_t* idx, const float* w, const void* dO, const float* ds,
                 const uint32_t* bm, int nwords, void* dK, void* dV, int* plan_ws,
                 float* part, hipStream_t st) {
    switch (dm.S) {
        case 16:
            launch_kv<T, D, 16>(dm, Q, K, V, idx, w, dO, ds, bm, nwords, dK, dV, plan_ws, part,
                              st);
            break;
        case 32:
            launch_kv<T, D, 32>(dm, Q, K, V, idx, w, dO, ds, bm, nwords, dK, dV, plan_ws, part,
                              st);
            break;
        case 64:
            launch_kv<T, D, 64>(dm, Q, K, V, idx, w, dO, ds, bm, nwords, dK, dV, plan_ws, part,
                              st);
            break;
        default:
            // fp32 with S = 128 and d = 128 exceeds the LDS of one workgroup; rejected by the
            // argument checks, so it is not instantiated.
            if constexpr (!(sizeof(T) == 4 && D == 128))
                launch_kv<T, D, 128>(dm, Q, K, V, idx, w, dO, ds, bm, nwords, dK, dV, plan_ws,
                                     part, st);
            break;
    }
}

void launch_bitmap(const Dims& dm, const int32_t* idx, uint32_t* bm, hipStream_t st) {
    if ((size_t)dm.B * dm.G * dm.C * dm.L == 0) return;
    HSA_TIMED("bitmap_build", st);
    hipLaunchKernelGGL(bitmap_build,
                       dim3((unsigned)cdiv(dm.L, 256), (unsigned)(dm.B * dm.G),
                            (unsigned)cdiv(dm.C, kBmRange)),
                       dim3(256), 0, st, dm, idx, bm, cdiv(dm.L, 32));
}

// selection bitmap, then the chunk-major key/value pass (ds already in the workspace)
template <typename T>
void launch_kv_pass(const Dims& dm, const void* Q, const void* K, const void* V,
                    const int32_t* idx, const float* w, const void* dO, void* dK, void* dV,
                    void* ws, hipStream_t st) {
    const int nwords = cdiv(dm.L, 32);
    const float* ds = (const float*)ws;
    uint32_t* bm = (uint32_t*)((char*)ws + align256((size_t)dm.B * dm.L * dm.G * dm.k * 4));
    const size_t nbm = (size_t)dm.B * dm.G * dm.C * nwords;
    launch_bitmap(dm, idx, bm, st);
    // the split's row counts, group prefix and plan, then the per-workgroup partials
    const size_t R = (size_t)dm.B * dm.G * dm.C;
    int* plan_ws = (int*)((char*)bm + align256(nbm * 4));
    float* part = (float*)((char*)plan_ws + align256((2 * R + 3) * 4));
    if (dm.d == 128)
        launch_kv_s<T, 128>(dm, Q, K, V, idx, w, dO, ds, bm, nwords, dK, dV, plan_ws, part, st);
    else
        launch_kv_s<T, 64>(dm, Q, K, V, idx, w, dO, ds, bm, nwords, dK, dV, plan_ws, part, st);
}

template <typename T>
hipError_t launch_t(const Dims& dm, const void* Q, const void* K, const void* V,
                    const float* Kbar, const int32_t* idx, const float* w, const void* dO,
                    void* dQ, void* dK, void* dV, void* ws, hipStream_t st) {
    float* ds = (float*)ws;
    dim3 g1(dm.L, dm.B * dm.G);
    // LDS sized for the chunk (so short chunks leave room for more workgroups per CU)
    auto q_pass = [&](auto dc, auto sc) {
        constexpr int DD = decltype(dc)::value, SS = decltype(sc)::value;
        HSA_TIMED("bwd_q_generic", st);
        hipLaunchKernelGGL((bwd_q_generic<T, DD, SS>), g1, dim3(kThreads), 0, st, dm, (const T*)Q,
                           (const T*)K, (const T*)V, Kbar, idx, w, (const T*)dO, (T*)dQ, ds);
    };
    auto q_pass_s = [&](auto dc) {
        switch (dm.S) {
            case 16: q_pass(dc, std::integral_constant<int, 16>{}); break;
            case 32: q_pass(dc, std::integral_constant<int, 32>{}); break;
            case 64: q_pass(dc, std::integral_constant<int, 64>{}); break;
            default:
                // float32 with S = 128 and d = 128 is rejected by the argument checks
                if constexpr (!(sizeof(T) == 4 && decltype(dc)::value == 128))
                    q_pass(dc, std::integral_constant<int, 128>{});
                break;
        }
    };
    if (dm.d == 128) q_pass_s(std::integral_constant<int, 128>{});
    else q_pass_s(std::integral_constant<int, 64>{});
    launch_kv_pass<T>(dm, Q, K, V, idx, w, dO, dK, dV, ws, st);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_selection_bitmap(const Dims& dm, const int32_t* idx, uint32_t* bm,
                                   hipStream_t st) {
    launch_bitmap(dm, idx, bm, st);
    return hipGetLastError();
}

size_t backward_generic_workspace(const Dims& dm) {
    const size_t nwords = (size_t)cdiv(dm.L, 32);
    const size_t R = (size_t)dm.B * dm.G * dm.C;
    const size_t part = (size_t)kGenWGs * 2 * 2 * dm.S * dm.d * 4;
    return align256((size_t)dm.B * dm.L * dm.G * dm.k * 4) + align256(R * nwords * 4) +
           align256((2 * R + 3) * 4) + align256(part);
}

size_t backward_workspace(const Dims& dm) {
    const size_t a = backward_generic_workspace(dm);
    const size_t b = backward_mfma_workspace(dm);
    const size_t f = backward_fused_workspace(dm);
    const size_t ab = a > b ? a : b;
    return ab > f ? ab : f;
}

hipError_t launch_backward_generic(const Dims& dm, bool in_bf16, const void* Q, const void* K,
                                   const void* V, const float* Kbar, const int32_t* idx,
                                   const float* w, const void* dO, void* dQ, void* dK, void* dV,
                                   void* ws, hipStream_t st) {
    if (dm.B == 0 || dm.L == 0) return hipSuccess;
    return in_bf16 ? launch_t<bf16>(dm, Q, K, V, Kbar, idx, w, dO, dQ, dK, dV, ws, st)
                   : launch_t<float>(dm, Q, K, V, Kbar, idx, w, dO, dQ, dK, dV, ws, st);
}

hipError_t launch_backward(const Dims& dm, bool in_bf16, const void* Q, const void* K,
                           const void* V, const float* Kbar, const int32_t* idx, const float* w,
                           const void* dO, void* dQ, void* dK, void* dV, void* ws,
                           hipStream_t st) {
    if (dm.B == 0 || dm.L == 0) return hipSuccess;
    if (backward_fused_supported(dm, in_bf16))
        return launch_backward_fused(dm, Q, K, V, Kbar, idx, w, dO, dQ, dK, dV, ws, st);
    if (backward_mfma_supported(dm, in_bf16))
        return launch_backward_mfma(dm, Q, K, V, Kbar, idx, w, dO, dQ, dK, dV, ws, st);
    return launch_backward_generic(dm, in_bf16, Q, K, V, Kbar, idx, w, dO, dQ, dK, dV, ws, st);
}

}  // namespace hsa
