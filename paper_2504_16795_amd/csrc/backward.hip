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

__host__ __device__ inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

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
    float acc[NACC];
#pragma unroll
    for (int r = 0; r < NACC; ++r) acc[r] = 0.f;

    for (int slot = 0; slot < k; ++slot) {
        const int c = idx[sel + slot];
        if (c < 0 || c >= ncand) continue;
        const float wi = w[sel + slot];
        __syncthreads();
        for (int i = tid; i < S * D; i += kThreads) {
            const int s = i / D, e = i % D;
            const size_t gi = (((size_t)b * dm.L + (size_t)c * S + s) * dm.G + g) * D + e;
            Ks[s * KP + e] = K[gi];
            Vs[s * KP + e] = V[gi];
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
            dwl[slot] = s;
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
    __shared__ uint32_t wlist[kThreads];
    __shared__ int tlist[HMAX];          // the tokens of a batch
    __shared__ float twt[HMAX], tds[HMAX];   // their weights and ds for this chunk

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int c = blockIdx.x;
    const int bg = blockIdx.y, b = bg / dm.G, g = bg % dm.G;
    const int h = dm.h, k = dm.k;
    const size_t rowbase = ((size_t)b * dm.L + (size_t)c * CS) * dm.G + g;   // row cS

    // split z of nsplit takes the chunk's tokens z, z + nsplit, ... (in increasing order) and,
    // with more than one split, writes fp32 partials that kv_generic_finish adds in split order
    const int z = blockIdx.z, nsplit = gridDim.z;
    if (c >= dm.C) {   // trailing partial chunk: never selected, zero gradient
        if (z != 0) return;
        const int rows = dm.L - c * CS;
        for (int i = tid; i < rows * D; i += kThreads) {
            const size_t gi = (rowbase + (size_t)(i / D) * dm.G) * D + i % D;
            dK[gi] = from_f32<T>(0.f);
            dV[gi] = from_f32<T>(0.f);
        }
        return;
    }
    for (int i = tid; i < CS * D; i += kThreads) {
        const int s = i / D, e = i % D;
        const size_t gi = (rowbase + (size_t)s * dm.G) * D + e;
        Ks[s * KP + e] = K[gi];
        Vs[s * KP + e] = V[gi];
    }
    float aK[NE], aV[NE];
#pragma unroll
    for (int r = 0; r < NE; ++r) aK[r] = aV[r] = 0.f;
    float dkbar = 0.f;   // thread tid < D owns element tid of dKbar

    // Tokens are taken TB = floor(HMAX / h) at a time: the batch's (token, head) rows fill
    // the HMAX-row LDS arrays, so a batch costs the barriers and memory round trips of one
    // token.
    const int TB = HMAX / h;
    auto batch = [&](int n) __attribute__((always_inline)) {
        const int nrows = n * h;
        __syncthreads();                  // the previous batch's rows are read
        for (int i = tid; i < nrows * D; i += kThreads) {
            const int tk = i / (h * D), r = i - tk * (h * D);
            const size_t qoff = (((size_t)b * dm.L + tlist[tk]) * dm.H + (size_t)g * h) * D;
            qf[i] = to_f32(Q[qoff + r]);
            gf[i] = to_f32(dO[qoff + r]);
        }
        if (tid < n) {                    // the token's slot holding c: its w and ds
            const size_t sel = (((size_t)b * dm.L + tlist[tid]) * dm.G + g) * k;
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
            if (lane < CS) {
                pw[j * CS + lane] = wt * p0;
                dz[j * CS + lane] = wt * p0 * (dp[0] - Dj);
            }
            if (lane + 64 < CS) {
                pw[j * CS + lane + 64] = wt * p1;
                dz[j * CS + lane + 64] = wt * p1 * (dp[1] - Dj);
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
            float av[NE], ak[NE];
#pragma unroll
            for (int r = 0; r < NE; ++r) av[r] = ak[r] = 0.f;
            for (int j = 0; j < nrows; ++j) {
                const float gv = gf[j * D + e], qv = qf[j * D + e];
#pragma unroll
                for (int r = 0; r < NE; ++r) {
                    const int s = (tid + r * kThreads) / D;
                    av[r] = fmaf(pw[j * CS + s], gv, av[r]);
                    ak[r] = fmaf(dz[j * CS + s], qv, ak[r]);
                }
            }
#pragma unroll
            for (int r = 0; r < NE; ++r) {
                aV[r] += av[r];
                aK[r] = fmaf(dm.beta, ak[r], aK[r]);
            }
        } else {
#pragma unroll
            for (int r = 0; r < NE; ++r) {
                const int i = tid + r * kThreads;
                const int s = i / D, e = i % D;
                float av = 0.f, ak = 0.f;
                for (int j = 0; j < nrows; ++j) {
                    av = fmaf(pw[j * CS + s], gf[j * D + e], av);
                    ak = fmaf(dz[j * CS + s], qf[j * D + e], ak);
                }
                aV[r] += av;
                aK[r] = fmaf(dm.beta, ak, aK[r]);
            }
        }
    };

    const uint32_t* row = bm + (((size_t)b * dm.G + g) * dm.C + c) * nwords;
    int ord = 0;                         // the token's place in the chunk's token list
    int nb = 0;                          // tokens of the current batch
    // the bitmap row is read kThreads words at a time into LDS (one load per thread), so
    // the walk over the words waits for no memory access of its own
    for (int wb = ((c + 1) * CS) >> 5; wb < nwords; wb += kThreads) {
        __syncthreads();                 // the previous batch of words is read
        if (wb + tid < nwords) wlist[tid] = row[wb + tid];
        __syncthreads();
        const int wend = min(nwords, wb + kThreads);
        for (int wi = wb; wi < wend; ++wi) {
            uint32_t word = wlist[wi - wb];
            while (word) {
                const int t = wi * 32 + (__ffs(word) - 1);
                word &= word - 1;
                if (ord++ % nsplit != z) continue;
                // the list is read by the batch only after its first barrier
                if (tid == 0) tlist[nb] = t;
                if (++nb == TB) {
                    batch(nb);
                    nb = 0;
                }
            }
        }
    }
    if (nb > 0) batch(nb);
    __syncthreads();
    if (tid < D) dkb[tid] = dkbar;
    __syncthreads();
    const float invS = 1.f / (float)CS;
    float* pk = nsplit > 1 ? part + (((size_t)z * dm.B * dm.G + bg) * dm.C + c) * (2 * CS * D)
                           : nullptr;
#pragma unroll
    for (int r = 0; r < NE; ++r) {
        const int i = tid + r * kThreads;
        const int s = i / D, e = i % D;
        if (nsplit > 1) {
            pk[i] = aK[r] + dkb[e] * invS;
            pk[CS * D + i] = aV[r];
        } else {
            const size_t gi = (rowbase + (size_t)s * dm.G) * D + e;
            dK[gi] = from_f32<T>(aK[r] + dkb[e] * invS);
            dV[gi] = from_f32<T>(aV[r]);
        }
    }
}

// dK, dV of a complete chunk from the key pass's per-split partials, added in split order
// (the chunk's elements spread over gridDim.z workgroups)
template <typename T, int D, int CS>
__global__ __launch_bounds__(kThreads) void kv_generic_finish(Dims dm, int nsplit,
                                                              const float* __restrict__ part,
                                                              T* __restrict__ dK,
                                                              T* __restrict__ dV) {
    const int c = blockIdx.x, bg = blockIdx.y, b = bg / dm.G, g = bg % dm.G;
    const size_t rowbase = ((size_t)b * dm.L + (size_t)c * CS) * dm.G + g;
    const size_t zstride = (size_t)dm.B * dm.G * dm.C * (2 * CS * D);
    const float* p0 = part + ((size_t)bg * dm.C + c) * (2 * CS * D);
    for (int i = blockIdx.z * kThreads + threadIdx.x; i < CS * D; i += gridDim.z * kThreads) {
        float sk = 0.f, sv = 0.f;
        // the loads of 8 splits in flight together, the sums still in split order
        for (int z0 = 0; z0 < nsplit; z0 += 8) {
            float vk[8], vv[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float* pk = p0 + (size_t)min(z0 + j, nsplit - 1) * zstride;
                vk[j] = pk[i];
                vv[j] = pk[CS * D + i];
            }
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (z0 + j < nsplit) {
                    sk += vk[j];
                    sv += vv[j];
                }
        }
        const size_t gi = (rowbase + (size_t)(i / D) * dm.G) * D + i % D;
        dK[gi] = from_f32<T>(sk);
        dV[gi] = from_f32<T>(sv);
    }
}

// Splits of the generic key pass: enough workgroups to fill the chip when the chunks are
// few (each chunk's tokens are otherwise walked by one workgroup, one after another), at
// most 32 (tiny fp32 workload, key pass and finish: 32 splits 109 us, 24 splits 132, 16
// splits 150, 48 splits 170, 64 splits 181: past two workgroups per CU the splits run in
// two rounds and the finish sums more partials).
inline int kv_splits(const Dims& dm) {
    const long rows = (long)dm.B * dm.G * dm.Call;
    long n = rows > 0 ? (1024 + rows - 1) / rows : 1;
    return (int)(n < 1 ? 1 : (n > 32 ? 32 : n));
}

template <typename T, int D, int CS>
void launch_kv(const Dims& dm, const void* Q, const void* K, const void* V, const int32_t* idx,
               const float* w, const void* dO, const float* ds, const uint32_t* bm, int nwords,
               void* dK, void* dV, float* part, hipStream_t st) {
    const int nsplit = kv_splits(dm);
    dim3 grid(dm.Call, dm.B * dm.G, nsplit);
    {
        HSA_TIMED("bwd_kv_generic", st);
        hipLaunchKernelGGL((bwd_kv_generic<T, D, CS>), grid, dim3(kThreads), 0, st, dm, (const T*)Q,
                           (const T*)K, (const T*)V, idx, w, (const T*)dO, ds, bm, nwords, (T*)dK,
                           (T*)dV, part);
    }
    if (nsplit > 1 && dm.C > 0) {
        HSA_TIMED("bwd_kv_finish", st);
        hipLaunchKernelGGL((kv_generic_finish<T, D, CS>), dim3(dm.C, dm.B * dm.G, 16),
                           dim3(kThreads), 0, st, dm, nsplit, (const float*)part, (T*)dK,
                           (T*)dV);
    }
}

template <typename T, int D>
void launch_kv_s(const Dims& dm, const void* Q, const void* K, const void* V,
                 const int32_t* idx, const float* w, const void* dO, const float* ds,
                 const uint32_t* bm, int nwords, void* dK, void* dV, float* part,
                 hipStream_t st) {
    switch (dm.S) {
        case 16: launch_kv<T, D, 16>(dm, Q, K, V, idx, w, dO, ds, bm, nwords, dK, dV, part, st); break;
        case 32: launch_kv<T, D, 32>(dm, Q, K, V, idx, w, dO, ds, bm, nwords, dK, dV, part, st); break;
        case 64: launch_kv<T, D, 64>(dm, Q, K, V, idx, w, dO, ds, bm, nwords, dK, dV, part, st); break;
        default:
            // fp32 with S = 128 and d = 128 exceeds the LDS of one workgroup; rejected by the
            // argument checks, so it is not instantiated.
            if constexpr (!(sizeof(T) == 4 && D == 128))
                launch_kv<T, D, 128>(dm, Q, K, V, idx, w, dO, ds, bm, nwords, dK, dV, part, st);
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
    // the key pass's per-split partials follow the bitmap
    float* part = (float*)((char*)bm + align256(nbm * 4));
    if (dm.d == 128)
        launch_kv_s<T, 128>(dm, Q, K, V, idx, w, dO, ds, bm, nwords, dK, dV, part, st);
    else
        launch_kv_s<T, 64>(dm, Q, K, V, idx, w, dO, ds, bm, nwords, dK, dV, part, st);
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
    const int nsplit = kv_splits(dm);
    const size_t part = nsplit > 1 ? (size_t)nsplit * dm.B * dm.G * dm.C * 2 * dm.S * dm.d * 4 : 0;
    return align256((size_t)dm.B * dm.L * dm.G * dm.k * 4) +
           align256((size_t)dm.B * dm.G * dm.C * nwords * 4) + align256(part);
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
