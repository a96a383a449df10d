// Single-token decode (Sec. 3.2 "Inference"): only the landmark cache is scanned and only
// the selected chunks' keys and values are read.
//
// Stage 1 (scan): workgroup = (b, slice of 256 chunks).  The slice's landmark rows for all
// G groups are one contiguous block of the [B, C, G, d] cache, streamed with 16-byte loads;
// D/VN consecutive lanes share a row and reduce their partial dot products with
// shuffles.  Each wave then extracts the slice's top-k of one group by k rounds of a
// wave-wide arg-max (ties to the lower chunk index) and writes k (score, chunk) candidates.
// Stage 2 (finish): workgroup = (b, g).  Wave 0 merges the slice candidates into the final
// top-k, computes the softmax chunk weights and the descending-chunk slot order; then the
// 8 waves take one slot each, compute the intra-chunk softmax for all h heads and the
// weighted P V, and the per-wave partial outputs are summed in a fixed order.
#include "common.h"

namespace hsa {
namespace {

constexpr int kScanThreads = 256;
constexpr int SL = 256;            // chunks per scan slice
constexpr int GMAX = 16;
constexpr int kFinThreads = 512;
constexpr int NW = kFinThreads / 64;
constexpr int HMAX = 16;
constexpr int KMAX = 32;

template <typename T> struct V16;
template <> struct V16<float> { static constexpr int n = 4; };
template <> struct V16<bf16> { static constexpr int n = 8; };

__device__ __forceinline__ void unpack16(const float* p, float* x) {
    const float4 r = *reinterpret_cast<const float4*>(p);
    x[0] = r.x; x[1] = r.y; x[2] = r.z; x[3] = r.w;
}
__device__ __forceinline__ void unpack16(const bf16* p, float* x) {
    const uint4 r = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[2 * i] = __uint_as_float(w[i] << 16);
        x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
}

__device__ __forceinline__ bool better(float s1, int c1, float s2, int c2) {
    return s1 > s2 || (s1 == s2 && c1 < c2);
}

// wave-wide arg-max of (s, c) pairs; ties to the lower c
__device__ __forceinline__ void wave_argmax(float& s, int& c) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float so = __shfl_xor(s, o, 64);
        const int co = __shfl_xor(c, o, 64);
        if (better(so, co, s, c)) {
            s = so;
            c = co;
        }
    }
}

__device__ __forceinline__ int cache_tokens(const int32_t* cache_len, int b, int ncap) {
    int n = cache_len ? cache_len[b] : ncap;
    return n < 0 ? 0 : (n > ncap ? ncap : n);
}

template <typename Tq, typename Tk, int D>
__global__ __launch_bounds__(kScanThreads) void decode_scan(
    Dims dm, const Tq* __restrict__ q, const Tk* __restrict__ Kbar,
    const int32_t* __restrict__ cache_len, float* __restrict__ cand_s,
    int32_t* __restrict__ cand_c, int nslices) {
    constexpr int VN = V16<Tk>::n;
    constexpr int LPR = D / VN;       // lanes per landmark row
    __shared__ float qs[GMAX * D];
    __shared__ float sc[SL * GMAX];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int b = blockIdx.y, slice = blockIdx.x;
    const int G = dm.G, h = dm.h, k = dm.k;
    const int ncand = cache_tokens(cache_len, b, dm.L) / dm.S;
    const int c0 = slice * SL;
    const int nch = max(0, min(SL, ncand - c0));

    for (int i = tid; i < G * D; i += kScanThreads) {
        const int g = i / D, e = i % D;
        float s = 0.f;
        for (int j = 0; j < h; ++j) s += to_f32(q[((size_t)b * dm.H + g * h + j) * D + e]);
        qs[i] = s;
    }
    __syncthreads();
    const Tk* base = Kbar + ((size_t)b * dm.C + c0) * G * D;
    const int nvec = nch * G * LPR;
    const int nit = cdiv(nvec, kScanThreads);
    for (int it = 0; it < nit; ++it) {
        const int v = it * kScanThreads + tid;
        const bool valid = v < nvec;
        const int row = v / LPR, part = v % LPR;
        float dot = 0.f;
        if (valid) {
            float x[VN];
            unpack16(base + (size_t)row * D + part * VN, x);
            const float* qg = qs + (row % G) * D + part * VN;
#pragma unroll
            for (int i = 0; i < VN; ++i) dot = fmaf(qg[i], x[i], dot);
        }
#pragma unroll
        for (int o = LPR / 2; o > 0; o >>= 1) dot += __shfl_xor(dot, o, 64);
        if (valid && part == 0) sc[row] = dm.alpha * dot;
    }
    __syncthreads();
    for (int g = wave; g < G; g += kScanThreads / 64) {
        float s[SL / 64];
#pragma unroll
        for (int m = 0; m < SL / 64; ++m) {
            const int cl = lane + 64 * m;
            s[m] = (cl < nch) ? sc[cl * G + g] : -INFINITY;
        }
        float* os = cand_s + (((size_t)b * G + g) * nslices + slice) * k;
        int32_t* oc = cand_c + (((size_t)b * G + g) * nslices + slice) * k;
        for (int i = 0; i < k; ++i) {
            float bs = -INFINITY;
            int bc = 0x7FFFFFFF;
#pragma unroll
            for (int m = 0; m < SL / 64; ++m) {
                const int cl = lane + 64 * m;
                if (better(s[m], cl, bs, bc)) {
                    bs = s[m];
                    bc = cl;
                }
            }
            wave_argmax(bs, bc);
            const bool found = bs > -INFINITY;
            if (lane == 0) {
                os[i] = bs;
                oc[i] = found ? c0 + bc : -1;
            }
#pragma unroll
            for (int m = 0; m < SL / 64; ++m)
                if (found && bc == lane + 64 * m) s[m] = -INFINITY;
        }
    }
}

template <typename T, int D>
__global__ __launch_bounds__(kFinThreads) void decode_finish(
    Dims dm, const T* __restrict__ q, const T* __restrict__ Kc, const T* __restrict__ Vc,
    const int32_t* __restrict__ cache_len, const float* __restrict__ cand_s,
    const int32_t* __restrict__ cand_c, int nslices, T* __restrict__ o,
    int32_t* __restrict__ idx_out, float* __restrict__ w_out) {
    constexpr int VN = V16<T>::n;
    constexpr int EPL = D / 64;       // output elements per lane in P V
    __shared__ float qf[HMAX * D];
    __shared__ int sel_c[KMAX];
    __shared__ float sel_w[KMAX];
    __shared__ float ow[NW][HMAX * D];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bg = blockIdx.x, b = bg / dm.G, g = bg % dm.G;
    const int h = dm.h, S = dm.S, k = dm.k;
    const int ncand = cache_tokens(cache_len, b, dm.L) / S;
    const int n = min(k, ncand);

    for (int i = tid; i < h * D; i += kFinThreads)
        qf[i] = to_f32(q[((size_t)b * dm.H + (size_t)g * h) * D + i]);
    if (wave == 0) {
        const int nc = nslices * k;
        const float* cs = cand_s + (size_t)bg * nc;
        const int32_t* cc = cand_c + (size_t)bg * nc;
        float ls = -INFINITY;      // lane i < n receives the i-th best candidate
        int lc = -1;
        // Candidates carry distinct chunk ids, so (score desc, chunk asc) is a strict total
        // order: round i takes the best candidate ranked below the winner of round i-1.
        float ps = INFINITY;
        int pc = -1;
        const int niter = cdiv(nc, 64);
        for (int i = 0; i < n; ++i) {
            float bs = -INFINITY;
            int bc = 0x7FFFFFFF;
            for (int it = 0; it < niter; ++it) {
                const int x = it * 64 + lane;
                if (x < nc) {
                    const int c = cc[x];
                    const float s = cs[x];
                    if (c >= 0 && better(ps, pc, s, c) && better(s, c, bs, bc)) {
                        bs = s;
                        bc = c;
                    }
                }
            }
            wave_argmax(bs, bc);
            if (lane == i) {
                ls = bs;
                lc = bc;
            }
            ps = bs;
            pc = bc;
        }
        const float m = __shfl(ls, 0, 64);
        const float ex = (lane < n) ? expf(ls - m) : 0.f;
        const float z = wave_sum(ex);
        int rank = 0;
        for (int j = 0; j < n; ++j) rank += (__shfl(lc, j, 64) > lc) ? 1 : 0;
        if (lane < n) {
            sel_c[rank] = lc;
            sel_w[rank] = ex / z;
            idx_out[(size_t)bg * k + rank] = lc;
            w_out[(size_t)bg * k + rank] = ex / z;
        } else if (lane < k) {
            sel_c[lane] = -1;
            sel_w[lane] = 0.f;
            idx_out[(size_t)bg * k + lane] = -1;
            w_out[(size_t)bg * k + lane] = 0.f;
        }
    }
    __syncthreads();

    float acc[HMAX][EPL];
#pragma unroll
    for (int j = 0; j < HMAX; ++j)
#pragma unroll
        for (int u = 0; u < EPL; ++u) acc[j][u] = 0.f;
    for (int slot = wave; slot < n; slot += NW) {
        const int c = sel_c[slot];
        const float wi = sel_w[slot];
        // logits: lane = key (two keys per lane for S = 128)
        float z[2][HMAX];
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int j = 0; j < HMAX; ++j) z[u][j] = 0.f;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int s = lane + 64 * u;
            if (s < S) {
                const T* kr = Kc + (((size_t)b * dm.L + (size_t)c * S + s) * dm.G + g) * D;
                for (int e0 = 0; e0 < D; e0 += VN) {
                    float x[VN];
                    unpack16(kr + e0, x);
#pragma unroll
                    for (int j = 0; j < HMAX; ++j) {
                        if (j < h) {
#pragma unroll
                            for (int i = 0; i < VN; ++i) z[u][j] = fmaf(qf[j * D + e0 + i], x[i], z[u][j]);
                        }
                    }
                }
            }
        }
        float pz[2][HMAX];
#pragma unroll
        for (int j = 0; j < HMAX; ++j) {
            pz[0][j] = pz[1][j] = 0.f;
            if (j < h) {
                const float z0 = (lane < S) ? dm.beta * z[0][j] : -INFINITY;
                const float z1 = (lane + 64 < S) ? dm.beta * z[1][j] : -INFINITY;
                const float m = wave_max(fmaxf(z0, z1));
                const float e0 = expf(z0 - m), e1 = expf(z1 - m);
                const float scale = wi / wave_sum(e0 + e1);
                pz[0][j] = e0 * scale;
                pz[1][j] = e1 * scale;
            }
        }
        // P V: lanes own output columns; the probability of key s is broadcast from lane s%64
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            for (int sl = 0; sl < 64 && u * 64 + sl < S; ++sl) {
                const int s = u * 64 + sl;
                const T* vr = Vc + (((size_t)b * dm.L + (size_t)c * S + s) * dm.G + g) * D;
                float v[EPL];
#pragma unroll
                for (int e = 0; e < EPL; ++e) v[e] = to_f32(vr[lane + 64 * e]);
#pragma unroll
                for (int j = 0; j < HMAX; ++j) {
                    if (j < h) {
                        const float p = __shfl(pz[u][j], sl, 64);
#pragma unroll
                        for (int e = 0; e < EPL; ++e) acc[j][e] = fmaf(p, v[e], acc[j][e]);
                    }
                }
            }
        }
    }
#pragma unroll
    for (int j = 0; j < HMAX; ++j)
        if (j < h)
#pragma unroll
            for (int u = 0; u < EPL; ++u) ow[wave][j * D + lane + 64 * u] = acc[j][u];
    __syncthreads();
    for (int i = tid; i < h * D; i += kFinThreads) {
        float s = 0.f;
        for (int wv = 0; wv < NW; ++wv) s += ow[wv][i];
        o[((size_t)b * dm.H + (size_t)g * h) * D + i] = from_f32<T>(s);
    }
}

template <typename T, typename Tk>
void launch_tk(const Dims& dm, const void* q, const void* Kc, const void* Vc, const void* Kbar,
               const int32_t* cache_len, void* o, int32_t* idx, float* w, void* ws,
               hipStream_t st) {
    const int nslices = cdiv(dm.C > 0 ? dm.C : 1, SL);
    float* cs = (float*)ws;
    int32_t* cc = (int32_t*)((char*)ws + (((size_t)dm.B * dm.G * nslices * dm.k * 4 + 255) & ~(size_t)255));
    dim3 g1(nslices, dm.B);
    if (dm.d == 128) {
        {
            HSA_TIMED("decode_scan", st);
            hipLaunchKernelGGL((decode_scan<T, Tk, 128>), g1, dim3(kScanThreads), 0, st, dm,
                               (const T*)q, (const Tk*)Kbar, cache_len, cs, cc, nslices);
        }
        {
            HSA_TIMED("decode_finish", st);
            hipLaunchKernelGGL((decode_finish<T, 128>), dim3(dm.B * dm.G), dim3(kFinThreads), 0, st,
                               dm, (const T*)q, (const T*)Kc, (const T*)Vc, cache_len, cs, cc,
                               nslices, (T*)o, idx, w);
        }
    } else {
        {
            HSA_TIMED("decode_scan", st);
            hipLaunchKernelGGL((decode_scan<T, Tk, 64>), g1, dim3(kScanThreads), 0, st, dm,
                               (const T*)q, (const Tk*)Kbar, cache_len, cs, cc, nslices);
        }
        {
            HSA_TIMED("decode_finish", st);
            hipLaunchKernelGGL((decode_finish<T, 64>), dim3(dm.B * dm.G), dim3(kFinThreads), 0, st,
                               dm, (const T*)q, (const T*)Kc, (const T*)Vc, cache_len, cs, cc,
                               nslices, (T*)o, idx, w);
        }
    }
}

}  // namespace

size_t decode_workspace(const Dims& dm) {
    const size_t nslices = (size_t)cdiv(dm.C > 0 ? dm.C : 1, SL);
    const size_t one = ((size_t)dm.B * dm.G * nslices * dm.k * 4 + 255) & ~(size_t)255;
    return 2 * one;
}

hipError_t launch_decode(const Dims& dm, bool in_bf16, const void* q, const void* Kc,
                         const void* Vc, const void* Kbar, bool kbar_bf16,
                         const int32_t* cache_len, void* o, int32_t* idx, float* w, void* ws,
                         hipStream_t st) {
    if (dm.B == 0) return hipSuccess;
    if (in_bf16) {
        if (kbar_bf16) launch_tk<bf16, bf16>(dm, q, Kc, Vc, Kbar, cache_len, o, idx, w, ws, st);
        else launch_tk<bf16, float>(dm, q, Kc, Vc, Kbar, cache_len, o, idx, w, ws, st);
    } else {
        if (kbar_bf16) launch_tk<float, bf16>(dm, q, Kc, Vc, Kbar, cache_len, o, idx, w, ws, st);
        else launch_tk<float, float>(dm, q, Kc, Vc, Kbar, cache_len, o, idx, w, ws, st);
    }
    return hipGetLastError();
}

}  // namespace hsa
