// Single-token decode (Sec. 3.2 "Inference"): only the landmark cache is scanned and only
// the selected chunks' keys and values are read.
//
// Stage 1 (scan): workgroup = (b, slice of 256 chunks).  The slice's landmark rows for all
// G groups are one contiguous block of the [B, C, G, d] cache, streamed with 16-byte loads
// (all of a thread's loads issued first); D/VN consecutive lanes share a row and reduce
// their partial dot products with DPP moves.  Each wave then extracts the slice's top-k of
// one group by k rounds of a wave-wide arg-max (ties to the lower chunk index) and writes
// k (score, chunk) candidates.
// Stage 2 (finish): workgroup = (slot, b, g): the k selected chunks are attended in
// parallel.  Stage 3 (combine): workgroup = (b, g), sums their weighted partial outputs in
// slot order.
#include "common.h"

namespace hsa {
namespace {

constexpr int kScanThreads = 256;
constexpr int SL = 256;            // chunks per scan slice
constexpr int GMAX = 16;
constexpr int kFinThreads = 256;
constexpr int NW = kFinThreads / 64;
constexpr int HMAX = 16;
constexpr int KMAX = 32;
constexpr int NCMAX = 4096;        // slice candidates merged from LDS (else from global memory)

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
    // U vectors per thread per pass, loads first; a row's LPR lanes reduce with DPP moves
    constexpr int U = 32;
    for (int v0 = 0; v0 < nvec; v0 += kScanThreads * U) {
        uint4 raw[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int v = v0 + u * kScanThreads + tid;
            raw[u] = v < nvec ? *reinterpret_cast<const uint4*>(base + (size_t)(v / LPR) * D +
                                                                (v % LPR) * VN)
                              : uint4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int v = v0 + u * kScanThreads + tid;
            const int row = v / LPR, part = v % LPR;
            const float* qg = qs + (row % G) * D + part * VN;
            float xu[VN];
            unpack16(reinterpret_cast<const Tk*>(&raw[u]), xu);
            float dot = 0.f;
#pragma unroll
            for (int i = 0; i < VN; ++i) dot = fmaf(qg[i], xu[i], dot);
            dot = group_sum<LPR>(dot);
            if (v < nvec && part == 0) sc[row] = dm.alpha * dot;
        }
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
            for (int m = 0; m < SL / 64; ++m) pick_better(bs, bc, s[m], lane + 64 * m);
            wave_argmax_dpp(bs, bc);
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

// Stage 2 (finish): workgroup = (slot, b, g), so the k selected chunks of a sequence are
// attended in parallel.  Wave 0 of every workgroup merges the slice candidates into the
// final top-k (the same deterministic merge in each), computes the softmax chunk weights and
// the descending-chunk slot order.  The workgroup of slot i stages its chunk's K and V in
// LDS, computes the intra-chunk softmax of the h heads and w_i P V, and stores that partial
// output.  Stage 3 (combine) sums the partials of a (b, g) in slot order.
template <typename T, int D>
__global__ __launch_bounds__(kFinThreads) void decode_finish(
    Dims dm, const T* __restrict__ q, const T* __restrict__ Kc, const T* __restrict__ Vc,
    const int32_t* __restrict__ cache_len, const float* __restrict__ cand_s,
    const int32_t* __restrict__ cand_c, int nslices, float* __restrict__ part,
    int32_t* __restrict__ idx_out, float* __restrict__ w_out) {
    constexpr int DP = D + 1;
    constexpr int SMAX = 128;
    constexpr int NE = sizeof(T) == 4 ? 8192 : SMAX * D;   // S * d <= 8192 for fp32 inputs
    __shared__ T ks[NE];
    __shared__ T vs[NE];
    __shared__ float qf[HMAX * DP];
    __shared__ float pz[HMAX * SMAX];
    __shared__ int sel_c[KMAX];
    __shared__ float sel_w[KMAX];
    __shared__ float lcs[NCMAX];
    __shared__ int lcc[NCMAX];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int slot = blockIdx.x;
    const int bg = blockIdx.y, b = bg / dm.G, g = bg % dm.G;
    const int h = dm.h, S = dm.S, k = dm.k;
    const int ncand = cache_tokens(cache_len, b, dm.L) / S;
    const int n = min(k, ncand);

    for (int i = tid; i < h * D; i += kFinThreads)
        qf[(i / D) * DP + i % D] = to_f32(q[((size_t)b * dm.H + (size_t)g * h) * D + i]);
    const int nc = nslices * k;
    const bool in_lds = nc <= NCMAX;
    if (in_lds) {
        for (int x = tid; x < nc; x += kFinThreads) {
            lcs[x] = cand_s[(size_t)bg * nc + x];
            lcc[x] = cand_c[(size_t)bg * nc + x];
        }
    }
    __syncthreads();
    if (wave == 0) {
        const float* cs = in_lds ? lcs : cand_s + (size_t)bg * nc;
        const int32_t* cc = in_lds ? lcc : cand_c + (size_t)bg * nc;
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
            wave_argmax_dpp(bs, bc);
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
        } else if (lane < k) {
            sel_c[lane] = -1;
            sel_w[lane] = 0.f;
        }
    }
    __syncthreads();
    if (slot == 0 && tid < k) {
        idx_out[(size_t)bg * k + tid] = sel_c[tid];
        w_out[(size_t)bg * k + tid] = sel_w[tid];
    }

    if (slot < n) {
        const int c = sel_c[slot];
        const float wi = sel_w[slot];
        // the chunk's S rows of K and V for group g
        constexpr int VN = V16<T>::n;
        for (int v = tid; v < S * D / VN; v += kFinThreads) {
            const int s = v / (D / VN), e = (v % (D / VN)) * VN;
            const size_t src = (((size_t)b * dm.L + (size_t)c * S + s) * dm.G + g) * D + e;
            *reinterpret_cast<uint4*>(&ks[s * D + e]) = *reinterpret_cast<const uint4*>(Kc + src);
            *reinterpret_cast<uint4*>(&vs[s * D + e]) = *reinterpret_cast<const uint4*>(Vc + src);
        }
        __syncthreads();
        // logits z[j][s] = beta q_j . k_s
        for (int x = tid; x < S * h; x += kFinThreads) {
            const int s = x / h, j = x % h;
            float a0 = 0.f, a1 = 0.f;
#pragma unroll 8
            for (int e = 0; e < D; e += 2) {
                a0 = fmaf(qf[j * DP + e], to_f32(ks[s * D + e]), a0);
                a1 = fmaf(qf[j * DP + e + 1], to_f32(ks[s * D + e + 1]), a1);
            }
            pz[j * SMAX + s] = dm.beta * (a0 + a1);
        }
        __syncthreads();
        // intra-chunk softmax of each head, scaled by the chunk weight
        for (int j = wave; j < h; j += NW) {
            const float z0 = lane < S ? pz[j * SMAX + lane] : -INFINITY;
            const float z1 = lane + 64 < S ? pz[j * SMAX + lane + 64] : -INFINITY;
            const float m = wave_max(fmaxf(z0, z1));
            const float e0 = lane < S ? expf(z0 - m) : 0.f;
            const float e1 = lane + 64 < S ? expf(z1 - m) : 0.f;
            const float scale = wi / wave_sum(e0 + e1);
            if (lane < S) pz[j * SMAX + lane] = e0 * scale;
            if (lane + 64 < S) pz[j * SMAX + lane + 64] = e1 * scale;
        }
        __syncthreads();
        // w_i P V for the h heads
        float* pp = part + (((size_t)bg * k + slot) * h) * D;
        for (int x = tid; x < h * D; x += kFinThreads) {
            const int j = x / D, d = x % D;
            float a0 = 0.f, a1 = 0.f;
            for (int s = 0; s < S; s += 2) {
                a0 = fmaf(pz[j * SMAX + s], to_f32(vs[s * D + d]), a0);
                a1 = fmaf(pz[j * SMAX + s + 1], to_f32(vs[(s + 1) * D + d]), a1);
            }
            pp[x] = a0 + a1;
        }
    }

}

template <typename T, int D>
__global__ __launch_bounds__(256) void decode_combine(Dims dm,
                                                      const int32_t* __restrict__ cache_len,
                                                      const float* __restrict__ part,
                                                      T* __restrict__ o) {
    const int bg = blockIdx.x, b = bg / dm.G, g = bg % dm.G;
    const int h = dm.h, k = dm.k;
    const int n = min(k, cache_tokens(cache_len, b, dm.L) / dm.S);
    for (int x = threadIdx.x; x < h * D; x += 256) {
        float s = 0.f;
        for (int i = 0; i < n; ++i) s += part[(((size_t)bg * k + i) * h) * D + x];
        o[((size_t)b * dm.H + (size_t)g * h) * D + x] = from_f32<T>(s);
    }
}

struct DecodeWs {
    size_t cs, cc, part, end;
};
DecodeWs decode_ws(const Dims& dm) {
    const size_t nslices = (size_t)cdiv(dm.C > 0 ? dm.C : 1, SL);
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    DecodeWs l;
    l.cs = 0;
    l.cc = al(l.cs + (size_t)dm.B * dm.G * nslices * dm.k * 4);
    l.part = al(l.cc + (size_t)dm.B * dm.G * nslices * dm.k * 4);
    l.end = al(l.part + (size_t)dm.B * dm.G * dm.k * dm.h * dm.d * 4);
    return l;
}

template <typename T, typename Tk, int D>
void launch_tkd(const Dims& dm, const void* q, const void* Kc, const void* Vc, const void* Kbar,
                const int32_t* cache_len, void* o, int32_t* idx, float* w, void* ws,
                hipStream_t st) {
    const int nslices = cdiv(dm.C > 0 ? dm.C : 1, SL);
    const DecodeWs l = decode_ws(dm);
    char* wb = (char*)ws;
    float* cs = (float*)(wb + l.cs);
    int32_t* cc = (int32_t*)(wb + l.cc);
    float* part = (float*)(wb + l.part);
    {
        HSA_TIMED("decode_scan", st);
        hipLaunchKernelGGL((decode_scan<T, Tk, D>), dim3(nslices, dm.B), dim3(kScanThreads), 0,
                           st, dm, (const T*)q, (const Tk*)Kbar, cache_len, cs, cc,
                           nslices);
    }
    {
        HSA_TIMED("decode_finish", st);
        hipLaunchKernelGGL((decode_finish<T, D>), dim3(dm.k, dm.B * dm.G), dim3(kFinThreads), 0,
                           st, dm, (const T*)q, (const T*)Kc, (const T*)Vc, cache_len, cs, cc,
                           nslices, part, idx, w);
    }
    {
        HSA_TIMED("decode_combine", st);
        hipLaunchKernelGGL((decode_combine<T, D>), dim3(dm.B * dm.G), dim3(256), 0, st, dm,
                           cache_len, part, (T*)o);
    }
}

template <typename T, typename Tk>
void launch_tk(const Dims& dm, const void* q, const void* Kc, const void* Vc, const void* Kbar,
               const int32_t* cache_len, void* o, int32_t* idx, float* w, void* ws,
               hipStream_t st) {
    if (dm.d == 128) launch_tkd<T, Tk, 128>(dm, q, Kc, Vc, Kbar, cache_len, o, idx, w, ws, st);
    else launch_tkd<T, Tk, 64>(dm, q, Kc, Vc, Kbar, cache_len, o, idx, w, ws, st);
}

}  // namespace

size_t decode_workspace(const Dims& dm) { return decode_ws(dm).end; }

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
