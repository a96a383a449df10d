// Gradient through the selection scores alone (Sec. 3.1: s_i = alpha q~ . Kbar_{c_i}; the
// weights of Sec. 3.1.1), for a selection over inputs of its own whose dw was summed over
// every layer that used it (Sec. 4.4 shares one selection across the HSA layers):
//   ds_i          from dw and w by the weight rule (softmax, or stick-breaking)
//   dQ[t, j, :]   = alpha sum_i ds_i Kbar_{c_i}               (each of the group's h rows)
//   dKbar[c, :]   = alpha sum over (t, i) with c_i = c of ds_i q~_t,  q~ = sum_j q_j
// Rows may be up to 1024 columns long (the group dimension d_g = h d_h of the paper's
// selection inputs).
//
// selbwd_rows: one wave per (b, t, g); lanes < k hold the slots, then every lane covers 4
// columns per 256.  selbwd_chunks: one workgroup per (b, g, c); the tokens that selected c
// are listed from the selection bitmap in increasing order (a batch of 64 words at a time,
// by a prefix sum of bit counts), their ds for c summed into LDS, and d / 16 lanes cover a
// token row (16 columns each), so a workgroup runs 4 to 64 token streams, each taking
// every nslot-th token with two rows in flight; the streams' sums are added in stream
// order: no atomics, a fixed order.
#include "common.h"

namespace hsa {

hipError_t launch_selection_bitmap(const Dims& dm, const int32_t* idx, uint32_t* bm,
                                   hipStream_t st);

namespace {

constexpr int NT = 256;
constexpr int NW_SEL = NT / 64;
constexpr int kWordsPerBatch = 64;          // bitmap words listed per batch (2048 tokens)
constexpr int kMaxD = 1024;

__host__ __device__ inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct SelBwdWs {
    size_t bitmap, ds, end;
};
inline SelBwdWs selbwd_ws(const Dims& dm) {
    SelBwdWs l;
    const size_t nwords = (size_t)cdiv(dm.L, 32);
    l.bitmap = 0;
    l.ds = align256((size_t)dm.B * dm.G * dm.C * nwords * 4);
    l.end = l.ds + align256((size_t)dm.B * dm.L * dm.G * dm.k * 4);
    return l;
}

__device__ __forceinline__ void store4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
__device__ __forceinline__ void store4(bf16* p, float4 v) {
    const uint32_t lo = (uint32_t)f32_to_bf16_bits(v.x) | ((uint32_t)f32_to_bf16_bits(v.y) << 16);
    const uint32_t hi = (uint32_t)f32_to_bf16_bits(v.z) | ((uint32_t)f32_to_bf16_bits(v.w) << 16);
    *reinterpret_cast<uint2*>(p) = uint2{lo, hi};
}
__device__ __forceinline__ float4 load4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 load4(const bf16* p) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    return float4{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                  __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u)};
}

__device__ __forceinline__ float lane_read(float v, int s) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), s));
}

template <typename T>
__global__ __launch_bounds__(NT) void selbwd_rows(Dims dm, const int32_t* __restrict__ idx,
                                                  const float* __restrict__ w,
                                                  const float* __restrict__ dw,
                                                  const float* __restrict__ Kbar,
                                                  T* __restrict__ dQ, float* __restrict__ ds) {
    const int lane = threadIdx.x & 63;
    const size_t item = (size_t)blockIdx.x * 4 + (threadIdx.x >> 6);     // ((b L) + t) G + g
    if (item >= (size_t)dm.B * dm.L * dm.G) return;
    const int g = (int)(item % dm.G);
    const size_t bt = item / dm.G;
    const int t = (int)(bt % dm.L);
    const int b = (int)(bt / dm.L);
    const int k = dm.k, d = dm.d;
    const size_t so = item * k;
    const int ncand = t / dm.S;

    int cl = -1;
    float wl = 0.f, dwl = 0.f;
    if (lane < k) {
        cl = idx[so + lane];
        wl = w[so + lane];
        dwl = dw[so + lane];
    }
    const bool valid = lane < k && cl >= 0 && cl < ncand;
    const float wd = valid ? wl * dwl : 0.f;
    float dsl;
    if (dm.stick) {
        // b = w / (1 - weight of the earlier valid slots);
        // ds = (1 - b) w dw - b (sum of w dw over the later valid slots)
        float before = 0.f, tail = 0.f;
        const float wv = valid ? wl : 0.f;
        for (int s = 0; s < k; ++s) {
            const float ws = lane_read(wv, s), wds = lane_read(wd, s);
            if (s < lane) before += ws;
            if (s > lane) tail += wds;
        }
        const float u = 1.f - before;
        const float bs = u > 0.f ? wl / u : 0.f;
        dsl = valid ? (1.f - bs) * wd - bs * tail : 0.f;
    } else {
        const float wdw = group_sum<64>(wd);
        dsl = valid ? wl * (dwl - wdw) : 0.f;
    }
    if (lane < k) ds[so + lane] = dsl;

    const size_t kbbase = (size_t)b * dm.C * dm.G + g;
    for (int e0 = 4 * lane; e0 < d; e0 += 256) {
        float4 a{0.f, 0.f, 0.f, 0.f};
        for (int s = 0; s < k; ++s) {
            const int cs = __builtin_amdgcn_readlane(cl, s);
            if (!(cs >= 0 && cs < ncand)) continue;            // the same on every lane
            const float coef = dm.alpha * lane_read(dsl, s);
            const float4 kv = load4(Kbar + (kbbase + (size_t)cs * dm.G) * d + e0);
            a.x = fmaf(coef, kv.x, a.x);
            a.y = fmaf(coef, kv.y, a.y);
            a.z = fmaf(coef, kv.z, a.z);
            a.w = fmaf(coef, kv.w, a.w);
        }
        T* q = dQ + (bt * dm.H + (size_t)g * dm.h) * d + e0;
        for (int j = 0; j < dm.h; ++j) store4(q + (size_t)j * d, a);
    }
}

// 16 consecutive columns of row q (+ h - 1 more rows, summed: q~) as floats
template <typename T>
__device__ __forceinline__ void load16(const T* q, int h, size_t rstride, float (&v)[16]) {
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = 0.f;
    for (int j = 0; j < h; ++j) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const float4 a = load4(q + (size_t)j * rstride + 4 * u);
            v[4 * u] += a.x;
            v[4 * u + 1] += a.y;
            v[4 * u + 2] += a.z;
            v[4 * u + 3] += a.w;
        }
    }
}

template <typename T>
__global__ __launch_bounds__(NT) void selbwd_chunks(Dims dm, const T* __restrict__ Q,
                                                    const int32_t* __restrict__ idx,
                                                    const float* __restrict__ ds,
                                                    const uint32_t* __restrict__ bm, int nwords,
                                                    float* __restrict__ dKbar) {
    __shared__ int list[kWordsPerBatch * 32];
    __shared__ float lsum[kWordsPerBatch * 32];
    __shared__ int ntot;
    __shared__ float part[NT * 16];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int c = blockIdx.x % dm.C;
    const int bg = blockIdx.x / dm.C, b = bg / dm.G, g = bg % dm.G;
    const int d = dm.d, k = dm.k;
    // token streams: lpt lanes per token row (16 columns each), tpw rows per wave
    const int lpt = d / 16, tpw = 64 / lpt, nslot = NW_SEL * tpw;
    const int slot = wave * tpw + lane / lpt, col = 16 * (lane % lpt);
    const uint32_t* row = bm + ((size_t)bg * dm.C + c) * nwords;
    const size_t rstride = (size_t)d;
    float acc[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = 0.f;
    // tokens before the end of chunk c cannot have selected it
    for (int w0 = ((c + 1) * dm.S) >> 5; w0 < nwords; w0 += kWordsPerBatch) {
        __syncthreads();                     // the previous batch's list is read
        if (wave == 0) {                     // list the batch: a prefix sum of bit counts
            const uint32_t word = w0 + lane < nwords ? row[w0 + lane] : 0u;
            const int cw = __popc(word);
            int incl = cw;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const int v = __shfl_up(incl, o, 64);
                if (lane >= o) incl += v;
            }
            int o = incl - cw;
            for (uint32_t wd = word; wd; wd &= wd - 1) list[o++] = (w0 + lane) * 32 + __ffs(wd) - 1;
            if (lane == 63) ntot = incl;
        }
        __syncthreads();
        const int n = ntot;
        for (int li = tid; li < n; li += NT) {   // each listed token's ds for chunk c
            const size_t so = (((size_t)b * dm.L + list[li]) * dm.G + g) * k;
            float sv = 0.f;
            for (int s2 = 0; s2 < k; ++s2)
                if (idx[so + s2] == c) sv += ds[so + s2];
            lsum[li] = sv;
        }
        __syncthreads();
        // stream `slot` takes tokens slot, slot + nslot, ...; two rows in flight
        int li = slot;
        for (; li + nslot < n; li += 2 * nslot) {
            float v0[16], v1[16];
            const T* q0 = Q + (((size_t)b * dm.L + list[li]) * dm.H + (size_t)g * dm.h) * rstride + col;
            const T* q1 = Q + (((size_t)b * dm.L + list[li + nslot]) * dm.H + (size_t)g * dm.h) * rstride + col;
            load16(q0, dm.h, rstride, v0);
            load16(q1, dm.h, rstride, v1);
            const float s0 = lsum[li], s1 = lsum[li + nslot];
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[i] = fmaf(s1, v1[i], fmaf(s0, v0[i], acc[i]));
        }
        if (li < n) {
            float v0[16];
            load16(Q + (((size_t)b * dm.L + list[li]) * dm.H + (size_t)g * dm.h) * rstride + col,
                   dm.h, rstride, v0);
            const float s0 = lsum[li];
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[i] = fmaf(s0, v0[i], acc[i]);
        }
    }
    // the streams' sums, added in stream order
#pragma unroll
    for (int i = 0; i < 16; ++i) part[slot * d + col + i] = acc[i];
    __syncthreads();
    for (int e = tid; e < d; e += NT) {
        float sv = 0.f;
        for (int s2 = 0; s2 < nslot; ++s2) sv += part[s2 * d + e];
        dKbar[(((size_t)b * dm.C + c) * dm.G + g) * d + e] = dm.alpha * sv;
    }
}

template <typename T>
hipError_t launch_t(const Dims& dm, const void* Q, const float* Kbar, const int32_t* idx,
                    const float* w, const float* dw, void* dQ, float* dKbar, void* ws,
                    hipStream_t st) {
    const SelBwdWs l = selbwd_ws(dm);
    char* wsb = (char*)ws;
    uint32_t* bm = (uint32_t*)(wsb + l.bitmap);
    float* dsb = (float*)(wsb + l.ds);
    const size_t items = (size_t)dm.B * dm.L * dm.G;
    {
        HSA_TIMED("selbwd_rows", st);
        hipLaunchKernelGGL((selbwd_rows<T>), dim3((unsigned)((items + 3) / 4)), dim3(NT), 0, st,
                           dm, idx, w, dw, Kbar, (T*)dQ, dsb);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || dm.C == 0) return e;
    e = launch_selection_bitmap(dm, idx, bm, st);
    if (e != hipSuccess) return e;
    {
        HSA_TIMED("selbwd_chunks", st);
        hipLaunchKernelGGL((selbwd_chunks<T>), dim3(dm.B * dm.G * dm.C), dim3(NT), 0, st, dm,
                           (const T*)Q, idx, (const float*)dsb, (const uint32_t*)bm,
                           cdiv(dm.L, 32), dKbar);
    }
    return hipGetLastError();
}

}  // namespace

size_t select_backward_workspace(const Dims& dm) { return selbwd_ws(dm).end; }

bool select_backward_supported(const Dims& dm) {
    return dm.d >= 64 && dm.d <= kMaxD && (dm.d & (dm.d - 1)) == 0;   // 64 .. 1024
}

hipError_t launch_select_backward(const Dims& dm, bool in_bf16, const void* Q,
                                  const float* Kbar, const int32_t* idx, const float* w,
                                  const float* dw, void* dQ, float* dKbar, void* ws,
                                  hipStream_t st) {
    if (dm.B == 0 || dm.L == 0) return hipSuccess;
    return in_bf16 ? launch_t<bf16>(dm, Q, Kbar, idx, w, dw, dQ, dKbar, ws, st)
                   : launch_t<float>(dm, Q, Kbar, idx, w, dw, dQ, dKbar, ws, st);
}

}  // namespace hsa
