// Single-token decode (Sec. 3.2 "Inference"): only the landmark cache is scanned and only
// the selected chunks' keys and values are read.
//
// Stage 1 (scan): workgroup = (b, slice of 256 chunks).  The slice's landmark rows for all
// G groups are one contiguous block of the [B, C, G, d] cache, streamed with 16-byte loads
// (all of a thread's loads issued first); D/VN consecutive lanes share a row and reduce
// their partial dot products with DPP moves.  Each wave then extracts the slice's top-k of
// one group by k rounds of a wave-wide arg-max (ties to the lower chunk index) and writes
// k (score, chunk) candidates.
// Stages 2 and 3, MFMA path (bf16, d = 128, h = 8, S = 64): workgroup = (slot, b, g).
// Each merges the slice candidates into the top-k, attends its slot's chunk with matrix
// cores (K fragments straight from global memory into registers, V rows copied into LDS
// and read transposed, as in the forward) and stores its weighted partial output; stage 3
// (combine) sums the partials in slot order.
// Other shapes: stage 2 (finish), workgroup = (slot, b, g), attends the k selected chunks
// in parallel; stage 3 (combine), workgroup = (b, g), sums their weighted partial outputs
// in slot order.
// With the key / value cache in host memory (Sec. 3.2: only the landmarks stay on the GPU):
// after the scan, decode_gather merges the selection and copies the selected
// chunks' rows from the host cache (read by the kernel over the host link) into a compact
// stage [B, G, k, S, d] in device memory, and the attend kernels run "staged": they take
// the merged selection and read slot i's rows from the stage.
#include "chunk_lds.h"

namespace hsa {
namespace {

constexpr int kScanThreads = 256;
constexpr int SL = 256;            // chunks per scan slice
constexpr int GMAX = 16;
constexpr int kFinThreads = 256;
constexpr int NW = kFinThreads / 64;
constexpr int HMAX = 16;
constexpr int KMAX = 32;
constexpr int NCMAX = 4096;        // slice candidates merged in registers (else sequentially)

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

// Query of group g summed over its h heads, qs[g D + e] (fp32).  Called by every thread of
// the scan workgroup; `issue` is run right after the loads of the first kScanThreads
// elements are issued and before their values are used, so loads it issues overlap them
// (vector-memory loads complete in order: the query's, issued first, land first; further
// elements, G d > kScanThreads, are loaded after it).  The loads are branch-free (indices
// clamped to valid elements, unused values dropped) so that they issue back to back.
template <typename Tq, int D, typename Issue>
__device__ __forceinline__ void scan_query(const Dims& dm, const Tq* __restrict__ q, int b,
                                           float* qs, Issue issue) {
    const int tid = threadIdx.x;
    const int G = dm.G, h = dm.h;
    for (int i00 = 0; i00 < G * D; i00 += kScanThreads) {
        const int i = i00 + tid;
        const int i0 = i < G * D ? i : 0;
        const int g = i0 / D, e = i0 % D;
        float qv[HMAX];
#pragma unroll
        for (int j = 0; j < HMAX; ++j)
            qv[j] = to_f32(q[((size_t)b * dm.H + g * h + min(j, h - 1)) * D + e]);
        if (i00 == 0) issue();
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < HMAX; ++j) s += (j < h) ? qv[j] : 0.f;
        if (i < G * D) qs[i] = s;
    }
}

// Scores with vector ALU dot products: U 16-byte vectors per thread per pass, loads first;
// D / VN consecutive lanes share a landmark row and reduce with DPP moves.
template <typename Tq, typename Tk, int D>
__device__ __forceinline__ void scan_scores_valu(const Dims& dm, const Tq* __restrict__ q,
                                                 const Tk* __restrict__ Kbar, int b, int c0,
                                                 int nch, float* qs, float* sc) {
    constexpr int VN = V16<Tk>::n;
    constexpr int LPR = D / VN;
    constexpr int U = 32;
    const int tid = threadIdx.x;
    const int G = dm.G;
    const Tk* base = Kbar + ((size_t)b * dm.C + c0) * G * D;
    const int nvec = nch * G * LPR;
    uint4 raw[U];
    auto load_pass = [&](int v0) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int v = v0 + u * kScanThreads + tid;
            raw[u] = v < nvec ? *reinterpret_cast<const uint4*>(base + (size_t)(v / LPR) * D +
                                                                (v % LPR) * VN)
                              : uint4{0u, 0u, 0u, 0u};
        }
    };
    scan_query<Tq, D>(dm, q, b, qs, [&]() __attribute__((always_inline)) { load_pass(0); });
    __syncthreads();
    for (int v0 = 0; v0 < nvec; v0 += kScanThreads * U) {
        if (v0 > 0) load_pass(v0);
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
}

// Scores of bf16 landmarks with packed dot products: the same contiguous loads as
// scan_scores_valu (a 16-byte vector per lane, D / 8 lanes per row), each vector reduced by
// four bf16 pair dot products (fp32 accumulation) against the summed query split into a
// bf16 pair hi + lo (16 mantissa bits together), then across the row's lanes.  A thread's
// slice of d and its group are the same for all its vectors when G divides the rows a
// pass covers per thread step (kScanThreads / (D / 8)), so its query fragments are loaded
// once.  Vectors are reduced as they land (loads complete in order).
template <typename Tq, int D>
__device__ __forceinline__ void scan_scores_dot2(const Dims& dm, const Tq* __restrict__ q,
                                                 const bf16* __restrict__ Kb, int b, int c0,
                                                 int nch, float* qs, float* sc) {
    constexpr int LPR = D / 8;
    constexpr int U = 32;
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    const int tid = threadIdx.x;
    const int G = dm.G;
    const bf16* base = Kb + ((size_t)b * dm.C + c0) * G * D;
    const int nvec = nch * G * LPR;
    uint4 raw[U];
    auto load_pass = [&](int v0) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int v = v0 + u * kScanThreads + tid;
            raw[u] = v < nvec ? *reinterpret_cast<const uint4*>(base + (size_t)(v / LPR) * D +
                                                                (v % LPR) * 8)
                              : uint4{0u, 0u, 0u, 0u};
        }
    };
    scan_query<Tq, D>(dm, q, b, qs, [&]() __attribute__((always_inline)) { load_pass(0); });
    __syncthreads();
    const int part = tid % LPR, g = (tid / LPR) % G;
    bf16x2_t qh[4], ql[4];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float v = qs[g * D + part * 8 + i];
        const __bf16 hi = f2bf(v);
        qh[i >> 1][i & 1] = hi;
        ql[i >> 1][i & 1] = f2bf(v - (float)hi);
    }
    for (int v0 = 0; v0 < nvec; v0 += kScanThreads * U) {
        if (v0 > 0) load_pass(v0);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int v = v0 + u * kScanThreads + tid;
            const uint32_t w[4] = {raw[u].x, raw[u].y, raw[u].z, raw[u].w};
            float dot = 0.f;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const bf16x2_t x = __builtin_bit_cast(bf16x2_t, w[i]);
                dot = __builtin_amdgcn_fdot2_f32_bf16(x, qh[i], dot, false);
                dot = __builtin_amdgcn_fdot2_f32_bf16(x, ql[i], dot, false);
            }
            dot = group_sum<LPR>(dot);
            if (v < nvec && part == 0) sc[v / LPR] = dm.alpha * dot;
        }
    }
}

template <typename Tk, int D>
constexpr bool kDot2Scan = sizeof(Tk) == 2 && (D == 128 || D == 64);

template <typename Tq, typename Tk, int D>
__global__ __launch_bounds__(kScanThreads, 2) void decode_scan(
    Dims dm, const Tq* __restrict__ q, const Tk* __restrict__ Kbar,
    const int32_t* __restrict__ cache_len, float* __restrict__ cand_s,
    int32_t* __restrict__ cand_c, int nslices) {
    __shared__ float qs[GMAX * D];
    __shared__ float sc[SL * GMAX];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int b = blockIdx.y, slice = blockIdx.x;
    const int G = dm.G, k = dm.k;
    const int ncand = cache_tokens(cache_len, b, dm.L) / dm.S;
    const int c0 = slice * SL;
    const int nch = max(0, min(SL, ncand - c0));

    // Scores sc[cl G + g] = alpha qbar_g . Kbar[c0 + cl, g] of the slice's rows.
    if constexpr (kDot2Scan<Tk, D>) {
        if ((kScanThreads / (D / 8)) % G == 0)
            scan_scores_dot2<Tq, D>(dm, q, reinterpret_cast<const bf16*>(Kbar), b, c0, nch, qs,
                                    sc);
        else scan_scores_valu<Tq, Tk, D>(dm, q, Kbar, b, c0, nch, qs, sc);
    } else {
        scan_scores_valu<Tq, Tk, D>(dm, q, Kbar, b, c0, nch, qs, sc);
    }
    __syncthreads();
    // top-k of the slice for each group: each lane sorts its SL / 64 order keys (descending);
    // round i takes the wave-wide maximum of the lanes' first keys and the lane holding it
    // drops its first key.
    static_assert(SL == 256, "four keys per lane");
    for (int g = wave; g < G; g += kScanThreads / 64) {
        uint64_t key[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int cl = lane + 64 * m;
            key[m] = (cl < nch) ? order_key(sc[cl * G + g], c0 + cl) : 0;
        }
        auto cx = [](uint64_t& x, uint64_t& y) __attribute__((always_inline)) {
            const uint64_t hi = max_u64(x, y), lo = x ^ y ^ hi;
            x = hi;
            y = lo;
        };
        cx(key[0], key[1]);
        cx(key[2], key[3]);
        cx(key[0], key[2]);
        cx(key[1], key[3]);
        cx(key[1], key[2]);
        float* os = cand_s + (((size_t)b * G + g) * nslices + slice) * k;
        int32_t* oc = cand_c + (((size_t)b * G + g) * nslices + slice) * k;
        for (int i = 0; i < k; ++i) {
            const uint64_t best = wave_max_key_hi(key[0]);
            if (lane == 0) {
                os[i] = best ? key_score(best) : -INFINITY;
                oc[i] = best ? key_chunk(best) : -1;
            }
            if (key[0] == best && best != 0) {
                key[0] = key[1];
                key[1] = key[2];
                key[2] = key[3];
                key[3] = 0;
            }
        }
    }
}

// Final top-k of (b, g) from the slice candidates, by wave 0 (lane i < n receives the
// i-th best; candidates carry distinct chunk ids, so (score desc, chunk asc) is a strict
// total order and round i takes the best candidate ranked below the winner of round
// i - 1), then the chunk weights (softmax, or stick-breaking with stick) and the
// descending-chunk slot order into sel_c / sel_w (slots n .. k - 1 empty).
__device__ __forceinline__ void merge_candidates(const float* cs, const int32_t* cc, int nc,
                                                 int n, int k, int lane, int* sel_c,
                                                 float* sel_w, bool stick) {
    float ls = -INFINITY;
    int lc = -1;
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
    float wt;
    int rank;
    lane_weights(ls, lc, lane < n, n, stick, wt, rank);
    if (lane < n) {
        sel_c[rank] = lc;
        sel_w[rank] = wt;
    } else if (lane < k) {
        sel_c[lane] = -1;
        sel_w[lane] = 0.f;
    }
}

// The same top-k by a two-level tournament over the whole workgroup (NWV waves), on order
// keys (score desc, chunk asc as one 64-bit integer, so every comparison is branch-free):
// each thread holds the keys of its candidates x = tid + j NT (j < NPL), each wave
// extracts the top n of its threads' keys by n rounds of a wave-wide maximum (the winner
// is knocked out of its lane) into tmp, and wave 0 extracts the top n of the NWV n
// survivors (NP2 per lane), then finishes as merge_candidates.  The top n of a union is the
// top n of the parts' top n, and the order is strict, so the result equals
// merge_candidates'.  Needs nc <= NPL NT and NWV n <= 64 NP2; every thread calls it; ends
// with a barrier.
template <int NWV, int NPL, int NP2>
__device__ __forceinline__ void merge_tournament(const float* __restrict__ cs,
                                                 const int32_t* __restrict__ cc, int nc, int n,
                                                 int k, uint64_t* tmp, int* sel_c,
                                                 float* sel_w, bool stick) {
    constexpr int NT = NWV * 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    float s[NPL];
    int c[NPL];
    // all loads first (neither depends on the other's value), keys afterwards
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
        const int x = tid + j * NT;
        c[j] = x < nc ? cc[x] : -1;
        s[j] = x < nc ? cs[x] : -INFINITY;
    }
    uint64_t key[NPL];
#pragma unroll
    for (int j = 0; j < NPL; ++j) key[j] = c[j] >= 0 ? order_key(s[j], c[j]) : 0;
    for (int r = 0; r < n; ++r) {
        uint64_t best = 0;
#pragma unroll
        for (int j = 0; j < NPL; ++j) best = max_u64(best, key[j]);
        best = wave_max_key(best);
#pragma unroll
        for (int j = 0; j < NPL; ++j)
            if (key[j] == best) key[j] = 0;
        if (lane == 0) tmp[wave * n + r] = best;
    }
    __syncthreads();
    if (wave == 0) {
        uint64_t key2[NP2];
#pragma unroll
        for (int j = 0; j < NP2; ++j) {
            const int x = lane + 64 * j;
            key2[j] = x < NWV * n ? tmp[x] : 0;
        }
        uint64_t mine = 0;               // lane r receives the r-th best
        for (int r = 0; r < n; ++r) {
            uint64_t best = 0;
#pragma unroll
            for (int j = 0; j < NP2; ++j) best = max_u64(best, key2[j]);
            best = wave_max_key(best);
#pragma unroll
            for (int j = 0; j < NP2; ++j)
                if (key2[j] == best) key2[j] = 0;
            if (lane == r) mine = best;
        }
        const float ls = mine ? key_score(mine) : -INFINITY;
        const int lc = mine ? key_chunk(mine) : -1;
        float wt;
        int rank;
        lane_weights(ls, lc, lane < n && lc >= 0, n, stick, wt, rank);
        if (lane < n) {
            sel_c[rank] = lc;
            sel_w[rank] = wt;
        } else if (lane < k) {
            sel_c[lane] = -1;
            sel_w[lane] = 0.f;
        }
    }
    __syncthreads();
}

// merge_tournament with the fewest registers that hold nc candidates and the survivors;
// false (nothing done) when nc exceeds NPLMAX per thread.
template <int NWV, int NPLMAX>
__device__ __forceinline__ bool merge_top(const float* __restrict__ cs,
                                          const int32_t* __restrict__ cc, int nc, int n, int k,
                                          uint64_t* tmp, int* sel_c, float* sel_w, bool stick) {
    constexpr int NT = NWV * 64;
    const bool s1 = NWV * n <= 64;
    if (nc <= NT) {
        if (s1) merge_tournament<NWV, 1, 1>(cs, cc, nc, n, k, tmp, sel_c, sel_w, stick);
        else merge_tournament<NWV, 1, NWV * KMAX / 64>(cs, cc, nc, n, k, tmp, sel_c, sel_w, stick);
    } else if (nc <= NPLMAX * NT) {
        if (s1) merge_tournament<NWV, NPLMAX, 1>(cs, cc, nc, n, k, tmp, sel_c, sel_w, stick);
        else merge_tournament<NWV, NPLMAX, NWV * KMAX / 64>(cs, cc, nc, n, k, tmp, sel_c, sel_w,
                                                             stick);
    } else {
        return false;
    }
    return true;
}

// The same top-k from at most 64 slice lists, each sorted by descending order key (the
// scan extracts them in that order) and padded with empty keys: lane l holds list l's
// first KC keys in registers; round r takes the wave-wide maximum of the lanes' first keys
// and the winning lane shifts its list up by one.  One wave, no barrier, no memory traffic
// inside the rounds; the order is strict, so the result equals merge_candidates'.
template <int KC>
__device__ __forceinline__ void merge_lists(const float* __restrict__ cs,
                                            const int32_t* __restrict__ cc, int nlists, int n,
                                            int k, int lane, int* sel_c, float* sel_w,
                                            bool stick) {
    int c[KC];
    float s[KC];
#pragma unroll
    for (int i = 0; i < KC; ++i) {       // all loads first
        const bool in = lane < nlists && i < k;
        c[i] = in ? cc[lane * k + i] : -1;
        s[i] = in ? cs[lane * k + i] : -INFINITY;
    }
    uint64_t key[KC];
#pragma unroll
    for (int i = 0; i < KC; ++i) key[i] = c[i] >= 0 ? order_key(s[i], c[i]) : 0;
    uint64_t mine = 0;                   // lane r receives the r-th best
    for (int r = 0; r < n; ++r) {
        const uint64_t best = wave_max_key_hi(key[0]);
        if (lane == r) mine = best;
        if (best != 0 && key[0] == best) {
#pragma unroll
            for (int i = 0; i + 1 < KC; ++i) key[i] = key[i + 1];
            key[KC - 1] = 0;
        }
    }
    const float ls = mine ? key_score(mine) : -INFINITY;
    const int lc = mine ? key_chunk(mine) : -1;
    float wt;
    int rank;
    lane_weights(ls, lc, lane < n && lc >= 0, n, stick, wt, rank);
    if (lane < n) {
        sel_c[rank] = lc;
        sel_w[rank] = wt;
    } else if (lane < k) {
        sel_c[lane] = -1;
        sel_w[lane] = 0.f;
    }
}

// Final top-k of (b, g) into sel_c / sel_w (LDS) from the slice candidates, by every thread
// of the workgroup; ends with a barrier.  Up to 64 slices: merge_lists by wave 0; more:
// the tournament over the whole workgroup, else wave 0 sequentially.
template <int NWV, int NPLMAX>
__device__ __forceinline__ void merge_slices(const float* __restrict__ cs,
                                             const int32_t* __restrict__ cc, int nslices,
                                             int n, int k, uint64_t* tmp, int* sel_c,
                                             float* sel_w, bool stick) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nc = nslices * k;
    if (nslices <= 64) {
        if (wave == 0) {
            if (k <= 8) merge_lists<8>(cs, cc, nslices, n, k, lane, sel_c, sel_w, stick);
            else if (k <= 16) merge_lists<16>(cs, cc, nslices, n, k, lane, sel_c, sel_w, stick);
            else merge_lists<KMAX>(cs, cc, nslices, n, k, lane, sel_c, sel_w, stick);
        }
        __syncthreads();
        return;
    }
    if (!merge_top<NWV, NPLMAX>(cs, cc, nc, n, k, tmp, sel_c, sel_w, stick)) {
        __syncthreads();
        if (wave == 0) merge_candidates(cs, cc, nc, n, k, lane, sel_c, sel_w, stick);
        __syncthreads();
    }
}

// Stage 2 (finish): workgroup = (slot, b, g), so the k selected chunks of a sequence are
// attended in parallel.  Wave 0 of every workgroup merges the slice candidates into the
// final top-k (the same deterministic merge in each), computes the chunk weights and
// the descending-chunk slot order.  The workgroup of slot i stages its chunk's K and V in
// LDS, computes the intra-chunk softmax of the h heads and w_i P V, and stores that partial
// output.  Stage 3 (combine) sums the partials of a (b, g) in slot order.
template <typename T, int D>
__global__ __launch_bounds__(kFinThreads) void decode_finish(
    Dims dm, const T* __restrict__ q, const T* __restrict__ Kc, const T* __restrict__ Vc,
    const int32_t* __restrict__ cache_len, const float* __restrict__ cand_s,
    const int32_t* __restrict__ cand_c, int nslices, float* __restrict__ part,
    int32_t* __restrict__ idx_out, float* __restrict__ w_out, int staged) {
    constexpr int DP = D + 1;
    constexpr int SMAX = 128;
    constexpr int NE = sizeof(T) == 4 ? 8192 : SMAX * D;   // S * d <= 8192 for fp32 inputs
    __shared__ T ks[NE];
    __shared__ T vs[NE];
    __shared__ float qf[HMAX * DP];
    __shared__ float pz[HMAX * SMAX];
    __shared__ int sel_c[KMAX];
    __shared__ float sel_w[KMAX];
    __shared__ uint64_t mtmp[NW * KMAX];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int slot = blockIdx.x;
    const int bg = blockIdx.y, b = bg / dm.G, g = bg % dm.G;
    const int h = dm.h, S = dm.S, k = dm.k;
    const int ncand = cache_tokens(cache_len, b, dm.L) / S;
    const int n = min(k, ncand);

    for (int i = tid; i < h * D; i += kFinThreads)
        qf[(i / D) * DP + i % D] = to_f32(q[((size_t)b * dm.H + (size_t)g * h) * D + i]);
    const int nc = nslices * k;
    if (staged) {                        // the selection is merged already (decode_gather)
        if (tid < k) {
            sel_c[tid] = idx_out[(size_t)bg * k + tid];
            sel_w[tid] = w_out[(size_t)bg * k + tid];
        }
        __syncthreads();
    } else {
        merge_slices<NW, NCMAX / kFinThreads>(cand_s + (size_t)bg * nc, cand_c + (size_t)bg * nc,
                                              nslices, n, k, mtmp, sel_c, sel_w, dm.stick != 0);
        if (slot == 0 && tid < k) {
            idx_out[(size_t)bg * k + tid] = sel_c[tid];
            w_out[(size_t)bg * k + tid] = sel_w[tid];
        }
    }

    // a chunk id outside the candidates (never produced by the scan) leaves the slot empty
    // rather than indexing the cache with it
    const bool live = slot < n && sel_c[slot] >= 0 && sel_c[slot] < ncand;
    if (slot < n && !live) {
        float* pp = part + (((size_t)bg * k + slot) * h) * D;
        for (int x = tid; x < h * D; x += kFinThreads) pp[x] = 0.f;
    }
    if (live) {
        const int c = sel_c[slot];
        const float wi = sel_w[slot];
        // the chunk's S rows of K and V for group g
        constexpr int VN = V16<T>::n;
        for (int v = tid; v < S * D / VN; v += kFinThreads) {
            const int s = v / (D / VN), e = (v % (D / VN)) * VN;
            const size_t src = staged ? (((size_t)bg * k + slot) * S + s) * D + e
                                      : (((size_t)b * dm.L + (size_t)c * S + s) * dm.G + g) * D + e;
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
            float m = wave_max(fmaxf(z0, z1));
            if (dm.off1) m = fmaxf(m, 0.f);
            const float e0 = lane < S ? expf(z0 - m) : 0.f;
            const float e1 = lane + 64 < S ? expf(z1 - m) : 0.f;
            const float scale = wi / (wave_sum(e0 + e1) + (dm.off1 ? expf(-m) : 0.f));
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

constexpr int kAttS = 64;
constexpr int kAttD = 128;
constexpr int kAttH = 8;

// Stage 2 on matrix cores, one workgroup per (slot, b, g) so that the k chunks of a sequence
// are read through k CUs: every workgroup of a (b, g) merges the slice candidates (the same
// deterministic merge; the slot-0 one writes idx and w), and wave 0 attends the slot's chunk
// (K fragments from global memory into registers, V rows copied into LDS and read
// transposed) and stores w_i P V (fp32) as the slot's partial; decode_combine sums them.
__global__ __launch_bounds__(kFinThreads) void decode_attend_slot(
    Dims dm, const __bf16* __restrict__ q, const __bf16* __restrict__ Kc,
    const __bf16* __restrict__ Vc, const int32_t* __restrict__ cache_len,
    const float* __restrict__ cand_s, const int32_t* __restrict__ cand_c, int nslices,
    float* __restrict__ part, int32_t* __restrict__ idx_out, float* __restrict__ w_out,
    int staged) {
    constexpr int S = kAttS, DD = kAttD, MB = S / 16, KS2 = S / 32;
    __shared__ __bf16 vst[S * DD];
    __shared__ int sel_c[KMAX];
    __shared__ float sel_w[KMAX];
    __shared__ uint64_t mtmp[NW * KMAX];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int row = lane & 15, grp = lane >> 4;
    const int slot = blockIdx.x;
    const int bg = blockIdx.y, b = bg / dm.G, g = bg % dm.G;
    const int k = dm.k;
    const int ncand = cache_tokens(cache_len, b, dm.L) / S;
    const int n = min(k, ncand);

    // Q^T operand of wave 0: columns 0-7 are the group's heads, 8-15 zero
    bf16x8_t qB[4];
    if (wave == 0) {
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)   // branch-free loads (rows 8-15 repeat 0-7), then zeroed
            qB[ks] = ld_bf16x8(q + ((size_t)b * dm.H + (size_t)g * kAttH + (row & 7)) * DD +
                               32 * ks + 8 * grp);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
            if (row >= kAttH) qB[ks] = bf16x8_t{};
    }
    const int nc = nslices * k;
    if (staged) {                        // the selection is merged already (decode_gather)
        if (tid < k) {
            sel_c[tid] = idx_out[(size_t)bg * k + tid];
            sel_w[tid] = w_out[(size_t)bg * k + tid];
        }
        __syncthreads();
    } else {
        merge_slices<NW, NCMAX / kFinThreads>(cand_s + (size_t)bg * nc, cand_c + (size_t)bg * nc,
                                              nslices, n, k, mtmp, sel_c, sel_w, dm.stick != 0);
        if (slot == 0 && tid < k) {
            idx_out[(size_t)bg * k + tid] = sel_c[tid];
            w_out[(size_t)bg * k + tid] = sel_w[tid];
        }
    }

    float* const pp = part + ((size_t)bg * k + slot) * kAttH * DD;
    if (wave == 0 && slot < n) {
        f32x4_t acc[8];
#pragma unroll
        for (int db = 0; db < 8; ++db) acc[db] = zero4();
        const int c = sel_c[slot];
        // a chunk id outside the candidates (never produced by the scan) leaves the slot empty
        if (c >= 0 && c < ncand) {
            const float wi = sel_w[slot];
            const size_t rowstride = staged ? (size_t)DD : (size_t)dm.G * DD;
            const size_t key0 = staged ? ((size_t)bg * k + slot) * S * DD
                                       : ((size_t)b * dm.L + (size_t)c * S) * rowstride +
                                             (size_t)g * DD;
            // V rows into LDS (copies, issued first), K fragments into registers
            chunk_to_lds<S, 1>(Vc + key0, rowstride, vst, 0, lane);
            bf16x8_t kf[4][MB];
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
                    kf[ks][mb] = ld_bf16x8(Kc + key0 + (size_t)(16 * mb + row) * rowstride +
                                           32 * ks + 8 * grp);
            f32x4_t z[MB];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) z[mb] = zero4();
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb) z[mb] = mfma16(kf[ks][mb], qB[ks], z[mb]);
            const float sl2 = dm.beta * 1.44269504088896341f;
            const bool off1 = dm.off1 != 0;
            float m = -INFINITY;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int i = 0; i < 4; ++i) m = fmaxf(m, z[mb][i]);
            const float msl = fmaxf(col_max(m), off1 ? 0.f : -INFINITY) * sl2;
            float ssum = 0.f;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    z[mb][i] = fast_exp2(fmaf(z[mb][i], sl2, -msl));
                    ssum += z[mb][i];
                }
            const float scale =
                wi * __builtin_amdgcn_rcpf(col_sum(ssum) + (off1 ? fast_exp2(-msl) : 0.f));
            int toff[8];
            tr_read_offsets(lane, toff);
            wait_loads_le<0>();
#pragma unroll
            for (int ks2 = 0; ks2 < KS2; ++ks2) {
                // w P as a bf16 pair hi + lo (about 16 bits), as in the forward
                f32x4_t pa, pc;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    pa[i] = z[2 * ks2][i] * scale;
                    pc[i] = z[2 * ks2 + 1][i] * scale;
                }
                bf16x8_t ph, pl;
                split8(pa, pc, ph, pl);
                // in halves of 4 column blocks: the hi products, then the lo ones
#pragma unroll
                for (int d0 = 0; d0 < 8; d0 += 4) {
                    bf16x8_t vt[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const __bf16* pv = vst + toff[d0 + j] + 32 * ks2 * DD;
                        vt[j] = cat(ld_tr16(pv), ld_tr16(pv + 16 * DD));
                    }
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[d0 + j] = mfma16(vt[j], ph, acc[d0 + j]);
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[d0 + j] = mfma16(vt[j], pl, acc[d0 + j]);
                }
            }
        }
        if (row < kAttH) {
#pragma unroll
            for (int db = 0; db < 8; ++db)
                *reinterpret_cast<f32x4_t*>(pp + row * DD + 16 * db + 4 * grp) = acc[db];
        }
    }
}

// The host-cache path's merge and gather: workgroup = (slot, b, g).  Every workgroup of a
// (b, g) merges the slice candidates (the same deterministic merge), the slot-0 one writes
// idx, w [B, G, k], and the workgroup of slot i copies its chunk's K and V rows from the
// cache in host memory [B, N, G, d] to the stage [B, G, k, S, d]; every thread issues all
// of its 16-byte loads (K and V) before its stores, so a workgroup keeps 2 S d elem bytes
// in flight over the host link.
template <typename T, int D>
__global__ __launch_bounds__(kFinThreads) void decode_gather(
    Dims dm, const T* __restrict__ Kh, const T* __restrict__ Vh,
    const int32_t* __restrict__ cache_len, const float* __restrict__ cand_s,
    const int32_t* __restrict__ cand_c, int nslices, int32_t* __restrict__ idx_out,
    float* __restrict__ w_out, T* __restrict__ Ks, T* __restrict__ Vs) {
    constexpr int VN = V16<T>::n;                 // elements per 16 bytes
    constexpr int PER = 128 * D / VN / kFinThreads;   // 16-byte vectors per thread, S <= 128
    __shared__ int sel_c[KMAX];
    __shared__ float sel_w[KMAX];
    __shared__ uint64_t mtmp[NW * KMAX];
    const int tid = threadIdx.x;
    const int slot = blockIdx.x;
    const int bg = blockIdx.y, b = bg / dm.G, g = bg % dm.G;
    const int S = dm.S, k = dm.k;
    const int ncand = cache_tokens(cache_len, b, dm.L) / S;
    const int n = min(k, ncand);
    const int nc = nslices * k;
    merge_slices<NW, NCMAX / kFinThreads>(cand_s + (size_t)bg * nc, cand_c + (size_t)bg * nc,
                                          nslices, n, k, mtmp, sel_c, sel_w, dm.stick != 0);
    if (slot == 0 && tid < k) {
        idx_out[(size_t)bg * k + tid] = sel_c[tid];
        w_out[(size_t)bg * k + tid] = sel_w[tid];
    }
    if (slot >= n) return;
    const int c = sel_c[slot];
    if (c < 0 || c >= ncand) return;              // never produced by the scan
    const int nv = S * D / VN;
    uint4 kr[PER], vr[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        const int v = threadIdx.x + u * kFinThreads;
        if (v < nv) {
            const int s = v / (D / VN), e = (v % (D / VN)) * VN;
            const size_t src = (((size_t)b * dm.L + (size_t)c * S + s) * dm.G + g) * D + e;
            kr[u] = *reinterpret_cast<const uint4*>(Kh + src);
            vr[u] = *reinterpret_cast<const uint4*>(Vh + src);
        }
    }
    const size_t dst0 = ((size_t)bg * k + slot) * S * D;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        const int v = threadIdx.x + u * kFinThreads;
        if (v < nv) {
            *reinterpret_cast<uint4*>(Ks + dst0 + (size_t)v * VN) = kr[u];
            *reinterpret_cast<uint4*>(Vs + dst0 + (size_t)v * VN) = vr[u];
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
    const size_t stride = (size_t)h * D;            // floats per slot
    const float* p0 = part + (size_t)bg * k * stride;
    // 4 consecutive outputs per thread; the slots' loads of 8 slots are issued together
    // (a loop carrying one load at a time waits for each in turn), then added in slot order
    for (int x = 4 * threadIdx.x; x < h * D; x += 4 * 256) {
        float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int i0 = 0; i0 < n; i0 += 8) {
            float4 v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j)
                v[j] = i0 + j < n ? *reinterpret_cast<const float4*>(p0 + (i0 + j) * stride + x)
                                  : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                s.x += v[j].x;
                s.y += v[j].y;
                s.z += v[j].z;
                s.w += v[j].w;
            }
        }
        T* op = o + ((size_t)b * dm.H + (size_t)g * h) * D + x;
        op[0] = from_f32<T>(s.x);
        op[1] = from_f32<T>(s.y);
        op[2] = from_f32<T>(s.z);
        op[3] = from_f32<T>(s.w);
    }
}

// The MFMA path of stages 2 and 3 applies to bf16 inputs with d = 128, 8 heads per group
// and chunks of 64 keys.
template <typename T, int D>
bool decode_mfma_shape(const Dims& dm) {
    return sizeof(T) == 2 && D == kAttD && dm.h == kAttH && dm.S == kAttS && dm.k <= KMAX &&
           path_override(HSA_OP_DECODE) != HSA_PATH_GENERIC;
}

struct DecodeWs {
    size_t cs, cc, part, kst, vst, end;
};
// elem: bytes per K / V element, when the stages of the host-cache path are included
DecodeWs decode_ws(const Dims& dm, int elem = 0) {
    const size_t nslices = (size_t)cdiv(dm.C > 0 ? dm.C : 1, SL);
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    DecodeWs l;
    l.cs = 0;
    l.cc = al(l.cs + (size_t)dm.B * dm.G * nslices * dm.k * 4);
    l.part = al(l.cc + (size_t)dm.B * dm.G * nslices * dm.k * 4);
    l.kst = al(l.part + (size_t)dm.B * dm.G * dm.k * dm.h * dm.d * 4);
    const size_t stage = (size_t)dm.B * dm.G * dm.k * dm.S * dm.d * elem;
    l.vst = al(l.kst + stage);
    l.end = al(l.vst + stage);
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
    const bool mfma = decode_mfma_shape<T, D>(dm);
    {
        HSA_TIMED("decode_scan", st);
        hipLaunchKernelGGL((decode_scan<T, Tk, D>), dim3(nslices, dm.B), dim3(kScanThreads), 0,
                           st, dm, (const T*)q, (const Tk*)Kbar, cache_len, cs, cc,
                           nslices);
    }
    if (mfma) {
        {
            HSA_TIMED("decode_attend_mfma", st);
            hipLaunchKernelGGL(decode_attend_slot, dim3(dm.k, dm.B * dm.G), dim3(kFinThreads), 0,
                               st, dm, (const __bf16*)q, (const __bf16*)Kc, (const __bf16*)Vc,
                               cache_len, cs, cc, nslices, part, idx, w, 0);
        }
        HSA_TIMED("decode_combine", st);
        hipLaunchKernelGGL((decode_combine<T, D>), dim3(dm.B * dm.G), dim3(256), 0, st, dm,
                           cache_len, part, (T*)o);
        return;
    }
    {
        HSA_TIMED("decode_finish", st);
        hipLaunchKernelGGL((decode_finish<T, D>), dim3(dm.k, dm.B * dm.G), dim3(kFinThreads), 0,
                           st, dm, (const T*)q, (const T*)Kc, (const T*)Vc, cache_len, cs, cc,
                           nslices, part, idx, w, 0);
    }
    {
        HSA_TIMED("decode_combine", st);
        hipLaunchKernelGGL((decode_combine<T, D>), dim3(dm.B * dm.G), dim3(256), 0, st, dm,
                           cache_len, part, (T*)o);
    }
}

// Host-cache path: scan, merge, gather into the stages, then the attend kernels on them.
template <typename T, typename Tk, int D>
void launch_tkd_host(const Dims& dm, const void* q, const void* Kh, const void* Vh,
                     const void* Kbar, const int32_t* cache_len, void* o, int32_t* idx, float* w,
                     void* ws, hipStream_t st) {
    const int nslices = cdiv(dm.C > 0 ? dm.C : 1, SL);
    const DecodeWs l = decode_ws(dm, (int)sizeof(T));
    char* wb = (char*)ws;
    float* cs = (float*)(wb + l.cs);
    int32_t* cc = (int32_t*)(wb + l.cc);
    float* part = (float*)(wb + l.part);
    const bool mfma = decode_mfma_shape<T, D>(dm);
    T* kst = (T*)(wb + l.kst);
    T* vst = (T*)(wb + l.vst);
    {
        HSA_TIMED("decode_scan", st);
        hipLaunchKernelGGL((decode_scan<T, Tk, D>), dim3(nslices, dm.B), dim3(kScanThreads), 0,
                           st, dm, (const T*)q, (const Tk*)Kbar, cache_len, cs, cc,
                           nslices);
    }
    {
        HSA_TIMED("decode_gather", st);
        hipLaunchKernelGGL((decode_gather<T, D>), dim3(dm.k, dm.B * dm.G), dim3(kFinThreads), 0,
                           st, dm, (const T*)Kh, (const T*)Vh, cache_len, cs, cc, nslices, idx,
                           w, kst, vst);
    }
    if (mfma) {
        {
            HSA_TIMED("decode_attend_mfma", st);
            hipLaunchKernelGGL(decode_attend_slot, dim3(dm.k, dm.B * dm.G), dim3(kFinThreads), 0,
                               st, dm, (const __bf16*)q, (const __bf16*)kst, (const __bf16*)vst,
                               cache_len, cs, cc, nslices, part, idx, w, 1);
        }
        HSA_TIMED("decode_combine", st);
        hipLaunchKernelGGL((decode_combine<T, D>), dim3(dm.B * dm.G), dim3(256), 0, st, dm,
                           cache_len, part, (T*)o);
        return;
    }
    {
        HSA_TIMED("decode_finish", st);
        hipLaunchKernelGGL((decode_finish<T, D>), dim3(dm.k, dm.B * dm.G), dim3(kFinThreads), 0,
                           st, dm, (const T*)q, (const T*)kst, (const T*)vst, cache_len, cs, cc,
                           nslices, part, idx, w, 1);
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
size_t decode_host_workspace(const Dims& dm, bool in_bf16) {
    return decode_ws(dm, in_bf16 ? 2 : 4).end;
}

hipError_t launch_decode_host(const Dims& dm, bool in_bf16, const void* q, const void* Kh,
                              const void* Vh, const void* Kbar, bool kbar_bf16,
                              const int32_t* cache_len, void* o, int32_t* idx, float* w,
                              void* ws, hipStream_t st) {
    if (dm.B == 0) return hipSuccess;
#define HSA_HOST_LAUNCH(T, Tk)                                                                  \
    (dm.d == 128 ? launch_tkd_host<T, Tk, 128>(dm, q, Kh, Vh, Kbar, cache_len, o, idx, w, ws, st) \
                 : launch_tkd_host<T, Tk, 64>(dm, q, Kh, Vh, Kbar, cache_len, o, idx, w, ws, st))
    if (in_bf16) {
        if (kbar_bf16) HSA_HOST_LAUNCH(bf16, bf16);
        else HSA_HOST_LAUNCH(bf16, float);
    } else {
        if (kbar_bf16) HSA_HOST_LAUNCH(float, bf16);
        else HSA_HOST_LAUNCH(float, float);
    }
#undef HSA_HOST_LAUNCH
    return hipGetLastError();
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
