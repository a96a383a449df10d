// Landmark pooling: Kbar[b, c, g, :] = mean of the S keys of chunk c (Fig. 1; Sec. 3.1).
//
// One workgroup per (b, chunk).  The S rows of a chunk are contiguous in [B, L, G, d]
// (S x G*d elements), so the workgroup streams one contiguous block with 16-byte loads:
// thread (row-group r, column-vector v) sums rows r, r+R, ... of column vector v, then
// the R partial sums are reduced in LDS in a fixed order (deterministic).  HBM-bound:
// reads S*G*d elements and writes G*d per chunk.
#include "common.h"

namespace hsa {
namespace {

constexpr int kThreads = 256;
constexpr int kLoads = 8;         // row loads a thread keeps in flight

template <typename T> struct Vec;
template <> struct Vec<float> { static constexpr int n = 4; using raw = float4; };
template <> struct Vec<bf16> { static constexpr int n = 8; using raw = uint4; };

__device__ __forceinline__ void unpack(const float4& r, float* x) {
    x[0] = r.x; x[1] = r.y; x[2] = r.z; x[3] = r.w;
}
__device__ __forceinline__ void unpack(const uint4& r, float* x) {
    const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[2 * i] = __uint_as_float(w[i] << 16);
        x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
}

template <typename Tin, typename Tout>
__global__ __launch_bounds__(kThreads) void landmarks_kernel(Dims dm, const Tin* __restrict__ K,
                                                             Tout* __restrict__ Kbar, int c0) {
    constexpr int VN = Vec<Tin>::n;
    const int b = blockIdx.y;
    const int c = c0 + blockIdx.x;
    const int row = dm.G * dm.d;           // elements per token row
    const int nvec = row / VN;             // vectors per row
    const int ncol = nvec < kThreads ? nvec : kThreads;
    const int R = kThreads / ncol;         // row groups
    const int tid = threadIdx.x;
    const int v_lane = tid % ncol;
    const int r = tid / ncol;
    __shared__ float part[kThreads * VN];

    const Tin* base = K + ((size_t)b * dm.L + (size_t)c * dm.S) * row;
    for (int v0 = 0; v0 < nvec; v0 += ncol) {
        const int v = v0 + v_lane;
        float acc[VN];
#pragma unroll
        for (int i = 0; i < VN; ++i) acc[i] = 0.f;
        if (r < R && v < nvec) {
            // rows r, r + R, ... in order; the loads of up to kLoads rows are issued before
            // any is added, so a thread has them in flight together
            for (int s0 = r; s0 < dm.S; s0 += kLoads * R) {
                typename Vec<Tin>::raw raw[kLoads];
#pragma unroll
                for (int u = 0; u < kLoads; ++u) {
                    const int s = s0 + u * R;
                    if (s < dm.S)
                        raw[u] = *reinterpret_cast<const typename Vec<Tin>::raw*>(
                            base + (size_t)s * row + (size_t)v * VN);
                }
#pragma unroll
                for (int u = 0; u < kLoads; ++u) {
                    if (s0 + u * R < dm.S) {
                        float x[VN];
                        unpack(raw[u], x);
#pragma unroll
                        for (int i = 0; i < VN; ++i) acc[i] += x[i];
                    }
                }
            }
        }
#pragma unroll
        for (int i = 0; i < VN; ++i) part[tid * VN + i] = acc[i];
        __syncthreads();
        // thread (v_lane, element i) reduces the R row-group partials in order
        const float inv = 1.0f / (float)dm.S;
        for (int e = tid; e < ncol * VN; e += kThreads) {
            const int vl = e / VN, i = e % VN;
            if (v0 + vl >= nvec) continue;
            float s = 0.f;
            for (int rr = 0; rr < R; ++rr) s += part[(rr * ncol + vl) * VN + i];
            const size_t col = (size_t)(v0 + vl) * VN + i;          // g*d + e
            Kbar[((size_t)b * dm.C + c) * row + col] = from_f32<Tout>(s * inv);
        }
        __syncthreads();
    }
}

template <typename Tin>
hipError_t launch_t(const Dims& dm, const void* K, void* Kbar, bool out_bf16, int c0, int c1,
                    hipStream_t st) {
    dim3 grid(c1 - c0, dm.B);
    if (out_bf16) {
        HSA_TIMED("landmarks_kernel", st);
        hipLaunchKernelGGL((landmarks_kernel<Tin, bf16>), grid, dim3(kThreads), 0, st, dm,
                           (const Tin*)K, (bf16*)Kbar, c0);
    } else {
        HSA_TIMED("landmarks_kernel", st);
        hipLaunchKernelGGL((landmarks_kernel<Tin, float>), grid, dim3(kThreads), 0, st, dm,
                           (const Tin*)K, (float*)Kbar, c0);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_landmarks(const Dims& dm, bool in_bf16, const void* K, void* Kbar,
                            bool out_bf16, int c0, int c1, hipStream_t st) {
    if (c1 <= c0 || dm.B == 0) return hipSuccess;
    return in_bf16 ? launch_t<bf16>(dm, K, Kbar, out_bf16, c0, c1, st)
                   : launch_t<float>(dm, K, Kbar, out_bf16, c0, c1, st);
}

}  // namespace hsa
