// Shared definitions of the HSA kernels for gfx950 (CDNA4, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hsa {

// Problem description passed by value to every kernel.
struct Dims {
    int B, L, H, G, h, d, S, k;
    int C;          // complete chunks, floor(L / S)
    int Call;       // chunks including a trailing partial one, ceil(L / S)
    float alpha;    // selection-score scale
    float beta;     // intra-chunk attention scale
};

// bfloat16 storage type of the generic kernels (bit pattern only).
struct bf16 {
    uint16_t v;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return __uint_as_float(((uint32_t)x.v) << 16); }

// Round to nearest even; inputs are finite by contract (NaN is kept quiet anyway).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u >> 16) | ((u & 0xFFFF) ? 0x40 : 0));
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return bf16{f32_to_bf16_bits(x)}; }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}

__host__ __device__ __forceinline__ int cdiv(int a, int b) { return (a + b - 1) / b; }

// RAII bracket of one kernel launch for the optional per-kernel timing (timing.hip).
class KernelTimer {
  public:
    KernelTimer(const char* name, hipStream_t st);
    ~KernelTimer();
    KernelTimer(const KernelTimer&) = delete;
    KernelTimer& operator=(const KernelTimer&) = delete;

  private:
    const char* name_;
    hipStream_t st_;
    hipEvent_t a_ = nullptr, b_ = nullptr;
};

#define HSA_TIMED(name, st) ::hsa::KernelTimer hsa_kernel_timer_(name, st)

}  // namespace hsa

// Host launchers implemented in the kernel translation units (called by hsa_api.hip).
namespace hsa {
hipError_t launch_landmarks(const Dims& dm, bool in_bf16, const void* K, void* Kbar,
                            bool out_bf16, int c0, int c1, hipStream_t st);
hipError_t launch_select(const Dims& dm, bool in_bf16, const void* Q, const float* Kbar,
                         int32_t* idx, float* w, hipStream_t st);
hipError_t launch_forward(const Dims& dm, bool in_bf16, const void* Q, const void* K,
                          const void* V, const int32_t* idx, const float* w, void* O,
                          void* ws, hipStream_t st);
size_t backward_workspace(const Dims& dm);
hipError_t launch_backward(const Dims& dm, bool in_bf16, const void* Q, const void* K,
                           const void* V, const float* Kbar, const int32_t* idx,
                           const float* w, const void* dO, void* dQ, void* dK, void* dV,
                           void* ws, hipStream_t st);
size_t decode_workspace(const Dims& dm);
hipError_t launch_decode(const Dims& dm, bool in_bf16, const void* q, const void* Kc,
                         const void* Vc, const void* Kbar, bool kbar_bf16,
                         const int32_t* cache_len, void* o, int32_t* idx, float* w,
                         void* ws, hipStream_t st);
}  // namespace hsa
