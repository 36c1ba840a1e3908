// Device fill of seeded synthetic inputs: the same counter-based definition
// as the host generator (paper_2608_22322_amd/synth.py), element for element.
// Holds none of the optimizer's or the codec's arithmetic.
//
//   w_k = mix64(key + (3e + k + 1) * GAMMA), k = 0, 1, 2   (mod 2^64)
//   S   = sum of the twelve 16-bit fields of w_0, w_1, w_2
//   v   = fl32(fl32(S - 393210) * scale)         (one binary32 multiply)
//   v   = 0 if mix64(mask_key + (e + 1) * GAMMA) < mask_threshold
// mix64 is the SplitMix64 output function (Steele, Lea & Flood, 2014).
#include "al_internal.hpp"

namespace al {

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

__global__ __launch_bounds__(256) void synth_normal_kernel(void* out, int out_bf16, int64_t n, uint64_t key,
                                                           float scale, uint64_t mask_key, uint64_t mask_thr) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += stride) {
        const uint64_t base = 3ull * (uint64_t)e;
        int64_t S = 0;
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            const uint64_t w = mix64(key + (base + (uint64_t)(k + 1)) * kGamma);
            S += (int64_t)(w & 0xFFFFull) + (int64_t)((w >> 16) & 0xFFFFull) + (int64_t)((w >> 32) & 0xFFFFull) +
                 (int64_t)(w >> 48);
        }
        float v = (float)(int32_t)(S - 393210) * scale;
        if (mask_thr != 0ull && mix64(mask_key + ((uint64_t)e + 1ull) * kGamma) < mask_thr) v = 0.0f;
        if (out_bf16) {
            const uint32_t b = __builtin_bit_cast(uint32_t, v);
            const uint32_t r = (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
            reinterpret_cast<uint16_t*>(out)[e] = (uint16_t)r;
        } else {
            reinterpret_cast<float*>(out)[e] = v;
        }
    }
}

hipError_t launch_synth_normal(void* out, int out_bf16, int64_t n, uint64_t key, float scale, uint64_t mask_key,
                               uint64_t mask_threshold, int grid_cap, hipStream_t s) {
    const int64_t want = (n + 255) / 256;
    const int grid = (int)(want < grid_cap ? want : grid_cap);
    if (grid <= 0) return hipSuccess;
    hipLaunchKernelGGL(synth_normal_kernel, dim3(grid), dim3(256), 0, s, out, out_bf16, n, key, scale, mask_key,
                       mask_threshold);
    return hipGetLastError();
}

}  // namespace al
