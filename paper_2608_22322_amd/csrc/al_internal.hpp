// Launch descriptors and launcher entry points shared between the C ABI
// (al_api.cpp) and the kernel translation units. Not a public header.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "al_device.hpp"

namespace al {

// ------------------------------------------------------------------ AdamW
// A launch covers up to kAdamWMaxTensors tensors; their descriptors travel
// in the kernel-argument segment, so a step needs no device-side table.
constexpr int kAdamWMaxTensors = 48;

struct AdamWDesc {
    float* p;
    const void* g;
    void* m;
    float* ms;  // UF8 absmax per 256-element block (unused for FP32 m)
    void* v;
    float* vm;  // AL {l_min, delta} per block (unused for FP32 v)
    int64_t n;
    int64_t tile_begin;  // first tile of this tensor within the launch
};

struct AdamWLaunch {
    double beta1, omb1, beta2, omb2;  // state EMA coefficients (binary64)
    float step_size;                  // lr / (1 - beta1^t)
    float inv_sqrt_bc2;               // 1 / sqrt(1 - beta2^t)
    float eps;
    float decay;                      // 1 - lr * weight_decay
    float v_floor;                    // l_floor of the second-moment code
    Exp2Coef cf;                      // decode polynomial
    int32_t nt;
    int64_t total_tiles;
    AdamWDesc t[kAdamWMaxTensors];
};

// Elements per tile: max(block of v, 256).
int adamw_tile_elems(int v_codec, int v_block);
hipError_t launch_adamw(const AdamWLaunch& a, int grad_dtype, int m_codec, int v_codec, int v_block,
                        int grid, hipStream_t s);

// ------------------------------------------------------------------ codec
hipError_t launch_quantize(int codec, const float* x, int64_t n, int block, float log_floor, void* codes,
                           float* meta, int grid_cap, hipStream_t s);
hipError_t launch_dequantize(int codec, const void* codes, const float* meta, int64_t n, int block,
                             float* out, int grid_cap, hipStream_t s);

hipError_t launch_diag_stream(int nt, float* p, const uint16_t* g, uint8_t* m, uint8_t* v, int64_t n,
                              hipStream_t s);
hipError_t launch_diag_math(int fn, const double* x, int64_t n, double* out, int grid_cap, hipStream_t s);

// ---------------------------------------------------- synthetic input fill
hipError_t launch_synth_normal(void* out, int out_bf16, int64_t n, uint64_t key, float scale,
                               uint64_t mask_key, uint64_t mask_threshold, int grid_cap, hipStream_t s);

// Taylor coefficients of the binary64 exp2 used by every decode.
const Exp2Coef& exp2_coef();

// Compute units of the current device (cached per device).
int device_cu_count();

}  // namespace al
