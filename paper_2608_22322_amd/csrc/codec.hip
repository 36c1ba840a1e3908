// Standalone block codecs (gfx950): AL8 / AL16 quantize and dequantize
// (section 4.1, Eq. al_bounds, al_quant, al_dequant; section 4.2) and the
// uniform signed 8-bit code UF8 (section 4.3).
//
// Quantize: a wavefront owns a tile of max(B, 256) consecutive elements,
// 4 per lane; the block reduction (positive min/max, or absmax) runs in
// registers and across lanes; each element is read once and its code
// written once. Dequantize is elementwise, 4 elements per lane.
#include "al_device.hpp"
#include "al_internal.hpp"

namespace al {

template <int C, int B, bool FULL>
__device__ __forceinline__ void quantize_tile(const float* __restrict__ x, int64_t e0, int64_t valid, int lane,
                                              float log_floor, void* codes, float* meta) {
    constexpr int T = B > kSub ? B : kSub;
    constexpr int K = T / kSub;
    constexpr int GL = B < kSub ? B / 4 : 64;  // lanes per block
    float xv[K][4];
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int rel = k * kSub + 4 * lane;
        if constexpr (FULL) {
            F4 t = load_f4(x + e0 + rel);
#pragma unroll
            for (int j = 0; j < 4; ++j) xv[k][j] = t.v[j];
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) xv[k][j] = (rel + j < valid) ? x[e0 + rel + j] : 0.0f;
        }
    }
    const int64_t blk = (e0 + (B < kSub ? 4 * lane : 0)) / B;
    const bool leader = (lane % GL) == 0;
    const bool blk_live = FULL || (B < kSub ? (4 * (lane - lane % GL) < valid) : true);

    if constexpr (C == UF8) {
        uint32_t am = 0u;
#pragma unroll
        for (int k = 0; k < K; ++k)
#pragma unroll
            for (int j = 0; j < 4; ++j) am = OpMax::f(am, abs_bits(xv[k][j]));
        am = group_reduce<OpMax, GL>(am);
        const float s = u2f(am);
        const double r = am != 0u ? 127.0 / (double)s : 0.0;
        if (leader && blk_live) meta[blk] = s;
#pragma unroll
        for (int k = 0; k < K; ++k) {
            uint32_t q[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) q[j] = (uint32_t)uf8_encode(xv[k][j], r) & 0xFFu;
            if (blk_live) store_codes4<UF8>(codes, e0 + k * kSub + 4 * lane, q);
        }
    } else {
        constexpr int LEVELS = levels_of<C>();
        uint32_t mn = 0xFFFFFFFFu, mx = 0u;
#pragma unroll
        for (int k = 0; k < K; ++k)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                mn = OpMin::f(mn, pos_min_key(xv[k][j]));
                mx = OpMax::f(mx, pos_max_key(xv[k][j]));
            }
        mn = group_reduce<OpMin, GL>(mn);
        mx = group_reduce<OpMax, GL>(mx);
        const ALFit f = al_fit(mn, mx, log_floor);
        if (leader && blk_live)
            *reinterpret_cast<float2*>(meta + 2 * blk) =
                make_float2(f.any ? (float)f.lmin : 0.0f, f.any ? (float)f.delta : 0.0f);
#pragma unroll
        for (int k = 0; k < K; ++k) {
            uint32_t q[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) q[j] = al_encode<LEVELS>(xv[k][j], f);
            if (blk_live) store_codes4<C>(codes, e0 + k * kSub + 4 * lane, q);
        }
    }
}

template <int C, int B>
__global__ __launch_bounds__(256) void quantize_kernel(const float* __restrict__ x, int64_t n, float log_floor,
                                                        void* codes, float* meta) {
    constexpr int T = B > kSub ? B : kSub;
    const int lane = threadIdx.x & 63;
    const int64_t wpb = blockDim.x >> 6;
    const int64_t wave = (int64_t)blockIdx.x * wpb + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nwaves = (int64_t)gridDim.x * wpb;
    const int64_t tiles = (n + T - 1) / T;
    for (int64_t tile = wave; tile < tiles; tile += nwaves) {
        const int64_t e0 = tile * T;
        const int64_t valid = n - e0;
        if (valid >= T)
            quantize_tile<C, B, true>(x, e0, T, lane, log_floor, codes, meta);
        else
            quantize_tile<C, B, false>(x, e0, valid, lane, log_floor, codes, meta);
    }
}

template <int C, int B>
__global__ __launch_bounds__(256) void dequantize_kernel(const void* __restrict__ codes,
                                                          const float* __restrict__ meta, int64_t n,
                                                          float* __restrict__ out) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; 4 * i < n; i += stride) {
        const int64_t e = 4 * i;
        const int64_t blk = e / B;
        uint32_t q[4];
        const bool full = e + 4 <= n;
        if (full) {
            load_codes4<C>(codes, e, q);
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) q[j] = (e + j < n) ? load_code1<C>(codes, e + j) : 0u;
        }
        F4 o;
        if constexpr (C == UF8) {
            const double step = (double)meta[blk] / 127.0;
#pragma unroll
            for (int j = 0; j < 4; ++j) o.v[j] = uf8_decode((int32_t)(int8_t)(uint8_t)q[j], step);
        } else {
            const float2 mm = *reinterpret_cast<const float2*>(meta + 2 * blk);
            const double l32 = (double)mm.x;
            const double step = (double)mm.y / (double)levels_of<C>();
#pragma unroll
            for (int j = 0; j < 4; ++j) o.v[j] = al_decode(q[j], l32, step);
        }
        if (full) {
            store_f4(out + e, o);
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (e + j < n) out[e + j] = o.v[j];
        }
    }
}

template <int C>
static hipError_t quant_b(const float* x, int64_t n, int block, float lf, void* codes, float* meta, int grid,
                          hipStream_t s) {
    switch (block) {
#define AL_Q(BB)                                                                                         \
    case BB:                                                                                             \
        hipLaunchKernelGGL((quantize_kernel<C, BB>), dim3(grid), dim3(256), 0, s, x, n, lf, codes, meta); \
        return hipGetLastError();
        AL_Q(64)
        AL_Q(128)
        AL_Q(256)
        AL_Q(512)
        AL_Q(1024)
        AL_Q(2048)
#undef AL_Q
    }
    return hipErrorInvalidValue;
}

template <int C>
static hipError_t dequant_b(const void* codes, const float* meta, int64_t n, int block, float* out, int grid,
                            hipStream_t s) {
    switch (block) {
#define AL_D(BB)                                                                                           \
    case BB:                                                                                               \
        hipLaunchKernelGGL((dequantize_kernel<C, BB>), dim3(grid), dim3(256), 0, s, codes, meta, n, out); \
        return hipGetLastError();
        AL_D(64)
        AL_D(128)
        AL_D(256)
        AL_D(512)
        AL_D(1024)
        AL_D(2048)
#undef AL_D
    }
    return hipErrorInvalidValue;
}

hipError_t launch_quantize(int codec, const float* x, int64_t n, int block, float log_floor, void* codes,
                           float* meta, int grid_cap, hipStream_t s) {
    const int64_t T = block > kSub ? block : kSub;
    const int64_t tiles = (n + T - 1) / T;
    const int64_t want = (tiles + 3) / 4;
    const int grid = (int)(want < grid_cap ? want : grid_cap);
    if (grid <= 0) return hipSuccess;
    switch (codec) {
        case AL8: return quant_b<AL8>(x, n, block, log_floor, codes, meta, grid, s);
        case AL16: return quant_b<AL16>(x, n, block, log_floor, codes, meta, grid, s);
        case UF8: return quant_b<UF8>(x, n, block, log_floor, codes, meta, grid, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_dequantize(int codec, const void* codes, const float* meta, int64_t n, int block, float* out,
                             int grid_cap, hipStream_t s) {
    const int64_t want = ((n + 3) / 4 + 255) / 256;
    const int grid = (int)(want < grid_cap ? want : grid_cap);
    if (grid <= 0) return hipSuccess;
    switch (codec) {
        case AL8: return dequant_b<AL8>(codes, meta, n, block, out, grid, s);
        case AL16: return dequant_b<AL16>(codes, meta, n, block, out, grid, s);
        case UF8: return dequant_b<UF8>(codes, meta, n, block, out, grid, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace al
