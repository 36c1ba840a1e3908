// Block encoder shared by the standalone codec and the factored-state
// finalize kernels: one wavefront encodes a tile of max(B, 256) consecutive
// fp32 values (4 per lane) into AL8 / AL16 / UF8 codes and block metadata.
#pragma once

#include "al_device.hpp"

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
        const double r = am != 0u ? rdiv127((double)s) : 0.0;
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
        const ALEnc enc = al_enc_params(f.lmin, f.any ? (double)LEVELS / f.delta : 1.0);
#pragma unroll
        for (int k = 0; k < K; ++k) {
            uint32_t q[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) q[j] = al_encode_fast<LEVELS>(xv[k][j], enc);
            if (blk_live) store_codes4<C>(codes, e0 + k * kSub + 4 * lane, q);
        }
    }
}

}  // namespace al
