// Fused multi-tensor AdamW step with block-quantized state (gfx950).
//
// One pass over HBM per step: read p (fp32), g (bf16/fp32), m (UF8 codes +
// absmax per 256, or fp32) and v (AL8/AL16 codes + {l_min, delta} per
// block, or fp32); write p, m, v and their metadata. Section 3.1 (Eq.
// adam_update) with PyTorch AdamW's decoupled weight decay and bias
// corrections; codes per section 4 (Eq. al_bounds, al_quant, al_dequant,
// exact_zero) and the uniform signed momentum code of section 4.3.
//
// Work decomposition: a tile is max(B_V, 256) consecutive elements of one
// tensor; a wavefront owns a tile at a time (4 elements per lane per
// 256-element sub-tile), so every block reduction stays inside the
// wavefront (DPP / swizzle / readlane) and each element is read once and
// written once. Waves stride over the launch's tiles; the tile -> tensor
// map is a binary search over the descriptor table in the kernel arguments.
#include "al_device.hpp"
#include "al_internal.hpp"

namespace al {

template <int G, int MC, int VC, int BV, bool FULL>
__device__ __forceinline__ void adamw_tile(const AdamWLaunch& a, const AdamWDesc& d, int64_t e0,
                                           int64_t valid, int lane) {
    constexpr int T = BV > kSub ? BV : kSub;
    constexpr int K = T / kSub;
    constexpr bool VQ = (VC == AL8 || VC == AL16);
    constexpr int LEVELS = levels_of<VC>();

    float vkeep[K][4];
    uint32_t vmin = 0xFFFFFFFFu, vmax = 0u;

    // second-moment metadata of the block(s) this lane decodes
    double v_lmin32 = 0.0, v_step = 0.0;
    if constexpr (VQ) {
        const int64_t vb = (e0 + (BV < kSub ? 4 * lane : 0)) / BV;
        const bool vb_live = FULL || (BV < kSub ? (4 * lane < valid) : true);
        if (vb_live) {
            float2 mm = *reinterpret_cast<const float2*>(d.vm + 2 * vb);
            v_lmin32 = (double)mm.x;
            v_step = (double)mm.y / (double)LEVELS;
        }
    }

#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int rel = k * kSub + 4 * lane;  // offset of this lane's first element in the tile
        const int64_t e = e0 + rel;
        const bool sub_live = FULL || (k * kSub < valid);

        // ---------------- loads
        F4 p, g, mh, vh;
        if constexpr (FULL) {
            p = load_f4(d.p + e);
            g = load_grad4<G>(d.g, e);
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const bool ok = rel + j < valid;
                p.v[j] = ok ? d.p[e + j] : 0.0f;
                g.v[j] = ok ? load_grad1<G>(d.g, e + j) : 0.0f;
            }
        }
        // momentum decode
        if constexpr (MC == UF8) {
            const double m_step = sub_live ? (double)d.ms[(e0 + k * kSub) / kSub] / 127.0 : 0.0;
            uint32_t q[4];
            if constexpr (FULL) {
                load_codes4<UF8>(d.m, e, q);
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) q[j] = (rel + j < valid) ? load_code1<UF8>(d.m, e + j) : 0u;
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) mh.v[j] = uf8_decode((int32_t)(int8_t)(uint8_t)q[j], m_step);
        } else {
            if constexpr (FULL) {
                mh = load_f4(reinterpret_cast<const float*>(d.m) + e);
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    mh.v[j] = (rel + j < valid) ? reinterpret_cast<const float*>(d.m)[e + j] : 0.0f;
            }
        }
        // second-moment decode
        if constexpr (VQ) {
            uint32_t q[4];
            if constexpr (FULL) {
                load_codes4<VC>(d.v, e, q);
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) q[j] = (rel + j < valid) ? load_code1<VC>(d.v, e + j) : 0u;
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) vh.v[j] = al_decode(q[j], v_lmin32, v_step);
        } else {
            if constexpr (FULL) {
                vh = load_f4(reinterpret_cast<const float*>(d.v) + e);
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    vh.v[j] = (rel + j < valid) ? reinterpret_cast<const float*>(d.v)[e + j] : 0.0f;
            }
        }

        // ---------------- moments (binary64, rounded once to fp32) and parameter (fp32)
        F4 mn, vn;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const double gd = (double)g.v[j];
            mn.v[j] = (float)(a.beta1 * (double)mh.v[j] + a.omb1 * gd);
            vn.v[j] = (float)(a.beta2 * (double)vh.v[j] + a.omb2 * (gd * gd));
            float pn = p.v[j] * a.decay;
            const float den = __builtin_amdgcn_sqrtf(vn.v[j]) * a.inv_sqrt_bc2 + a.eps;
            pn = pn - a.step_size * mn.v[j] * __builtin_amdgcn_rcpf(den);
            p.v[j] = pn;
        }
        if constexpr (!FULL) {
            // elements past the end are absent: no state, no contribution to reductions
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (rel + j >= valid) mn.v[j] = vn.v[j] = 0.0f;
        }
        if constexpr (FULL) {
            store_f4(d.p + e, p);
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (rel + j < valid) d.p[e + j] = p.v[j];
        }

        // ---------------- momentum encode (block = this 256-element sub-tile)
        if constexpr (MC == UF8) {
            uint32_t am = abs_bits(mn.v[0]);
#pragma unroll
            for (int j = 1; j < 4; ++j) am = OpMax::f(am, abs_bits(mn.v[j]));
            am = group_reduce<OpMax, 64>(am);
            const float s = u2f(am);
            const double r = am != 0u ? 127.0 / (double)s : 0.0;
            uint32_t q[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) q[j] = (uint32_t)uf8_encode(mn.v[j], r) & 0xFFu;
            if (sub_live) {
                store_codes4<UF8>(d.m, e, q);
                if (lane == 0) d.ms[(e0 + k * kSub) / kSub] = s;
            }
        } else {
            if constexpr (FULL) {
                store_f4(reinterpret_cast<float*>(d.m) + e, mn);
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (rel + j < valid) reinterpret_cast<float*>(d.m)[e + j] = mn.v[j];
            }
        }

        // ---------------- second moment: keep for the block encode
        if constexpr (VQ) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                vkeep[k][j] = vn.v[j];
                vmin = OpMin::f(vmin, pos_min_key(vn.v[j]));
                vmax = OpMax::f(vmax, pos_max_key(vn.v[j]));
            }
        } else {
            if constexpr (FULL) {
                store_f4(reinterpret_cast<float*>(d.v) + e, vn);
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (rel + j < valid) reinterpret_cast<float*>(d.v)[e + j] = vn.v[j];
            }
        }
    }

    // ---------------- second-moment block fit and encode
    if constexpr (VQ) {
        constexpr int GL = BV < kSub ? BV / 4 : 64;  // lanes per block
        vmin = group_reduce<OpMin, GL>(vmin);
        vmax = group_reduce<OpMax, GL>(vmax);
        const ALFit f = al_fit(vmin, vmax, a.v_floor);
        const int64_t vb = (e0 + (BV < kSub ? 4 * lane : 0)) / BV;
        const bool leader = (BV < kSub) ? ((lane % GL) == 0) : (lane == 0);
        const bool blk_live = FULL || (BV < kSub ? (4 * (lane - lane % GL) < valid) : true);
        if (leader && blk_live) {
            float2 mm = make_float2(f.any ? (float)f.lmin : 0.0f, f.any ? (float)f.delta : 0.0f);
            *reinterpret_cast<float2*>(d.vm + 2 * vb) = mm;
        }
#pragma unroll
        for (int k = 0; k < K; ++k) {
            uint32_t q[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) q[j] = al_encode<LEVELS>(vkeep[k][j], f);
            if (blk_live) store_codes4<VC>(d.v, e0 + k * kSub + 4 * lane, q);
        }
    }
}

template <int G, int MC, int VC, int BV>
__global__ __launch_bounds__(256) void adamw_kernel(const AdamWLaunch a) {
    constexpr int T = BV > kSub ? BV : kSub;
    const int lane = threadIdx.x & 63;
    const int64_t wpb = blockDim.x >> 6;
    const int64_t wave = (int64_t)blockIdx.x * wpb + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nwaves = (int64_t)gridDim.x * wpb;
    for (int64_t tile = wave; tile < a.total_tiles; tile += nwaves) {
        // largest ti with t[ti].tile_begin <= tile
        int lo = 0, hi = a.nt - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (a.t[mid].tile_begin <= tile)
                lo = mid;
            else
                hi = mid - 1;
        }
        const AdamWDesc& d = a.t[lo];
        const int64_t e0 = (tile - d.tile_begin) * T;
        const int64_t valid = d.n - e0;
        if (valid >= T)
            adamw_tile<G, MC, VC, BV, true>(a, d, e0, T, lane);
        else
            adamw_tile<G, MC, VC, BV, false>(a, d, e0, valid, lane);
    }
}

int adamw_tile_elems(int v_codec, int v_block) {
    if (v_codec == FP32) return kSub;
    return v_block > kSub ? v_block : kSub;
}

template <int G, int MC, int VC, int BV>
static hipError_t launch_t(const AdamWLaunch& a, int grid, hipStream_t s) {
    hipLaunchKernelGGL((adamw_kernel<G, MC, VC, BV>), dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int G, int MC, int VC>
static hipError_t launch_bv(const AdamWLaunch& a, int bv, int grid, hipStream_t s) {
    if constexpr (VC == FP32) {
        return launch_t<G, MC, VC, 256>(a, grid, s);
    } else {
        switch (bv) {
            case 64: return launch_t<G, MC, VC, 64>(a, grid, s);
            case 128: return launch_t<G, MC, VC, 128>(a, grid, s);
            case 256: return launch_t<G, MC, VC, 256>(a, grid, s);
            case 512: return launch_t<G, MC, VC, 512>(a, grid, s);
            case 1024: return launch_t<G, MC, VC, 1024>(a, grid, s);
            case 2048: return launch_t<G, MC, VC, 2048>(a, grid, s);
        }
        return hipErrorInvalidValue;
    }
}

template <int G, int MC>
static hipError_t launch_vc(const AdamWLaunch& a, int vc, int bv, int grid, hipStream_t s) {
    switch (vc) {
        case AL8: return launch_bv<G, MC, AL8>(a, bv, grid, s);
        case AL16: return launch_bv<G, MC, AL16>(a, bv, grid, s);
        case FP32: return launch_bv<G, MC, FP32>(a, bv, grid, s);
    }
    return hipErrorInvalidValue;
}

template <int G>
static hipError_t launch_mc(const AdamWLaunch& a, int mc, int vc, int bv, int grid, hipStream_t s) {
    switch (mc) {
        case UF8: return launch_vc<G, UF8>(a, vc, bv, grid, s);
        case FP32: return launch_vc<G, FP32>(a, vc, bv, grid, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_adamw(const AdamWLaunch& a, int grad_dtype, int m_codec, int v_codec, int v_block, int grid,
                        hipStream_t s) {
    if (grad_dtype == G_BF16) return launch_mc<G_BF16>(a, m_codec, v_codec, v_block, grid, s);
    return launch_mc<G_F32>(a, m_codec, v_codec, v_block, grid, s);
}

}  // namespace al
