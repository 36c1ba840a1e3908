// Factored-state optimizer steps on gfx950: Adafactor (factored second
// moment) and CAME (factored second moment + factored confidence + dense
// momentum), section 3.1, with AL/UF8/FP32 codes per state role (section 4).
//
// Kernel sequence of one Adafactor step (2-D tensors):
//   marg   row and column sums of G2 = g^2 + eps1, exact (double-double)
//   fin    one wavefront per code block of R and C: EMA of the exact means,
//          rounded to fp32, re-encoded; then per tensor mean(R) and the
//          factors r_i = (R_i / mean R)^-1/2, c_j = C_j^-1/2
//   rms    partial sums of u^2, u_ij = (r_i c_j) g_ij, per 256x256 unit
//   clip   per tensor: max(1, RMS(u) / d)
//   apply  p <- p (1 - lr wd) - lr u / clip
// 1-D tensors run their whole step in one workgroup (vec1d).
// CAME adds: res (sums of (uhat - m)^2 + eps2 with the in-step momentum),
// fin over the confidence, and apply (recompute uhat and m, encode m, update p).
//
// Marginal sums. A wavefront owns a 256x256 unit, walked as 16 groups of 16
// rows x 4 tiles of 64 columns. It loads a 16x64 tile in the natural layout
// (16 lanes x 4 columns x 4 rows, coalesced row segments), adds each term to
// in-lane column accumulators, and stages its binary64 terms in LDS (8.4 KB
// per wave, plus 4 KB of row accumulators: 12 waves per CU); 4 lanes then
// sum each tile row out of LDS.
// Each lane sums its terms in runs of at most 4 plain binary64 additions
// (relative error <= 3u) accumulated double-double, so every partial is within
// 3u of its exact sum. The finalize step keeps the fast sum only where that
// cannot change the fp32 rounding of the state's EMA and otherwise sums the
// element's row or column again exactly, so the fp32 states (and their codes)
// are the ones of the exactly rounded means.
#include "al_codec_dev.hpp"
#include "al_device.hpp"
#include "al_internal.hpp"

namespace al {

// ------------------------------------------------------------------ helpers
__device__ __forceinline__ int locate_unit(const FacDesc* D, int n, int64_t unit) {
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (D[mid].unit_begin <= unit)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

__device__ __forceinline__ int locate_chunk(const FacDesc* D, int n, int64_t chunk) {
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (D[mid].chunk_begin <= chunk)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// Global-address-space view of the data pointers of a descriptor (the
// descriptors are read from the workspace, so their pointers are generic to
// the compiler; see gp in al_device.hpp).
struct GD {
    gp<float> p;
    gp<const void> g;
    gp<void> m;
    gp<float> mm;
    gp<double> colpart, rowpart;
    gp<const double> rfac, cfac, sr, sc;
    gp<const double> scal;
    int64_t rows, cols, unit_begin;
    int32_t nru, ncu;
};

__device__ __forceinline__ GD gview(const FacDesc& d) {
    GD v;
    v.p = to_g(d.p);
    v.g = to_g(d.g);
    v.m = to_g(d.m);
    v.mm = to_g(d.mm);
    v.colpart = to_g(d.colpart);
    v.rowpart = to_g(d.rowpart);
    v.rfac = to_g((const double*)d.rfac);
    v.cfac = to_g((const double*)d.cfac);
    v.sr = to_g((const double*)d.sr);
    v.sc = to_g((const double*)d.sc);
    v.scal = to_g((const double*)d.scal);
    v.rows = d.rows;
    v.cols = d.cols;
    v.unit_begin = d.unit_begin;
    v.nru = d.nru;
    v.ncu = d.ncu;
    return v;
}

// Term of the second moment's marginal sums: fl64(g^2 + eps1).
__device__ __forceinline__ double marg_term(float g, double eps1) {
    const double x = (double)g;
    return x * x + eps1;
}

// Term of CAME's confidence marginal sums, from the decoded momentum and the
// clipped update: m = fl32(beta1 mhat + (1 - beta1) uhat), (uhat - m)^2 + eps2.
__device__ __forceinline__ double res_term(const FacArgs& a, float mh, float uh) {
    const float m = (float)(a.beta1 * (double)mh + a.omb1 * (double)uh);
    const double df = (double)uh - (double)m;
    return df * df + a.eps2;
}

// uhat - m of the same term (exact in binary64): the whole-unit residual pass
// accumulates its square with fused multiply-adds and adds eps2 to the mean.
__device__ __forceinline__ double res_diff(const FacArgs& a, float mh, float uh) {
    const float m = (float)(a.beta1 * (double)mh + a.omb1 * (double)uh);
    return (double)uh - (double)m;
}

template <int G>
__device__ __forceinline__ float grad1(const void* g, int64_t e) {
    if constexpr (G == G_BF16)
        return bf16_to_f32(reinterpret_cast<const uint16_t*>(g)[e]);
    else
        return reinterpret_cast<const float*>(g)[e];
}

// 4 consecutive gradients at element e (the caller guarantees alignment).
template <int G>
__device__ __forceinline__ void grad4(const void* g, int64_t e, float out[4]) {
    if constexpr (G == G_BF16) {
        const uint2 w = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(g) + e);
        out[0] = bf16_to_f32(w.x & 0xFFFFu);
        out[1] = bf16_to_f32(w.x >> 16);
        out[2] = bf16_to_f32(w.y & 0xFFFFu);
        out[3] = bf16_to_f32(w.y >> 16);
    } else {
        const float4 w = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(g) + e);
        out[0] = w.x;
        out[1] = w.y;
        out[2] = w.z;
        out[3] = w.w;
    }
}

// Decode element i of a vector state (runtime codec / block).
__device__ __forceinline__ float vec_decode(int codec, int B, const void* codes, const float* meta, int64_t i,
                                            const Exp2Coef& cf) {
    if (codec == FP32) return reinterpret_cast<const float*>(codes)[i];
    if (codec == UF8) {
        const int32_t q = reinterpret_cast<const int8_t*>(codes)[i];
        return uf8_decode(q, div127((double)meta[i / B]));
    }
    const uint32_t q = codec == AL16 ? reinterpret_cast<const uint16_t*>(codes)[i]
                                     : reinterpret_cast<const uint8_t*>(codes)[i];
    if (q == 0u) return 0.0f;
    const int64_t b = i / B;
    const double step = (double)meta[2 * b + 1] / (codec == AL16 ? 65534.0 : 254.0);
    return al_decode_fast(q, (double)meta[2 * b], step, cf);
}

// Encode x[0, n) into a vector state, one block per wavefront at a time
// (runtime codec / block; the vectors are small). Padding codes are 0.
__device__ void vec_encode(int codec, int B, const float* x, int64_t n, float log_floor, void* codes, float* meta,
                           int wave, int nwaves, int lane) {
    if (codec == FP32) {
        for (int64_t i = (int64_t)wave * 64 + lane; i < n; i += (int64_t)nwaves * 64)
            reinterpret_cast<float*>(codes)[i] = x[i];
        return;
    }
    const int64_t nb = (n + B - 1) / B;
    for (int64_t b = wave; b < nb; b += nwaves) {
        const int64_t s = b * B;
        const int64_t e = s + B < n ? s + B : n;
        if (codec == UF8) {
            uint32_t am = 0u;
            for (int64_t i = s + lane; i < e; i += 64) am = OpMax::f(am, abs_bits(x[i]));
            am = group_reduce<OpMax, 64>(am);
            const double r = am != 0u ? rdiv127((double)u2f(am)) : 0.0;
            if (lane == 0) meta[b] = u2f(am);
            for (int64_t i = s + lane; i < s + B; i += 64) {
                const int32_t q = i < e ? (int32_t)__builtin_rint((double)x[i] * r) : 0;
                reinterpret_cast<int8_t*>(codes)[i] = (int8_t)q;
            }
        } else {
            uint32_t mn = 0xFFFFFFFFu, mx = 0u;
            for (int64_t i = s + lane; i < e; i += 64) {
                mn = OpMin::f(mn, pos_min_key(x[i]));
                mx = OpMax::f(mx, pos_max_key(x[i]));
            }
            mn = group_reduce<OpMin, 64>(mn);
            mx = group_reduce<OpMax, 64>(mx);
            const ALFit f = al_fit(mn, mx, log_floor);
            if (lane == 0) {
                meta[2 * b] = f.any ? (float)f.lmin : 0.0f;
                meta[2 * b + 1] = f.any ? (float)f.delta : 0.0f;
            }
            const int levels = codec == AL16 ? 65534 : 254;
            const ALEnc enc = al_enc_params(f.lmin, f.any ? (double)levels / f.delta : 1.0);
            for (int64_t i = s + lane; i < s + B; i += 64) {
                const float v = i < e ? x[i] : 0.0f;
                const uint32_t q = codec == AL16 ? al_encode_fast<65534>(v, enc) : al_encode_fast<254>(v, enc);
                if (codec == AL16)
                    reinterpret_cast<uint16_t*>(codes)[i] = (uint16_t)q;
                else
                    reinterpret_cast<uint8_t*>(codes)[i] = (uint8_t)q;
            }
        }
    }
}

// Block-wide (256 threads) double-double total in a fixed order.
__device__ DD block_dd_sum(DD v, DD* sh) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    v = dd_wave_sum(v);
    if (lane == 0) sh[w] = v;
    __syncthreads();
    DD t = sh[0];
    for (int k = 1; k < (int)(blockDim.x >> 6); ++k) t = dd_merge(t, sh[k]);
    __syncthreads();
    return t;
}

// --------------------------------------------------------------- descriptors
__global__ void fac_desc_copy_kernel(const FacDescBatch b, FacDesc* dst) {
    constexpr int W = sizeof(FacDesc) / 8;
    const int total = b.count * W;
    const uint64_t* src = reinterpret_cast<const uint64_t*>(b.d);
    uint64_t* out = reinterpret_cast<uint64_t*>(dst + b.offset);
    for (int i = threadIdx.x; i < total; i += blockDim.x) out[i] = src[i];
}

hipError_t fac_copy_desc(const FacDesc* host, int count, FacDesc* dev, hipStream_t s) {
    static_assert(sizeof(FacDesc) % 8 == 0, "descriptor size");
    for (int off = 0; off < count; off += kFacCopyBatch) {
        FacDescBatch b;
        b.count = count - off < kFacCopyBatch ? count - off : kFacCopyBatch;
        b.offset = off;
        for (int i = 0; i < b.count; ++i) b.d[i] = host[off + i];
        hipLaunchKernelGGL(fac_desc_copy_kernel, dim3(1), dim3(256), 0, s, b, dev);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// ------------------------------------------------------- marginal sums of G2
// Lane roles in a 16x64 tile of a 256x256 unit. Load layout: lane (lr, lc) =
// (lane / 16, lane % 16) holds rows lr + 4i (i < 4), columns 4 lc .. 4 lc + 3
// (16 lanes cover a coalesced 64-column row segment). Row layout: lane
// (rrow, rq) = (lane / 4, lane % 4) sums row rrow, columns 16 rq .. 16 rq + 15
// of the tile out of LDS. Column sums stay in the loading lanes across the
// unit's rows; a row's partial is merged over its 4 lanes after the unit's 4
// column tiles. Every wave owns one unit, so the kernel has no unit loop.
constexpr int kTileRows = 16;

// Raw gradient words of one lane's 4 rows x 4 columns of a tile (bf16 pairs or
// fp32), loaded one tile ahead of the arithmetic; absent elements read as 0.
template <int G>
struct GRaw {
    uint2 w[4];
};
template <>
struct GRaw<G_F32> {
    float4 w[4];
};

// Tile width TC = 64: 16 lanes per row, lane rows lr + 4i of a 16-row group;
// TC = 128: 32 lanes per row, lane rows lr + 2i of an 8-row group.
// lane_off = lr * cols + 4 lc, the lane's part of every element index (formed
// once per unit), so each address is a wave-uniform base plus that offset.
template <int G, bool FULL, int TC = 64>
__device__ __forceinline__ void load_graw(GRaw<G>& r, const GD& d, int64_t r0, int64_t c0, int nr, int nc,
                                          int rg, int ct, int lr, int lc, bool vec, int64_t lane_off) {
    constexpr int LS = 256 / TC, TR = 4 * LS;
    const int cc = ct * TC + 4 * lc;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int rr = rg * TR + lr + LS * i;
        const int64_t e = (r0 + rg * TR + LS * i) * d.cols + c0 + ct * TC + lane_off;
        if constexpr (G == G_BF16) {
            const gp<const uint16_t> g = g_as<const uint16_t>(d.g);
            if (FULL || (rr < nr && vec && cc + 4 <= nc)) {
                r.w[i] = ld_u2<false>(g_as<const void>(g + e));
            } else {
                uint32_t h[4] = {0u, 0u, 0u, 0u};
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (rr < nr && cc + j < nc) h[j] = g[e + j];
                r.w[i] = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
            }
        } else {
            const gp<const float> g = g_as<const float>(d.g);
            if (FULL || (rr < nr && vec && cc + 4 <= nc)) {
                r.w[i] = ld_f4<false>(g + e);
            } else {
                float h[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (rr < nr && cc + j < nc) h[j] = g[e + j];
                r.w[i] = make_float4(h[0], h[1], h[2], h[3]);
            }
        }
    }
}

template <int G>
__device__ __forceinline__ void unpack_graw(const GRaw<G>& r, int i, float gv[4]) {
    if constexpr (G == G_BF16) {
        gv[0] = bf16_to_f32(r.w[i].x & 0xFFFFu);
        gv[1] = bf16_to_f32(r.w[i].x >> 16);
        gv[2] = bf16_to_f32(r.w[i].y & 0xFFFFu);
        gv[3] = bf16_to_f32(r.w[i].y >> 16);
    } else {
        gv[0] = r.w[i].x;
        gv[1] = r.w[i].y;
        gv[2] = r.w[i].z;
        gv[3] = r.w[i].w;
    }
}

// Column tiles outermost, 16-row groups inside: the column sums of the current
// 64-column tile stay in registers, each row's running sum over the column
// tiles in LDS (owned by one lane), and the next tile's gradients are loaded
// while the current one is summed.
template <int G, bool FULL>
__device__ __forceinline__ void marg_unit(const FacArgs& a, const GD& d, int64_t ru, int64_t cu, int nr_, int nc_,
                                          bool vec_, double (*tile)[66], DD* racc) {
    const int lane = threadIdx.x, lc = lane & 15, lr = lane >> 4, rrow = lane >> 2, rq = lane & 3;
    const int64_t r0 = ru * 256, c0 = cu * 256;
    const int nr = FULL ? 256 : nr_, nc = FULL ? 256 : nc_;
    const bool vec = FULL || vec_;
    const double eps1 = a.eps1;
    const int nrg = (nr + kTileRows - 1) / kTileRows, nct = (nc + 63) / 64, total = nrg * nct;
#pragma unroll
    for (int k = 0; k < 4; ++k) racc[lane + 64 * k] = DD{0.0, 0.0};
    DD cacc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) cacc[j] = DD{0.0, 0.0};
    GRaw<G> cur;
    const int64_t lane_off = (int64_t)lr * d.cols + 4 * lc;
    load_graw<G, FULL>(cur, d, r0, c0, nr, nc, 0, 0, lr, lc, vec, lane_off);
    for (int it = 0; it < total; ++it) {
        const int ct = it / nrg, rg = it - ct * nrg;
        GRaw<G> nxt = cur;
        if (it + 1 < total) {
            const int ct1 = (it + 1) / nrg;
            load_graw<G, FULL>(nxt, d, r0, c0, nr, nc, it + 1 - ct1 * nrg, ct1, lr, lc, vec, lane_off);
        }
        const int cc = ct * 64 + 4 * lc;
        double gs[4] = {0.0, 0.0, 0.0, 0.0};  // the lane's 4 rows of each column, summed in row order
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float gv[4];
            unpack_graw<G>(cur, i, gv);
            double t[4] = {0.0, 0.0, 0.0, 0.0};
            if (FULL || rg * kTileRows + lr + 4 * i < nr) {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (FULL || cc + j < nc) t[j] = marg_term(gv[j], eps1);
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) gs[j] += t[j];
            // the binary64 terms are staged once for the row sums
            double* tp = &tile[lr + 4 * i][4 * lc];
            *reinterpret_cast<double2*>(tp) = make_double2(t[0], t[1]);
            *reinterpret_cast<double2*>(tp + 2) = make_double2(t[2], t[3]);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) dd_add(cacc[j], gs[j]);
        __syncthreads();
        DD rsum{0.0, 0.0};
        const int rr = rg * kTileRows + rrow;
        const int cq = ct * 64 + 16 * rq;  // first column of this lane's quarter
        if (FULL || (rr < nr && cq < nc)) {
            if (FULL || cq + 16 <= nc) {
#pragma unroll
                for (int c = 0; c < 16; c += 4) {
                    const double2 t0 = *reinterpret_cast<const double2*>(&tile[rrow][16 * rq + c]);
                    const double2 t1 = *reinterpret_cast<const double2*>(&tile[rrow][16 * rq + c + 2]);
                    dd_add(rsum, ((t0.x + t0.y) + t1.x) + t1.y);
                }
            } else {
                for (int c = 0; c < nc - cq; ++c) dd_add(rsum, tile[rrow][16 * rq + c]);
            }
        }
        rsum = dd_merge(rsum, dd_quad_xor<kDppQuadXor1>(rsum));
        rsum = dd_merge(rsum, dd_quad_xor<kDppQuadXor2>(rsum));
        if (rq == 0 && (FULL || rr < nr)) racc[rr] = dd_merge(racc[rr], rsum);
        __syncthreads();
        if (rg == nrg - 1) {
            // column tile done: its column partials over the unit's rows
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                DD v = cacc[j];
                v = dd_merge(v, dd_shfl_xor(v, 16));
                v = dd_merge(v, dd_shfl_xor(v, 32));
                const int col = cc + j;
                if (lr == 0 && (FULL || col < nc)) {
                    const gp<double> cp = d.colpart + 2 * (ru * d.cols + c0 + col);
                    cp[0] = v.hi;
                    cp[1] = v.lo;
                }
                cacc[j] = DD{0.0, 0.0};
            }
        }
        cur = nxt;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int row = lane + 64 * k;
        if (FULL || row < nr) {
            const gp<double> rp = d.rowpart + 2 * (cu * d.rows + r0 + row);
            rp[0] = racc[row].hi;
            rp[1] = racc[row].lo;
        }
    }
}

// Interior units (256x256, width a multiple of 4) take a guard-free body.
template <int G>
__global__ __launch_bounds__(64) void fac_marg_g2_kernel(const FacArgs a, int64_t base) {
    __shared__ __attribute__((aligned(16))) double tile[kTileRows][66];
    __shared__ DD racc[256];
    const int64_t unit = base + xcd_order(blockIdx.x, gridDim.x);
    if (unit >= a.total_units) return;
    const FacDesc& d = a.D[locate_unit(a.D, a.n2, unit)];
    const int64_t u = unit - d.unit_begin;
    const int64_t ru = u / d.ncu, cu = u % d.ncu;
    const int nr = (int)(d.rows - ru * 256 < 256 ? d.rows - ru * 256 : 256);
    const int nc = (int)(d.cols - cu * 256 < 256 ? d.cols - cu * 256 : 256);
    const bool vec = (d.cols & 3) == 0;
    if (nr == 256 && nc == 256 && vec)
        marg_unit<G, true>(a, gview(d), ru, cu, nr, nc, vec, tile, racc);
    else
        marg_unit<G, false>(a, gview(d), ru, cu, nr, nc, vec, tile, racc);
}

// One 64-thread workgroup per unit of [begin, end); lists beyond 2^31 units
// take several launches. Each kernel checks unit < end itself.
template <class K>
static hipError_t launch_per_unit(K kernel, const FacArgs& a, int64_t begin, int64_t end, hipStream_t s) {
    constexpr int64_t kMaxGrid = int64_t(1) << 31;
    for (int64_t base = begin; base < end; base += kMaxGrid) {
        const int64_t left = end - base;
        const int64_t grid = left < kMaxGrid ? left : kMaxGrid;
        hipLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(64), 0, s, a, base);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// One wavefront per unit (4 per 256-thread workgroup); lists beyond 2^33 units
// take several launches.
template <class K>
static hipError_t launch_wave_per_unit(K kernel, const FacArgs& a, int64_t begin, int64_t end, hipStream_t s) {
    constexpr int64_t kMaxGrid = int64_t(1) << 31;
    for (int64_t base = begin; base < end; base += 4 * kMaxGrid) {
        const int64_t left = (end - base + 3) / 4;
        const int64_t grid = left < kMaxGrid ? left : kMaxGrid;
        hipLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(256), 0, s, a, base);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// ------------------------------ marginal sums over whole units (streaming)
// Units of the tensors whose rows and columns are both multiples of 256: no
// guards, and every unit row starts 16-byte aligned. A batch is 8 unit rows.
// Lane l = 32 h + q reads columns 8q .. 8q + 7 of rows 2k + h (k < 4) of the
// batch: 16 bytes of bf16 gradients per lane, one load instruction per pair of
// unit rows, the next batch's loads issued before the current batch's
// arithmetic. Rows: each lane adds its 8 terms pairwise (relative error <= 3u
// for non-negative terms) and stages that partial in LDS; 8 lanes then finish
// each row from 4 partials apiece (pairwise, then a quad and a half-row DPP
// merge), so a row's partial over the unit has relative error <= 8u and needs
// no further merge inside the unit. Columns: with all terms of a batch formed
// at once (the second moment's terms), the loading lanes add them in plain runs
// over 16 of their rows (<= 15u) and add the 8 runs of the unit (<= 7u more).
// CAME's residual terms (uhat - m)^2 + eps2 are formed one row pair at a time
// (they need the registers) and summed without eps2: each lane accumulates the
// squares of its 128 rows' differences by fused multiply-adds (<= 128u, one
// rounding per term) and its row partials likewise (8 terms), and the finalize
// adds eps2 to the mean; the oracle's terms fl64(fl64(d^2) + eps2) are within
// 2u of d^2 + eps2. The even- and odd-row halves merge at the end (1u): a
// column partial has relative error <= 23u or <= 131u against the exact sum
// of the terms. The finalize step's robustness margin covers these bounds.
constexpr int kWStride = 34;  // LDS stride of a staged row, in doubles (16-byte aligned rows)
constexpr int kWRunRows = 32; // unit rows per plain column run (16 rows of each lane)

template <int G>
struct Raw8 {
    uint4 w;  // 8 bf16
};
template <>
struct Raw8<G_F32> {
    float4 a, b;
};

template <int G>
__device__ __forceinline__ void unpack8(const Raw8<G>& r, float gv[8]) {
    if constexpr (G == G_BF16) {
        const uint32_t w[4] = {r.w.x, r.w.y, r.w.z, r.w.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            gv[2 * i] = u2f(w[i] << 16);
            gv[2 * i + 1] = u2f(w[i] & 0xFFFF0000u);
        }
    } else {
        gv[0] = r.a.x, gv[1] = r.a.y, gv[2] = r.a.z, gv[3] = r.a.w;
        gv[4] = r.b.x, gv[5] = r.b.y, gv[6] = r.b.z, gv[7] = r.b.w;
    }
}

__device__ __forceinline__ double sum8(const double t[8]) {
    return ((t[0] + t[1]) + (t[2] + t[3])) + ((t[4] + t[5]) + (t[6] + t[7]));
}

// Gradients of a batch of NR unit rows (NR / 2 row pairs) of one lane.
template <int G, int NR>
struct WBatch {
    Raw8<G> r[NR / 2];
};

// Batch at unit row rb: the wave-uniform part of each address (row base) plus
// the lane's 32-bit offset lo, so the loads take the scalar-base form.
template <int G, int NR>
__device__ __forceinline__ void load_wbatch(WBatch<G, NR>& b, gp<const void> g, int64_t rb, int64_t cols, uint32_t lo) {
#pragma unroll
    for (int k = 0; k < NR / 2; ++k) {
        if constexpr (G == G_BF16) {
            const gp<const uint16_t> row = g_as<const uint16_t>(g) + (rb + 2 * k) * cols;
            b.r[k].w = ld_u4<false>(g_as<const void>(row + lo));
        } else {
            const gp<const float> row = g_as<const float>(g) + (rb + 2 * k) * cols;
            b.r[k].a = ld_f4<false>(row + lo);
            b.r[k].b = ld_f4<false>(row + lo + 4);
        }
    }
}

// Shared part of the whole-unit marginal kernels, batches of P::NR unit rows
// (4, 8 or 16). The policy P supplies the batch type, load(batch, rb) for the
// rows from rb, and terms(batch, k, t): the 8 binary64 terms of the lane's
// row 2k + h of that batch (with P::SQUARES, 8 values whose squares are the
// terms, summed by fused multiply-adds); P::DEPTH batches are in flight (2: the next
// batch's loads are issued before the current batch's arithmetic; 3: the
// next two). Row partials go to rowpart, column partials to colpart, one
// binary64 sum each (the other tensors' partials are (hi, lo) pairs); stage
// holds NR x kWStride doubles.
template <class P>
__device__ __forceinline__ void whole_unit_sums(const P& pol, const GD& d, int64_t ru, int64_t cu, double* stage) {
    // row partials are finished P::FR rows (FB batches) at a time
    constexpr int NR = P::NR, NP = NR / 2, FR = P::FR, FB = FR / NR;
    constexpr int LPR = 64 / FR, PPL = 32 / LPR;  // lanes per finished row, partials per lane
    constexpr int SZ = FR * kWStride;  // one stage buffer; finish groups alternate between two
    static_assert(NR == 4 || NR == 8 || NR == 16, "batch rows");
    static_assert(FR % NR == 0 && (FR == 4 || FR == 8 || FR == 16), "finish group rows");
    const int lane = threadIdx.x & 63, h = lane >> 5, q = lane & 31;
    const int64_t r0 = ru * 256, c0 = cu * 256, cols = d.cols;
    const int rrow = lane / LPR, rpart = lane % LPR;  // row finishing: row rrow of a group, partials PPL rpart ..
    // column sums: runs in crun added into cacc (all terms of a batch at once), else one plain sum in cacc
    double cacc[8], crun[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        cacc[j] = 0.0;
        crun[j] = 0.0;
    }
    // Row rrow of finish group gi from its staged partials PPL rpart .. PPL rpart + PPL - 1, pairwise,
    // then merged over the row's LPR lanes. Called one batch late (with the next group's first batch),
    // so the LDS round trip overlaps that batch's arithmetic.
    auto finish_rows = [&](int gi) {
        const double* st = stage + (gi & 1) * SZ + rrow * kWStride + PPL * rpart;
        double rs;
        const double2 p0 = *reinterpret_cast<const double2*>(st);
        if constexpr (PPL == 8) {
            const double2 p1 = *reinterpret_cast<const double2*>(st + 2);
            const double2 p2 = *reinterpret_cast<const double2*>(st + 4);
            const double2 p3 = *reinterpret_cast<const double2*>(st + 6);
            rs = ((p0.x + p0.y) + (p1.x + p1.y)) + ((p2.x + p2.y) + (p3.x + p3.y));
        } else if constexpr (PPL == 4) {
            const double2 p1 = *reinterpret_cast<const double2*>(st + 2);
            rs = (p0.x + p0.y) + (p1.x + p1.y);
        } else {
            rs = p0.x + p0.y;
        }
        rs += dpp_d<kDppQuadXor1>(rs);
        rs += dpp_d<kDppQuadXor2>(rs);
        if constexpr (LPR >= 8) rs += dpp_d<kDppRowHalfMirror>(rs);
        if constexpr (LPR == 16) rs += dpp_d<kDppRowMirror>(rs);
        if (rpart == 0) d.rowpart[cu * d.rows + r0 + FR * gi + rrow] = rs;
    };
    typename P::Batch A, B;
    pol.load(A, 0);
    auto step = [&](const typename P::Batch& cur, int bi) {
        double* sb = stage + ((bi / FB) & 1) * SZ + (bi % FB) * NR * kWStride;
        if constexpr (P::ILP) {
            // all terms of the batch at once (more registers, fewer waves per SIMD, more independent
            // work per wave): the batch's column terms are added first, then into the run
            double cs[8];
#pragma unroll
            for (int k = 0; k < NP; ++k) {
                double t[8];
                pol.terms(cur, k, t);
#pragma unroll
                for (int j = 0; j < 8; ++j) cs[j] = k == 0 ? t[j] : cs[j] + t[j];
                sb[(2 * k + h) * kWStride + q] = sum8(t);
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) crun[j] += cs[j];
        } else if constexpr (P::SQUARES) {
            // column sums and the lane's row partial take the squares by fused multiply-adds (one
            // rounding per term)
#pragma unroll
            for (int k = 0; k < NP; ++k) {
                double t[8];
                pol.terms(cur, k, t);
                double rs = t[0] * t[0];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    cacc[j] = __builtin_fma(t[j], t[j], cacc[j]);
                    if (j > 0) rs = __builtin_fma(t[j], t[j], rs);
                    if (k & 1) __asm__ volatile("" : "+v"(cacc[j]));
                }
                sb[(2 * k + h) * kWStride + q] = rs;
            }
        } else {
#pragma unroll
            for (int k = 0; k < NP; ++k) {
                double t[8];
                pol.terms(cur, k, t);
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    cacc[j] += t[j];
                    // two row pairs' terms live at a time: without the fence the compiler forms all terms
                    // of the batch before the column additions
                    if (k & 1) __asm__ volatile("" : "+v"(cacc[j]));
                }
                sb[(2 * k + h) * kWStride + q] = sum8(t);
            }
        }
        // the stages belong to this wavefront alone and its LDS accesses
        // execute in order: only the compiler must keep them in order
        __builtin_amdgcn_wave_barrier();
        if (bi > 0 && bi % FB == 0) finish_rows(bi / FB - 1);
        __builtin_amdgcn_wave_barrier();
        if (P::ILP && (bi + 1) % (kWRunRows / NR) == 0) {
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                cacc[j] += crun[j];
                crun[j] = 0.0;
            }
        }
    };
    // The last pair of batches is peeled: with a conditional load inside the
    // loop the compiler's wait counts would have to hold for both paths, and
    // every odd batch would wait for the next even batch's loads.
    constexpr int NB = 256 / NR;
    if constexpr (P::DEPTH == 2) {
#pragma unroll 1
        for (int bi = 0; bi < NB - 2; bi += 2) {
            pol.load(B, (bi + 1) * NR);
            step(A, bi);
            pol.load(A, (bi + 2) * NR);
            step(B, bi + 1);
        }
        pol.load(B, (NB - 1) * NR);
        step(A, NB - 2);
        step(B, NB - 1);
    } else {
        // three batches rotate, two in flight ahead of the one being formed
        static_assert(P::DEPTH == 3 && NB % 3 == 1, "three-deep rotation over NB = 1 mod 3 batches");
        typename P::Batch C;
        pol.load(B, NR);
#pragma unroll 1
        for (int bi = 0; bi < NB - 4; bi += 3) {
            pol.load(C, (bi + 2) * NR);
            step(A, bi);
            pol.load(A, (bi + 3) * NR);
            step(B, bi + 1);
            pol.load(B, (bi + 4) * NR);
            step(C, bi + 2);
        }
        pol.load(C, (NB - 2) * NR);
        step(A, NB - 4);
        pol.load(A, (NB - 1) * NR);
        step(B, NB - 3);
        step(C, NB - 2);
        step(A, NB - 1);
    }
    __builtin_amdgcn_wave_barrier();
    finish_rows(NB / FB - 1);
    // the two halves hold the even and the odd rows of the same columns
#pragma unroll
    for (int j = 0; j < 8; ++j) cacc[j] += __shfl_xor(cacc[j], 32);
    // through LDS, so that each store instruction writes 64 consecutive
    // column partials (512 bytes) instead of 8 bytes in every 64
    static_assert(2 * SZ >= 256, "the stages hold a unit's 256 column sums");
    __builtin_amdgcn_wave_barrier();
    if (h == 0) {
#pragma unroll
        for (int j = 0; j < 8; ++j) stage[8 * q + j] = cacc[j];
    }
    __builtin_amdgcn_wave_barrier();
    const gp<double> cp = d.colpart + (ru * cols + c0 + lane);
#pragma unroll
    for (int i = 0; i < 4; ++i) cp[64 * i] = stage[lane + 64 * i];
}

// The lane's place in a whole unit: the unit's first gradient element as a
// wave-uniform byte address and the lane's element offset from it.
struct WholeLane {
    int64_t r0, c0, cols;
    uint32_t lo;  // h * cols + 8 q
    int h, q;
};

__device__ __forceinline__ WholeLane whole_lane(const GD& d, int64_t u) {
    WholeLane w;
    w.h = (int)(threadIdx.x >> 5) & 1;
    w.q = (int)threadIdx.x & 31;
    w.r0 = (u / d.ncu) * 256;
    w.c0 = (u % d.ncu) * 256;
    w.cols = d.cols;
    w.lo = (uint32_t)(w.h * d.cols + 8 * w.q);
    return w;
}

template <int G>
__device__ __forceinline__ gp<const void> unit_base(const GD& d, const WholeLane& w) {
    return g_as<const void>(g_as<const uint8_t>(d.g) + (G == G_BF16 ? 2 : 4) * (w.r0 * w.cols + w.c0));
}

// Terms of the second moment's marginals: fl64(g^2 + eps1).
template <int G>
struct MargTerms {
    // 8-row batches, all terms of a batch at once: the cheap terms gain more from independent work per
    // wave than from occupancy (200 registers, 2 waves per SIMD: 2.53 against 2.68 ms on the 7B list)
    static constexpr int NR = 8;
    static constexpr int FR = NR;
    static constexpr bool ILP = true;
    static constexpr bool SQUARES = false;
    static constexpr int DEPTH = 2;
    using Batch = WBatch<G, NR>;
    gp<const void> gu;
    int64_t cols;
    uint32_t lo;
    double eps1;
    __device__ void load(Batch& b, int rb) const { load_wbatch<G, NR>(b, gu, rb, cols, lo); }
    __device__ void terms(const Batch& b, int k, double t[8]) const {
        float gv[8];
        unpack8<G>(b.r[k], gv);
#pragma unroll
        for (int j = 0; j < 8; ++j) t[j] = marg_term(gv[j], eps1);
    }
};

// One wavefront per unit, 4 per 256-thread workgroup (each with its own
// LDS stage), as in the other streaming kernels.
__device__ __forceinline__ int64_t whole_unit_of_wave(int64_t base) {
    return base + xcd_order(blockIdx.x, gridDim.x) * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
}

template <int G>
__global__ __launch_bounds__(256) void fac_marg_whole_kernel(const FacArgs a, int64_t base) {
    __shared__ __attribute__((aligned(16))) double stages[4][2 * MargTerms<G>::NR * kWStride];
    double* stage = stages[threadIdx.x >> 6];
    const int64_t unit = whole_unit_of_wave(base);
    if (unit >= a.whole_units) return;
    const GD d = gview(a.D[locate_unit(a.D, a.n2, unit)]);
    const WholeLane w = whole_lane(d, unit - d.unit_begin);
    const MargTerms<G> pol{unit_base<G>(d, w), w.cols, w.lo, a.eps1};
    whole_unit_sums(pol, d, w.r0 / 256, w.c0 / 256, stage);
}

hipError_t launch_fac_marg_g2(const FacArgs& a, int grad_dtype, hipStream_t s) {
    if (a.total_units == 0) return hipSuccess;
    hipError_t e;
    if (grad_dtype == G_BF16) {
        if ((e = launch_wave_per_unit(fac_marg_whole_kernel<G_BF16>, a, 0, a.whole_units, s)) != hipSuccess) return e;
        return launch_per_unit(fac_marg_g2_kernel<G_BF16>, a, a.whole_units, a.total_units, s);
    }
    if ((e = launch_wave_per_unit(fac_marg_whole_kernel<G_F32>, a, 0, a.whole_units, s)) != hipSuccess) return e;
    return launch_per_unit(fac_marg_g2_kernel<G_F32>, a, a.whole_units, a.total_units, s);
}

// ------------------------------------------------------------- finalize
// role 0: second moment (EMA beta, codes vr/vc, factors rfac/cfac);
// role 1: CAME confidence (EMA beta3, codes cr/cc, factors sr/sc).
// fin_block: one wavefront per code block of a factor vector (R blocks, then C
// blocks, of every 2-D tensor): merge the unit partials of each element into
// its mean, EMA with the decoded old value, round to fp32, re-encode the
// block; R blocks also leave their double-double sum for mean(R), C blocks
// their factors C_j^-1/2. fin_rows: one workgroup per tensor merges the R
// block sums in order into mean(R) and writes r_i = (R_i / mean R)^-1/2.
struct FinRole {
    int codec, B;
    void *rc, *cc;
    float *rm, *cm;
    double *fr, *fc;
    double beta, omb;
    float lf;
};

__device__ __forceinline__ FinRole fin_role(const FacArgs& a, const FacDesc& d, int role) {
    FinRole r;
    r.codec = role ? a.c_codec : a.v_codec;
    r.B = role ? a.c_block : a.v_block;
    r.rc = role ? d.cr : d.vr;
    r.rm = role ? d.crm : d.vrm;
    r.cc = role ? d.cc : d.vc;
    r.cm = role ? d.ccm : d.vcm;
    r.fr = role ? d.sr : d.rfac;
    r.fc = role ? d.sc : d.cfac;
    r.beta = role ? a.beta3 : a.beta;
    r.omb = role ? a.omb3 : a.omb;
    r.lf = role ? a.c_floor : a.v_floor;
    return r;
}

__device__ __forceinline__ int locate_blk(const FacDesc* D, int n, int64_t blk, int role) {
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (D[mid].blk_begin[role] <= blk)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// fl32(y) is the same for every binary64 y' within tol of y >= 0: y lies
// farther than tol from both fp32 rounding midpoints around fl32(y) (the
// midpoint of two adjacent fp32 values is exact in binary64).
__device__ __forceinline__ bool f32_round_robust(double y, double tol) {
    const float f = (float)y;
    const uint32_t b = f2u(f);
    if (b >= 0x7F7FFFFFu) return false;  // FLT_MAX, +inf, NaN, negative: take the exact path
    const float up = u2f(b + 1u);
    const float dn = b == 0u ? -u2f(1u) : u2f(b - 1u);
    const double mhi = 0.5 * ((double)f + (double)up), mlo = 0.5 * ((double)f + (double)dn);
    return (y - mlo > tol) & (mhi - y > tol);
}

// The decoded momentum of element e (UF8 or fp32).
__device__ __forceinline__ float came_mhat(const FacArgs& a, const GD& v, int64_t e) {
    if (a.m_codec == UF8) return uf8_decode(g_as<const int8_t>(v.m)[e], div127((double)v.mm[e / a.m_block]));
    return g_as<const float>(v.m)[e];
}

// Exact (double-double) sum of the marginal terms of row idx (isrow) or
// column idx of a 2-D tensor -- role 0: fl64(g^2 + eps1); role 1: CAME's
// residual terms -- by the whole wavefront; each term is formed exactly as the
// marginal kernels form it.
template <int G>
__device__ DD exact_line_sum(const FacArgs& a, const FacDesc& d, int role, bool isrow, int64_t idx, int lane) {
    const GD v = gview(d);
    const int64_t len = isrow ? d.cols : d.rows;
    const double clip = role ? v.scal[0] : 1.0;
    const double rclip = 1.0 / clip;
    DD acc{0.0, 0.0};
#pragma unroll 4
    for (int64_t k = lane; k < len; k += 64) {
        const int64_t i = isrow ? idx : k, j = isrow ? k : idx;
        const int64_t e = i * d.cols + j;
        float g;
        if constexpr (G == G_BF16)
            g = bf16_to_f32(g_as<const uint16_t>(v.g)[e]);
        else
            g = g_as<const float>(v.g)[e];
        double t;
        if (role == 0) {
            t = marg_term(g, a.eps1);
        } else {
            const double uu = (v.rfac[i] * v.cfac[j]) * (double)g;
            t = res_term(a, came_mhat(a, v, e), div_to_f32(uu, clip, rclip));
        }
        dd_add(acc, t);
    }
    return dd_wave_sum(acc);
}

// Relative distance from an fp32 rounding midpoint below which the EMA value
// from the fast partial sums may round differently from the one from the exact
// sum. A partial is within 131u (u = 2^-53) of its exact sum: the whole-unit
// kernels' column partials (the second moment's: plain runs of 16 binary64
// additions of non-negative terms, 8 runs added, two halves merged, 23u;
// CAME's residual: fused multiply-add sums of 128 squared differences per
// lane, two halves merged, eps2 added to the mean, 131u against the sum of
// the oracle's terms; their row partials: 16u), the other units' runs of at
// most 4 (3u) accumulated double-double; the partials are merged
// double-double, and the mean, eps2 and the EMA add at most 5u. 32u bounds
// the second moment's total (role 0), 160u CAME's confidence (role 1); an EMA
// value that close to a midpoint is about one in ten million (one in a
// million) of the elements (the exact sum of its line is then taken).
constexpr double kRobustTol[2] = {32.0 * 0x1p-53, 160.0 * 0x1p-53};

template <int G>
__global__ __launch_bounds__(256) void fac_fin_block_kernel(const FacArgs a, int role) {
    const int lane = threadIdx.x & 63;
    const int64_t blk = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (blk >= a.total_blk[role]) return;
    const FacDesc& d = a.D[locate_blk(a.D, a.n2, blk, role)];
    const FinRole R = fin_role(a, d, role);
    const int64_t lb = blk - d.blk_begin[role];
    const int64_t nbr = (d.rows + R.B - 1) / R.B;
    const bool isrow = lb < nbr;
    const int64_t n = isrow ? d.rows : d.cols;
    const int64_t b = isrow ? lb : lb - nbr;
    const int64_t s = b * R.B, e = s + R.B < n ? s + R.B : n;
    void* codes = isrow ? R.rc : R.cc;
    float* meta = isrow ? R.rm : R.cm;
    float* x = isrow ? d.rtmp : d.ctmp;
    const double cnt = (double)(isrow ? d.cols : d.rows);
    const bool whole = d.unit_begin < a.whole_units;  // the tensor's units are all whole
    // 1. EMA of the means (each lane handles the elements it encodes). The
    // marginal kernels' partials are within 3u of the exact sums; where that
    // could change the fp32 rounding of the EMA (or with exact_all), the
    // wavefront sums the element's row or column again, exactly.
    const int64_t nk = (e - s + 63) / 64;
    for (int64_t k = 0; k < nk; ++k) {
        const int64_t i = s + lane + 64 * k;
        const bool act = i < e;
        float old = 0.0f;
        double y = 0.0;
        if (act) {
            DD acc{0.0, 0.0};
            // the partials' loads do not depend on the running sum: unrolled, they are issued ahead
            // (the embedding's column blocks merge 125 row-unit partials per element)
            // whole-unit tensors' partials are single binary64 sums, the others' (hi, lo) pairs
            const int st = whole ? 1 : 2;
            if (isrow) {
#pragma unroll 8
                for (int cu = 0; cu < d.ncu; ++cu) {
                    const double* rp = d.rowpart + st * ((int64_t)cu * d.rows + i);
                    acc = dd_merge(acc, DD{rp[0], whole ? 0.0 : rp[1]});
                }
            } else {
#pragma unroll 8
                for (int ru = 0; ru < d.nru; ++ru) {
                    const double* cp = d.colpart + st * ((int64_t)ru * d.cols + i);
                    acc = dd_merge(acc, DD{cp[0], whole ? 0.0 : cp[1]});
                }
            }
            old = vec_decode(R.codec, R.B, codes, meta, i, a.cf);
            // whole-unit residual partials sum (uhat - m)^2 alone: eps2 joins the mean
            const double mean = role == 1 && whole ? dd_value(acc) / cnt + a.eps2 : dd_value(acc) / cnt;
            y = R.beta * (double)old + R.omb * mean;
        }
        const bool robust = !act || (!a.exact_all && f32_round_robust(y, kRobustTol[role] * y));
        uint64_t pend = __ballot(!robust);
        while (pend) {
            const int src = __builtin_ctzll(pend);
            pend &= pend - 1;
            const DD S = exact_line_sum<G>(a, d, role, isrow, s + src + 64 * k, lane);
            if (lane == src) y = R.beta * (double)old + R.omb * (dd_value(S) / cnt);
        }
        if (act) x[i] = (float)y;
    }
    __threadfence_block();  // the encode below reads x[] back (each lane its own elements)
    // 2. re-encode the block
    if (R.codec == FP32) {
        for (int64_t i = s + lane; i < e; i += 64) reinterpret_cast<float*>(codes)[i] = x[i];
    } else {
        uint32_t mn = 0xFFFFFFFFu, mx = 0u;
        for (int64_t i = s + lane; i < e; i += 64) {
            mn = OpMin::f(mn, pos_min_key(x[i]));
            mx = OpMax::f(mx, pos_max_key(x[i]));
        }
        mn = group_reduce<OpMin, 64>(mn);
        mx = group_reduce<OpMax, 64>(mx);
        const ALFit f = al_fit(mn, mx, R.lf);
        if (lane == 0) {
            meta[2 * b] = f.any ? (float)f.lmin : 0.0f;
            meta[2 * b + 1] = f.any ? (float)f.delta : 0.0f;
        }
        const int levels = R.codec == AL16 ? 65534 : 254;
        const ALEnc enc = al_enc_params(f.lmin, f.any ? (double)levels / f.delta : 1.0);
        for (int64_t i = s + lane; i < s + R.B; i += 64) {
            const float v = i < e ? x[i] : 0.0f;
            if (R.codec == AL16)
                reinterpret_cast<uint16_t*>(codes)[i] = (uint16_t)al_encode_fast<65534>(v, enc);
            else
                reinterpret_cast<uint8_t*>(codes)[i] = (uint8_t)al_encode_fast<254>(v, enc);
        }
    }
    // 3. R: block sum for mean(R); C: factors
    if (isrow) {
        DD acc{0.0, 0.0};
        for (int64_t i = s + lane; i < e; i += 64) dd_add(acc, (double)x[i]);
        acc = dd_wave_sum(acc);
        if (lane == 0) {
            d.rsum[2 * b] = acc.hi;
            d.rsum[2 * b + 1] = acc.lo;
        }
    } else {
        for (int64_t i = s + lane; i < e; i += 64) R.fc[i] = 1.0 / sqrt((double)x[i]);
    }
}

__global__ __launch_bounds__(256) void fac_fin_rows_kernel(const FacArgs a, int role) {
    __shared__ DD sh[4];
    const FacDesc& d = a.D[blockIdx.x];
    const FinRole R = fin_role(a, d, role);
    const int tid = threadIdx.x;
    const int64_t nbr = (d.rows + R.B - 1) / R.B;
    DD acc{0.0, 0.0};
    for (int64_t k = tid; k < nbr; k += blockDim.x) acc = dd_merge(acc, DD{d.rsum[2 * k], d.rsum[2 * k + 1]});
    acc = block_dd_sum(acc, sh);
    const double mr = dd_value(acc) / (double)d.rows;
    for (int64_t i = tid; i < d.rows; i += blockDim.x) R.fr[i] = 1.0 / sqrt((double)d.rtmp[i] / mr);
}

hipError_t launch_fac_fin(const FacArgs& a, int role, int grad_dtype, hipStream_t s) {
    if (a.n2 == 0) return hipSuccess;
    const int64_t grid = (a.total_blk[role] + 3) / 4;
    if (grad_dtype == G_BF16)
        hipLaunchKernelGGL(fac_fin_block_kernel<G_BF16>, dim3((unsigned)grid), dim3(256), 0, s, a, role);
    else
        hipLaunchKernelGGL(fac_fin_block_kernel<G_F32>, dim3((unsigned)grid), dim3(256), 0, s, a, role);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fac_fin_rows_kernel, dim3(a.n2), dim3(256), 0, s, a, role);
    return hipGetLastError();
}

// ------------------------------------------------ RMS partials (per unit)
// Natural layout: lane = 4 consecutive columns of a 256-column segment; the
// wave walks the unit's rows, kRowBatch rows at a time with all their loads
// issued before the arithmetic. u_ij = (r_i c_j) g_ij, exactly the oracle's
// operation order; u^2 summed double-double. One wave per unit.
constexpr int kRowBatch = 8;

template <int G>
__device__ __forceinline__ void load_row4(const GD& d, int64_t e, bool vec, int nc, int c, GRaw<G>& r, int k) {
    if constexpr (G == G_BF16) {
        const gp<const uint16_t> g = g_as<const uint16_t>(d.g);
        if (vec) {
            r.w[k] = ld_u2<true>(g_as<const void>(g + e));
        } else {
            uint32_t h[4] = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (c + j < nc) h[j] = g[e + j];
            r.w[k] = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
        }
    } else {
        const gp<const float> g = g_as<const float>(d.g);
        if (vec) {
            r.w[k] = ld_f4<true>(g + e);
        } else {
            float h[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (c + j < nc) h[j] = g[e + j];
            r.w[k] = make_float4(h[0], h[1], h[2], h[3]);
        }
    }
}

// Gradient words of R rows (the GRaw layout, R / 4 x 4 rows).
template <int G, int R = kRowBatch>
struct GRows {
    GRaw<G> h[R / 4];
};

// The Adafactor apply pass streams p in and out as well as g: 16-row batches
// (all loads of a batch issued before its stores, 180 registers, 2 waves per
// SIMD) run 7% faster than 8-row ones at 4-5 waves per SIMD.
constexpr int kApplyRows = 16;

// Interior units (256 x 256, width a multiple of 4) take the guard-free body.
template <int G, bool FULL>
__device__ __forceinline__ DD rms_unit(const GD& d, int64_t r0, int64_t c0, int nr_, int nc_, int lane) {
    const int nr = FULL ? 256 : nr_, nc = FULL ? 256 : nc_;
    const int c = 4 * lane;
    const bool vec = FULL || ((d.cols & 3) == 0 && c + 4 <= nc);
    const bool live = FULL || c < nc;
    double cf[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) cf[j] = (FULL || c + j < nc) ? d.cfac[c0 + c + j] : 0.0;
    DD acc{0.0, 0.0};
    for (int r = 0; r < nr; r += kRowBatch) {
        GRows<G> g;
        double ri[kRowBatch];
#pragma unroll
        for (int k = 0; k < kRowBatch; ++k) {
            const int rr = (FULL || r + k < nr) ? r + k : nr - 1;  // rows past the end repeat the last one, unused
            ri[k] = d.rfac[r0 + rr];
            if (live) load_row4<G>(d, (r0 + rr) * d.cols + c0 + c, vec, nc, c, g.h[k / 4], k % 4);
        }
#pragma unroll
        for (int k = 0; k < kRowBatch; ++k) {
            if (!FULL && (r + k >= nr || !live)) continue;
            float gv[4];
            unpack_graw<G>(g.h[k / 4], k % 4, gv);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (FULL || c + j < nc) {
                    const double uu = (ri[k] * cf[j]) * (double)gv[j];
                    dd_add(acc, uu * uu);
                }
            }
        }
    }
    return acc;
}

template <int G>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(6))) void fac_rms_kernel(const FacArgs a, int64_t base) {
    const int lane = threadIdx.x & 63;
    const int64_t unit = base + xcd_order(blockIdx.x, gridDim.x) * 4 +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (unit >= a.total_units) return;
    const GD d = gview(a.D[locate_unit(a.D, a.n2, unit)]);
    const int64_t u = unit - d.unit_begin;
    const int64_t ru = u / d.ncu, cu = u % d.ncu;
    const int64_t r0 = ru * 256, c0 = cu * 256;
    const int nr = (int)(d.rows - r0 < 256 ? d.rows - r0 : 256);
    const int nc = (int)(d.cols - c0 < 256 ? d.cols - c0 : 256);
    DD acc = (nr == 256 && nc == 256 && (d.cols & 3) == 0) ? rms_unit<G, true>(d, r0, c0, nr, nc, lane)
                                                           : rms_unit<G, false>(d, r0, c0, nr, nc, lane);
    acc = dd_wave_sum(acc);
    if (lane == 0) {
        a.rmspart[2 * unit] = acc.hi;
        a.rmspart[2 * unit + 1] = acc.lo;
    }
}


// Whole units (the marginal kernels' streaming layout): lane 32 h + q holds
// columns 8q .. 8q + 7 of rows 2k + h of each 8-row batch, 16-byte gradient
// loads, the next batch loaded before the current one's arithmetic. The 8
// terms u^2 of a lane's row are added pairwise (relative error <= 3u) and
// those sums accumulated double-double, so a unit's partial is within 3u of
// its exact sum (the other units sum term by term). The clip divisor then
// carries a relative error of at most about 2u: it scales Adafactor's update
// (inside the parameter tolerance), and for CAME it can move fl32(u / clip)
// by one fp32 ulp only where u / clip lies within that distance of an fp32
// rounding midpoint, about one element in 10^8.
template <int G>
__global__ __launch_bounds__(256) void fac_rms_whole_kernel(const FacArgs a, int64_t base) {
    const int64_t unit = whole_unit_of_wave(base);
    if (unit >= a.whole_units) return;
    const GD d = gview(a.D[locate_unit(a.D, a.n2, unit)]);
    const WholeLane w = whole_lane(d, unit - d.unit_begin);
    const gp<const void> gu = unit_base<G>(d, w);
    const int64_t cols = w.cols;
    const uint32_t lo = w.lo;
    double cf[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) cf[j] = d.cfac[w.c0 + 8 * w.q + j];
    const gp<const double> rf = d.rfac + w.r0 + w.h;  // row factor of row 2k + h of a batch: rf[rb + 2k]
    constexpr int NR = 8;
    DD acc{0.0, 0.0};
    WBatch<G, NR> A, B;
    double ra[4], rb_[4];
    load_wbatch<G, NR>(A, gu, 0, cols, lo);
#pragma unroll
    for (int k = 0; k < 4; ++k) ra[k] = rf[2 * k];
    auto step = [&](const WBatch<G, NR>& cur, const double ri[4]) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            float gv[8];
            unpack8<G>(cur.r[k], gv);
            double t[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const double uu = (ri[k] * cf[j]) * (double)gv[j];
                t[j] = uu * uu;
            }
            dd_add(acc, sum8(t));
        }
    };
    constexpr int NB = 256 / NR;
    auto load = [&](WBatch<G, NR>& b, double ri[4], int bi) {
        load_wbatch<G, NR>(b, gu, bi * NR, cols, lo);
#pragma unroll
        for (int k = 0; k < 4; ++k) ri[k] = rf[bi * NR + 2 * k];
    };
    // last pair of batches peeled (see whole_unit_sums)
#pragma unroll 1
    for (int bi = 0; bi < NB - 2; bi += 2) {
        load(B, rb_, bi + 1);
        step(A, ra);
        load(A, ra, bi + 2);
        step(B, rb_);
    }
    load(B, rb_, NB - 1);
    step(A, ra);
    step(B, rb_);
    acc = dd_wave_sum(acc);
    if ((threadIdx.x & 63) == 0) {
        a.rmspart[2 * unit] = acc.hi;
        a.rmspart[2 * unit + 1] = acc.lo;
    }
}

hipError_t launch_fac_rms(const FacArgs& a, int grad_dtype, hipStream_t s) {
    if (a.total_units == 0) return hipSuccess;
    hipError_t e;
    if (grad_dtype == G_BF16) {
        if ((e = launch_wave_per_unit(fac_rms_whole_kernel<G_BF16>, a, 0, a.whole_units, s)) != hipSuccess) return e;
        return launch_wave_per_unit(fac_rms_kernel<G_BF16>, a, a.whole_units, a.total_units, s);
    }
    if ((e = launch_wave_per_unit(fac_rms_whole_kernel<G_F32>, a, 0, a.whole_units, s)) != hipSuccess) return e;
    return launch_wave_per_unit(fac_rms_kernel<G_F32>, a, a.whole_units, a.total_units, s);
}

// ------------------------------------------------ clip divisor (wave / tensor)
__global__ __launch_bounds__(64) void fac_clip_kernel(const FacArgs a) {
    const FacDesc& d = a.D[blockIdx.x];
    const int lane = threadIdx.x;
    const int64_t nu = (int64_t)d.nru * d.ncu;
    DD s{0.0, 0.0};
    for (int64_t k = lane; k < nu; k += 64) {
        const int64_t unit = d.unit_begin + k;
        s = dd_merge(s, DD{a.rmspart[2 * unit], a.rmspart[2 * unit + 1]});
    }
    s = dd_wave_sum(s);
    if (lane == 0) {
        const double rms = sqrt(dd_value(s) / (double)(d.rows * d.cols));
        d.scal[0] = rms / a.clip_d > 1.0 ? rms / a.clip_d : 1.0;
    }
}

hipError_t launch_fac_clip(const FacArgs& a, hipStream_t s) {
    if (a.n2 == 0) return hipSuccess;
    hipLaunchKernelGGL(fac_clip_kernel, dim3(a.n2), dim3(64), 0, s, a);
    return hipGetLastError();
}

// --------------------------------------------------- Adafactor apply (2-D)
// The RMS pass's layout in kApplyRows-row batches; p <- p (1 - lr wd) - lr u / clip.
template <int G>
__global__ __launch_bounds__(256) void ada_apply_kernel(const FacArgs a, int64_t base) {
    const int lane = threadIdx.x & 63;
    const int64_t unit = base + xcd_order(blockIdx.x, gridDim.x) * 4 +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (unit >= a.total_units) return;
    const GD d = gview(a.D[locate_unit(a.D, a.n2, unit)]);
    const int64_t u = unit - d.unit_begin;
    const int64_t ru = u / d.ncu, cu = u % d.ncu;
    const int64_t r0 = ru * 256, c0 = cu * 256;
    const int nr = (int)(d.rows - r0 < 256 ? d.rows - r0 : 256);
    const int nc = (int)(d.cols - c0 < 256 ? d.cols - c0 : 256);
    const int c = 4 * lane;
    const bool vec = (d.cols & 3) == 0 && c + 4 <= nc;
    if (c >= nc) return;
    const double rclip = 1.0 / d.scal[0];
    double cf[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) cf[j] = c + j < nc ? d.cfac[c0 + c + j] : 0.0;
    for (int r = 0; r < nr; r += kApplyRows) {
        GRows<G, kApplyRows> g;
        double ri[kApplyRows];
        float4 pv[kApplyRows];
#pragma unroll
        for (int k = 0; k < kApplyRows; ++k) {
            const int rr = r + k < nr ? r + k : nr - 1;
            const int64_t e = (r0 + rr) * d.cols + c0 + c;
            ri[k] = d.rfac[r0 + rr];
            load_row4<G>(d, e, vec, nc, c, g.h[k / 4], k % 4);
            if (vec) {
                pv[k] = ld_f4<true>(d.p + e);
            } else {
                float h[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (c + j < nc) h[j] = d.p[e + j];
                pv[k] = make_float4(h[0], h[1], h[2], h[3]);
            }
        }
#pragma unroll
        for (int k = 0; k < kApplyRows; ++k) {
            if (r + k >= nr) continue;
            const int64_t e = (r0 + r + k) * d.cols + c0 + c;
            float gv[4];
            unpack_graw<G>(g.h[k / 4], k % 4, gv);
            const float pin[4] = {pv[k].x, pv[k].y, pv[k].z, pv[k].w};
            float out[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const double uu = (ri[k] * cf[j]) * (double)gv[j];
                const double pd = (double)pin[j] * a.decay;
                out[j] = (float)(pd - a.lr * (uu * rclip));  // p carries a tolerance: multiply by 1 / clip
            }
            if (vec) {
                st_f4<true>(d.p + e, make_float4(out[0], out[1], out[2], out[3]));
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (c + j < nc) d.p[e + j] = out[j];
            }
        }
    }
}

// Whole units, one wavefront per chunk of 2048 elements (32 per unit, 4 per
// 256-thread workgroup) with no loop: the grid itself streams, as in the
// AdamW step. Lanes take 4 consecutive columns of each 256-column row
// segment, so every load and store instruction covers a contiguous 1 KB of
// parameters (512 bytes of bf16 gradients); 16-byte non-temporal parameter
// accesses.
constexpr int kChunksPerUnit = 32;

template <int G>
__device__ __forceinline__ void load_g4(gp<const void> g, int64_t e, float gv[4]) {
    if constexpr (G == G_BF16) {
        const uint2 w = ld_u2<true>(g_as<const void>(g_as<const uint16_t>(g) + e));
        gv[0] = u2f(w.x << 16), gv[1] = u2f(w.x & 0xFFFF0000u), gv[2] = u2f(w.y << 16), gv[3] = u2f(w.y & 0xFFFF0000u);
    } else {
        const float4 w = ld_f4<true>(g_as<const float>(g) + e);
        gv[0] = w.x, gv[1] = w.y, gv[2] = w.z, gv[3] = w.w;
    }
}

// A whole-unit chunk as rows and columns: 8 / W rows from row0, 256 W
// columns from col0 (W units side by side; the unit columns left over in a
// unit row, ncu mod W, take W = 1: 8 rows x 256). A unit row holds 32 ncu
// chunks.
struct RowChunk {
    int64_t row0, col0;
    bool full;  // W units (else one)
};

template <int W>
__device__ __forceinline__ RowChunk row_chunk(const GD& d, int64_t chunk) {
    const int64_t t_ch = chunk - d.unit_begin * kChunksPerUnit;
    const int64_t cpr = (int64_t)d.ncu * kChunksPerUnit;  // chunks per unit row
    const int64_t ur = t_ch / cpr, r = t_ch - ur * cpr;
    const int64_t ng = d.ncu / W;             // groups of W units in a unit row
    RowChunk c;
    c.full = r < ng * W * kChunksPerUnit;
    if (c.full) {
        const int64_t grp = r / (W * kChunksPerUnit), ci = r - grp * (W * kChunksPerUnit);
        c.row0 = ur * 256 + ci * (8 / W);
        c.col0 = grp * (256 * W);
    } else {
        const int64_t x = r - ng * W * kChunksPerUnit;
        c.row0 = ur * 256 + (x % kChunksPerUnit) * 8;
        c.col0 = (ng * W + x / kChunksPerUnit) * 256;
    }
    return c;
}

// Adafactor apply over a row chunk (lane l: columns 4l .. 4l + 3 of each
// 256-column segment): every load of the chunk is issued before the
// arithmetic.
template <int G, int W>
__device__ __forceinline__ void ada_apply_rows(const FacArgs& a, const GD& d, int64_t row0, int64_t col0) {
    constexpr int R = 8 / W;
    const int64_t cb = col0 + 4 * (threadIdx.x & 63);
    const double rclip = 1.0 / d.scal[0], lr = a.lr, decay = a.decay;
    float gv[R][W][4];
    float4 pv[R][W];
    double ri[R], cf[W][4];
#pragma unroll
    for (int k = 0; k < R; ++k) {
        ri[k] = d.rfac[row0 + k];
#pragma unroll
        for (int sg = 0; sg < W; ++sg) {
            const int64_t e = (row0 + k) * d.cols + cb + 256 * sg;
            load_g4<G>(d.g, e, gv[k][sg]);
            pv[k][sg] = ld_f4<true>(d.p + e);
        }
    }
#pragma unroll
    for (int sg = 0; sg < W; ++sg)
#pragma unroll
        for (int j = 0; j < 4; ++j) cf[sg][j] = d.cfac[cb + 256 * sg + j];
#pragma unroll
    for (int k = 0; k < R; ++k) {
#pragma unroll
        for (int sg = 0; sg < W; ++sg) {
            const float pin[4] = {pv[k][sg].x, pv[k][sg].y, pv[k][sg].z, pv[k][sg].w};
            float out[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const double uu = (ri[k] * cf[sg][j]) * (double)gv[k][sg][j];
                const double pd = (double)pin[j] * decay;
                out[j] = (float)(pd - lr * (uu * rclip));  // p carries a tolerance: multiply by 1 / clip
            }
            st_f4<true>(d.p + (row0 + k) * d.cols + cb + 256 * sg, make_float4(out[0], out[1], out[2], out[3]));
        }
    }
}

constexpr int kAdaApplyW = 2;

template <int G>
__global__ __launch_bounds__(256) void ada_apply_whole_kernel(const FacArgs a, int64_t base) {
    const int64_t chunk = base + xcd_order(blockIdx.x, gridDim.x) * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t unit = chunk / kChunksPerUnit;
    if (unit >= a.whole_units) return;
    const GD d = gview(a.D[locate_unit(a.D, a.n2, unit)]);
    const RowChunk c = row_chunk<kAdaApplyW>(d, chunk);
    if (c.full)
        ada_apply_rows<G, kAdaApplyW>(a, d, c.row0, c.col0);
    else
        ada_apply_rows<G, 1>(a, d, c.row0, c.col0);
}

// One wavefront per whole-unit chunk, 4 per 256-thread workgroup; grids
// beyond 2^31 workgroups take several launches.
template <class K>
static hipError_t launch_per_chunk(K kernel, const FacArgs& a, hipStream_t s) {
    constexpr int64_t kMaxGrid = int64_t(1) << 31;
    const int64_t end = a.whole_units * kChunksPerUnit;
    for (int64_t base = 0; base < end; base += 4 * kMaxGrid) {
        const int64_t left = (end - base + 3) / 4;
        const int64_t grid = left < kMaxGrid ? left : kMaxGrid;
        hipLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(256), 0, s, a, base);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_ada_apply(const FacArgs& a, int grad_dtype, hipStream_t s) {
    if (a.total_units == 0) return hipSuccess;
    hipError_t e;
    if (grad_dtype == G_BF16) {
        if ((e = launch_per_chunk(ada_apply_whole_kernel<G_BF16>, a, s)) != hipSuccess) return e;
        return launch_wave_per_unit(ada_apply_kernel<G_BF16>, a, a.whole_units, a.total_units, s);
    }
    if ((e = launch_per_chunk(ada_apply_whole_kernel<G_F32>, a, s)) != hipSuccess) return e;
    return launch_wave_per_unit(ada_apply_kernel<G_F32>, a, a.whole_units, a.total_units, s);
}

// ------------------------------------------- Adafactor 1-D tensors (WG each)
template <int G>
__global__ __launch_bounds__(256) void ada_vec1d_kernel(const FacArgs a) {
    __shared__ DD sh[4];
    __shared__ double clip_s;
    const FacDesc& d = a.D[a.n2 + blockIdx.x];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t n = d.rows * d.cols;
    for (int64_t i = tid; i < n; i += blockDim.x) {
        const double gi = (double)grad1<G>(d.g, i);
        const float old = vec_decode(a.v_codec, a.v_block, d.v, d.vm, i, a.cf);
        d.rtmp[i] = (float)(a.beta * (double)old + a.omb * (gi * gi + a.eps1));
    }
    __syncthreads();
    vec_encode(a.v_codec, a.v_block, d.rtmp, n, a.v_floor, d.v, d.vm, wave, 4, lane);
    DD s{0.0, 0.0};
    for (int64_t i = tid; i < n; i += blockDim.x) {
        const double uu = (1.0 / sqrt((double)d.rtmp[i])) * (double)grad1<G>(d.g, i);
        dd_add(s, uu * uu);
    }
    s = block_dd_sum(s, sh);
    if (tid == 0) {
        const double rms = sqrt(dd_value(s) / (double)n);
        clip_s = rms / a.clip_d > 1.0 ? rms / a.clip_d : 1.0;
    }
    __syncthreads();
    const double clip = clip_s;
    for (int64_t i = tid; i < n; i += blockDim.x) {
        const double uu = (1.0 / sqrt((double)d.rtmp[i])) * (double)grad1<G>(d.g, i);
        const double pd = (double)d.p[i] * a.decay;
        d.p[i] = (float)(pd - a.lr * (uu / clip));
    }
}

hipError_t launch_ada_vec1d(const FacArgs& a, int grad_dtype, hipStream_t s) {
    if (a.n1 == 0) return hipSuccess;
    if (grad_dtype == G_BF16)
        hipLaunchKernelGGL(ada_vec1d_kernel<G_BF16>, dim3(a.n1), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(ada_vec1d_kernel<G_F32>, dim3(a.n1), dim3(256), 0, s, a);
    return hipGetLastError();
}

// ---------------------------------------------------------- CAME momentum
// In-step momentum of element e of tensor d from its uhat (binary64 EMA,
// rounded to fp32): m = fl32(beta1 * mhat + (1 - beta1) * uhat).
__device__ __forceinline__ float came_momentum(const FacArgs& a, const FacDesc& d, int64_t e, float uh) {
    float mh;
    if (a.m_codec == UF8) {
        const int32_t q = reinterpret_cast<const int8_t*>(d.m)[e];
        mh = uf8_decode(q, div127((double)d.mm[e / a.m_block]));
    } else {
        mh = reinterpret_cast<const float*>(d.m)[e];
    }
    return (float)(a.beta1 * (double)mh + a.omb1 * (double)uh);
}

// --------------------------- CAME residual marginal sums (tile layout, fp64)
// Term (uhat - m)^2 + eps2 with uhat = fl32(u / clip), m the in-step
// momentum; the loop order and one-tile-ahead loads of the marginals of G2,
// on 8x128 tiles: lane (lr, lc) = (lane / 32, lane % 32) holds rows lr + 2i
// (i < 4), columns 4 lc .. 4 lc + 3, so each row's 128 momentum codes are one
// full 128-byte line; the binary64 terms are staged in LDS and 8 lanes sum
// each tile row (16 columns each, merged with DPP).
constexpr int kResRows = 8, kResCols = 128;

template <int G>
struct ResRaw {
    GRaw<G> g;
    uint32_t mw[4];  // UF8 codes of the 4 columns (fp32 momentum: read directly)
    double ri[4];
    float ms[4];
};

template <int G, bool FULL, bool UF>
__device__ __forceinline__ void load_resraw(ResRaw<G>& r, const FacArgs& a, const GD& d, int64_t r0,
                                            int64_t c0, int nr, int nc, int rg, int ct, int lr, int lc, bool vec,
                                            int64_t lane_off) {
    load_graw<G, FULL, kResCols>(r.g, d, r0, c0, nr, nc, rg, ct, lr, lc, vec, lane_off);
    const int cc = ct * kResCols + 4 * lc;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int rr = rg * kResRows + lr + 2 * i;
        const int64_t e = (r0 + rg * kResRows + 2 * i) * d.cols + c0 + ct * kResCols + lane_off;
        r.ri[i] = (FULL || rr < nr) ? d.rfac[r0 + rr] : 0.0;
        r.mw[i] = 0u;
        r.ms[i] = 0.0f;
        if (UF && (FULL || rr < nr)) {
            if (FULL || (vec && cc + 4 <= nc)) {
                // e % 4 == 0: the 4 codes are one word of one momentum block
                r.mw[i] = *g_as<const uint32_t>(g_as<const uint8_t>(d.m) + e);
                r.ms[i] = d.mm[(uint64_t)e >> 8];
            }
        }
    }
}

template <int G, bool FULL, bool UF>
__device__ __forceinline__ void res_unit(const FacArgs& a, const GD& d, double clip, int64_t ru, int64_t cu, int nr_,
                                         int nc_, bool vec_, double (*tile)[kResCols + 2], DD* racc) {
    const int lane = threadIdx.x, lc = lane & 31, lr = lane >> 5, rrow = lane >> 3, re = lane & 7;
    const int64_t r0 = ru * 256, c0 = cu * 256;
    const int nr = FULL ? 256 : nr_, nc = FULL ? 256 : nc_;
    const bool vec = FULL || vec_;
    const double rclip = 1.0 / clip;
    constexpr bool uf8 = UF;
    const int nrg = (nr + kResRows - 1) / kResRows, nct = (nc + kResCols - 1) / kResCols, total = nrg * nct;
#pragma unroll
    for (int k = 0; k < 4; ++k) racc[lane + 64 * k] = DD{0.0, 0.0};
    DD cacc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) cacc[j] = DD{0.0, 0.0};
    double cf[4] = {0.0, 0.0, 0.0, 0.0};
    ResRaw<G> cur;
    const int64_t lane_off = (int64_t)lr * d.cols + 4 * lc;
    load_resraw<G, FULL, UF>(cur, a, d, r0, c0, nr, nc, 0, 0, lr, lc, vec, lane_off);
    for (int it = 0; it < total; ++it) {
        const int ct = it / nrg, rg = it - ct * nrg;
        const int cc = ct * kResCols + 4 * lc;
        if (rg == 0) {
#pragma unroll
            for (int j = 0; j < 4; ++j) cf[j] = (FULL || cc + j < nc) ? d.cfac[c0 + cc + j] : 0.0;
        }
        ResRaw<G> nxt = cur;
        if (it + 1 < total) {
            const int ct1 = (it + 1) / nrg;
            load_resraw<G, FULL, UF>(nxt, a, d, r0, c0, nr, nc, it + 1 - ct1 * nrg, ct1, lr, lc, vec, lane_off);
        }
        double gs[4] = {0.0, 0.0, 0.0, 0.0};  // the lane's 4 rows of each column, summed in row order
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int rr = rg * kResRows + lr + 2 * i;
            double term[4] = {0.0, 0.0, 0.0, 0.0};
            if (FULL || rr < nr) {
                const int64_t e = (r0 + rg * kResRows + 2 * i) * d.cols + c0 + ct * kResCols + lane_off;
                float gv[4], mh[4] = {0.0f, 0.0f, 0.0f, 0.0f};
                unpack_graw<G>(cur.g, i, gv);
                if (FULL || (vec && cc + 4 <= nc)) {
                    if constexpr (uf8) {
                        const double st = div127((double)cur.ms[i]);
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            mh[j] = uf8_decode((int32_t)(int8_t)(uint8_t)(cur.mw[i] >> (8 * j)), st);
                    } else {
                        const float4 t = ld_f4<false>(g_as<const float>(d.m) + e);
                        mh[0] = t.x;
                        mh[1] = t.y;
                        mh[2] = t.z;
                        mh[3] = t.w;
                    }
                } else {
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        if (cc + j < nc) {
                            if constexpr (uf8)
                                mh[j] = uf8_decode(g_as<const int8_t>(d.m)[e + j],
                                                   div127((double)d.mm[(e + j) / 256]));
                            else
                                mh[j] = g_as<const float>(d.m)[e + j];
                        }
                    }
                }
                double uu[4];
                float uh[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) uu[j] = (cur.ri[i] * cf[j]) * (double)gv[j];
                div4_to_f32(uu, clip, rclip, uh);
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (FULL || cc + j < nc) term[j] = res_term(a, mh[j], uh[j]);
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) gs[j] += term[j];
            double* tp = &tile[lr + 2 * i][4 * lc];
            *reinterpret_cast<double2*>(tp) = make_double2(term[0], term[1]);
            *reinterpret_cast<double2*>(tp + 2) = make_double2(term[2], term[3]);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) dd_add(cacc[j], gs[j]);
        __syncthreads();
        DD rsum{0.0, 0.0};
        const int rr = rg * kResRows + rrow;
        const int cq = ct * kResCols + 16 * re;  // first column of this lane's sixteenth
        if (FULL || (rr < nr && cq < nc)) {
            const int cnt = nc - cq < 16 ? nc - cq : 16;
            if (FULL || cnt == 16) {
#pragma unroll
                for (int c = 0; c < 16; c += 4) {
                    const double2 t0 = *reinterpret_cast<const double2*>(&tile[rrow][16 * re + c]);
                    const double2 t1 = *reinterpret_cast<const double2*>(&tile[rrow][16 * re + c + 2]);
                    dd_add(rsum, ((t0.x + t0.y) + t1.x) + t1.y);
                }
            } else {
                for (int c = 0; c < cnt; ++c) dd_add(rsum, tile[rrow][16 * re + c]);
            }
        }
        rsum = dd_merge(rsum, dd_quad_xor<kDppQuadXor1>(rsum));
        rsum = dd_merge(rsum, dd_quad_xor<kDppQuadXor2>(rsum));
        rsum = dd_merge(rsum, dd_quad_xor<kDppRowHalfMirror>(rsum));  // the other quad of the 8 lanes
        if (re == 0 && (FULL || rr < nr)) racc[rr] = dd_merge(racc[rr], rsum);
        __syncthreads();
        if (rg == nrg - 1) {
            // column tile done: merge the two lanes of each column
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                DD v = cacc[j];
                v = dd_merge(v, dd_shfl_xor(v, 32));
                const int col = cc + j;
                if (lr == 0 && (FULL || col < nc)) {
                    const gp<double> cp = d.colpart + 2 * (ru * d.cols + c0 + col);
                    cp[0] = v.hi;
                    cp[1] = v.lo;
                }
                cacc[j] = DD{0.0, 0.0};
            }
        }
        cur = nxt;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int row = lane + 64 * k;
        if (FULL || row < nr) {
            const gp<double> rp = d.rowpart + 2 * (cu * d.rows + r0 + row);
            rp[0] = racc[row].hi;
            rp[1] = racc[row].lo;
        }
    }
}

// UF: UF8 momentum codes (else fp32 momentum).
template <int G, bool UF>
__global__ __launch_bounds__(64) void came_res_kernel(const FacArgs a, int64_t base) {
    __shared__ __attribute__((aligned(16))) double tile[kResRows][kResCols + 2];
    __shared__ DD racc[256];
    const int64_t unit = base + xcd_order(blockIdx.x, gridDim.x);
    if (unit >= a.total_units) return;
    const FacDesc& d = a.D[locate_unit(a.D, a.n2, unit)];
    const int64_t u = unit - d.unit_begin;
    const int64_t ru = u / d.ncu, cu = u % d.ncu;
    const int nr = (int)(d.rows - ru * 256 < 256 ? d.rows - ru * 256 : 256);
    const int nc = (int)(d.cols - cu * 256 < 256 ? d.cols - cu * 256 : 256);
    const bool vec = (d.cols & 3) == 0;
    if (nr == 256 && nc == 256 && vec)
        res_unit<G, true, UF>(a, gview(d), d.scal[0], ru, cu, nr, nc, vec, tile, racc);
    else
        res_unit<G, false, UF>(a, gview(d), d.scal[0], ru, cu, nr, nc, vec, tile, racc);
}

// Whole units: the marginal kernels' streaming layout (whole_unit_sums) with
// CAME's residual terms. Each unit row is one 256-element momentum block
// (the width is a multiple of 256), so a row's codes share one scale; the
// lane's 8 momentum values of a row are one 8-byte word of codes (or two
// 16-byte fp32 loads), loaded with the gradients one batch ahead.
constexpr int kResNR = 4;  // unit rows per batch of the residual kernel (its terms need more registers)
template <int G, bool UF>
struct ResBatch;
template <int G>
struct ResBatch<G, true> {
    WBatch<G, kResNR> g;
    uint2 mc[kResNR / 2];  // 8 UF8 codes of the lane's row in each row pair
    float ms[kResNR / 2];  // their block's absmax
    double ri[kResNR / 2];
};
template <int G>
struct ResBatch<G, false> {
    WBatch<G, kResNR> g;
    float4 ma[kResNR / 2], mb[kResNR / 2];  // fp32 momentum
    double ri[kResNR / 2];
};

template <int G, bool UF>
struct ResTerms {
    static constexpr int NR = kResNR;
    static constexpr int FR = 16;  // row partials finished 16 rows at a time (4 batches)
    static constexpr bool ILP = false;  // the residual terms need the registers for occupancy
    // terms() gives uhat - m; the sums take its square (eps2 is added to the means in the finalize)
    static constexpr bool SQUARES = true;
    // the registers the single column sum frees (against runs) hold a third batch: 3 waves per SIMD either way
    static constexpr int DEPTH = 3;
    using Batch = ResBatch<G, UF>;
    const FacArgs* a;
    gp<const void> gu;   // the unit's first gradient
    gp<const void> mu;   // the unit's first momentum element (codes or fp32)
    gp<const float> msu;  // absmax of the unit's first row's block (UF8)
    gp<const double> rf;  // row factor of the lane's first row
    int64_t cols, hcols;  // hcols = h * cols: the lane's row within a pair
    uint32_t lo;
    double cf[8];
    double cfmin;  // the smallest of the lane's column factors
    double clip, rclip;
    __device__ void load(Batch& b, int rb) const {
        load_wbatch<G, NR>(b.g, gu, rb, cols, lo);
#pragma unroll
        for (int k = 0; k < NR / 2; ++k) {
            const int64_t off = (int64_t)(rb + 2 * k) * cols;  // row rb + 2k + h, with lo
            b.ri[k] = rf[rb + 2 * k];
            if constexpr (UF) {
                b.mc[k] = ld_u2<false>(g_as<const void>(g_as<const uint8_t>(mu) + off + lo));
                b.ms[k] = msu[(off + hcols) >> 8];  // the row's momentum block
            } else {
                const gp<const float> m = g_as<const float>(mu) + off + lo;
                b.ma[k] = ld_f4<false>(m);
                b.mb[k] = ld_f4<false>(m + 4);
            }
        }
    }
    __device__ void terms(const Batch& b, int k, double t[8]) const {
        float gv[8], mh[8], uh[8];
        unpack8<G>(b.g.r[k], gv);
        if constexpr (UF) {
            const double st = div127((double)b.ms[k]);
            const uint32_t w[2] = {b.mc[k].x, b.mc[k].y};
#pragma unroll
            for (int j = 0; j < 8; ++j) mh[j] = uf8_decode((int32_t)(int8_t)(uint8_t)(w[j >> 2] >> (8 * (j & 3))), st);
        } else {
            mh[0] = b.ma[k].x, mh[1] = b.ma[k].y, mh[2] = b.ma[k].z, mh[3] = b.ma[k].w;
            mh[4] = b.mb[k].x, mh[5] = b.mb[k].y, mh[6] = b.mb[k].z, mh[7] = b.mb[k].w;
        }
        // uhat = fl32(u / clip), u = fl64(fl64(r c) g): from the quotient with 1 / clip folded into the
        // row factor (two multiplications), the exact division where its rounding is not decided
        const double rk = b.ri[k] * rclip;
        double qv[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) qv[j] = (rk * cf[j]) * (double)gv[j];
        // A nonzero bf16 gradient has |g| >= 2^-133, so when rk * min_j c_j >= 2^7 (1 + 2^-18) on every
        // lane each q_j is zero or above 2^-126 (1 + 2^-19) (three roundings of at most u each): only the
        // midpoint test remains. The condition is taken wave-wide, so the branch is uniform.
        bool ok;
        if (G == G_BF16 && __builtin_expect(__all(rk * cfmin >= 0x1.00004p7), 1))
            ok = f32_midpoints_decided<8>(qv, uh);
        else
            ok = f32_roundings_decided<8>(qv, uh);
        if (__builtin_expect(!ok, 0)) {
#pragma unroll
            for (int j = 0; j < 8; ++j) uh[j] = (float)(((b.ri[k] * cf[j]) * (double)gv[j]) / clip);
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) t[j] = res_diff(*a, mh[j], uh[j]);
    }
};

template <int G, bool UF>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3))) void came_res_whole_kernel(const FacArgs a, int64_t base) {
    __shared__ __attribute__((aligned(16))) double stages[4][2 * ResTerms<G, UF>::FR * kWStride];
    double* stage = stages[threadIdx.x >> 6];
    const int64_t unit = whole_unit_of_wave(base);
    if (unit >= a.whole_units) return;
    const GD d = gview(a.D[locate_unit(a.D, a.n2, unit)]);
    const WholeLane w = whole_lane(d, unit - d.unit_begin);
    ResTerms<G, UF> pol;
    pol.a = &a;
    pol.gu = unit_base<G>(d, w);
    const int64_t e0 = w.r0 * w.cols + w.c0;
    pol.mu = UF ? g_as<const void>(g_as<const uint8_t>(d.m) + e0) : g_as<const void>(g_as<const float>(d.m) + e0);
    pol.msu = d.mm + (e0 >> 8);
    pol.rf = d.rfac + w.r0 + w.h;
    pol.cols = w.cols;
    pol.hcols = w.h * w.cols;
    pol.lo = w.lo;
#pragma unroll
    for (int j = 0; j < 8; ++j) pol.cf[j] = d.cfac[w.c0 + 8 * w.q + j];
    pol.cfmin = pol.cf[0];
#pragma unroll
    for (int j = 1; j < 8; ++j) pol.cfmin = pol.cf[j] < pol.cfmin ? pol.cf[j] : pol.cfmin;
    pol.clip = d.scal[0];
    pol.rclip = 1.0 / pol.clip;
    whole_unit_sums(pol, d, w.r0 / 256, w.c0 / 256, stage);
}

hipError_t launch_came_res(const FacArgs& a, int grad_dtype, hipStream_t s) {
    if (a.total_units == 0) return hipSuccess;
    const bool uf = a.m_codec == UF8;
    hipError_t e;
    if (grad_dtype == G_BF16) {
        if ((e = uf ? launch_wave_per_unit(came_res_whole_kernel<G_BF16, true>, a, 0, a.whole_units, s)
                    : launch_wave_per_unit(came_res_whole_kernel<G_BF16, false>, a, 0, a.whole_units, s)) != hipSuccess)
            return e;
        return uf ? launch_per_unit(came_res_kernel<G_BF16, true>, a, a.whole_units, a.total_units, s)
                  : launch_per_unit(came_res_kernel<G_BF16, false>, a, a.whole_units, a.total_units, s);
    }
    if ((e = uf ? launch_wave_per_unit(came_res_whole_kernel<G_F32, true>, a, 0, a.whole_units, s)
                : launch_wave_per_unit(came_res_whole_kernel<G_F32, false>, a, 0, a.whole_units, s)) != hipSuccess)
        return e;
    return uf ? launch_per_unit(came_res_kernel<G_F32, true>, a, a.whole_units, a.total_units, s)
              : launch_per_unit(came_res_kernel<G_F32, false>, a, a.whole_units, a.total_units, s);
}

// ------------------------------------------------------ CAME apply (2-D)
// Recompute uhat and m, encode m, and p <- p (1 - lr wd) - lr (s_i s_j) m.
// Widths that are a multiple of 256: one wave per unit in the RMS pass's
// layout, so each unit row is exactly one 256-element momentum block (one
// wave-wide absmax per row); rows in batches with their loads issued first.
template <int G, bool UF>
__global__ __launch_bounds__(256) void came_apply_unit_kernel(const FacArgs a, int64_t base) {
    const int lane = threadIdx.x & 63;
    const int64_t unit = base + xcd_order(blockIdx.x, gridDim.x) * 4 +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (unit >= a.total_units) return;
    const GD d = gview(a.D[locate_unit(a.D, a.n2, unit)]);
    if (d.cols & 255) return;  // other widths: the chunk kernel
    const int64_t u = unit - d.unit_begin;
    const int64_t ru = u / d.ncu, cu = u % d.ncu;
    const int64_t r0 = ru * 256, c0 = cu * 256;
    const int nr = (int)(d.rows - r0 < 256 ? d.rows - r0 : 256);
    const int c = 4 * lane;
    const double clip = d.scal[0], rclip = 1.0 / clip;
    constexpr bool uf8 = UF;
    double cf[4], sf[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        cf[j] = d.cfac[c0 + c + j];
        sf[j] = d.sc[c0 + c + j];
    }
    constexpr int RB = 8;  // rows per batch: 165 registers, 3 waves per SIMD (4% faster than 4 rows; 16 slower)
    for (int r = 0; r < nr; r += RB) {
        GRows<G, RB> g;
        float4 pv[RB];
        uint32_t mw[UF ? RB : 1];
        float4 mf[UF ? 1 : RB];
        double ri[RB], si[RB];
        float ms[RB];
#pragma unroll
        for (int k = 0; k < RB; ++k) {
            const int rr = r + k < nr ? r + k : nr - 1;  // rows past the end repeat the last one, unused
            const int64_t e = (r0 + rr) * d.cols + c0 + c;
            ri[k] = d.rfac[r0 + rr];
            si[k] = d.sr[r0 + rr];
            load_row4<G>(d, e, true, 256, c, g.h[k / 4], k % 4);
            pv[k] = ld_f4<true>(d.p + e);
            if constexpr (uf8) {
                mw[k] = ld_u1<true>(g_as<const void>(g_as<const uint8_t>(d.m) + e));
                ms[k] = d.mm[(e - c) / 256];
            } else {
                mf[k] = ld_f4<true>(g_as<const float>(d.m) + e);
            }
        }
#pragma unroll
        for (int k = 0; k < RB; ++k) {
            if (r + k >= nr) break;
            const int64_t e = (r0 + r + k) * d.cols + c0 + c;
            float gv[4], mh[4];
            unpack_graw<G>(g.h[k / 4], k % 4, gv);
            if constexpr (uf8) {
                const double st = div127((double)ms[k]);
#pragma unroll
                for (int j = 0; j < 4; ++j) mh[j] = uf8_decode((int32_t)(int8_t)(uint8_t)(mw[k] >> (8 * j)), st);
            } else {
                mh[0] = mf[k].x;
                mh[1] = mf[k].y;
                mh[2] = mf[k].z;
                mh[3] = mf[k].w;
            }
            const float pin[4] = {pv[k].x, pv[k].y, pv[k].z, pv[k].w};
            float mnew[4], pout[4], uh[4];
            double uu[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) uu[j] = (ri[k] * cf[j]) * (double)gv[j];
            div4_to_f32(uu, clip, rclip, uh);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                mnew[j] = (float)(a.beta1 * (double)mh[j] + a.omb1 * (double)uh[j]);
                const double upd = (si[k] * sf[j]) * (double)mnew[j];
                pout[j] = (float)((double)pin[j] * a.decay - a.lr * upd);
            }
            st_f4<true>(d.p + e, make_float4(pout[0], pout[1], pout[2], pout[3]));
            if constexpr (uf8) {
                uint32_t am = 0u;
#pragma unroll
                for (int j = 0; j < 4; ++j) am = OpMax::f(am, abs_bits(mnew[j]));
                am = group_reduce<OpMax, 64>(am);
                const double rs = am != 0u ? rdiv127((double)u2f(am)) : 0.0;
                uint32_t q[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) q[j] = rint_low_bits((double)mnew[j] * rs) & 0xFFu;
                const uint32_t w = (q[0] & 0xFFu) | ((q[1] & 0xFFu) << 8) | ((q[2] & 0xFFu) << 16) | (q[3] << 24);
                st_u1<true>(g_as<void>(g_as<uint8_t>(d.m) + e), w);
                if (lane == 0) d.mm[(e - c) / 256] = u2f(am);
            } else {
                st_f4<true>(g_as<float>(d.m) + e, make_float4(mnew[0], mnew[1], mnew[2], mnew[3]));
            }
        }
    }
}

// Other widths: flattened 1024-element chunks, 4 sub-tiles of 256 per wave,
// so each momentum block (256) is one sub-tile; element by element.
template <int G>
__global__ __launch_bounds__(256) void came_apply_chunk_kernel(const FacArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t wave = xcd_order(blockIdx.x, gridDim.x) * 4 + (threadIdx.x >> 6);
    const int64_t nw = (int64_t)gridDim.x * 4;
    for (int64_t chunk = wave; chunk < a.total_chunks; chunk += nw) {
        const FacDesc& d = a.D[locate_chunk(a.D, a.n2, chunk)];
        const int64_t n = d.rows * d.cols;
        const int64_t e0 = (chunk - d.chunk_begin) * 1024;
        const double clip = d.scal[0], rclip = 1.0 / clip;
        for (int k = 0; k < 4; ++k) {
            const int64_t sb = e0 + 256 * k;
            if (sb >= n) break;
            const int64_t eb = sb + 4 * lane;
            // row / column of the lane's first element (binary64 estimate, then exact correction)
            int64_t i = (int64_t)((double)eb / (double)d.cols);
            int64_t jc = eb - i * d.cols;
            while (jc < 0) {
                --i;
                jc += d.cols;
            }
            while (jc >= d.cols) {
                ++i;
                jc -= d.cols;
            }
            float mnew[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t e = eb + j;
                if (e < n) {
                    const double uu = (d.rfac[i] * d.cfac[jc]) * (double)grad1<G>(d.g, e);
                    const float uh = div_to_f32(uu, clip, rclip);
                    const float m = came_momentum(a, d, e, uh);
                    mnew[j] = m;
                    const double upd = (d.sr[i] * d.sc[jc]) * (double)m;
                    const double pd = (double)d.p[e] * a.decay;
                    d.p[e] = (float)(pd - a.lr * upd);
                }
                if (++jc == d.cols) {
                    jc = 0;
                    ++i;
                }
            }
            if (a.m_codec == UF8) {
                uint32_t am = 0u;
#pragma unroll
                for (int j = 0; j < 4; ++j) am = OpMax::f(am, abs_bits(mnew[j]));
                am = group_reduce<OpMax, 64>(am);
                const double r = am != 0u ? rdiv127((double)u2f(am)) : 0.0;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int32_t q = (int32_t)__builtin_rint((double)mnew[j] * r);
                    reinterpret_cast<int8_t*>(d.m)[eb + j] = (int8_t)q;  // padded to whole blocks
                }
                if (lane == 0) d.mm[sb / 256] = u2f(am);
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (eb + j < n) reinterpret_cast<float*>(d.m)[eb + j] = mnew[j];
            }
        }
    }
}

// Whole units: a wavefront takes a chunk of 8 / W rows x 256 W columns, W
// units side by side (lane l: columns 4l .. 4l + 3 of each 256-column
// segment), one row at a time: each row is one contiguous segment of 256 W
// elements. A unit row holds 32 chunks' worth of the unit columns; the unit
// columns left over in a row (ncu mod W) take W = 1 (8 rows x 256). Each
// 256-column segment of a row is one momentum block over all 64 lanes.
// W = 2 (2 KB parameter segments, 88 registers) measured 1.8% faster than
// 8 rows x 256 columns in two 32-lane halves; W = 1 and 4 no faster, W = 8
// (232 registers) 21% slower.
constexpr int kCameApplyW = 2;
template <int G, bool UF, int W>
__device__ __forceinline__ void came_apply_rows(const FacArgs& a, const GD& d, int64_t row0, int64_t col0) {
    constexpr int R = 8 / W;
    const int lane = threadIdx.x & 63;
    const int64_t cb = col0 + 4 * lane;
    const int64_t cols = d.cols;
    const double clip = d.scal[0], rclip = 1.0 / clip;
    const gp<uint8_t> mc = g_as<uint8_t>(d.m);
    const gp<float> mf = g_as<float>(d.m);
    // The parameter update runs in fp32 (the states never depend on p, which is held to a relative
    // tolerance): p' = fma(-lr, (s_i s_j) m, p (1 - lr wd)) on the fp32 roundings of the factors.
    const float lrf = (float)a.lr, decayf = (float)a.decay;
    double cf[W][4];
    float sf[W][4];
#pragma unroll
    for (int sg = 0; sg < W; ++sg)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            cf[sg][j] = d.cfac[cb + 256 * sg + j];
            sf[sg][j] = (float)d.sc[cb + 256 * sg + j];
        }
#pragma unroll 1
    for (int k = 0; k < R; ++k) {
        const int64_t row = row0 + k;
        const double ri = d.rfac[row], rk = ri * rclip;
        const float si = (float)d.sr[row];
        float gv[W][4], ms[W];
        float4 pv[W], mv[UF ? 1 : W];
        uint32_t mw[W];
#pragma unroll
        for (int sg = 0; sg < W; ++sg) {
            const int64_t e = row * cols + cb + 256 * sg;
            load_g4<G>(d.g, e, gv[sg]);
            pv[sg] = ld_f4<true>(d.p + e);
            if constexpr (UF) {
                mw[sg] = ld_u1<true>(g_as<const void>(mc + e));
                ms[sg] = d.mm[e >> 8];
            } else {
                mv[sg] = ld_f4<true>(mf + e);
            }
        }
#pragma unroll
        for (int sg = 0; sg < W; ++sg) {
            const int64_t e = row * cols + cb + 256 * sg;
            float mh[4], uh[4], mnew[4];
            if constexpr (UF) {
                const double st = div127((double)ms[sg]);
#pragma unroll
                for (int j = 0; j < 4; ++j) mh[j] = uf8_decode((int32_t)(int8_t)(uint8_t)(mw[sg] >> (8 * j)), st);
            } else {
                mh[0] = mv[sg].x, mh[1] = mv[sg].y, mh[2] = mv[sg].z, mh[3] = mv[sg].w;
            }
            double qv[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) qv[j] = (rk * cf[sg][j]) * (double)gv[sg][j];
            if (__builtin_expect(!f32_roundings_decided<4>(qv, uh), 0)) {
#pragma unroll
                for (int j = 0; j < 4; ++j) uh[j] = (float)(((ri * cf[sg][j]) * (double)gv[sg][j]) / clip);
            }
            const float pin[4] = {pv[sg].x, pv[sg].y, pv[sg].z, pv[sg].w};
            float pout[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                mnew[j] = (float)(a.beta1 * (double)mh[j] + a.omb1 * (double)uh[j]);
                const float upd = (si * sf[sg][j]) * mnew[j];
                pout[j] = __builtin_fmaf(-lrf, upd, pin[j] * decayf);
            }
            st_f4<true>(d.p + e, make_float4(pout[0], pout[1], pout[2], pout[3]));
            if constexpr (UF) {
                uint32_t am = 0u;
#pragma unroll
                for (int j = 0; j < 4; ++j) am = OpMax::f(am, abs_bits(mnew[j]));
                am = group_reduce<OpMax, 64>(am);
                const double rs = am != 0u ? rdiv127((double)u2f(am)) : 0.0;
                uint32_t qv[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) qv[j] = rint_low_bits((double)mnew[j] * rs) & 0xFFu;
                st_u1<true>(g_as<void>(mc + e), qv[0] | (qv[1] << 8) | (qv[2] << 16) | (qv[3] << 24));
                if (lane == 0) d.mm[e >> 8] = u2f(am);
            } else {
                st_f4<true>(mf + e, make_float4(mnew[0], mnew[1], mnew[2], mnew[3]));
            }
        }
    }
}

template <int G, bool UF>
__global__ __launch_bounds__(256) void came_apply_whole_kernel(const FacArgs a, int64_t base) {
    const int64_t chunk = base + xcd_order(blockIdx.x, gridDim.x) * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t unit = chunk / kChunksPerUnit;
    if (unit >= a.whole_units) return;
    const GD d = gview(a.D[locate_unit(a.D, a.n2, unit)]);
    const RowChunk c = row_chunk<kCameApplyW>(d, chunk);
    if (c.full)
        came_apply_rows<G, UF, kCameApplyW>(a, d, c.row0, c.col0);
    else
        came_apply_rows<G, UF, 1>(a, d, c.row0, c.col0);
}

hipError_t launch_came_apply(const FacArgs& a, int grad_dtype, hipStream_t s) {
    if (a.total_units == 0) return hipSuccess;
    const bool uf = a.m_codec == UF8;
    const bool bf = grad_dtype == G_BF16;
    hipError_t e = bf ? (uf ? launch_per_chunk(came_apply_whole_kernel<G_BF16, true>, a, s)
                            : launch_per_chunk(came_apply_whole_kernel<G_BF16, false>, a, s))
                      : (uf ? launch_per_chunk(came_apply_whole_kernel<G_F32, true>, a, s)
                            : launch_per_chunk(came_apply_whole_kernel<G_F32, false>, a, s));
    if (e != hipSuccess) return e;
    const int64_t b0 = a.whole_units, b1 = a.total_units;
    e = bf ? (uf ? launch_wave_per_unit(came_apply_unit_kernel<G_BF16, true>, a, b0, b1, s)
                 : launch_wave_per_unit(came_apply_unit_kernel<G_BF16, false>, a, b0, b1, s))
           : (uf ? launch_wave_per_unit(came_apply_unit_kernel<G_F32, true>, a, b0, b1, s)
                 : launch_wave_per_unit(came_apply_unit_kernel<G_F32, false>, a, b0, b1, s));
    if (e != hipSuccess || a.total_chunks == 0) return e;
    const int64_t cap = int64_t(1) << 30;
    const int64_t want = (a.total_chunks + 3) / 4;
    const int grid = (int)(want < cap ? want : cap);
    if (grad_dtype == G_BF16)
        hipLaunchKernelGGL(came_apply_chunk_kernel<G_BF16>, dim3(grid), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(came_apply_chunk_kernel<G_F32>, dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

// ------------------------------------------------ CAME 1-D tensors (WG each)
template <int G>
__global__ __launch_bounds__(256) void came_vec1d_kernel(const FacArgs a) {
    __shared__ DD sh[4];
    __shared__ double clip_s;
    const FacDesc& d = a.D[a.n2 + blockIdx.x];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t n = d.rows * d.cols;
    for (int64_t i = tid; i < n; i += blockDim.x) {
        const double gi = (double)grad1<G>(d.g, i);
        const float old = vec_decode(a.v_codec, a.v_block, d.v, d.vm, i, a.cf);
        d.rtmp[i] = (float)(a.beta * (double)old + a.omb * (gi * gi + a.eps1));
    }
    __syncthreads();
    vec_encode(a.v_codec, a.v_block, d.rtmp, n, a.v_floor, d.v, d.vm, wave, 4, lane);
    DD s{0.0, 0.0};
    for (int64_t i = tid; i < n; i += blockDim.x) {
        const double uu = (1.0 / sqrt((double)d.rtmp[i])) * (double)grad1<G>(d.g, i);
        dd_add(s, uu * uu);
    }
    s = block_dd_sum(s, sh);
    if (tid == 0) {
        const double rms = sqrt(dd_value(s) / (double)n);
        clip_s = rms / a.clip_d > 1.0 ? rms / a.clip_d : 1.0;
    }
    __syncthreads();
    const double clip = clip_s;
    for (int64_t i = tid; i < n; i += blockDim.x) {
        const double uu = (1.0 / sqrt((double)d.rtmp[i])) * (double)grad1<G>(d.g, i);
        const float uh = (float)(uu / clip);
        const float m = came_momentum(a, d, i, uh);
        d.ctmp[i] = m;
        const double pd = (double)d.p[i] * a.decay;
        d.p[i] = (float)(pd - a.lr * (double)m);
    }
    __syncthreads();
    vec_encode(a.m_codec, a.m_block, d.ctmp, n, 0.0f, d.m, d.mm, wave, 4, lane);
}

hipError_t launch_came_vec1d(const FacArgs& a, int grad_dtype, hipStream_t s) {
    if (a.n1 == 0) return hipSuccess;
    if (grad_dtype == G_BF16)
        hipLaunchKernelGGL(came_vec1d_kernel<G_BF16>, dim3(a.n1), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(came_vec1d_kernel<G_F32>, dim3(a.n1), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace al
