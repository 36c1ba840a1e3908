// APOLLO projected-state step on gfx950 (section 3.1: moments kept in a
// low-rank projection of the gradient derive a channel-wise scale of the
// original gradient; section 6 setup: rank 256, channel-wise scaling).
//
// Kernel sequence of one step (the fused AdamW step over the projected
// moments runs between proj and scale, launched by the C ABI):
//   proj    R = fl32(A Pi) for a tile of 32 channels and all r columns, in
//           binary64 on the matrix cores (v_mfma_f64_16x16x4f64): A (bf16 or
//           fp32 gradient, as C x L) and Pi (fp32) are staged through LDS in
//           slices of 16 inputs (Pi by LDS DMA) and widened to binary64 as the
//           operands are read; the products are
//           exact and the accumulation is binary64, so fl32 of the result is
//           the exactly rounded value except within ~L ulps of binary64 of an
//           fp32 midpoint. Also sums g^2 per channel and clears Rt (below
//           rank 256).
//   scale   16 lanes per channel: s_c = ||Rt_c|| / (||R_c|| + 1e-8) (below rank
//           256; at rank 256 a channel is one sub-tile of the AdamW step, which
//           forms s_c itself and never writes Rt).
//   norm    one wavefront per tensor: ||G~||^2 = sum_c s_c^2 ||G_c||^2 and the
//           norm-growth limiter.
//   update  p = fl32(p (1 - lr wd) - lr g (s_c / lam)): one wavefront per
//           8-row chunk of a 256x256 unit (per unit for tensors of other
//           shapes).
// The projection is the one dense contraction of the path (2 r flops per
// parameter); everything else streams.
#include "al_device.hpp"
#include "al_internal.hpp"

namespace al {

typedef double d4v __attribute__((ext_vector_type(4)));

template <int64_t ApolloDesc::*F>
__device__ __forceinline__ int apollo_locate(const ApolloDesc* D, int n, int64_t x) {
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (D[mid].*F <= x)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// Fixed-order butterfly sum of a double over the wavefront (every lane gets the total).
__device__ __forceinline__ double wave_sum_d(double x) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m);
    return x;
}

template <int G>
__device__ __forceinline__ double grad_d(const void* g, int64_t e) {
    if constexpr (G == G_BF16)
        return (double)bf16_to_f32(reinterpret_cast<const uint16_t*>(g)[e]);
    else
        return (double)reinterpret_cast<const float*>(g)[e];
}

// --------------------------------------------------------------- descriptors
__global__ void apollo_desc_copy_kernel(const ApolloDescBatch b, ApolloDesc* dst) {
    constexpr int W = sizeof(ApolloDesc) / 8;
    const int total = b.count * W;
    const uint64_t* src = reinterpret_cast<const uint64_t*>(b.d);
    uint64_t* out = reinterpret_cast<uint64_t*>(dst + b.offset);
    for (int i = threadIdx.x; i < total; i += blockDim.x) out[i] = src[i];
}

hipError_t apollo_copy_desc(const ApolloDesc* host, int count, ApolloDesc* dev, hipStream_t s) {
    static_assert(sizeof(ApolloDesc) % 8 == 0, "descriptor size");
    for (int off = 0; off < count; off += kApolloCopyBatch) {
        ApolloDescBatch b;
        b.count = count - off < kApolloCopyBatch ? count - off : kApolloCopyBatch;
        b.offset = off;
        for (int i = 0; i < b.count; ++i) b.d[i] = host[off + i];
        hipLaunchKernelGGL(apollo_desc_copy_kernel, dim3(1), dim3(256), 0, s, b, dev);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// ---------------------------------------------------------------- projection
constexpr int kLK = 16;  // inputs per LDS slice

// One workgroup of 4 wavefronts per tile of 32 channels; wave w computes output
// columns [64 w, 64 w + 64) of the tile (2 x 4 MFMA tiles of 16 x 16, eight
// binary64 accumulators) when 64 w < r. Four such workgroups share a CU (one
// wavefront of each per SIMD), so one workgroup's barrier leaves three to feed
// the matrix cores. (Eight wavefronts on 64 channels: 2 workgroups per CU,
// projection 2% slower; four wavefronts of 64 x 64 outputs -- 16 accumulators,
// 230 VGPRs, 2 waves per SIMD -- 14% slower.) Slices of 16 inputs are
// double-buffered in LDS with one barrier per slice: while the matrix cores
// work on slice n, slice n + 1 of Pi is copied straight from global memory into
// the other buffer (LDS DMA, one row of Pi per wavefront instruction; rows past
// L repeat row L - 1, whose products meet zero inputs) and slice n + 1 of A is
// loaded into registers, then stored to the other buffer after the matrix work.
// A stays fp32 in LDS (row pitch 18 floats: each half-wavefront of an operand
// read hits 32 distinct banks; pitch 20, distinct over 64 banks, measured 1%
// slower) and is widened to binary64 with Pi when the operands are read; the
// four 4-input steps of a slice are unrolled, each step's operands read during
// the previous step's matrix work, one read per matrix instruction (scheduling
// groups: 0.7% faster than the compiler's own order). MFMA f64 16x16x4 operand
// layout: lane l supplies A[l % 16][l / 16] and B[l / 16][l % 16]; result
// register v of lane l is D[l / 16 + 4 v][l % 16].
constexpr int kProjWaves = 4;                                     // wavefronts per workgroup
constexpr int kProjThreads = 64 * kProjWaves;
constexpr int kProjIT = kApolloTileCh / 16;                       // 16-channel MFMA tiles per wavefront
constexpr int kProjCW = 256 / kProjWaves;                         // output columns per wavefront
constexpr int kProjJT = kProjCW / 16;                             // 16-column MFMA tiles per wavefront
constexpr int kProjRows = kLK / kProjWaves;                       // rows of Pi each wavefront copies per slice
constexpr int kAPer = kApolloTileCh * kLK / kProjThreads;         // A values per thread and slice
constexpr int kAsPitch = 18;                                      // A row pitch in LDS (floats)
constexpr int kBsPitch = 256 + 16;                                // Pi row pitch in LDS (floats)
static_assert(kProjIT * kProjJT == 8 && kLK % kProjWaves == 0 && kAPer * kProjThreads == kApolloTileCh * kLK,
              "projection tiling");

// A pointer known to be the same on every lane, made scalar, so that a load
// from it plus a 32-bit lane offset needs no vector address arithmetic.
template <class P>
__device__ __forceinline__ P uniform_ptr(P p) {
    const uint64_t v = (uint64_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return (P)(((uint64_t)hi << 32) | lo);
}

// One thread's share of the A slices of a tile, fixed for the whole tile:
// value q of every slice is input (c_q, l0 + l_q), stored at As[c_q][l_q].
// Every slice loads from a uniform slice base plus a fixed 32-bit byte offset
// per value (no vector address work): one offset for slices wholly inside the
// tensor, one for a ragged last slice, which clamps l to L - 1 (and zeroes it).
template <int G>
struct ProjA {
    using T = typename std::conditional<G == G_BF16, uint16_t, uint32_t>::type;
    gp<const T> tile;       // element (c0, 0): the tile's first channel, first input
    int64_t stride;         // distance between consecutive inputs of a channel
    uint32_t off[kAPer];    // bytes from the slice base to (c_q clamped to C - 1, l_q)
    uint32_t offt[kAPer];   // the same in the last slice, l_q clamped to L - 1
    int l[kAPer];           // l_q
    int slot[kAPer];        // c_q * kAsPitch + l_q
    bool cval[kAPer];       // c_q inside the tensor
    bool cfull;             // every channel of the tile inside the tensor (uniform)
};

template <int G>
__device__ __forceinline__ void proj_a_setup(ProjA<G>& A, const void* g, int64_t cols, int64_t C, int64_t c0,
                                             int L, bool right, int tid) {
    using T = typename ProjA<G>::T;
    A.stride = right ? 1 : cols;
    A.tile = to_g(reinterpret_cast<const T*>(g)) + (right ? c0 * cols : c0);
    A.cfull = c0 + kApolloTileCh <= C;
#pragma unroll
    for (int q = 0; q < kAPer; ++q) {
        const int e = tid + kProjThreads * q;
        const int c = right ? e / kLK : e % kApolloTileCh;
        const int l = right ? e % kLK : e / kApolloTileCh;
        const int64_t cc = c0 + c < C ? c : C - 1 - c0;
        const int64_t coff = right ? cc * cols : cc;
        const int llast = ((L - 1) / kLK) * kLK;  // first input of the last slice
        const int lt = llast + l < L ? l : L - 1 - llast;
        A.off[q] = (uint32_t)((coff + l * A.stride) * (int64_t)sizeof(T));
        A.offt[q] = (uint32_t)((coff + lt * A.stride) * (int64_t)sizeof(T));
        A.l[q] = l;
        A.slot[q] = c * kAsPitch + l;
        A.cval[q] = c0 + c < C;
    }
}

// Slice l0 of A as raw bits into registers (the wait for them falls after the
// matrix work, where proj_store_a consumes them).
template <int G>
__device__ __forceinline__ void proj_fetch_a(const ProjA<G>& A, int l0, int L, uint32_t (&ra)[kAPer]) {
    using T = typename ProjA<G>::T;
    const bool inside = l0 + kLK <= L;  // otherwise the last slice
    const gp<const char> sb = uniform_ptr(g_as<const char>(A.tile + (int64_t)l0 * A.stride));
#pragma unroll
    for (int q = 0; q < kAPer; ++q) ra[q] = *g_as<const T>(sb + (inside ? A.off[q] : A.offt[q]));
}

// The slice into LDS as fp32, inputs outside the tensor as zero; each thread
// also accumulates the squares of the values it stores (binary64, exact products).
template <int G>
__device__ __forceinline__ void proj_store_a(const ProjA<G>& A, int l0, int L, float* As,
                                             const uint32_t (&ra)[kAPer], double (&gq)[kAPer]) {
    const bool full = A.cfull && l0 + kLK <= L;
#pragma unroll
    for (int q = 0; q < kAPer; ++q) {
        const float x = G == G_BF16 ? __uint_as_float(ra[q] << 16) : __uint_as_float(ra[q]);
        const float v = (full || (A.cval[q] && l0 + A.l[q] < L)) ? x : 0.0f;
        As[A.slot[q]] = v;
        gq[q] = __builtin_fma((double)v, (double)v, gq[q]);
    }
}

// Rows l0 + kProjRows w + t of Pi (r floats each, lanes < r / 4 copy 16 B) into
// the same rows of the LDS buffer; rows past L repeat row L - 1. w is uniform,
// so the row addresses are scalar (32-bit row arithmetic: a 64-bit compare has no
// scalar form). Completion is counted by vmcnt.
__device__ __forceinline__ void proj_copy_pi(const float* proj, int L, int l0, int r, int w, int lane,
                                             float (*Bs)[kBsPitch]) {
    if (4 * lane >= r) return;
#pragma unroll
    for (int t = 0; t < kProjRows; ++t) {
        int row = l0 + kProjRows * w + t;
        row = row < L ? row : L - 1;
        const float* rp = uniform_ptr(proj + (int64_t)row * r);
        __builtin_amdgcn_global_load_lds(rp + 4 * lane, &Bs[kProjRows * w + t][0], 16, 0, 0);
    }
}

template <int G>
__global__ __launch_bounds__(kProjThreads) __attribute__((amdgpu_waves_per_eu(4)))
void apollo_proj_kernel(const ApolloArgs a) {
    // Two buffers of each operand as four separate LDS objects, named statically
    // in each half of the unrolled slice loop: the compiler then knows that the
    // copy into one buffer does not alias the reads of the other and does not
    // wait for the copy before the matrix work.
    __shared__ __attribute__((aligned(16))) float As0[kApolloTileCh][kAsPitch];
    __shared__ __attribute__((aligned(16))) float As1[kApolloTileCh][kAsPitch];
    __shared__ __attribute__((aligned(16))) float Bs0[kLK][kBsPitch];
    __shared__ __attribute__((aligned(16))) float Bs1[kLK][kBsPitch];
    const int64_t tile = blockIdx.x;
    const ApolloDesc& d = a.D[apollo_locate<&ApolloDesc::tile_begin>(a.D, a.nt, tile)];
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, l4 = lane >> 4;
    const int r = a.rank;
    // the descriptor's fields, read once (read through the descriptor they are
    // fetched again every slice, and those fetches wait for the copies in flight)
    const int64_t C = d.C;
    // the projected length is at most 2^20 (rows * cols <= 2^40): slice arithmetic in
    // 32 bits and uniform, so its compares are scalar
    const int L = __builtin_amdgcn_readfirstlane((int)d.L);
    const int64_t c0 = (tile - d.tile_begin) * kApolloTileCh;
    const float* proj = d.proj;
    float* const Rp = d.R;
    float* const Rtp = d.Rt;
    double* const gn2 = d.gn2;
    const bool right = d.right != 0;
    ProjA<G> A;
    proj_a_setup<G>(A, d.g, d.cols, C, c0, L, right, tid);
    const bool active = kProjCW * w < r;
    d4v acc[kProjIT][kProjJT];
#pragma unroll
    for (int i = 0; i < kProjIT; ++i)
#pragma unroll
        for (int j = 0; j < kProjJT; ++j) acc[i][j] = d4v{0.0, 0.0, 0.0, 0.0};
    double gq[kAPer];  // this thread's sums of squares, value q of every slice
#pragma unroll
    for (int q = 0; q < kAPer; ++q) gq[q] = 0.0;
    uint32_t ra[kAPer];
    const int ns = (L + kLK - 1) / kLK;
    // Slice n from (Ac, Bc) while slice n + 1 is brought into (An, Bn).
    auto slice = [&](int n, float (*Ac)[kAsPitch], float (*Bc)[kBsPitch], float (*An)[kAsPitch],
                     float (*Bn)[kBsPitch]) {
        const bool more = n + 1 < ns;
        if (more) {
            proj_copy_pi(proj, L, (n + 1) * kLK, r, w, lane, Bn);
            proj_fetch_a<G>(A, (n + 1) * kLK, L, ra);
        }
        if (active) {
            // the operands of step kk + 4 are read before the matrix work of step kk
            float xa[2][kProjIT], xb[2][kProjJT];
            auto rd = [&](int st, int kk) {
#pragma unroll
                for (int i = 0; i < kProjIT; ++i) xa[st][i] = Ac[16 * i + l16][kk + l4];
#pragma unroll
                for (int j = 0; j < kProjJT; ++j) xb[st][j] = Bc[kk + l4][kProjCW * w + 16 * j + l16];
            };
            rd(0, 0);
#pragma unroll
            for (int kk = 0; kk < kLK; kk += 4) {
                const int st = (kk >> 2) & 1;
                if (kk + 4 < kLK) rd(st ^ 1, kk + 4);
                double af[kProjIT], bf[kProjJT];
#pragma unroll
                for (int i = 0; i < kProjIT; ++i) af[i] = (double)xa[st][i];
#pragma unroll
                for (int j = 0; j < kProjJT; ++j) bf[j] = (double)xb[st][j];
#pragma unroll
                for (int i = 0; i < kProjIT; ++i)
#pragma unroll
                    for (int j = 0; j < kProjJT; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(af[i], bf[j], acc[i][j], 0, 0, 0);
                // issue order: one matrix instruction, then one read of the next step's operands
#pragma unroll
                for (int x = 0; x < kProjIT + kProjJT; ++x) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x008, kProjIT * kProjJT - kProjIT - kProjJT, 0);
            }
        }
        if (more) proj_store_a<G>(A, (n + 1) * kLK, L, &An[0][0], ra, gq);
        // the copies into the other buffers have landed and every read of these is done
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
    };
    if (ns > 0) {
        proj_copy_pi(proj, L, 0, r, w, lane, Bs0);
        proj_fetch_a<G>(A, 0, L, ra);
        proj_store_a<G>(A, 0, L, &As0[0][0], ra, gq);
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
    }
    for (int n = 0; n < ns; n += 2) {
        slice(n, As0, Bs0, As1, Bs1);
        if (n + 1 < ns) slice(n + 1, As1, Bs1, As0, Bs0);
    }
    // Channel sums of g^2 in a fixed order: the per-thread sums go to LDS (the
    // first Pi buffer, free after the last barrier), then thread c adds the 16
    // of channel c -- value q of threads c + kApolloTileCh m (channels along the
    // rows of g) or value c / G16 of threads 16 (c % G16) + m, G16 = threads / 16
    // (channels along the columns).
    constexpr int kG16 = kProjThreads / 16;
    static_assert(kAPer * kProjThreads / kApolloTileCh == 16 && kProjThreads % kApolloTileCh == 0 &&
                      kAPer * kProjThreads * 8 <= (int)sizeof(Bs0),
                  "the reduction below takes 16 values per channel");
    double* red = reinterpret_cast<double*>(&Bs0[0][0]);
#pragma unroll
    for (int q = 0; q < kAPer; ++q) red[q * kProjThreads + tid] = gq[q];
    __syncthreads();
    if (tid < kApolloTileCh && c0 + tid < C) {
        double x = 0.0;
        if (right) {
            const int q = tid / kG16, t0 = 16 * (tid % kG16);
            for (int m = 0; m < 16; ++m) x += red[q * kProjThreads + t0 + m];
        } else {
            for (int q = 0; q < kAPer; ++q)
                for (int m = 0; m < kProjThreads / kApolloTileCh; ++m)
                    x += red[q * kProjThreads + tid + kApolloTileCh * m];
        }
        to_g(gn2)[c0 + tid] = x;
    }
    // Rt exists below rank 256 only (it is then the AdamW step's parameter, cleared here)
    const bool clear_rt = Rtp != nullptr;
    const gp<float> Rg = to_g(Rp);
    const gp<float> Rtg = to_g(Rtp);
    if (active) {
#pragma unroll
        for (int i = 0; i < kProjIT; ++i)
#pragma unroll
            for (int j = 0; j < kProjJT; ++j)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int64_t c = c0 + 16 * i + l4 + 4 * v;
                    const int k = kProjCW * w + 16 * j + l16;
                    if (c < C) {
                        Rg[c * r + k] = (float)acc[i][j][v];
                        if (clear_rt) Rtg[c * r + k] = 0.0f;
                    }
                }
    }
}

hipError_t launch_apollo_proj(const ApolloArgs& a, int grad_dtype, hipStream_t s) {
    if (a.total_tiles == 0) return hipSuccess;
    // an active wavefront stores all kProjCW of its columns, and Pi rows are copied 16 B per lane
    if (a.rank <= 0 || a.rank > 256 || a.rank % kProjCW != 0) return hipErrorInvalidValue;
    if (grad_dtype == G_BF16)
        hipLaunchKernelGGL(apollo_proj_kernel<G_BF16>, dim3((unsigned)a.total_tiles), dim3(kProjThreads), 0, s, a);
    else
        hipLaunchKernelGGL(apollo_proj_kernel<G_F32>, dim3((unsigned)a.total_tiles), dim3(kProjThreads), 0, s, a);
    return hipGetLastError();
}

// ------------------------------------------------------------ channel scales
// A wavefront takes kScaleCh consecutive channels of the list (one tensor's
// channels are consecutive, so a group may span two tensors), 4 at a time:
// 16 lanes per channel, 16-byte loads of R and Rt covering 4 KB of each, and
// each channel's two sums of squares merged over its 16 lanes with DPP in a
// fixed order. Rt holds the negated direction (the AdamW kernel's parameter
// output from zero); only squares are used.
constexpr int kScaleCh = 16;

__device__ __forceinline__ double row16_sum_d(double x) {
    x += dpp_d<kDppQuadXor1>(x);
    x += dpp_d<kDppQuadXor2>(x);
    x += dpp_d<kDppRowHalfMirror>(x);
    x += dpp_d<kDppRowMirror>(x);
    return x;
}

__global__ __launch_bounds__(256) void apollo_scale_kernel(const ApolloArgs a) {
    const int lane = threadIdx.x & 63, sub = lane >> 4, l16 = lane & 15;
    const int64_t ch0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * kScaleCh;
    const int r = a.rank;
    for (int q = 0; q < kScaleCh; q += 4) {
        const int64_t ch = ch0 + q + sub;  // this lane's channel
        const bool live = ch < a.total_chans;
        if (__builtin_amdgcn_readfirstlane(ch0 + q) >= a.total_chans) return;
        double st = 0.0, sr = 0.0;
        int64_t c = 0;
        const ApolloDesc* dp = nullptr;
        if (live) {
            dp = &a.D[apollo_locate<&ApolloDesc::chan_begin>(a.D, a.nt, ch)];
            c = ch - dp->chan_begin;
            const gp<const float> rt = to_g((const float*)dp->Rt) + c * r;
            const gp<const float> rr = to_g((const float*)dp->R) + c * r;
            for (int k = 4 * l16; k < r; k += 64) {
                const float4 x = ld_f4<false>(rt + k);
                const float4 y = ld_f4<false>(rr + k);
                st += ((double)x.x * x.x + (double)x.y * x.y) + ((double)x.z * x.z + (double)x.w * x.w);
                sr += ((double)y.x * y.x + (double)y.y * y.y) + ((double)y.z * y.z + (double)y.w * y.w);
            }
        }
        st = row16_sum_d(st);
        sr = row16_sum_d(sr);
        if (live && l16 == 0) {
            const double sc = sqrt(st) / (sqrt(sr) + 1e-8);
            dp->s[c] = sc;
            dp->sg[c] = sc * sc * dp->gn2[c];
        }
    }
}

hipError_t launch_apollo_scale(const ApolloArgs& a, hipStream_t s) {
    if (a.total_chans == 0) return hipSuccess;
    const int64_t waves = (a.total_chans + kScaleCh - 1) / kScaleCh;
    hipLaunchKernelGGL(apollo_scale_kernel, dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s, a);
    return hipGetLastError();
}

// --------------------------------------------------------- limiter per tensor
__global__ __launch_bounds__(64) void apollo_norm_kernel(const ApolloArgs a) {
    const ApolloDesc& d = a.D[blockIdx.x];
    const int lane = threadIdx.x;
    double acc = 0.0;
    for (int64_t c = lane; c < d.C; c += 64) acc += d.sg[c];
    acc = wave_sum_d(acc);
    if (lane == 0) {
        const double n = sqrt(acc);
        double lam = 1.0;
        if (a.gamma > 0.0) {
            if (a.step >= 2) {
                const double q = n / ((double)d.norm_state[0] + 1e-8);
                lam = (q > a.gamma ? q : a.gamma) / a.gamma;
                d.norm_state[0] = (float)(n / lam);
            } else {
                d.norm_state[0] = (float)n;
            }
        }
        d.lam[0] = lam;
    }
}

hipError_t launch_apollo_norm(const ApolloArgs& a, hipStream_t s) {
    if (a.nt == 0) return hipSuccess;
    hipLaunchKernelGGL(apollo_norm_kernel, dim3(a.nt), dim3(64), 0, s, a);
    return hipGetLastError();
}

// ------------------------------------------------------------ parameter update
// One wave per 256 x 256 unit, lane = 4 consecutive columns, rows in batches of
// kUpdRows with all their loads issued before the stores (non-temporal: p and g
// are touched once). The row scales s_r / lambda of the unit's 256 rows are
// divided once per unit (4 per lane) and read back from LDS as broadcasts, so a
// row costs no binary64 division.
constexpr int kUpdRows = 16;

template <int G>
__global__ __launch_bounds__(256) void apollo_update_kernel(const ApolloArgs a) {
    __shared__ double srow_all[4][256];
    const int lane = threadIdx.x & 63;
    double* srow = srow_all[threadIdx.x >> 6];
    const int64_t unit = xcd_order(blockIdx.x, gridDim.x) * 4 +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (unit >= a.total_units) return;
    const ApolloDesc& d = a.D[apollo_locate<&ApolloDesc::unit_begin>(a.D, a.nt, unit)];
    if (d.whole) return;  // the chunk kernel's
    const int64_t u = unit - d.unit_begin;
    const int64_t ru = u / d.ncu, cu = u % d.ncu;
    const int64_t r0 = ru * 256, c0 = cu * 256, cols = d.cols;
    const int nr = (int)(d.rows - r0 < 256 ? d.rows - r0 : 256);
    const int nc = (int)(cols - c0 < 256 ? cols - c0 : 256);
    const int c = 4 * lane;
    const bool right = d.right != 0;
    const double lam = d.lam[0];
    const gp<const double> sv = to_g((const double*)d.s);
    if (right) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int r = lane + 64 * k;
            srow[r] = r < nr ? sv[r0 + r] / lam : 0.0;
        }
    }
    if (c >= nc) return;
    const bool vec = (cols & 3) == 0 && c + 4 <= nc;
    const gp<float> pp = to_g(d.p);
    double sc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) sc[j] = (!right && c + j < nc) ? sv[c0 + c + j] / lam : 0.0;
    for (int rb = 0; rb < nr; rb += kUpdRows) {
        float4 pv[kUpdRows];
        float gv[kUpdRows][4];
#pragma unroll
        for (int k = 0; k < kUpdRows; ++k) {
            const int rr = rb + k < nr ? rb + k : nr - 1;  // rows past the end repeat the last one, unused
            const int64_t e = (r0 + rr) * cols + c0 + c;
            if (vec) {
                pv[k] = ld_f4<true>(gp<const float>(pp + e));
                if constexpr (G == G_BF16) {
                    const uint2 w = ld_u2<true>(g_as<const void>(to_g((const uint16_t*)d.g) + e));
                    gv[k][0] = bf16_to_f32(w.x & 0xFFFFu);
                    gv[k][1] = bf16_to_f32(w.x >> 16);
                    gv[k][2] = bf16_to_f32(w.y & 0xFFFFu);
                    gv[k][3] = bf16_to_f32(w.y >> 16);
                } else {
                    const float4 y = ld_f4<true>(to_g((const float*)d.g) + e);
                    gv[k][0] = y.x;
                    gv[k][1] = y.y;
                    gv[k][2] = y.z;
                    gv[k][3] = y.w;
                }
            } else {
                float h[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    h[j] = c + j < nc ? pp[e + j] : 0.0f;
                    gv[k][j] = c + j < nc ? (float)grad_d<G>(d.g, e + j) : 0.0f;
                }
                pv[k] = make_float4(h[0], h[1], h[2], h[3]);
            }
        }
#pragma unroll
        for (int k = 0; k < kUpdRows; ++k) {
            if (rb + k >= nr) continue;
            const int64_t e = (r0 + rb + k) * cols + c0 + c;
            const double sr = right ? srow[rb + k] : 0.0;
            const float pin[4] = {pv[k].x, pv[k].y, pv[k].z, pv[k].w};
            float out[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const double upd = (double)gv[k][j] * (right ? sr : sc[j]);
                out[j] = (float)((double)pin[j] * a.decay - a.lr * upd);
            }
            if (vec) {
                st_f4<true>(pp + e, make_float4(out[0], out[1], out[2], out[3]));
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (c + j < nc) pp[e + j] = out[j];
            }
        }
    }
}

// Tensors of whole 256x256 units: one wavefront per chunk of 8 unit rows
// (2048 elements, 4 per 256-thread workgroup) with no loop, lane 32 h + q on
// rows 2k + h and columns 4q .. 4q + 3 and 128 + 4q .. 128 + 4q + 3, so every
// access covers contiguous row segments; all loads of the chunk before its
// stores. A chunk of another tensor returns (the unit kernel takes those).
constexpr int kUpdChunkRows = 8;

template <int G, bool RIGHT>
__device__ __forceinline__ void apollo_update_chunk(const ApolloArgs& a, const ApolloDesc& d, int64_t row0, int64_t c0,
                                                    int q) {
    const int64_t cols = d.cols;
    const double lam = d.lam[0];
    const gp<const double> sv = to_g((const double*)d.s);
    const gp<float> pp = to_g(d.p);
    constexpr int NP = kUpdChunkRows / 2;
    float4 pv[NP][2];
    uint2 gw[NP][2];
    float4 gf[NP][2];
#pragma unroll
    for (int k = 0; k < NP; ++k) {
#pragma unroll
        for (int sg = 0; sg < 2; ++sg) {
            const int64_t e = (row0 + 2 * k) * cols + c0 + 128 * sg + 4 * q;
            pv[k][sg] = ld_f4<true>(gp<const float>(pp + e));
            if constexpr (G == G_BF16)
                gw[k][sg] = ld_u2<true>(g_as<const void>(to_g((const uint16_t*)d.g) + e));
            else
                gf[k][sg] = ld_f4<true>(to_g((const float*)d.g) + e);
        }
    }
    // channel scales s_c / lambda: one per row pair (channels are rows) or per column
    double sr[RIGHT ? NP : 1], sc[RIGHT ? 1 : 2][4];
    if constexpr (RIGHT) {
#pragma unroll
        for (int k = 0; k < NP; ++k) sr[k] = sv[row0 + 2 * k] / lam;
    } else {
#pragma unroll
        for (int sg = 0; sg < 2; ++sg)
#pragma unroll
            for (int j = 0; j < 4; ++j) sc[sg][j] = sv[c0 + 128 * sg + 4 * q + j] / lam;
    }
#pragma unroll
    for (int k = 0; k < NP; ++k) {
#pragma unroll
        for (int sg = 0; sg < 2; ++sg) {
            float gv[4];
            if constexpr (G == G_BF16) {
                gv[0] = bf16_to_f32(gw[k][sg].x & 0xFFFFu), gv[1] = bf16_to_f32(gw[k][sg].x >> 16);
                gv[2] = bf16_to_f32(gw[k][sg].y & 0xFFFFu), gv[3] = bf16_to_f32(gw[k][sg].y >> 16);
            } else {
                gv[0] = gf[k][sg].x, gv[1] = gf[k][sg].y, gv[2] = gf[k][sg].z, gv[3] = gf[k][sg].w;
            }
            const float pin[4] = {pv[k][sg].x, pv[k][sg].y, pv[k][sg].z, pv[k][sg].w};
            float out[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const double upd = (double)gv[j] * (RIGHT ? sr[k] : sc[RIGHT ? 0 : sg][j]);
                out[j] = (float)((double)pin[j] * a.decay - a.lr * upd);
            }
            const int64_t e = (row0 + 2 * k) * cols + c0 + 128 * sg + 4 * q;
            st_f4<true>(pp + e, make_float4(out[0], out[1], out[2], out[3]));
        }
    }
}

template <int G>
__global__ __launch_bounds__(256) void apollo_update_chunk_kernel(const ApolloArgs a) {
    const int lane = threadIdx.x & 63, h = lane >> 5, q = lane & 31;
    const int64_t chunk = xcd_order(blockIdx.x, gridDim.x) * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t unit = chunk / (256 / kUpdChunkRows);
    if (unit >= a.total_units) return;
    const ApolloDesc& d = a.D[apollo_locate<&ApolloDesc::unit_begin>(a.D, a.nt, unit)];
    if (!d.whole) return;
    const int64_t u = unit - d.unit_begin;
    const int64_t r0 = (u / d.ncu) * 256, c0 = (u % d.ncu) * 256;
    const int64_t row0 = r0 + (chunk % (256 / kUpdChunkRows)) * kUpdChunkRows + h;
    if (d.right)
        apollo_update_chunk<G, true>(a, d, row0, c0, q);
    else
        apollo_update_chunk<G, false>(a, d, row0, c0, q);
}

hipError_t launch_apollo_update(const ApolloArgs& a, int grad_dtype, hipStream_t s) {
    if (a.total_units == 0) return hipSuccess;
    if (a.any_whole) {
        const unsigned grid = (unsigned)((a.total_units * (256 / kUpdChunkRows) + 3) / 4);
        if (grad_dtype == G_BF16)
            hipLaunchKernelGGL(apollo_update_chunk_kernel<G_BF16>, dim3(grid), dim3(256), 0, s, a);
        else
            hipLaunchKernelGGL(apollo_update_chunk_kernel<G_F32>, dim3(grid), dim3(256), 0, s, a);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (!a.any_ragged) return hipSuccess;
    const unsigned grid = (unsigned)((a.total_units + 3) / 4);
    if (grad_dtype == G_BF16)
        hipLaunchKernelGGL(apollo_update_kernel<G_BF16>, dim3(grid), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(apollo_update_kernel<G_F32>, dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace al
