// Fused multi-tensor AdamW step with block-quantized state (gfx950).
//
// One pass over HBM per step: read p (fp32), g (bf16/fp32), m (UF8 codes +
// absmax per 256, or fp32) and v (AL8/AL16 codes + {l_min, delta} per
// block, or fp32); write p, m, v and their metadata. Section 3.1 (Eq.
// adam_update) with PyTorch AdamW's decoupled weight decay and bias
// corrections; codes per section 4 (Eq. al_bounds, al_quant, al_dequant,
// exact_zero) and the uniform signed momentum code of section 4.3.
//
// Work decomposition. A chunk is max(2048, B_V) consecutive elements of one
// tensor for AL8 blocks of 128+, else max(1024, B_V), owned by one wavefront:
// 4 consecutive elements per lane in each of K = chunk/256 sub-tiles, so every
// load and store is a coalesced 16/8/4-byte access and every block reduction
// stays inside the wavefront (DPP, swizzle, readlane). The momentum block
// (256) is one sub-tile and is encoded as soon as that sub-tile's moments are
// computed; the second moment is held in registers until its block is
// complete, and a block of whole sub-tiles has its min/max keys reduced as
// soon as its last sub-tile is done (smaller blocks: reduced over their lane
// group after every sub-tile and parked in LDS). Per-block scalar work of the second
// moment (the binary64 divisions and endpoint logarithms of up to 16 blocks)
// runs once per chunk with one block per lane pair, and the results are
// broadcast back (readlane for blocks that span whole sub-tiles, ds_bpermute
// for smaller ones). The grid holds one wave per chunk over the whole tensor
// list, and the chunk -> tensor map is a binary search over the descriptor
// table in device memory (one launch per step). Full chunks use non-temporal
// loads and stores: every byte of the step is touched exactly once.
#include <mutex>

#include "al_device.hpp"
#include "al_internal.hpp"

#ifndef AL_ADAMW_NT_LOAD
#define AL_ADAMW_NT_LOAD 1
#endif
#ifndef AL_ADAMW_NT_STORE
#define AL_ADAMW_NT_STORE 1
#endif

namespace al {

// The decode polynomial's coefficients, in constant memory: scalar loads at the
// point of use (as kernel arguments they would be held in scalar registers for
// the whole chunk, next to the descriptor read from the table, and spill).
__constant__ Exp2Coef kExp2 = AL_EXP2_TAYLOR;

// Split-table decode of AL8 levels. A code q >= 1 stands for level q - 1,
// fl32(2^(l32 + (q - 1) st)) with l32 = fl32(l_min) and st = delta32 / 254 in
// binary64 (Eq. al_dequant). Two factors (blocks of 128+): q = 16 a + b and
// 2^(l32 + (q - 1) st) = 2^(l32 + (16 a - 1) st) * 2^(b st), table entries
// j < 16 the first factor, 16 + j the second. Three factors (blocks of 64):
// q = 64 a + 8 b + c, entries [0, 4) 2^(l32 + (64 a - 1) st), [4, 12) 2^(8 b st),
// [12, 20) 2^(c st). The binary64 value before the fp32 rounding is the
// product; al_diag_levels evaluates the same functions.
__device__ __forceinline__ double split2_entry(double l32, double st, int j) {
    const double arg = j < 16 ? l32 + (double)(16 * j - 1) * st : (double)(j - 16) * st;
    return exp2_d(arg, kExp2);
}
// An empty register constraint: the compiler cannot move work across it.
__device__ __forceinline__ void opaque_f(float& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ double split2_product(double f1, double f2) { return f1 * f2; }
__device__ __forceinline__ double split2_level(const double* t, uint32_t q) {
    return split2_product(t[q >> 4], t[16 + (q & 15u)]);
}
// The three-factor entries' arguments share one conversion, product and sum
// (the lanes of one pass take different entry kinds): base + fl64(m st) with
// base = l32 for the first factor and +0.0 otherwise, which adds exactly
// (m st >= 0); 1% faster at B_V 64. (The same form for the two-factor
// entries raised the B_V 256 kernel's spills and ran 1% slower there.)
__device__ __forceinline__ double split3_entry(double l32, double st, int j) {
    const int m = j < 4 ? 64 * j - 1 : (j < 12 ? 8 * (j - 4) : j - 12);
    const double base = j < 4 ? l32 : 0.0;
    return exp2_d(base + (double)m * st, kExp2);
}
__device__ __forceinline__ double split3_product(double f1, double f2, double f3) { return (f1 * f2) * f3; }
__device__ __forceinline__ double split3_level(const double* t, uint32_t q) {
    return split3_product(t[q >> 6], t[4 + ((q >> 3) & 7u)], t[12 + (q & 7u)]);
}

// Every byte the step touches is read once and written once, so the full-chunk
// path may mark its loads and stores non-temporal (streaming).
constexpr bool kNtLoad = AL_ADAMW_NT_LOAD != 0;
constexpr bool kNtStore = AL_ADAMW_NT_STORE != 0;

__host__ __device__ constexpr int chunk_elems(int vc, int bv) {
    return vc == FP32 ? 1024 : (vc == AL8 && bv >= 128) ? (bv > 2048 ? bv : 2048) : (bv > 1024 ? bv : 1024);
}

template <int MC, int VC, int BV>
struct Geo {
    static constexpr bool VQ = (VC == AL8 || VC == AL16);
    // elements per chunk: AL8 blocks of 128+ take 2048 (the per-chunk work amortised over twice
    // the elements; blocks of 128 then need 138 registers and run 3 waves per SIMD, 1% faster
    // than 1024-element chunks at 4); blocks of 64 (no gain at 2048), AL16 (wider codes) and an
    // fp32 second moment take max(1024, B_V)
    static constexpr int C = chunk_elems(VC, BV);
    static constexpr int K = C / kSub;                       // sub-tiles per chunk
    static constexpr int NB = VQ ? C / BV : 1;               // v blocks per chunk
    static constexpr int GL = BV < kSub ? BV / 4 : 64;       // lanes per v block within a sub-tile
    static constexpr int PER = kSub / BV > 0 ? kSub / BV : 1;  // v blocks per sub-tile (BV < 256)
    static constexpr int LEVELS = VQ ? levels_of<VC>() : 1;
    static constexpr int NSLOT = BV < kSub ? 1 : NB;         // wave-uniform min/max slots (blocks of 256+)
    static constexpr bool LUT = (VC == AL8) && BV >= 512;     // decode through an LDS level table
    // decode through per-block split tables: 16 + 16 binary64 factors per block
    static constexpr bool SPLIT = (VC == AL8) && (BV == 128 || BV == 256);
    // blocks of 64: three factors (4 + 8 + 8 binary64 entries per block)
    static constexpr bool SPLIT3 = (VC == AL8) && BV == 64;
};

template <bool C_, class A, class B>
struct Pick {
    using T = A;
};
template <class A, class B>
struct Pick<false, A, B> {
    using T = B;
};

__device__ __forceinline__ float f4_at(const float4& v, int j) {
    return j == 0 ? v.x : j == 1 ? v.y : j == 2 ? v.z : v.w;
}

// Raw inputs of up to 4 sub-tiles as loaded from HBM (packed: a bf16 pair or
// four 8-bit codes per register).
template <int G, int MC, int VC, int BV>
struct Raw {
    using Q = Geo<MC, VC, BV>;
    using GT = typename Pick<G == G_BF16, uint2, float4>::T;
    using MT = typename Pick<MC == UF8, uint32_t, float4>::T;
    using VT = typename Pick<VC == AL16, uint2, typename Pick<VC == AL8, uint32_t, float4>::T>::T;
    static constexpr int P = Q::K < 4 ? Q::K : 4;  // sub-tiles per load phase
    float4 p[P];
    GT g[P];
    MT m[P];
    VT v[P];
};

// Old block metadata, one block per lane: lanes [0, K) hold the momentum
// scales of the K sub-tiles, lanes [32, 32 + NB) the {l_min, delta} of the NB
// second-moment blocks.
struct OldMeta {
    float a;  // momentum absmax (lanes < K) or v delta (lanes 32..)
    float l;  // v l_min (lanes 32..)
};

// A descriptor's streams as global-address-space pointers: the descriptors
// are read from memory, so the compiler would otherwise treat their pointers
// as generic and issue flat loads and stores.
struct DescG {
    gp<float> p;
    gp<const uint8_t> g;
    gp<uint8_t> m;
    gp<float> ms;
    gp<uint8_t> v;
    gp<float> vm;
    int64_t n;
    gp<double> cs, csg;   // APOLLO: channel scales and s_c^2 gn2_c (rank 256: one channel per sub-tile)
    gp<const double> cg2;  // APOLLO: per-channel sums of g^2
};

// The table is read-only during the step, so it is read through the constant
// address space: its loads are invariant and the compiler may repeat them
// instead of holding every field in a scalar register for the whole chunk.
template <class T>
using cp = __attribute__((address_space(4))) T*;

__device__ __forceinline__ DescG gview(cp<const AdamWDesc> D, int i) {
    return DescG{to_g(D[i].p), (gp<const uint8_t>)to_g(D[i].g), (gp<uint8_t>)to_g(D[i].m), to_g(D[i].ms),
                 (gp<uint8_t>)to_g(D[i].v), to_g(D[i].vm), D[i].n, nullptr, nullptr, nullptr};
}

typedef float f2v __attribute__((ext_vector_type(2)));

template <int G, int MC, int VC, int BV, bool FULL, bool APO>
__device__ __forceinline__ void load_raw(Raw<G, MC, VC, BV>& r, const DescG& d, int64_t e0, int64_t valid,
                                         int lane, int ph) {
    using R = Raw<G, MC, VC, BV>;
#pragma unroll
    for (int k = 0; k < R::P; ++k) {
        const int rel = (ph * R::P + k) * kSub + 4 * lane;
        const int64_t e = e0 + rel;
        if constexpr (APO) r.p[k] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);  // no parameter stream
        if constexpr (FULL) {
            if constexpr (!APO) r.p[k] = ld_f4<kNtLoad>(d.p + e);
            if constexpr (G == G_BF16)
                r.g[k] = ld_u2<kNtLoad>(g_as<const uint16_t>(d.g) + e);
            else
                r.g[k] = ld_f4<kNtLoad>(g_as<const float>(d.g) + e);
            if constexpr (MC == UF8)
                r.m[k] = ld_u1<kNtLoad>(g_as<const uint8_t>(d.m) + e);
            else
                r.m[k] = ld_f4<kNtLoad>(g_as<const float>(d.m) + e);
            if constexpr (VC == AL16)
                r.v[k] = ld_u2<kNtLoad>(g_as<const uint16_t>(d.v) + e);
            else if constexpr (VC == AL8)
                r.v[k] = ld_u1<kNtLoad>(g_as<const uint8_t>(d.v) + e);
            else
                r.v[k] = ld_f4<kNtLoad>(g_as<const float>(d.v) + e);
        } else {
            float pp[4];
            uint32_t gb[4], mb[4], vb[4];
            float gf[4], mf[4], vf[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const bool ok = rel + j < valid;
                pp[j] = (ok && !APO) ? d.p[e + j] : 0.0f;
                if constexpr (G == G_BF16) gb[j] = ok ? g_as<const uint16_t>(d.g)[e + j] : 0u;
                else gf[j] = ok ? g_as<const float>(d.g)[e + j] : 0.0f;
                if constexpr (MC == UF8) mb[j] = ok ? g_as<const uint8_t>(d.m)[e + j] : 0u;
                else mf[j] = ok ? g_as<const float>(d.m)[e + j] : 0.0f;
                if constexpr (VC == AL16) vb[j] = ok ? g_as<const uint16_t>(d.v)[e + j] : 0u;
                else if constexpr (VC == AL8) vb[j] = ok ? g_as<const uint8_t>(d.v)[e + j] : 0u;
                else vf[j] = ok ? g_as<const float>(d.v)[e + j] : 0.0f;
            }
            r.p[k] = make_float4(pp[0], pp[1], pp[2], pp[3]);
            if constexpr (G == G_BF16) r.g[k] = make_uint2(gb[0] | (gb[1] << 16), gb[2] | (gb[3] << 16));
            else r.g[k] = make_float4(gf[0], gf[1], gf[2], gf[3]);
            if constexpr (MC == UF8) r.m[k] = mb[0] | (mb[1] << 8) | (mb[2] << 16) | (mb[3] << 24);
            else r.m[k] = make_float4(mf[0], mf[1], mf[2], mf[3]);
            if constexpr (VC == AL16) r.v[k] = make_uint2(vb[0] | (vb[1] << 16), vb[2] | (vb[3] << 16));
            else if constexpr (VC == AL8) r.v[k] = vb[0] | (vb[1] << 8) | (vb[2] << 16) | (vb[3] << 24);
            else r.v[k] = make_float4(vf[0], vf[1], vf[2], vf[3]);
        }
    }
}

template <int MC, int VC, int BV, bool FULL>
__device__ __forceinline__ OldMeta load_meta(const DescG& d, int64_t e0, int64_t valid, int lane) {
    using Q = Geo<MC, VC, BV>;
    OldMeta r;
    r.a = 0.0f;
    r.l = 0.0f;
    if constexpr (MC == UF8) {
        if (lane < Q::K && (FULL || lane * kSub < valid)) r.a = d.ms[e0 / kSub + lane];
    }
    if constexpr (Q::VQ) {
        const int b = lane - 32;
        if (b >= 0 && b < Q::NB && (FULL || (int64_t)b * BV < valid)) {
            const f2v mm = *g_as<const f2v>(d.vm + 2 * (e0 / BV + b));
            r.l = mm.x;
            r.a = mm.y;
        }
    }
    return r;
}

template <int G>
__device__ __forceinline__ float grad_at(const typename Pick<G == G_BF16, uint2, float4>::T& w, int j) {
    if constexpr (G == G_BF16)
        return bf16_to_f32(((j < 2 ? w.x : w.y) >> (16 * (j & 1))) & 0xFFFFu);
    else
        return f4_at(w, j);
}

// The min/max keys of two second-moment blocks (A, B: each lane's running
// minimum of bits - 1 and maximum of bits) reduced over the wavefront by one
// reduce-scatter: the minima travel complemented, so every step is a maximum.
// After the two quad steps lane L holds key (L & 1 ? maximum : minimum) of
// block (L & 2 ? B : A) over its quad; four more steps (lane xor 4, 8, 16,
// 32) complete it over the wavefront. Lanes 4 pair .. 4 pair + 3 take the
// result into their slot: lane 2b then holds block b's minimum (bits; 0 when
// the block has no positive value) and 2b + 1 its maximum.
__device__ __forceinline__ uint32_t key_pair_reduce(uint32_t amn, uint32_t amx, uint32_t bmn, uint32_t bmx, int lane,
                                                    int pair, uint32_t slot) {
    const bool b0 = lane & 1, b1 = lane & 2;
    const uint32_t wa0 = ~amn, wb0 = ~bmn;
    // step 1 (lane xor 1): keep this lane's kind (minimum / maximum) of both blocks
    uint32_t ka = b0 ? amx : wa0, kb = b0 ? bmx : wb0;
    const uint32_t sa = b0 ? wa0 : amx, sb = b0 ? wb0 : bmx;
    ka = OpMax::f(ka, dpp<kDppQuadXor1>(sa));
    kb = OpMax::f(kb, dpp<kDppQuadXor1>(sb));
    // step 2 (lane xor 2): keep this lane's block
    uint32_t v = b1 ? kb : ka;
    v = OpMax::f(v, dpp<kDppQuadXor2>(b1 ? ka : kb));
    v = OpMax::f(v, (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, kSwzXor4));
    v = OpMax::f(v, (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, kSwzXor8));
    v = OpMax::f(v, (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, kSwzXor16));
    v = OpMax::f(v, (uint32_t)__shfl_xor((int)v, 32));
    const uint32_t key = b0 ? v : ~v + 1u;
    return (lane >> 2) == pair ? key : slot;
}

// A binary64 sum over each row of 16 lanes in a fixed order (DPP); every lane
// of the row gets it.
__device__ __forceinline__ double row16_sum(double x) {
    x += dpp_d<kDppQuadXor1>(x);
    x += dpp_d<kDppQuadXor2>(x);
    x += dpp_d<kDppRowHalfMirror>(x);
    x += dpp_d<kDppRowMirror>(x);
    return x;
}

// APO: APOLLO's moments on the projected gradient R (rank 256): the parameter
// stream is absent (a zero parameter, lr 1: the output would be the negated
// direction Rt), and each sub-tile -- one channel of 256 -- reduces sum Rt^2
// and sum R^2 over its rows of 16 lanes into LDS (csum); after the last
// sub-tile, lane k adds its channel's four row sums and forms the channel
// scale.
template <int G, int MC, int VC, int BV, bool FULL, bool APO>
__device__ __forceinline__ void adamw_compute(const AdamWLaunch& a, const DescG& d, int64_t e0, int64_t valid,
                                              int lane, double* lut, double* stab, uint2* skey, uint4* encp,
                                              double2* encd, double2* csum) {
    using Q = Geo<MC, VC, BV>;
    constexpr int K = Q::K;
    constexpr int NB = Q::NB;
    constexpr bool VQ = Q::VQ;
    constexpr int LEVELS = Q::LEVELS;

    using R = Raw<G, MC, VC, BV>;
    // first load phase and the old metadata are issued before any arithmetic
    R r;
    load_raw<G, MC, VC, BV, FULL, APO>(r, d, e0, valid, lane, 0);
    const OldMeta om = load_meta<MC, VC, BV, FULL>(d, e0, valid, lane);

    // ------------------------------------------------ 1. decode steps of the old metadata, one block per lane
    double num = 1.0, den = 1.0;
    if constexpr (MC == UF8) {
        if (lane < K) {
            num = (double)om.a;
            den = 127.0;
        }
    }
    if constexpr (VQ) {
        if (lane >= 32 && lane < 32 + NB) {
            num = (double)om.a;
            den = (double)LEVELS;
        }
    }
    const double q1 = num / den;  // UF8: absmax / 127; AL: delta / (L - 2)

    // Blocks of 512+ elements: decode through a per-block table of the 255
    // positive levels fl32(2^(l_min + k step)), k = 0..254, built in this
    // wavefront's LDS slice (4 levels per lane) from the block's 16 + 16
    // split factors below (32 evaluations per block instead of 255; a level is
    // one binary64 product, relative error below (ln 2 (|l_min| + 3 k st) + 5)
    // 2^-53 before the fp32 rounding). LDS traffic of one wavefront is ordered, so no barrier is
    // needed between building and reading its own tables.
    // Entry 0 holds 0.0 (code 0 is exact zero), entry q the level of code q,
    // kept in binary64 (the fp32 value widened) for the binary64 EMA.
    if constexpr (Q::LUT) {
        constexpr int NF = NB * 32;  // factor entries of the chunk (32 for one 2048 block)
#pragma unroll
        for (int i = 0; i < (NF + kWave - 1) / kWave; ++i) {
            // entry lane + 64 i belongs to block 2 i (lanes < 32) or 2 i + 1
            const int b0 = 2 * i, b1 = 2 * i + 1 < NB ? 2 * i + 1 : 2 * i;
            const double st0 = readlane_d(q1, 32 + b0), st1 = readlane_d(q1, 32 + b1);
            const float l0 = u2f(readlane_u(f2u(om.l), 32 + b0));
            const float l1 = u2f(readlane_u(f2u(om.l), 32 + b1));
            const double st = lane < 32 ? st0 : st1;
            const double v = split2_entry((double)(lane < 32 ? l0 : l1), st, lane & 31);
            if (lane + kWave * i < NF) stab[lane + kWave * i] = v;
        }
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const double* t = stab + b * 32;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int k = lane + 64 * i;
                const float lv = (float)split2_level(t, (uint32_t)k);
                lut[b * 256 + k] = k == 0 ? 0.0 : (double)lv;
            }
        }
    }

    // Blocks of 128 and 256 elements: a level table would cost one evaluation
    // per element. Instead, with the code q = 16 a + b (a, b in 0..15) of level
    // q - 1, 2^(l_min + (q - 1) step) = 2^(l_min + (16 a - 1) step) * 2^(b step):
    // entries [0, 16) of a block's split table hold the first factor, [16, 32)
    // the second, so a block costs 32 evaluations and an element one binary64
    // product indexed by the code's two nibbles (relative error below
    // (ln 2 (|l_min| + 3 (q - 1) st) + 5) 2^-53 against 2^E, then rounded to
    // fp32; code 0 is replaced by exact zero).
    if constexpr (Q::SPLIT) {
        static_assert(NB * 32 % kWave == 0, "split tables fill whole wavefront passes");
#pragma unroll
        for (int i = 0; i < NB * 32 / kWave; ++i) {
            // entry lane + 64 i belongs to block 2 i (lanes < 32) or 2 i + 1
            const double st0 = readlane_d(q1, 32 + 2 * i), st1 = readlane_d(q1, 33 + 2 * i);
            const float l0 = u2f(readlane_u(f2u(om.l), 32 + 2 * i));
            const float l1 = u2f(readlane_u(f2u(om.l), 33 + 2 * i));
            const double st = lane < 32 ? st0 : st1;
            stab[lane + kWave * i] = split2_entry((double)(lane < 32 ? l0 : l1), st, lane & 31);
        }
    }

    // Blocks of 64: with the code q = 64 a + 8 b + c (a < 4, b, c < 8),
    // 2^(l_min + (q - 1) step) = 2^(l_min + (64 a - 1) step) * 2^(8 b step) *
    // 2^(c step): 20 entries per block ([0, 4) first factor, [4, 12) second,
    // [12, 20) third), 5 evaluations per lane for the chunk's 16 blocks, and two
    // binary64 products per element (relative error below (ln 2 (|l_min| + 3 (q - 1)
    // st) + 7) 2^-53, then rounded to fp32).
    if constexpr (Q::SPLIT3) {
        static_assert(NB * 20 % kWave == 0, "three-factor tables fill whole wavefront passes");
#pragma unroll
        for (int i = 0; i < NB * 20 / kWave; ++i) {
            const int e = lane + kWave * i;
            const int b = e / 20, j = e - 20 * b;
            const double st = shfl_d(q1, 32 + b);
            const double l32 = (double)__shfl(om.l, 32 + b);
            stab[e] = split3_entry(l32, st, j);
        }
    }

    // ------------------------------------------------ 2. per sub-tile: decode, moments, parameter, momentum code
    // the new second moment waits in registers for its block's interval
    float vk[K][4];
    uint32_t vmn[Q::NSLOT], vmx[Q::NSLOT];
    uint32_t pmn = 0xFFFFFFFFu, pmx = 0u;
    // blocks of 256: the previous block's lane keys, and this lane's slot of
    // the chunk's reduced keys (lane 2b: block b's minimum, 2b + 1: its maximum)
    uint32_t qmn = 0xFFFFFFFFu, qmx = 0u, fitkey = 0u;
#pragma unroll
    for (int s = 0; s < Q::NSLOT; ++s) {
        vmn[s] = 0xFFFFFFFFu;
        vmx[s] = 0u;
    }
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int rel = k * kSub + 4 * lane;
        const int64_t e = e0 + rel;
        const int kk = k % R::P;  // slot of this sub-tile in the current load phase
        if (k > 0 && kk == 0) {
            __builtin_amdgcn_sched_barrier(0);  // keep the next phase's loads after this phase's arithmetic
            load_raw<G, MC, VC, BV, FULL, APO>(r, d, e0, valid, lane, k / R::P);
        }
        float mh[4], vh[4], mn[4], vn[4], pn[4];
        double vhd[4];  // the decoded second moment, widened for the EMA
        double r2 = 0.0;  // APO: this lane's sum of R^2
        if constexpr (MC == UF8) {
            const double mstep = readlane_d(q1, k);
#pragma unroll
            for (int j = 0; j < 4; ++j) mh[j] = uf8_decode((int32_t)(int8_t)(uint8_t)(r.m[kk] >> (8 * j)), mstep);
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) mh[j] = f4_at(r.m[kk], j);
        }
        if constexpr (Q::LUT) {
            const double* t = lut + (k * kSub / BV) * 256;
#pragma unroll
            for (int j = 0; j < 4; ++j) vhd[j] = t[(r.v[kk] >> (8 * j)) & 0xFFu];
        } else if constexpr (Q::SPLIT) {
            const double* t = stab + ((k * kSub + 4 * lane) / BV) * 32;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t q = (r.v[kk] >> (8 * j)) & 0xFFu;
                float lv = (float)split2_level(t, q);
                lv = q == 0u ? 0.0f : lv;
                opaque_f(lv);  // the code-0 select stays on the fp32 value (one select, not two after widening)
                vh[j] = lv;
            }
        } else if constexpr (Q::SPLIT3) {
            const double* t = stab + ((k * kSub + 4 * lane) / BV) * 20;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t q = (r.v[kk] >> (8 * j)) & 0xFFu;
                float lv = (float)split3_level(t, q);
                lv = q == 0u ? 0.0f : lv;
                opaque_f(lv);  // the code-0 select stays on the fp32 value (one select, not two after widening)
                vh[j] = lv;
            }
        } else if constexpr (VQ) {
            double vstep, vl32;
            if constexpr (BV >= kSub) {
                const int b = k * kSub / BV;
                vstep = readlane_d(q1, 32 + b);
                vl32 = (double)u2f(readlane_u(f2u(om.l), 32 + b));
            } else {
                const int src = 32 + (k * kSub + 4 * lane) / BV;
                vstep = shfl_d(q1, src);
                vl32 = (double)__shfl(om.l, src);
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                uint32_t q;
                if constexpr (VC == AL16)
                    q = ((j < 2 ? r.v[kk].x : r.v[kk].y) >> (16 * (j & 1))) & 0xFFFFu;
                else
                    q = (r.v[kk] >> (8 * j)) & 0xFFu;
                vh[j] = al_decode_fast(q, vl32, vstep, kExp2);
            }
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) vh[j] = f4_at(r.v[kk], j);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const double gd = (double)grad_at<G>(r.g[kk], j);
            if constexpr (APO) r2 += gd * gd;
            mn[j] = (float)(a.beta1 * (double)mh[j] + a.omb1 * gd);
            if constexpr (!Q::LUT) vhd[j] = (double)vh[j];
            vn[j] = (float)(a.beta2 * vhd[j] + a.omb2 * (gd * gd));
            const float den_p = __builtin_fmaf(__builtin_amdgcn_sqrtf(vn[j]), a.inv_sqrt_bc2, a.eps);
            const float upd = mn[j] * __builtin_amdgcn_rcpf(den_p);
            pn[j] = __builtin_fmaf(-a.step_size, upd, f4_at(r.p[kk], j) * a.decay);
        }
        if constexpr (!FULL) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (rel + j >= valid) mn[j] = vn[j] = 0.0f;  // absent: no state, no reduction input
        }
        if constexpr (APO) {
            // the channel of this sub-tile: sums of Rt^2 (Rt the fp32 direction) and R^2 per row of 16
            // lanes (absent elements have R = 0 and a zero direction)
            double t2 = 0.0;
#pragma unroll
            for (int j = 0; j < 4; ++j) t2 += (double)pn[j] * (double)pn[j];
            t2 = row16_sum(t2);
            r2 = row16_sum(r2);
            if ((lane & 15) == 0) csum[4 * k + (lane >> 4)] = make_double2(t2, r2);
        } else if constexpr (FULL) {
            st_f4<kNtStore>(d.p + e, make_float4(pn[0], pn[1], pn[2], pn[3]));
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (rel + j < valid) d.p[e + j] = pn[j];
        }
        // momentum: the UF8 block is this sub-tile
        if constexpr (MC == UF8) {
            uint32_t am = abs_bits(mn[0]);
#pragma unroll
            for (int j = 1; j < 4; ++j) am = OpMax::f(am, abs_bits(mn[j]));
            am = group_reduce<OpMax, 64>(am);
            const double rr = am != 0u ? rdiv127((double)u2f(am)) : 0.0;
            uint32_t q[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) q[j] = rint_low_bits((double)mn[j] * rr) & 0xFFu;
            if (FULL || k * kSub < valid) {
                store_codes4<UF8, FULL && kNtStore>(d.m, e, q);
                if (lane == 0) d.ms[e0 / kSub + k] = u2f(am);
            }
        } else if constexpr (FULL) {
            st_f4<kNtStore>(g_as<float>(d.m) + e, make_float4(mn[0], mn[1], mn[2], mn[3]));
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (rel + j < valid) g_as<float>(d.m)[e + j] = mn[j];
        }
        if constexpr (VQ) {
            // vn >= 0 here, so its bit pattern orders it; bits - 1 sends +0 to
            // the largest key, out of the positive minimum
            if constexpr (BV >= kSub) {
                // a block of whole sub-tiles: one running key pair, reduced over
                // the wavefront (to wave-uniform values) as soon as the block ends
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    vk[k][j] = vn[j];
                    pmn = OpMin::f(pmn, f2u(vn[j]) - 1u);
                    pmx = OpMax::f(pmx, f2u(vn[j]));
                }
                if constexpr (BV == kSub) {
                    // one block per sub-tile: the keys of two blocks at a time go
                    // through one reduce-scatter (below) instead of four reductions
                    if (k & 1) {
                        fitkey = key_pair_reduce(qmn, qmx, pmn, pmx, lane, k >> 1, fitkey);
                    } else {
                        qmn = pmn;
                        qmx = pmx;
                    }
                    pmn = 0xFFFFFFFFu;
                    pmx = 0u;
                } else if ((k + 1) * kSub % BV == 0) {
                    const int s = k * kSub / BV;
                    vmn[s] = group_reduce<OpMin, 64>(pmn) + 1u;  // back to bits; 0 when no positive
                    vmx[s] = group_reduce<OpMax, 64>(pmx);
                    pmn = 0xFFFFFFFFu;
                    pmx = 0u;
                }
            } else {
                // blocks inside the sub-tile: reduce each GL-lane group now and park
                // the keys in LDS, slot = block index within the chunk
                uint32_t tmn = 0xFFFFFFFFu, tmx = 0u;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    vk[k][j] = vn[j];
                    tmn = OpMin::f(tmn, f2u(vn[j]) - 1u);
                    tmx = OpMax::f(tmx, f2u(vn[j]));
                }
                tmn = group_reduce<OpMin, Q::GL>(tmn) + 1u;
                tmx = group_reduce<OpMax, Q::GL>(tmx);
                if (lane % Q::GL == 0) skey[k * Q::PER + lane / Q::GL] = make_uint2(tmn, tmx);
            }
        } else if constexpr (FULL) {
            st_f4<kNtStore>(g_as<float>(d.v) + e, make_float4(vn[0], vn[1], vn[2], vn[3]));
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (rel + j < valid) g_as<float>(d.v)[e + j] = vn[j];
        }
    }
    if constexpr (APO) {
        // ||Rt_c|| / (||R_c|| + 1e-8) and s_c^2 gn2_c of the chunk's K channels, lane k channel k
        __builtin_amdgcn_wave_barrier();  // this wavefront's LDS accesses run in order
        if (lane < K && (FULL || lane * kSub < valid)) {
            const double2 q0 = csum[4 * lane], q1 = csum[4 * lane + 1], q2 = csum[4 * lane + 2],
                          q3 = csum[4 * lane + 3];
            const double st = (q0.x + q1.x) + (q2.x + q3.x), sr = (q0.y + q1.y) + (q2.y + q3.y);
            const int64_t c = (e0 + lane * kSub) / kSub;
            const double sc = sqrt(st) / (sqrt(sr) + 1e-8);
            d.cs[c] = sc;
            d.csg[c] = sc * sc * d.cg2[c];
        }
    }
    if constexpr (VQ) {
        // -------------------------------------------- 3. block fits, one block per lane pair
        // lanes 2b, 2b+1 hold block b's min / max key; both compute its interval.
        uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
        const int b = lane >> 1;
        if constexpr (BV == kSub) {
            const uint32_t other = dpp<kDppQuadXor1>(fitkey);
            kmin = (lane & 1) ? other : fitkey;
            kmax = (lane & 1) ? fitkey : other;
        } else if constexpr (BV >= kSub) {
#pragma unroll
            for (int s = 0; s < NB; ++s) {
                kmin = (b == s) ? vmn[s] : kmin;
                kmax = (b == s) ? vmx[s] : kmax;
            }
        } else if (b < NB) {
            const uint2 kk = skey[b];
            kmin = kk.x;
            kmax = kk.y;
        }
        const bool any = kmax != 0u && b < NB;
        const uint32_t key = (lane & 1) ? kmax : kmin;
        const double lg = fit_log2(any ? u2f(key) : 1.0f);
        const double lg_other = __shfl_xor(lg, 1);
        const double lo = (lane & 1) ? lg_other : lg;
        const double hi = (lane & 1) ? lg : lg_other;
        const double l0 = lo > (double)a.v_floor ? lo : (double)a.v_floor;
        double l1 = hi < 126.0 ? hi : 126.0;
        if (kmin == kmax) l1 = l0 + 1.0;
        double dl = l1 - l0;
        dl = dl < 1e-12 ? 1e-12 : dl;
        if ((lane & 1) == 0 && b < NB && (FULL || (int64_t)b * BV < valid)) {
            *g_as<f2v>(d.vm + 2 * (e0 / BV + b)) = any ? f2v{(float)l0, (float)dl} : f2v{0.0f, 0.0f};
        }
        const double q2 = any ? (double)LEVELS / dl : 1.0;  // (L - 2) / delta
        if constexpr (VC == AL8 && BV < kSub) {
            // blocks inside a sub-tile: each block's encode parameters once, to LDS
            // (lane 2b), instead of two shuffles and the derivation per element group
            if ((lane & 1) == 0 && b < NB) {
                const ALEnc p = al_enc_params(l0, q2);
                encp[b] = make_uint4((uint32_t)p.I, f2u(p.fr32), f2u(p.inv32), f2u(p.guard32));
                encd[b] = make_double2(l0, q2);
            }
            __builtin_amdgcn_wave_barrier();  // this wavefront's LDS accesses run in order
        }

        // -------------------------------------------- 5. second-moment codes
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const int64_t e = e0 + k * kSub + 4 * lane;
            ALEnc enc;
            bool live;
            if constexpr (BV >= kSub) {
                const int bb = k * kSub / BV;
                enc = al_enc_params(readlane_d(l0, 2 * bb), readlane_d(q2, 2 * bb));
                live = FULL || (int64_t)bb * BV < valid;
            } else if constexpr (VC == AL8) {
                const int bb = (k * kSub + 4 * lane) / BV;
                live = FULL || (int64_t)bb * BV < valid;
                const uint4 pw = encp[bb];
                uint32_t q[4];
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    q[j] = al_encode_f32(vk[k][j], (int)pw.x, u2f(pw.y), u2f(pw.z), u2f(pw.w),
                                         [&] { return encd[bb]; });
                if (live) store_codes4<VC, FULL && kNtStore>(d.v, e, q);
                continue;
            } else {
                const int bb = (k * kSub + 4 * lane) / BV;
                enc = al_enc_params(shfl_d(l0, 2 * bb), shfl_d(q2, 2 * bb));
                live = FULL || (int64_t)bb * BV < valid;
            }
            uint32_t q[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                q[j] = VC == AL8 ? al_encode_f32(vk[k][j], enc) : al_encode_fast<LEVELS>(vk[k][j], enc);
            if (live) store_codes4<VC, FULL && kNtStore>(d.v, e, q);
        }
    }
}

// At least 4 waves per SIMD (at most 128 VGPRs) with a UF8 momentum: with one
// chunk per wave the step needs about 95-127 registers, and the extra resident
// waves hide HBM latency behind the per-element decode/encode arithmetic. An
// fp32 momentum carries 12 more registers per sub-tile and gets 3 (168), or 2
// with 2048-element AL16 chunks; AL8 blocks of 128 in 2048-element chunks get 3.
template <int MC, int VC, int BV>
constexpr int adamw_waves_per_eu() {
    return (MC == UF8 && !(VC == AL8 && BV == 128)) ? 4 : (VC == AL16 && Geo<MC, VC, BV>::C >= 2048 ? 2 : 3);
}

// largest ti with tb[ti] <= chunk (tb ascending, tb[0] = 0); wave-uniform, so
// every probe is a scalar load of the packed offsets (a few cache lines)
__device__ __forceinline__ int locate(cp<const int64_t> tb, int nt, int64_t chunk) {
    int lo = 0, hi = nt - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (tb[mid] <= chunk)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// One chunk per wave; each wave issues the loads of up to 4 sub-tiles
// (packed, 8 registers per sub-tile for bf16/UF8/AL8) before it computes on
// them. A chunk that ends a tensor takes the guarded path.
template <int G, int MC, int VC, int BV, bool APO>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(adamw_waves_per_eu<MC, VC, BV>())))
void adamw_kernel(const AdamWLaunch a) {
    constexpr int C = Geo<MC, VC, BV>::C;
    const int lane = threadIdx.x & 63;
    const int64_t chunk = a.chunk_base + xcd_order(blockIdx.x, gridDim.x) * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    constexpr int NT = Geo<MC, VC, BV>::LUT ? Geo<MC, VC, BV>::NB * 256 : 1;
    constexpr int NS = (Geo<MC, VC, BV>::SPLIT || Geo<MC, VC, BV>::LUT) ? Geo<MC, VC, BV>::NB * 32 : Geo<MC, VC, BV>::SPLIT3 ? Geo<MC, VC, BV>::NB * 20 : 1;
    constexpr int NK = (Geo<MC, VC, BV>::VQ && BV < kSub) ? Geo<MC, VC, BV>::NB : 1;
    __shared__ double lut_all[4][NT];
    __shared__ double stab_all[4][NS];
    __shared__ uint2 skey_all[4][NK];
    __shared__ uint4 encp_all[4][NK];     // blocks inside a sub-tile: fp32 encode parameters
    __shared__ double2 encd_all[4][NK];   // and {l_min, (L - 2) / delta} for the binary64 recheck
    __shared__ double2 csum_all[4][APO ? 4 * C / kSub : 1];  // APO: row sums of each channel
    double* lut = lut_all[threadIdx.x >> 6];
    double* stab = stab_all[threadIdx.x >> 6];
    uint2* skey = skey_all[threadIdx.x >> 6];
    uint4* encp = encp_all[threadIdx.x >> 6];
    double2* encd = encd_all[threadIdx.x >> 6];
    double2* csum = csum_all[threadIdx.x >> 6];
    if (chunk >= a.total_tiles) return;
    // the descriptor's pointers come from memory: mark them global so the
    // streams use global (not flat) loads and stores
    const cp<const AdamWDesc> D = (cp<const AdamWDesc>)a.D;
    const int ti = locate((cp<const int64_t>)a.tb, a.nt, chunk);
    DescG d = gview(D, ti);
    if constexpr (APO) {
        d.cs = to_g(a.apollo[ti].s);
        d.csg = to_g(a.apollo[ti].sg);
        d.cg2 = to_g((const double*)a.apollo[ti].gn2);
    }
    const int64_t e0 = (chunk - D[ti].tile_begin) * C;
    const int64_t valid = d.n - e0;
    if (valid >= C)
        adamw_compute<G, MC, VC, BV, true, APO>(a, d, e0, C, lane, lut, stab, skey, encp, encd, csum);
    else
        adamw_compute<G, MC, VC, BV, false, APO>(a, d, e0, valid, lane, lut, stab, skey, encp, encd, csum);
}

int adamw_tile_elems(int v_codec, int v_block) { return chunk_elems(v_codec, v_block); }

// al_diag_levels: every positive AL8 level of each block through the step
// kernel's split-table functions, as the binary64 product before the fp32
// rounding (kind 0: two factors, kind 1: three factors).
__global__ __launch_bounds__(256) void diag_levels_kernel(int kind, const float* __restrict__ meta, int64_t nblocks,
                                                          double* __restrict__ out) {
    const int64_t total = nblocks * 255;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
        const int64_t b = i / 255;
        const uint32_t q = 1u + (uint32_t)(i - b * 255);
        const double l32 = (double)meta[2 * b], st = (double)meta[2 * b + 1] / 254.0;
        if (kind == 0)
            out[i] = split2_product(split2_entry(l32, st, (int)(q >> 4)), split2_entry(l32, st, 16 + (int)(q & 15u)));
        else
            out[i] = split3_product(split3_entry(l32, st, (int)(q >> 6)),
                                    split3_entry(l32, st, 4 + (int)((q >> 3) & 7u)),
                                    split3_entry(l32, st, 12 + (int)(q & 7u)));
    }
}

hipError_t launch_diag_levels(int kind, const float* meta, int64_t nblocks, double* out, int grid_cap, hipStream_t s) {
    if (nblocks == 0) return hipSuccess;
    const int64_t want = (nblocks * 255 + 255) / 256;
    const int grid = (int)(want < grid_cap ? want : grid_cap);
    hipLaunchKernelGGL(diag_levels_kernel, dim3(grid), dim3(256), 0, s, kind, meta, nblocks, out);
    return hipGetLastError();
}

// ------------------------------------------------------------ descriptor table
struct AdamWDescBatch {
    int32_t count, offset;
    AdamWDesc d[kAdamWCopyBatch];
};

__global__ void adamw_desc_copy_kernel(const AdamWDescBatch b, AdamWDesc* dst, int64_t* tb) {
    constexpr int W = sizeof(AdamWDesc) / 8;
    const uint64_t* src = reinterpret_cast<const uint64_t*>(b.d);
    uint64_t* out = reinterpret_cast<uint64_t*>(dst + b.offset);
    for (int i = threadIdx.x; i < b.count * W; i += blockDim.x) out[i] = src[i];
    for (int i = threadIdx.x; i < b.count; i += blockDim.x) tb[b.offset + i] = b.d[i].tile_begin;
}

static constexpr size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

size_t adamw_table_bytes(int64_t nt) {
    return nt <= 0 ? 0 : align256((size_t)nt * sizeof(AdamWDesc)) + align256((size_t)nt * sizeof(int64_t));
}

static AdamWDesc* table_desc(void* table) { return static_cast<AdamWDesc*>(table); }
static int64_t* table_tb(void* table, int64_t nt) {
    return reinterpret_cast<int64_t*>(static_cast<char*>(table) + align256((size_t)nt * sizeof(AdamWDesc)));
}

hipError_t adamw_write_batch(const AdamWDesc* host, int count, int offset, void* table, int64_t nt, hipStream_t s) {
    static_assert(sizeof(AdamWDesc) % 8 == 0, "descriptor size");
    static_assert(sizeof(AdamWDescBatch) <= 4096 - 64, "copy arguments");
    AdamWDescBatch b;
    b.count = count;
    b.offset = offset;
    for (int i = 0; i < count; ++i) b.d[i] = host[i];
    hipLaunchKernelGGL(adamw_desc_copy_kernel, dim3(1), dim3(256), 0, s, b, table_desc(table), table_tb(table, nt));
    return hipGetLastError();
}

void adamw_bind_table(void* table, int64_t nt, AdamWLaunch& a) {
    a.D = table_desc(table);
    a.tb = table_tb(table, nt);
    a.nt = (int32_t)nt;
}

hipError_t adamw_write_table(const AdamWDesc* host, int nt, void* table, AdamWLaunch& a, hipStream_t s) {
    for (int off = 0; off < nt; off += kAdamWCopyBatch) {
        const hipError_t e = adamw_write_batch(host + off, nt - off < kAdamWCopyBatch ? nt - off : kAdamWCopyBatch,
                                               off, table, nt, s);
        if (e != hipSuccess) return e;
    }
    adamw_bind_table(table, nt, a);
    return hipSuccess;
}

// The descriptor table of the allocation-free entry point: a fixed device
// array (one copy per GPU, alive until the process ends). Host code reaches
// it only through the device address hipGetSymbolAddress returns; the array's
// name in host code is a stand-in, not a device pointer.
static __device__ __align__(256) unsigned char scratch[kAdamWScratchBytes];
static_assert(kAdamWScratchBytes == align256((size_t)kAdamWStaticTensors * sizeof(AdamWDesc)) +
                                        align256((size_t)kAdamWStaticTensors * sizeof(int64_t)),
              "static table size");

hipError_t adamw_static_table(void** table) {
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(mu);
    if (!addr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = p;
    }
    *table = addr[dev];
    return hipSuccess;
}

// One wave per chunk: the grid covers every chunk of the launch and the
// hardware dispatcher refills each CU as its waves retire; each XCD walks a
// contiguous eighth of the chunks (xcd_order). (A persistent grid
// sized by occupancy moves the same byte mix about 6% slower on gfx950, and a
// chunk loop lets the compiler hoist per-chunk constants into spilled
// registers.) Lists beyond 2^32 chunks take several launches.
template <int G, int MC, int VC, int BV, bool APO>
static hipError_t launch_t(const AdamWLaunch& a, hipStream_t s) {
    constexpr int64_t kMaxGrid = int64_t(1) << 30;  // workgroups (4 waves each) per launch
    AdamWLaunch b = a;
    for (b.chunk_base = 0; b.chunk_base < a.total_tiles; b.chunk_base += 4 * kMaxGrid) {
        const int64_t left = (a.total_tiles - b.chunk_base + 3) / 4;
        const int64_t grid = left < kMaxGrid ? left : kMaxGrid;
        hipLaunchKernelGGL((adamw_kernel<G, MC, VC, BV, APO>), dim3((unsigned)grid), dim3(256), 0, s, b);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <int G, int MC, int VC, bool APO>
static hipError_t launch_bv(const AdamWLaunch& a, int bv, hipStream_t s) {
    if constexpr (VC == FP32) {
        return launch_t<G, MC, VC, 256, APO>(a, s);
    } else {
        switch (bv) {
            case 64: return launch_t<G, MC, VC, 64, APO>(a, s);
            case 128: return launch_t<G, MC, VC, 128, APO>(a, s);
            case 256: return launch_t<G, MC, VC, 256, APO>(a, s);
            case 512: return launch_t<G, MC, VC, 512, APO>(a, s);
            case 1024: return launch_t<G, MC, VC, 1024, APO>(a, s);
            case 2048: return launch_t<G, MC, VC, 2048, APO>(a, s);
        }
        return hipErrorInvalidValue;
    }
}

template <int G, int MC, bool APO>
static hipError_t launch_vc(const AdamWLaunch& a, int vc, int bv, hipStream_t s) {
    switch (vc) {
        case AL8: return launch_bv<G, MC, AL8, APO>(a, bv, s);
        case AL16: return launch_bv<G, MC, AL16, APO>(a, bv, s);
        case FP32: return launch_bv<G, MC, FP32, APO>(a, bv, s);
    }
    return hipErrorInvalidValue;
}

template <int G, bool APO>
static hipError_t launch_mc(const AdamWLaunch& a, int mc, int vc, int bv, hipStream_t s) {
    switch (mc) {
        case UF8: return launch_vc<G, UF8, APO>(a, vc, bv, s);
        case FP32: return launch_vc<G, FP32, APO>(a, vc, bv, s);
    }
    return hipErrorInvalidValue;
}

// apollo: APOLLO's projected moments at rank 256 (fp32 gradient R, no parameter
// stream, channel scales out; see AdamWLaunch::apollo).
hipError_t launch_adamw(const AdamWLaunch& a, int grad_dtype, int m_codec, int v_codec, int v_block, hipStream_t s,
                        bool apollo) {
    if (apollo) {
        if (grad_dtype != G_F32 || !a.apollo) return hipErrorInvalidValue;
        return launch_mc<G_F32, true>(a, m_codec, v_codec, v_block, s);
    }
    if (grad_dtype == G_BF16) return launch_mc<G_BF16, false>(a, m_codec, v_codec, v_block, s);
    return launch_mc<G_F32, false>(a, m_codec, v_codec, v_block, s);
}

}  // namespace al
