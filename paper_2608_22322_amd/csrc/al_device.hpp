// Device helpers shared by the gfx950 kernels: cross-lane reductions on a
// 64-wide wavefront, bfloat16 unpacking, and the per-element / per-block
// pieces of the AL and UF8 codes.
//
// Every kernel maps 4 consecutive elements to a lane, so a wavefront covers
// 256 consecutive elements (a "sub-tile"). A block of B <= 256 elements then
// spans B/4 lanes (16, 32 or 64); a larger block spans B/256 sub-tiles held
// in registers by one wavefront.
//
// The sources are built with -ffp-contract=off: every binary64 expression
// below rounds after each operation, in the order written, which is what
// makes the fp32-rounded states reproducible bit for bit.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace al {

constexpr int kWave = 64;
constexpr int kSub = 256;  // elements per wavefront sub-tile (4 per lane)

enum Codec : int { FP32 = 0, AL8 = 1, AL16 = 2, UF8 = 3 };
enum GradT : int { G_F32 = 0, G_BF16 = 1 };

// ---------------------------------------------------------------- bit casts
__device__ __forceinline__ uint32_t f2u(float x) { return __builtin_bit_cast(uint32_t, x); }
__device__ __forceinline__ float u2f(uint32_t x) { return __builtin_bit_cast(float, x); }
__device__ __forceinline__ float bf16_to_f32(uint32_t b16) { return u2f(b16 << 16); }

// ------------------------------------------------------- cross-lane helpers
// DPP control words (GCN/CDNA "dpp_ctrl"): quad permutations, row mirrors.
constexpr int kDppQuadXor1 = 0xB1;      // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;      // quad_perm [2,3,0,1]
constexpr int kDppRowHalfMirror = 0x141;  // lane i -> 7-i within 8
constexpr int kDppRowMirror = 0x140;      // lane i -> 15-i within 16
// ds_swizzle bit mode: and_mask 0x1F, xor_mask m -> lane ^ m within 32
constexpr int kSwzXor4 = 0x101F;
constexpr int kSwzXor8 = 0x201F;
constexpr int kSwzXor16 = 0x401F;

// Every control word above reads a lane of the same row, so no lane is out of
// range and bound_ctrl changes nothing; with it set the compiler folds the move
// into the consuming operation (v_min_u32_dpp etc.), one instruction per step.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, true);
}

struct OpMax {
    __device__ static uint32_t f(uint32_t a, uint32_t b) { return a > b ? a : b; }
};
struct OpMin {
    __device__ static uint32_t f(uint32_t a, uint32_t b) { return a < b ? a : b; }
};

// Reduce over aligned groups of LANES lanes (16, 32 or 64). Every lane gets
// its group's result; for 64 the result is wave-uniform.
template <class Op, int LANES>
__device__ __forceinline__ uint32_t group_reduce(uint32_t x) {
    static_assert(LANES == 16 || LANES == 32 || LANES == 64, "group size");
    x = Op::f(x, dpp<kDppQuadXor1>(x));
    x = Op::f(x, dpp<kDppQuadXor2>(x));
    x = Op::f(x, dpp<kDppRowHalfMirror>(x));
    x = Op::f(x, dpp<kDppRowMirror>(x));
    if constexpr (LANES >= 32) x = Op::f(x, (uint32_t)__builtin_amdgcn_ds_swizzle((int)x, kSwzXor16));
    if constexpr (LANES == 64) {
        uint32_t a = (uint32_t)__builtin_amdgcn_readlane((int)x, 0);
        uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)x, 32);
        x = Op::f(a, b);
    }
    return x;
}

// ------------------------------------------------------------------ AL code
// Fitted interval of one block from its exact positive min / max bit
// patterns (0 max means "no positive value").
struct ALFit {
    double lmin;   // unrounded binary64 l_min
    double delta;  // unrounded binary64 width
    bool any;
};

__device__ __forceinline__ ALFit al_fit(uint32_t min_bits, uint32_t max_bits, float log_floor) {
    ALFit f;
    f.any = max_bits != 0u;
    if (!f.any) {
        f.lmin = 0.0;
        f.delta = 0.0;
        return f;
    }
    double lo = log2((double)u2f(min_bits));
    double hi = log2((double)u2f(max_bits));
    double l0 = lo > (double)log_floor ? lo : (double)log_floor;
    double l1 = hi < 126.0 ? hi : 126.0;
    if (min_bits == max_bits) l1 = l0 + 1.0;
    double d = l1 - l0;
    if (d < 1e-12) d = 1e-12;
    f.lmin = l0;
    f.delta = d;
    return f;
}

// Code of one element under a fitted interval; LEVELS = L - 2.
template <int LEVELS>
__device__ __forceinline__ uint32_t al_encode(float x, const ALFit& f) {
    if (!(x > 0.0f)) return 0u;
    double z = (log2((double)x) - f.lmin) / f.delta;
    z = z < 0.0 ? 0.0 : z;
    z = z > 1.0 ? 1.0 : z;
    double y = (double)LEVELS * z;
    return 1u + (uint32_t)__builtin_rint(y);
}

// Decode of one code from the stored fp32 metadata: step = delta32 / (L-2),
// value = fl32(2^(lmin32 + (q-1) * step)).
__device__ __forceinline__ float al_decode(uint32_t q, double lmin32, double step) {
    if (q == 0u) return 0.0f;
    double e = lmin32 + (double)(q - 1u) * step;
    return (float)exp2(e);
}

// ------------------------------------------------- fast binary64 exp2 / encode
// 2^E in binary64 for |E| < 1000: E = n + f with n = rint(E), |f| <= 1/2, and
// 2^f = e^(f ln 2) by its Taylor series to degree 13 (coefficients
// (ln 2)^k / k!, rounded to binary64); relative error <= 1.4e-16 over the
// range, i.e. about one ulp, so fl32 of it equals fl32 of a faithfully
// rounded exp2 except within ~1e-16 of an fp32 rounding midpoint.
// The coefficients travel in the kernel arguments or in constant memory, so
// they are read with scalar loads and each Horner step is one v_fma_f64 with a
// scalar-register addend (there are no 64-bit literal operands on this ISA; as
// immediates the compiler keeps them in vector registers and copies one per
// step).
struct Exp2Coef {
    double c[14];  // (ln 2)^k / k!, k = 0..13, rounded to binary64
};

// (ln 2)^k / k!, k = 0..13, rounded to binary64: the Taylor coefficients of
// 2^f = e^(f ln 2).
#define AL_EXP2_TAYLOR                                                                                      \
    {                                                                                                       \
        {1.0, 0x1.62e42fefa39efp-1, 0x1.ebfbdff82c58fp-3, 0x1.c6b08d704a0c0p-5, 0x1.3b2ab6fba4e77p-7,         \
         0x1.5d87fe78a6731p-10, 0x1.430912f86c787p-13, 0x1.ffcbfc588b0c7p-17, 0x1.62c0223a5c824p-20,          \
         0x1.b5253d395e7c4p-24, 0x1.e4cf5158b8ecap-28, 0x1.e8cac7351bb25p-32, 0x1.c3bd650fc2986p-36,          \
         0x1.816193166d0f9p-40}                                                                             \
    }

__device__ __forceinline__ double exp2_d(double E, const Exp2Coef& cf) {
    const double n = __builtin_rint(E);
    const double f = E - n;
    double p = cf.c[13];
#pragma unroll
    for (int k = 12; k >= 0; --k) p = __builtin_fma(p, f, cf.c[k]);
    return __builtin_amdgcn_ldexp(p, (int)n);
}

// Branch-free: code 0 evaluates level 0 and is then replaced by exact zero.
__device__ __forceinline__ float al_decode_fast(uint32_t q, double lmin32, double step, const Exp2Coef& cf) {
    const uint32_t k = q == 0u ? 0u : q - 1u;
    const float v = (float)exp2_d(lmin32 + (double)k * step, cf);
    return q == 0u ? 0.0f : v;
}

// Bound on |log2f_hw(m) - log2(m)| for m in [1/2, 1), the hardware fp32 log2
// on a mantissa (measured exhaustively on the device by the diagnostic test,
// which requires the measured maximum to stay below a quarter of this).
constexpr double kLog2MantErr = 0x1p-21;

// log2 x in binary64 for x a positive fp32 value (the block endpoints of the
// second-moment codes), in well under half the instructions of the general
// binary64 log2: x = 2^e m with m in [sqrt(1/2), sqrt(2)), s = (m - 1) / (m + 1)
// (m - 1 and m + 1 exact; the quotient by a refined reciprocal and one
// remainder correction, its residual carried as s_lo), and
// ln m = 2 atanh s = 2 s (1 + z Q(z)), z = s^2, Q(z) = 1/3 + z/5 + ... + z^9/21
// (|s| <= 0.1716: the first omitted term is below 2^-57 relative). With
// K = 2 / ln 2 = Kh + Kl, log2 x = e + K s (1 + z Q): the leading product
// Kh s and its sum with e are carried exactly (FMA product error, Fast2Sum),
// the small remainder terms (Kl s, Kh s_lo, Kh s z Q) are added to the error
// terms, and the result is rounded once: correctly rounded except within a
// few hundredths of an ulp of a rounding midpoint. The device test holds it to
// the host's log2 on every fp32 significand of three binades and on random
// fp32 values.
__device__ __forceinline__ double fit_log2(float xf) {
    const double x = (double)xf;
    double m = __builtin_amdgcn_frexp_mant(x);  // [1/2, 1)
    int e = __builtin_amdgcn_frexp_exp(x);
    const bool lo = m < 0x1.6a09e667f3bcdp-1;
    m = lo ? 2.0 * m : m;
    e = lo ? e - 1 : e;
    const double num = m - 1.0, den = m + 1.0;
    double r = __builtin_amdgcn_rcp(den);
    r = __builtin_fma(__builtin_fma(-den, r, 1.0), r, r);
    r = __builtin_fma(__builtin_fma(-den, r, 1.0), r, r);
    const double s0 = num * r;
    const double s = __builtin_fma(__builtin_fma(-den, s0, num), r, s0);
    const double s_lo = __builtin_fma(-den, s, num) * r;  // num / den - s, to first order
    const double z = s * s;
    double q = 1.0 / 21.0;
    q = __builtin_fma(q, z, 1.0 / 19.0);
    q = __builtin_fma(q, z, 1.0 / 17.0);
    q = __builtin_fma(q, z, 1.0 / 15.0);
    q = __builtin_fma(q, z, 1.0 / 13.0);
    q = __builtin_fma(q, z, 1.0 / 11.0);
    q = __builtin_fma(q, z, 1.0 / 9.0);
    q = __builtin_fma(q, z, 1.0 / 7.0);
    q = __builtin_fma(q, z, 1.0 / 5.0);
    q = __builtin_fma(q, z, 1.0 / 3.0);
    constexpr double kKh = 0x1.71547652b82fep+1;   // 2 / ln 2 rounded to binary64
    constexpr double kKl = 0x1.777d0ffda0d24p-55;  // 2 / ln 2 - kKh
    const double hi = s * kKh;
    double tail = __builtin_fma(s, kKh, -hi);  // exact error of hi
    tail += __builtin_fma(s_lo, kKh, s * kKl);
    tail = __builtin_fma(hi, z * q, tail);
    const double ed = (double)e;
    const double sum = ed + hi;
    const double err = (ed - sum) + hi;  // Fast2Sum: |e| >= |hi| or e = 0
    return sum + (err + tail);
}

// Per-block encode parameters: the binary64 interval start, LEVELS/delta,
// and a guard band on the code position (binary64 and fp32 arithmetic).
struct ALEnc {
    double lmin;
    double inv;    // (L - 2) / delta
    double fr;     // lmin - floor(lmin), exact
    double guard;  // bound on |fast position - binary64 position|
    int I;         // floor(lmin)
    float inv32, fr32, guard32;  // the fp32 path (AL8): fl32(inv), fl32(fr), its guard
};

__device__ __forceinline__ ALEnc al_enc_params(double lmin, double inv) {
    ALEnc p;
    p.lmin = lmin;
    p.inv = inv;
    const double I = __builtin_floor(lmin);
    p.I = (int)I;
    p.fr = lmin - I;
    p.guard = inv * kLog2MantErr + 1e-9;
    // fp32 path: |y32 - y| <= inv (kLog2MantErr + 2^-24 + 2^-25) + 3 * 2^-24 |y| (the mantissa log,
    // the fp32 rounding of fr and of l - fr, and three relative roundings of at most 2^-24: d, inv, the
    // product); only |y| <= 255 decides a code (beyond it both sides clamp), so 1.25 * 2^-21 inv +
    // 2^-14 bounds it
    p.inv32 = (float)inv;
    p.fr32 = (float)p.fr;
    p.guard32 = (float)(inv * 0x1.4p-21 + 0x1p-14);
    return p;
}

// Code of x > 0 (0 for x <= 0). The position y = LEVELS * (log2 x - lmin) /
// delta comes from x = mant * 2^ex: y = ((ex - I) + (log2f_hw(mant) - fr)) *
// inv, whose only sizeable error is the fp32 mantissa log (kLog2MantErr); a
// position within that guard of a rounding boundary is recomputed with the
// binary64 log2, so the rounding decision is the binary64 one.
template <int LEVELS>
__device__ __forceinline__ uint32_t al_encode_fast(float x, const ALEnc& p) {
    const float mant = __builtin_amdgcn_frexp_mantf(x);
    const int ex = __builtin_amdgcn_frexp_expf(x);
    const float l = __builtin_amdgcn_logf(mant);
    const double d = (double)(ex - p.I) + ((double)l - p.fr);
    double yc = __builtin_fmin(__builtin_fmax(d * p.inv, 0.0), (double)LEVELS);
    double r = __builtin_rint(yc);
    if (__builtin_fabs(yc - r) > 0.5 - p.guard) {
        const double ys = (log2((double)x) - p.lmin) * p.inv;
        yc = __builtin_fmin(__builtin_fmax(ys, 0.0), (double)LEVELS);
        r = __builtin_rint(yc);
    }
    return x > 0.0f ? 1u + (uint32_t)r : 0u;
}

// AL8 code of x with the fast position in fp32 arithmetic (AL8 positions are
// at most 254, so fp32 carries them to about 2^-16); the guard band of
// al_enc_params covers the fp32 roundings, and positions inside it take the
// same binary64 recheck as al_encode_fast, so every rounding decision is the
// binary64 one.
// SLOW() returns {lmin, inv} for the recheck (read only when it is needed).
template <class Slow>
__device__ __forceinline__ uint32_t al_encode_f32(float x, int I, float fr32, float inv32, float guard32, Slow slow) {
    constexpr float L = 254.0f;
    const float mant = __builtin_amdgcn_frexp_mantf(x);
    const int ex = __builtin_amdgcn_frexp_expf(x);
    const float l = __builtin_amdgcn_logf(mant);
    const float d = (float)(ex - I) + (l - fr32);
    float yc = __builtin_fminf(__builtin_fmaxf(d * inv32, 0.0f), L);
    float r = __builtin_rintf(yc);
    if (__builtin_fabsf(yc - r) > 0.5f - guard32) {
        const double2 li = slow();
        const double ys = (log2((double)x) - li.x) * li.y;
        r = (float)__builtin_rint(__builtin_fmin(__builtin_fmax(ys, 0.0), 254.0));
    }
    return x > 0.0f ? 1u + (uint32_t)r : 0u;
}

__device__ __forceinline__ uint32_t al_encode_f32(float x, const ALEnc& p) {
    return al_encode_f32(x, p.I, p.fr32, p.inv32, p.guard32, [&] { return make_double2(p.lmin, p.inv); });
}

// fl32(x / d) from a precomputed rd = fl64(1 / d). q = fl64(x * rd) lies
// within 2.5 binary64 ulps of fl64(x / d), so the two round to the same fp32
// value unless q is that close to an fp32 rounding midpoint (its 29 low
// mantissa bits near 2^28) or |fl32(q)| is not above FLT_MIN (subnormal
// results round on a coarser grid; FLT_MIN itself may be the rounding of a
// subnormal-range q); those rare cases take the binary64 division. An
// infinite fl32(q) passes: the overflow threshold is the midpoint above
// FLT_MAX, which the low-bit test catches; a NaN fails. The conditions
// combine as lane masks, with no short-circuit branches.
__device__ __forceinline__ bool quotient_ok(double q, float f) {
    const uint32_t low = (uint32_t)__builtin_bit_cast(uint64_t, q) & 0x1FFFFFFFu;
    return (q == 0.0) | ((__builtin_fabsf(f) > 0x1p-126f) & (low - 0x0FFFFFF8u > 16u));
}

__device__ __forceinline__ float div_to_f32(double x, double d, double rd) {
    const double q = x * rd;
    const float f = (float)q;
    if (__builtin_expect(quotient_ok(q, f), 1)) return f;
    return (float)(x / d);
}

// Four quotients at once, with one (rarely taken) branch for the fallbacks.
__device__ __forceinline__ void div4_to_f32(const double x[4], double d, double rd, float out[4]) {
    bool ok[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const double q = x[j] * rd;
        out[j] = (float)q;
        ok[j] = quotient_ok(q, out[j]);
    }
    if (__builtin_expect(!(ok[0] & ok[1] & ok[2] & ok[3]), 0)) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (!ok[j]) out[j] = (float)(x[j] / d);
    }
}

// fp32 roundings of N approximate quotients. Each q_j lies within 8 binary64
// ulps of the binary64 quotient fl64(x_j / d) whose fp32 rounding is wanted
// (q_j = fl64(fl64(fl64(r * fl64(1 / d)) * c_j) * g_j) against x_j =
// fl64(fl64(r * c_j) * g_j): four roundings against three, 7 ulps). f_j =
// fl32(q_j), and the result is true when every f_j is that rounding: bits
// 0..28 of q_j (the ones the fp32 rounding drops) are more than kQuotW from
// the halfway pattern 2^28, and |q_j| is at least 2^-126 (1 + 2^-20) (the fp32
// normal range with a margin) or below the binary64 normal range (zero, or a
// quotient that rounds to zero either way). Both tests are unsigned minima
// over the N quotients (v_min3 chains), one compare each, with no per-element
// lane masks. Infinities pass (the overflow threshold is the midpoint above
// FLT_MAX, caught by the first test), NaNs pass and stay NaN.
constexpr uint32_t kQuotW = 32;
__device__ __forceinline__ uint32_t umin32(uint32_t a, uint32_t b) { return a < b ? a : b; }
template <int N>
__device__ __forceinline__ bool f32_roundings_decided(const double q[N], float f[N]) {
    uint32_t mk = 0xFFFFFFFFu, mz = 0xFFFFFFFFu;
#pragma unroll
    for (int j = 0; j < N; ++j) {
        f[j] = (float)q[j];
        const uint2 b = __builtin_bit_cast(uint2, q[j]);  // (low word, high word)
        // ((bits 0..28) - (2^28 - W)) mod 2^29, times 8: at most 16 W iff within W of 2^28
        mk = umin32(mk, (b.x << 3) - ((0x10000000u - kQuotW) << 3));
        // 2 |high word| - 1: 2^32 - 1 for a zero high word; above 0x70200000 iff |q| >= 2^-126 (1 + 2^-20).
        // Written as the instruction: from C the compiler sees bits 32..63 of q shifted, and emits a
        // 64-bit funnel shift, a mask and an add.
        uint32_t z;
        __asm__("v_lshl_add_u32 %0, %1, 1, -1" : "=v"(z) : "v"(b.y));
        mz = umin32(mz, z);
    }
    return (mk > 16u * kQuotW) & (mz > 0x70200000u);
}

// As f32_roundings_decided, with the range test known to pass for every q_j
// (each q_j zero or at least 2^-126 (1 + 2^-20) in magnitude): the midpoint
// test alone.
template <int N>
__device__ __forceinline__ bool f32_midpoints_decided(const double q[N], float f[N]) {
    uint32_t mk = 0xFFFFFFFFu;
#pragma unroll
    for (int j = 0; j < N; ++j) {
        f[j] = (float)q[j];
        const uint2 b = __builtin_bit_cast(uint2, q[j]);
        mk = umin32(mk, (b.x << 3) - ((0x10000000u - kQuotW) << 3));
    }
    return mk > 16u * kQuotW;
}

// Cross-lane moves of 64-bit values.
__device__ __forceinline__ double shfl_d(double v, int src) { return __shfl(v, src); }
__device__ __forceinline__ double readlane_d(double v, int lane) {
    const uint64_t b = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, lane);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), lane);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ uint32_t readlane_u(uint32_t v, int lane) {
    return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}

// ---------------------------------------------------- double-double sums
// Sums of non-negative binary64 terms carried as (hi, lo) with TwoSum
// (Knuth): hi + lo equals the exact sum up to ~n 2^-106 relative, so
// fl64(hi + lo) is the correctly rounded exact sum except within that of a
// rounding boundary, whatever the order of accumulation.
struct DD {
    double hi, lo;
};

__device__ __forceinline__ void dd_add(DD& a, double x) {
    const double s = a.hi + x;
    const double bp = s - a.hi;
    const double e = (a.hi - (s - bp)) + (x - bp);
    a.hi = s;
    a.lo += e;
}

__device__ __forceinline__ DD dd_merge(DD a, DD b) {
    const double s = a.hi + b.hi;
    const double bp = s - a.hi;
    double e = (a.hi - (s - bp)) + (b.hi - bp);
    e += a.lo + b.lo;
    const double hi = s + e;
    return DD{hi, e - (hi - s)};
}

__device__ __forceinline__ double dd_value(DD a) { return a.hi + a.lo; }

__device__ __forceinline__ DD dd_shfl_xor(DD a, int m) { return DD{__shfl_xor(a.hi, m), __shfl_xor(a.lo, m)}; }

// Double-double of the partner lane within a quad (DPP, no LDS traffic):
// CTRL = kDppQuadXor1 or kDppQuadXor2.
template <int CTRL>
__device__ __forceinline__ DD dd_quad_xor(DD a) {
    const uint64_t h = __builtin_bit_cast(uint64_t, a.hi), l = __builtin_bit_cast(uint64_t, a.lo);
    const uint64_t h2 = ((uint64_t)dpp<CTRL>((uint32_t)(h >> 32)) << 32) | dpp<CTRL>((uint32_t)h);
    const uint64_t l2 = ((uint64_t)dpp<CTRL>((uint32_t)(l >> 32)) << 32) | dpp<CTRL>((uint32_t)l);
    return DD{__builtin_bit_cast(double, h2), __builtin_bit_cast(double, l2)};
}

// A binary64 value of another lane of the same DPP row (CTRL: a quad
// permutation or a row mirror).
template <int CTRL>
__device__ __forceinline__ double dpp_d(double x) {
    const uint64_t b = __builtin_bit_cast(uint64_t, x);
    return __builtin_bit_cast(double, ((uint64_t)dpp<CTRL>((uint32_t)(b >> 32)) << 32) | dpp<CTRL>((uint32_t)b));
}

// Wave-wide merge; every lane gets the total (fixed butterfly order).
__device__ __forceinline__ DD dd_wave_sum(DD a) {
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) a = dd_merge(a, dd_shfl_xor(a, m));
    return a;
}

// ----------------------------------------------------------------- UF8 code
// The low byte of rint(y) in two's complement, for |y| <= 2^51: adding
// 1.5 2^52 rounds y to an integer in the sum's last place (to nearest even,
// as rint does), and the sum's low word is then 2^51 + rint(y). One binary64
// addition in place of a rounding and a conversion.
__device__ __forceinline__ uint32_t rint_low_bits(double y) {
    return (uint32_t)__builtin_bit_cast(uint64_t, y + 0x1.8p52);
}

// Encode with r = 127 / absmax (binary64), y = x * r, round to nearest even,
// clamp to [-127, 127].
__device__ __forceinline__ int32_t uf8_encode(float x, double r) {
    double y = (double)x * r;
    double q = __builtin_rint(y);
    q = q > 127.0 ? 127.0 : q;
    q = q < -127.0 ? -127.0 : q;
    return (int32_t)q;
}

// fl64(x / 127) without a division, for x a finite fp32 value held in
// binary64. q = fl64(x * R), R = fl64(1/127), is within about an ulp of the
// quotient; the remainder x - 127 q is a small multiple of ulp(q), so the fma
// forms it exactly, and one correction step q + rem * R gives the correctly
// rounded quotient (Markstein's correction; R's significand is not all ones).
// Scaling x by 2^k scales every step exactly, so the device test over all fp32
// significands covers every such x.
__device__ __forceinline__ double div127(double x) {
    constexpr double R = 1.0 / 127.0;
    const double q = x * R;
    const double rem = __builtin_fma(-q, 127.0, x);
    return __builtin_fma(rem, R, q);
}

// fl64(127 / x) for x a positive finite fp32 value held in binary64: the
// hardware reciprocal, two Newton steps, and the same remainder correction
// as div127 (a third of the instructions of the general binary64 division,
// whose scaling steps guard ranges an fp32 x never reaches). Checked against
// the IEEE quotient on the device over all fp32 significands.
__device__ __forceinline__ double rdiv127(double x) {
    double r = __builtin_amdgcn_rcp(x);
    r = __builtin_fma(__builtin_fma(-x, r, 1.0), r, r);
    r = __builtin_fma(__builtin_fma(-x, r, 1.0), r, r);
    const double q = 127.0 * r;
    const double rem = __builtin_fma(-x, q, 127.0);
    return __builtin_fma(rem, r, q);
}

// Decode with step = absmax / 127 (binary64): fl32(q * step).
__device__ __forceinline__ float uf8_decode(int32_t q, double step) { return (float)((double)q * step); }

__device__ __forceinline__ uint32_t abs_bits(float x) { return f2u(x) & 0x7FFFFFFFu; }
// For the positive minimum: zero (and -0) map to the largest key.
__device__ __forceinline__ uint32_t pos_min_key(float x) {
    uint32_t b = f2u(x);
    return (b == 0u || (b & 0x80000000u)) ? 0xFFFFFFFFu : b;
}
__device__ __forceinline__ uint32_t pos_max_key(float x) {
    uint32_t b = f2u(x);
    return (b & 0x80000000u) ? 0u : b;
}

// ------------------------------------------------------- packed 4-wide I/O
struct F4 {
    float v[4];
};

__device__ __forceinline__ F4 load_f4(const float* p) {
    float4 t = *reinterpret_cast<const float4*>(p);
    return F4{{t.x, t.y, t.z, t.w}};
}
__device__ __forceinline__ void store_f4(float* p, const F4& x) {
    *reinterpret_cast<float4*>(p) = make_float4(x.v[0], x.v[1], x.v[2], x.v[3]);
}

// Gradients: 4 consecutive elements as fp32.
template <int G>
__device__ __forceinline__ F4 load_grad4(const void* g, int64_t e) {
    if constexpr (G == G_BF16) {
        uint2 w = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(g) + e);
        return F4{{bf16_to_f32(w.x & 0xFFFFu), bf16_to_f32(w.x >> 16), bf16_to_f32(w.y & 0xFFFFu),
                   bf16_to_f32(w.y >> 16)}};
    } else {
        return load_f4(reinterpret_cast<const float*>(g) + e);
    }
}

template <int G>
__device__ __forceinline__ float load_grad1(const void* g, int64_t e) {
    if constexpr (G == G_BF16)
        return bf16_to_f32(reinterpret_cast<const uint16_t*>(g)[e]);
    else
        return reinterpret_cast<const float*>(g)[e];
}

// Codes: 4 consecutive codes as unsigned (AL) or signed (UF8) integers.
template <int C>
__device__ __forceinline__ void load_codes4(const void* c, int64_t e, uint32_t q[4]) {
    if constexpr (C == AL8 || C == UF8) {
        uint32_t w = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const uint8_t*>(c) + e);
        q[0] = w & 0xFFu;
        q[1] = (w >> 8) & 0xFFu;
        q[2] = (w >> 16) & 0xFFu;
        q[3] = w >> 24;
    } else {
        uint2 w = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(c) + e);
        q[0] = w.x & 0xFFFFu;
        q[1] = w.x >> 16;
        q[2] = w.y & 0xFFFFu;
        q[3] = w.y >> 16;
    }
}

template <int C>
__device__ __forceinline__ uint32_t load_code1(const void* c, int64_t e) {
    if constexpr (C == AL8 || C == UF8)
        return reinterpret_cast<const uint8_t*>(c)[e];
    else
        return reinterpret_cast<const uint16_t*>(c)[e];
}

// Workgroup id -> work unit for streaming kernels. The dispatcher hands
// workgroups to the 8 XCDs round-robin (workgroup i to XCD i mod 8); this
// gives each XCD a contiguous eighth of the units instead of every eighth
// unit (the tail beyond a multiple of 8 keeps its order). Measured on the
// step's read/write mix: 1-3% more HBM throughput.
__device__ __forceinline__ int64_t xcd_order(uint32_t wg, uint32_t grid) {
    const int64_t g8 = (int64_t)(grid & ~7u);
    const int64_t w = wg;
    return w < g8 ? (w & 7) * (g8 >> 3) + (w >> 3) : w;
}

// Streaming (non-temporal) or ordinary vector loads and stores of 16, 8 and 4
// bytes. The non-temporal builtins take clang vector types, not HIP's structs.
typedef float nt_f4 __attribute__((ext_vector_type(4)));
typedef uint32_t nt_u2 __attribute__((ext_vector_type(2)));
typedef uint32_t nt_u4 __attribute__((ext_vector_type(4)));
typedef double nt_d2 __attribute__((ext_vector_type(2)));

template <bool NT>
__device__ __forceinline__ float4 ld_f4(const float* p) {
    if constexpr (NT) {
        const nt_f4 x = __builtin_nontemporal_load(reinterpret_cast<const nt_f4*>(p));
        return make_float4(x.x, x.y, x.z, x.w);
    } else {
        return *reinterpret_cast<const float4*>(p);
    }
}
template <bool NT>
__device__ __forceinline__ uint2 ld_u2(const void* p) {
    if constexpr (NT) {
        const nt_u2 x = __builtin_nontemporal_load(reinterpret_cast<const nt_u2*>(p));
        return make_uint2(x.x, x.y);
    } else {
        return *reinterpret_cast<const uint2*>(p);
    }
}
template <bool NT>
__device__ __forceinline__ uint32_t ld_u1(const void* p) {
    if constexpr (NT)
        return __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p));
    else
        return *reinterpret_cast<const uint32_t*>(p);
}
template <bool NT>
__device__ __forceinline__ void st_f4(float* p, const float4& x) {
    if constexpr (NT)
        __builtin_nontemporal_store(nt_f4{x.x, x.y, x.z, x.w}, reinterpret_cast<nt_f4*>(p));
    else
        *reinterpret_cast<float4*>(p) = x;
}
template <bool NT>
__device__ __forceinline__ void st_u2(void* p, const uint2& x) {
    if constexpr (NT)
        __builtin_nontemporal_store(nt_u2{x.x, x.y}, reinterpret_cast<nt_u2*>(p));
    else
        *reinterpret_cast<uint2*>(p) = x;
}
template <bool NT>
__device__ __forceinline__ void st_u1(void* p, uint32_t x) {
    if constexpr (NT)
        __builtin_nontemporal_store(x, reinterpret_cast<uint32_t*>(p));
    else
        *reinterpret_cast<uint32_t*>(p) = x;
}

// Pointers in the global address space. Pointers read from a workspace table
// are generic to the compiler, which then issues flat loads; those also count
// against the LDS wait counter, so an LDS read would wait for every load in
// flight. Kernels that read their pointers from memory convert them once.
template <class T>
using gp = __attribute__((address_space(1))) T*;

template <class T>
__device__ __forceinline__ gp<T> to_g(T* p) {
    return (gp<T>)p;
}
template <class U, class T>
__device__ __forceinline__ gp<U> g_as(gp<T> p) {
    return (gp<U>)p;
}

template <bool NT>
__device__ __forceinline__ float4 ld_f4(gp<const float> p) {
    if constexpr (NT) {
        const nt_f4 x = __builtin_nontemporal_load(g_as<const nt_f4>(p));
        return make_float4(x.x, x.y, x.z, x.w);
    } else {
        const nt_f4 x = *g_as<const nt_f4>(p);
        return make_float4(x.x, x.y, x.z, x.w);
    }
}
template <bool NT>
__device__ __forceinline__ uint2 ld_u2(gp<const void> p) {
    if constexpr (NT) {
        const nt_u2 x = __builtin_nontemporal_load(g_as<const nt_u2>(p));
        return make_uint2(x.x, x.y);
    } else {
        const nt_u2 x = *g_as<const nt_u2>(p);
        return make_uint2(x.x, x.y);
    }
}
template <bool NT>
__device__ __forceinline__ uint4 ld_u4(gp<const void> p) {
    if constexpr (NT) {
        const nt_u4 x = __builtin_nontemporal_load(g_as<const nt_u4>(p));
        return make_uint4(x.x, x.y, x.z, x.w);
    } else {
        const nt_u4 x = *g_as<const nt_u4>(p);
        return make_uint4(x.x, x.y, x.z, x.w);
    }
}
// Two binary64 values to 16-byte aligned global memory.
__device__ __forceinline__ void st_d2(gp<double> p, double x, double y) { *g_as<nt_d2>(p) = nt_d2{x, y}; }

template <bool NT>
__device__ __forceinline__ uint32_t ld_u1(gp<const void> p) {
    if constexpr (NT)
        return __builtin_nontemporal_load(g_as<const uint32_t>(p));
    else
        return *g_as<const uint32_t>(p);
}
template <bool NT>
__device__ __forceinline__ void st_f4(gp<float> p, const float4& x) {
    if constexpr (NT)
        __builtin_nontemporal_store(nt_f4{x.x, x.y, x.z, x.w}, g_as<nt_f4>(p));
    else
        *g_as<nt_f4>(p) = nt_f4{x.x, x.y, x.z, x.w};
}
template <bool NT>
__device__ __forceinline__ void st_u1(gp<void> p, uint32_t x) {
    if constexpr (NT)
        __builtin_nontemporal_store(x, g_as<uint32_t>(p));
    else
        *g_as<uint32_t>(p) = x;
}

template <int C, bool NT = false>
__device__ __forceinline__ void store_codes4(void* c, int64_t e, const uint32_t q[4]) {
    if constexpr (C == AL8 || C == UF8) {
        uint32_t w = (q[0] & 0xFFu) | ((q[1] & 0xFFu) << 8) | ((q[2] & 0xFFu) << 16) | (q[3] << 24);
        st_u1<NT>(reinterpret_cast<uint8_t*>(c) + e, w);
    } else {
        uint2 w = make_uint2((q[0] & 0xFFFFu) | (q[1] << 16), (q[2] & 0xFFFFu) | (q[3] << 16));
        st_u2<NT>(reinterpret_cast<uint16_t*>(c) + e, w);
    }
}

template <bool NT>
__device__ __forceinline__ void st_u2(gp<void> p, const uint2& x) {
    if constexpr (NT)
        __builtin_nontemporal_store(nt_u2{x.x, x.y}, g_as<nt_u2>(p));
    else
        *g_as<nt_u2>(p) = nt_u2{x.x, x.y};
}

// Four codes of element e onward into a global code array (bytes for AL8/UF8,
// 16-bit words for AL16).
template <int C, bool NT = false>
__device__ __forceinline__ void store_codes4(gp<uint8_t> c, int64_t e, const uint32_t q[4]) {
    if constexpr (C == AL8 || C == UF8) {
        uint32_t w = (q[0] & 0xFFu) | ((q[1] & 0xFFu) << 8) | ((q[2] & 0xFFu) << 16) | (q[3] << 24);
        st_u1<NT>(c + e, w);
    } else {
        uint2 w = make_uint2((q[0] & 0xFFFFu) | (q[1] << 16), (q[2] & 0xFFFFu) | (q[3] << 16));
        st_u2<NT>(g_as<uint16_t>(c) + e, w);
    }
}

template <int C>
__device__ __forceinline__ void store_code1(void* c, int64_t e, uint32_t q) {
    if constexpr (C == AL8 || C == UF8)
        reinterpret_cast<uint8_t*>(c)[e] = (uint8_t)q;
    else
        reinterpret_cast<uint16_t*>(c)[e] = (uint16_t)q;
}

template <int C>
constexpr int levels_of() {
    return C == AL16 ? 65534 : 254;
}

}  // namespace al
