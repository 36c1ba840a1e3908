/*
 * al.h -- C ABI of the MI355X (gfx950) quantized optimizer-step library
 * (libal.so).
 *
 * The library implements the fused quantized optimizer step of "Beyond Dense
 * Adam States: Adaptive Log-Space Quantization for Memory-Efficient
 * Optimizers": each step decodes block-wise optimizer state, applies the
 * optimizer update and re-encodes the state, for AdamW (dense M, V), Adafactor
 * (factored V) and CAME (dense M, factored V and factored confidence C),
 * section 3.1.
 *
 * Codes (section 4):
 *   AL8 / AL16  non-negative states. Per block of B consecutive elements of
 *               the row-major flattening: l_min = max(l_floor, log2 of the
 *               smallest positive value), l_max = log2 of the largest,
 *               capped at 126 (Eq. al_bounds); positive x -> 1 +
 *               round((L-2) clip((log2 x - l_min)/(l_max - l_min), 0, 1)),
 *               zero -> 0 (Eq. al_quant); decode 2^(l_min + (q-1)/(L-2) *
 *               delta) (Eq. al_dequant). L = 256 (AL8, uint8 codes) or
 *               65,536 (AL16, uint16 codes). q = 0 iff x = 0 (Eq.
 *               exact_zero). Equal positives widen the interval upward by
 *               one log2 unit; the width is at least 1e-12.
 *               Metadata: 2 floats per block, {l_min, delta}.
 *   UF8         signed momentum (section 4.3): symmetric int8 in
 *               [-127, 127] with a per-block absmax scale; code =
 *               round(127 x / absmax), decode code * absmax / 127.
 *               Metadata: 1 float per block, {absmax}.
 *   FP32        the state is a plain float array (no metadata).
 *
 * Storage (section 4.4, Eq. al_memory): a state of n elements under block B
 * holds ceil(n/B)*B codes -- padded per tensor; padded codes are written as
 * 0 -- plus its metadata. al_code_bytes / al_meta_floats / al_state_bytes
 * give the sizes.
 *
 * Numeric contract. State arithmetic (decode, EMA, marginal means, factor
 * reconstruction, residuals) is binary64, each state rounded once to fp32
 * per step, sums exact to binary64 rounding; codes are decided from binary64
 * positions. The parameter update itself is fp32.
 *
 * Memory and execution. Every pointer argument is device memory owned by
 * the caller, except that tensor lists and config structs are host memory
 * read during the call. The library keeps no pointer after a call returns.
 * All device work is enqueued on `stream` (a hipStream_t; NULL = the null
 * stream) in order; calls return without synchronizing. The library never
 * allocates device memory: each step takes a caller workspace whose size the
 * matching *_workspace_bytes query returns. Calls on distinct streams with
 * distinct buffers may run concurrently; calls that share a workspace or
 * state buffers must be ordered by the caller.
 *
 * Fresh state: all codes and metadata zero (code 0 is exact zero).
 *
 * Errors. Every call returns an al_status. All argument checks run on the
 * host before any HIP call, so a rejected call has enqueued nothing.
 * al_last_error() returns a thread-local description of the last failure on
 * the calling thread. Non-finite or negative values in a non-negative state
 * are not detected; their codes are unspecified.
 *
 * Alignment. Every device pointer must be 16-byte aligned (AL_EALIGN).
 */
#ifndef AL_H
#define AL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum al_status {
    AL_OK = 0,
    AL_EINVAL = 1,       /* bad argument: NULL, n < 0, bad codec/block/dtype, rows*cols mismatch */
    AL_EALIGN = 2,       /* a device pointer is not 16-byte aligned */
    AL_EWORKSPACE = 3,   /* workspace missing or smaller than the query returned */
    AL_EUNSUPPORTED = 4, /* a valid combination the library does not implement */
    AL_EHIP = 5          /* a HIP runtime call or launch failed */
} al_status;

typedef enum al_codec {
    AL_CODEC_FP32 = 0,
    AL_CODEC_AL8 = 1,
    AL_CODEC_AL16 = 2,
    AL_CODEC_UF8 = 3
} al_codec;

typedef enum al_dtype { AL_DTYPE_F32 = 0, AL_DTYPE_BF16 = 1 } al_dtype;

/* Which code a state gets ("representation and state policy", section 4.3).
 * block: 64, 128, 256, 512, 1024 or 2048 (ignored for FP32).
 * log_floor: l_floor of Eq. al_bounds (AL codecs only); the optimizer path
 * supplies it, typically log2 of its squared numerical floor (section 4.1). */
typedef struct al_state_spec {
    int32_t codec;
    int32_t block;
    float log_floor;
} al_state_spec;

/* One parameter tensor and its optimizer state buffers.
 * rows, cols: the row-major shape; a 1-D tensor has rows == 1 (such tensors,
 * and any tensor with rows == 1, keep an unfactored second moment in `v`).
 * param: rows*cols fp32, updated in place. grad: rows*cols of the call's
 * grad dtype.
 * m, m_meta:       momentum (AdamW, CAME).
 * v, v_meta:       dense second moment (AdamW), or the unfactored second
 *                  moment of a rows == 1 tensor (Adafactor, CAME).
 * vr/vc (+meta):   factored second moment, row (len rows) / column (len cols)
 *                  statistics (Adafactor, CAME; rows > 1 only).
 * cr/cc (+meta):   CAME factored confidence, row / column (rows > 1 only).
 * Slots a path does not use must be NULL. Metadata pointers are NULL for
 * FP32 states. */
typedef struct al_tensor {
    float* param;
    const void* grad;
    int64_t rows;
    int64_t cols;
    void* m;
    float* m_meta;
    void* v;
    float* v_meta;
    void* vr;
    float* vr_meta;
    void* vc;
    float* vc_meta;
    void* cr;
    float* cr_meta;
    void* cc;
    float* cc_meta;
} al_tensor;

/* AdamW (section 3.1, Eq. adam_update; decoupled weight decay and bias
 * corrections as in PyTorch AdamW). m: UF8 (block 256) or FP32.
 * v: AL8, AL16 or FP32. */
typedef struct al_adamw_cfg {
    double lr, beta1, beta2, eps, weight_decay;
    int32_t grad_dtype;
    int32_t reserved;
    al_state_spec m, v;
} al_adamw_cfg;

/* Flags of the factored steps (al_adafactor_cfg / al_came_cfg .flags).
 * AL_FLAG_EXACT_SUMS: every row and column mean behind the factored states is
 * recomputed with exact sums (slow). The default path already yields the same
 * fp32 states bit for bit -- its fast sums are kept only where they provably
 * round the same way -- so this flag is a check of that path, not a
 * different result. */
#define AL_FLAG_EXACT_SUMS 1

/* Adafactor (factored second moment, section 3.1): beta2_t = 1 - t^decay_rate,
 * G2 = g^2 + eps1, R/C = EMA of row/column means of G2, update
 * u = g / sqrt(R_i C_j / mean(R)), clipped by max(1, RMS(u)/clip_threshold);
 * no first moment, no relative step, no parameter scaling.
 * v: AL8, AL16 or FP32 for R, C and 1-D v. flags: 0 or AL_FLAG_EXACT_SUMS. */
typedef struct al_adafactor_cfg {
    double lr, eps1, clip_threshold, decay_rate, weight_decay;
    int32_t grad_dtype;
    int32_t flags;
    al_state_spec v;
} al_adafactor_cfg;

/* CAME (confidence-guided factored optimizer, section 3.1): factored V as
 * Adafactor with a constant beta2 and no bias correction; clipped update
 * uhat; m = EMA(beta1) of uhat; residual (uhat - m)^2 + eps2 feeds factored
 * confidence R', C' (EMA beta3); update m / sqrt(R'_i C'_j / mean(R')).
 * 1-D tensors: unfactored v, update = m, no confidence.
 * m: UF8 (block 256) or FP32; v and conf: AL8, AL16 or FP32.
 * flags: 0 or AL_FLAG_EXACT_SUMS. */
typedef struct al_came_cfg {
    double lr, beta1, beta2, beta3, eps1, eps2, clip_threshold, weight_decay;
    int32_t grad_dtype;
    int32_t flags;
    al_state_spec m, v, conf;
} al_came_cfg;

/* APOLLO, the projected-state path (section 3.1: first and second moments
 * kept in a low-rank projection of the gradient derive a channel-wise scale
 * of the original gradient; section 6 setup: rank 256, channel-wise scaling,
 * projection refreshed every 200 steps; Table 4: UF8 momentum, AL8 second
 * moment). A rows x cols tensor has C = max(rows, cols) channels of
 * L = min(rows, cols) inputs: rows >= cols projects the columns (channel c is
 * row c), otherwise the rows (channel c is column c). Per step:
 *   R   = fl32(A Pi) in binary64, A = G (rows >= cols) or G^T as C x L,
 *         Pi = proj (L x rank, row-major fp32; the caller draws it, N(0, 1/rank),
 *         and refreshes it every gap steps);
 *   m, v: the AdamW moments of R (rank * C elements, channel-major: element
 *         c * rank + k), with AdamW's codes, bias corrections and eps; the
 *         direction Rt = (m / bc1) / (sqrt(v / bc2) + eps) is fp32;
 *   s_c = ||Rt_c|| / (||R_c|| + 1e-8), G~ = G with channel c scaled by s_c;
 *   limiter (gamma > 0): from step 2, lam = max(||G~|| / (*norm_state + 1e-8),
 *         gamma) / gamma and *norm_state = fl32(||G~|| / lam); at step 1
 *         lam = 1 and *norm_state = fl32(||G~||);
 *   param = fl32(param (1 - lr wd) - lr g (s_c / lam)), binary64.
 * The token embedding, LM head and 1-D tensors are not projected: they take
 * al_adamw_step with the same codes. */
typedef struct al_apollo_tensor {
    float* param;
    const void* grad;
    int64_t rows;
    int64_t cols;
    const float* proj; /* L x rank fp32 */
    void* m;           /* projected momentum, rank * C elements */
    float* m_meta;
    void* v;           /* projected second moment, rank * C elements */
    float* v_meta;
    float* norm_state; /* 1 float: the limiter's last update norm (unused when gamma <= 0) */
} al_apollo_tensor;

/* rank: 64, 128 or 256. gamma: the limiter's growth bound (<= 0: no limiter).
 * m: UF8 (block 256) or FP32; v: AL8, AL16 or FP32. */
typedef struct al_apollo_cfg {
    double lr, beta1, beta2, eps, weight_decay, gamma;
    int32_t rank;
    int32_t grad_dtype;
    al_state_spec m, v;
} al_apollo_cfg;

/* Library version string, e.g. "0.1.0 gfx950". */
const char* al_version(void);

/* Thread-local text of the last failure on this thread ("" if none). */
const char* al_last_error(void);

/* Storage accounting (section 4.4). Bytes of the code array of an n-element
 * state (padded to whole blocks), metadata floats, and their total in bytes.
 * Return -1 for an invalid codec, block or n < 0. */
int64_t al_code_bytes(int32_t codec, int64_t n, int32_t block);
int64_t al_meta_floats(int32_t codec, int64_t n, int32_t block);
int64_t al_state_bytes(int32_t codec, int64_t n, int32_t block);

/* Encode n fp32 values x (non-negative for AL codecs) into codes + meta
 * (Eq. al_bounds and al_quant for AL8/AL16; section 4.3 for UF8).
 * codec: AL8, AL16 or UF8. codes: al_code_bytes(codec, n, block) bytes;
 * meta: al_meta_floats(codec, n, block) floats. log_floor is ignored for
 * UF8. n == 0 is a no-op. */
al_status al_quantize(int32_t codec, const float* x, int64_t n, int32_t block, float log_floor,
                      void* codes, float* meta, void* stream);

/* Decode n values (Eq. al_dequant for AL8/AL16; section 4.3 for UF8) into
 * out (n floats). */
al_status al_dequantize(int32_t codec, const void* codes, const float* meta, int64_t n,
                        int32_t block, float* out, void* stream);

/* Workspace size (bytes) that al_adamw_step needs for this tensor list and
 * config: the step's tensor descriptor table (64 + 8 bytes per non-empty
 * tensor, 256-byte aligned parts). 0 for a list with no elements. */
al_status al_adamw_workspace_bytes(const al_tensor* tensors, int32_t nt, const al_adamw_cfg* cfg, size_t* bytes);

/* One fused AdamW step over a list of nt tensors (section 3.1, Eq.
 * adam_update, with PyTorch AdamW's decoupled weight decay and bias
 * corrections; codes of section 4). step = the 1-based step count after
 * increment. One pass over HBM: read p, g, m, v (+meta), write p, m, v
 * (+meta). Uses per tensor: param, grad, m, m_meta, v, v_meta; the other
 * slots must be NULL. ws: device workspace of at least
 * al_adamw_workspace_bytes, 256-byte aligned (AL_EWORKSPACE otherwise); the
 * call writes the descriptor table there on the stream (small copy kernels)
 * and runs the whole list in one launch of the step kernel (several for
 * lists beyond 2^32 chunks of 1024-2048 elements). ws is scratch: its
 * contents need not survive between calls, and calls that share it must be
 * ordered on one stream. */
al_status al_adamw_step(const al_tensor* tensors, int32_t nt, const al_adamw_cfg* cfg, int64_t step, void* ws,
                        size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory or hand over a workspace
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): al_adamw_step without ws, same arguments otherwise and the
 * same results bit for bit (the same kernels). The descriptor table lives in
 * a fixed device array of the library instead, 288 KiB per GPU, held until
 * the process ends: at most 4096 non-empty tensors per call (more:
 * AL_EUNSUPPORTED, before any HIP call). The first call on a device looks up
 * that array's address once (hipGetSymbolAddress). The call allocates
 * nothing (no hipMalloc, hipFree or host heap). Every call on one GPU writes
 * the same array: calls in order on one stream are safe, calls that may
 * overlap on one GPU (several streams or threads) race and must be
 * serialized by the caller. */
al_status al_adamw_step_noalloc(const al_tensor* tensors, int32_t nt, const al_adamw_cfg* cfg, int64_t step,
                                void* stream);

/* Workspace size (bytes) that al_adafactor_step / al_came_step need for this
 * tensor list and config. */
al_status al_adafactor_workspace_bytes(const al_tensor* tensors, int32_t nt,
                                       const al_adafactor_cfg* cfg, size_t* bytes);
al_status al_came_workspace_bytes(const al_tensor* tensors, int32_t nt, const al_came_cfg* cfg,
                                  size_t* bytes);

/* One Adafactor step over nt tensors. Uses per tensor: param, grad and
 * (rows > 1) vr, vr_meta, vc, vc_meta or (rows == 1) v, v_meta.
 * ws: device workspace of at least the queried size, 256-byte aligned. */
al_status al_adafactor_step(const al_tensor* tensors, int32_t nt, const al_adafactor_cfg* cfg,
                            int64_t step, void* ws, size_t ws_bytes, void* stream);

/* One CAME step over nt tensors. Uses per tensor: param, grad, m, m_meta and
 * (rows > 1) vr, vc, cr, cc with metadata or (rows == 1) v, v_meta. */
al_status al_came_step(const al_tensor* tensors, int32_t nt, const al_came_cfg* cfg,
                       int64_t step, void* ws, size_t ws_bytes, void* stream);

/* Workspace size (bytes) that al_apollo_step needs for this list and config:
 * per tensor R (rank * C floats), below rank 256 also Rt (as many floats),
 * per-channel binary64 sums, and the descriptor tables of the step's
 * launches. */
al_status al_apollo_workspace_bytes(const al_apollo_tensor* tensors, int32_t nt, const al_apollo_cfg* cfg,
                                    size_t* bytes);

/* One APOLLO step over nt projected tensors (rows, cols >= 1). Kernels, in
 * stream order: the binary64 projection on the matrix cores (also sums of
 * squares per channel of G), the fused AdamW step over the projected moments
 * (fp32 R as its gradient, lr 1, no weight decay; at rank 256 it forms the
 * channel scales itself, one channel per 256-element sub-tile, from the
 * direction it computes; below rank 256 it writes the direction as its
 * parameter Rt in the workspace and a separate pass forms the channel
 * scales), the limiter per tensor, and the parameter update. ws: device
 * workspace of at least the queried size, 256-byte aligned. */
al_status al_apollo_step(const al_apollo_tensor* tensors, int32_t nt, const al_apollo_cfg* cfg, int64_t step,
                         void* ws, size_t ws_bytes, void* stream);

/* Diagnostic: evaluate, elementwise on the device, a math primitive the
 * codes rely on, so tests can bound it against the host: fn 0 = hardware
 * fp32 log2 of (float)x (the fast code position uses it on mantissas in
 * [1/2, 1)), 1 = the binary64 exp2 used by decoding, 2 = binary64 log2 (block
 * endpoints and near-boundary positions), 3 = binary64 sqrt, 4 = 1/sqrt(x)
 * (factored second-moment reconstruction), 5 = x / 127 and 6 = 127 / x by
 * the division-free sequences of the UF8 code (exact for x a finite fp32
 * value, x > 0 for 6), 7 = fl32(x / 3) by the multiply-and-check quotient of
 * the clipped updates, 8 = the binary64 log2 of (float)x that fits the AdamW
 * step's second-moment blocks (x > 0), 9 = the clipped update of the CAME
 * passes, fl32(fl64(fl64(r c) x) / d) for fixed binary64 r, c, d from the
 * quotient with fl64(1 / d) folded into r and the decision test over eight
 * consecutive inputs (n a multiple of 8), 10 = the same for bf16 values x with
 * r = d = 1 and c = 0x1.00008c3a4f91dp7 (about 2^7 (1 + 2^-17)), where the residual pass's range test is
 * known to pass and only the midpoint test runs. x, out: n doubles (device). */
al_status al_diag_math(int32_t fn, const double* x, int64_t n, double* out, void* stream);

/* The AL8 levels of the fused AdamW step's split-table decode (section 4.1,
 * Eq. al_dequant): for each of nblocks blocks with metadata {l_min, delta}
 * (fp32 pairs, the AL8 layout), out[255 b + q - 1] is the binary64 value of
 * the level of code q = 1..255 before its rounding to fp32, computed by the
 * same device functions as the step: kind 0 = two factors (blocks of 128 and
 * more), 1 = three factors (blocks of 64). meta, out: device, 16-byte
 * aligned; out holds 255 nblocks doubles. For measuring the decode's error
 * against 2^E. */
al_status al_diag_levels(int32_t kind, const float* meta, int64_t nblocks, double* out, void* stream);

/* Sums of squares behind the relative update error of section 3.2 (Eq.
 * update_error): with U = a, U_ref = b (two updates of the same n elements,
 * fp32 device arrays), writes out[0] = sum_i (a_i - b_i)^2 and out[1] =
 * sum_i b_i^2, each term formed in binary64 and summed double-double (fixed
 * order: the result is reproducible and within an ulp of the exact sum).
 * out: device buffer of at least AL_DIFF_NORMS_OUT doubles, 16-byte aligned;
 * out[2 ..] is scratch. n = 0 writes zeros. Enqueued on stream; allocates
 * nothing. The error is sqrt(out[0]) / (sqrt(out[1]) + eps). */
#define AL_DIFF_NORMS_OUT 4098
al_status al_diff_norms(const float* a, const float* b, int64_t n, double* out, void* stream);

/* Diagnostic: streaming rates of the fused AdamW byte mix. Reads p (n fp32),
 * g (n bf16), m and v (n bytes each) and writes p, m, v with no optimizer
 * arithmetic. mode selects the access shape:
 *   0, 1  the shape of al_adamw_step (one 2048-element chunk per wavefront in
 *         two load phases, 4 consecutive elements per lane, XCD-contiguous
 *         workgroup order); mode 1 uses non-temporal loads and stores. Writes
 *         p[4i] += g[4i], p[4i+3] += g[4i+3] (g as bf16), m ^= v, v += 1 per
 *         byte. n must be a multiple of 2048.
 *   2, 3  the fastest shape found for the mix (one 4096-element chunk per
 *         wavefront, 16 bytes per lane from every stream, all loads before any
 *         store, non-temporal): a reference rate, not the step's layout.
 *         Writes p += 1, m ^= v, v += 1 per byte; g is only read. n must be a
 *         multiple of 4096.
 * v += 1 carries into the next byte where a byte is 0xFF. Timing it gives the
 * achievable HBM bandwidth for the step's exact byte mix. Enqueued on stream;
 * allocates nothing. AL_EINVAL for a bad mode, n or NULL buffer, AL_EALIGN
 * for a buffer not 16-byte aligned. */
al_status al_diag_stream(int32_t mode, float* p, const void* g, void* m, void* v, int64_t n, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* AL_H */
