/*
 * al_oracle.c -- TEST INFRASTRUCTURE. Not part of the product path.
 *
 * Plain, slow, obviously-correct binary64 CPU reference for the quantized
 * optimizer step of "Beyond Dense Adam States: Adaptive Log-Space
 * Quantization for Memory-Efficient Optimizers". Only the tests, the smoke
 * check and the benchmark's CPU baseline may load it; the product path never
 * does. Single-threaded loops in index order, no blocking or fusion.
 *
 * Numeric convention (the paper fixes no precision; these are the readings
 * the parity tests hold the GPU to):
 *   N1 storage: params fp32; grads bf16 or fp32; codes uint8/uint16/int8;
 *      metadata fp32.
 *   N2 arithmetic: binary64, round-to-nearest-even, built without
 *      contraction (-ffp-contract=off), libm log2/exp2/sqrt/pow.
 *   N3 each optimizer state is rounded to fp32 once per step; that fp32
 *      value is both what gets encoded and what the update uses.
 *   N4 block min/max/absmax are exact; sums are exact and rounded once to
 *      binary64 (Shewchuk's partials method, as Python's math.fsum).
 *   N5 hyperparameters are binary64; derived scalars are computed here.
 *
 * Pin status (the CPU tests hold each function to something other than
 * itself): the codes to worked examples, invariants and brute force; AdamW
 * to torch.optim.AdamW; Adafactor to Hugging Face's Adafactor. CAME's
 * official implementation is not available: the CAME step is pinned through
 * closed forms (beta1 = 0 against the clipped update, the second-moment path
 * at t = 1, and 20 steps with beta1 = 0.9 for constant uniform and rank-1
 * gradients, sign flips at one step or at element-specific steps, and a
 * rows == 1 tensor) and, for gradients whose row and column magnitudes
 * vary from step to step, by symmetries its definition implies over 20 steps
 * with beta1 = 0.9 (row and column permutations and negation commute with
 * the step bit for bit, scaling the gradient by 2 leaves the update unchanged,
 * transposition swaps the factors); against CAME's own implementation the
 * values for such gradients stay parity unpinned.
 */
#include "al_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

enum { C_FP32 = 0, C_AL8 = 1, C_AL16 = 2, C_UF8 = 3 };

/* ------------------------------------------------------------------------ */
/* Exact summation. Shewchuk, "Adaptive precision floating-point arithmetic  */
/* and fast robust geometric predicates" (1997): keep a list of non-         */
/* overlapping partial sums whose exact total is the exact running sum; the  */
/* final step rounds that total once, resolving half-way cases.              */
/* ------------------------------------------------------------------------ */
typedef struct {
    int n;
    double p[160];
} xsum_t;

static void xsum_init(xsum_t* s) { s->n = 0; }

static void xsum_add(xsum_t* s, double x) {
    int kept = 0;
    for (int i = 0; i < s->n; i++) {
        double y = s->p[i];
        if (fabs(x) < fabs(y)) {
            double t = x;
            x = y;
            y = t;
        }
        double hi = x + y;          /* rounded sum            */
        double lo = y - (hi - x);   /* its exact error (|x|>=|y|) */
        if (lo != 0.0) s->p[kept++] = lo;
        x = hi;
    }
    s->p[kept++] = x;
    s->n = kept;
    if (s->n > 150) abort(); /* cannot happen for finite binary64 input */
}

static double xsum_round(const xsum_t* s) {
    int n = s->n;
    if (n == 0) return 0.0;
    double hi = s->p[--n];
    double lo = 0.0;
    while (n > 0) {
        double x = hi;
        double y = s->p[--n];
        hi = x + y;
        lo = y - (hi - x);
        if (lo != 0.0) break;
    }
    /* If the remaining partials push the discarded part past half an ulp in
     * the direction of lo, the rounding of hi must move. */
    if (n > 0 && ((lo < 0.0 && s->p[n - 1] < 0.0) || (lo > 0.0 && s->p[n - 1] > 0.0))) {
        double y = lo * 2.0;
        double x = hi + y;
        if (y == x - hi) hi = x;
    }
    return hi;
}

double orc_exact_sum(const double* x, int64_t n) {
    xsum_t s;
    xsum_init(&s);
    for (int64_t i = 0; i < n; i++) xsum_add(&s, x[i]);
    return xsum_round(&s);
}

/* ------------------------------------------------------------------------ */
/* Small helpers                                                             */
/* ------------------------------------------------------------------------ */
static int valid_block(int32_t b) {
    return b == 64 || b == 128 || b == 256 || b == 512 || b == 1024 || b == 2048 ||
           b == 8 || b == 16 || b == 32; /* tiny blocks: brute-force pins only */
}

static int64_t nblocks(int64_t n, int32_t b) { return (n + b - 1) / b; }

static double grad_at(const void* g, int32_t g_bf16, int64_t i) {
    if (g_bf16) {
        uint32_t bits = (uint32_t)((const uint16_t*)g)[i] << 16;
        float f;
        memcpy(&f, &bits, 4);
        return (double)f;
    }
    return (double)((const float*)g)[i];
}

/* ------------------------------------------------------------------------ */
/* AL codec: section 4.1, Eq. al_bounds / al_quant / al_dequant; the         */
/* degenerate-range rules after them; the exact-zero invariant of 4.2.       */
/* L = 2^bits codes; code 0 only for exact zero; positive values use codes   */
/* 1 .. L-1 spread uniformly in log2 over the block's interval.              */
/* ------------------------------------------------------------------------ */

/* Fit one block's interval. Returns 0 if the block holds no positive value.
 * lmin = max(floor, log2 of the smallest positive value) -- log2 is
 * increasing, so the log of the smallest value is the smallest log.
 * lmax = log2 of the largest positive value, capped at 126.
 * Equal positives: the interval is widened upward by one log2 unit.
 * The width is clamped to at least 1e-12 (this also covers a block lying
 * entirely below the floor, where lmax < lmin). */
static int al_fit(const float* x, int64_t nb, float log_floor, double* lmin, double* delta) {
    int any = 0;
    float xmin = 0.0f, xmax = 0.0f;
    for (int64_t i = 0; i < nb; i++) {
        if (x[i] > 0.0f) {
            if (!any || x[i] < xmin) xmin = x[i];
            if (!any || x[i] > xmax) xmax = x[i];
            any = 1;
        }
    }
    if (!any) return 0;
    double lo = log2((double)xmin);
    double hi = log2((double)xmax);
    double l0 = lo > (double)log_floor ? lo : (double)log_floor;
    double l1 = hi < 126.0 ? hi : 126.0;
    if (xmin == xmax) l1 = l0 + 1.0;
    double d = l1 - l0;
    if (d < 1e-12) d = 1e-12;
    *lmin = l0;
    *delta = d;
    return 1;
}

int orc_al_quantize(int32_t bits, const float* x, int64_t n, int32_t block, float log_floor,
                    void* codes, float* meta, double* y) {
    if ((bits != 8 && bits != 16) || n < 0 || !valid_block(block)) return -1;
    const double levels = (bits == 8) ? 254.0 : 65534.0; /* L - 2 */
    int64_t nbk = nblocks(n, block);
    for (int64_t b = 0; b < nbk; b++) {
        int64_t s = b * block;
        int64_t e = s + block < n ? s + block : n;
        double lmin = 0.0, delta = 0.0;
        int any = al_fit(x + s, e - s, log_floor, &lmin, &delta);
        meta[2 * b] = any ? (float)lmin : 0.0f;
        meta[2 * b + 1] = any ? (float)delta : 0.0f;
        for (int64_t i = s; i < s + block; i++) {
            uint32_t q = 0;
            double yy = NAN;
            if (i < n && x[i] > 0.0f) {
                double z = (log2((double)x[i]) - lmin) / delta;
                if (z < 0.0) z = 0.0;
                if (z > 1.0) z = 1.0;
                yy = levels * z;
                q = 1u + (uint32_t)rint(yy);
            }
            if (bits == 8)
                ((uint8_t*)codes)[i] = (uint8_t)q;
            else
                ((uint16_t*)codes)[i] = (uint16_t)q;
            if (y && i < n) y[i] = yy;
        }
    }
    return 0;
}

int orc_al_dequantize(int32_t bits, const void* codes, const float* meta, int64_t n,
                      int32_t block, float* out) {
    if ((bits != 8 && bits != 16) || n < 0 || !valid_block(block)) return -1;
    const double levels = (bits == 8) ? 254.0 : 65534.0;
    for (int64_t i = 0; i < n; i++) {
        int64_t b = i / block;
        uint32_t q = bits == 8 ? ((const uint8_t*)codes)[i] : ((const uint16_t*)codes)[i];
        if (q == 0) {
            out[i] = 0.0f;
            continue;
        }
        double step = (double)meta[2 * b + 1] / levels;
        double e = (double)meta[2 * b] + (double)(q - 1) * step;
        out[i] = (float)exp2(e);
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* UF8: uniform signed 8-bit momentum code with a per-block absmax scale     */
/* (section 4.3). Codes are symmetric in [-127, 127]; 0 encodes 0.           */
/* ------------------------------------------------------------------------ */
int orc_uf8_quantize(const float* x, int64_t n, int32_t block, int8_t* codes, float* meta,
                     double* y) {
    if (n < 0 || !valid_block(block)) return -1;
    int64_t nbk = nblocks(n, block);
    for (int64_t b = 0; b < nbk; b++) {
        int64_t s = b * block;
        int64_t e = s + block < n ? s + block : n;
        float amax = 0.0f;
        for (int64_t i = s; i < e; i++) {
            float a = fabsf(x[i]);
            if (a > amax) amax = a;
        }
        meta[b] = amax;
        double r = amax > 0.0f ? 127.0 / (double)amax : 0.0;
        for (int64_t i = s; i < s + block; i++) {
            int q = 0;
            double yy = NAN;
            if (i < n && amax > 0.0f) {
                yy = (double)x[i] * r;
                double qq = rint(yy);
                if (qq > 127.0) qq = 127.0;
                if (qq < -127.0) qq = -127.0;
                q = (int)qq;
            }
            codes[i] = (int8_t)q;
            if (y && i < n) y[i] = yy;
        }
    }
    return 0;
}

int orc_uf8_dequantize(const int8_t* codes, const float* meta, int64_t n, int32_t block,
                       float* out) {
    if (n < 0 || !valid_block(block)) return -1;
    for (int64_t i = 0; i < n; i++) {
        double step = (double)meta[i / block] / 127.0;
        out[i] = (float)((double)codes[i] * step);
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* A state under a spec (FP32 / AL8 / AL16 / UF8)                            */
/* ------------------------------------------------------------------------ */
int orc_state_decode(orc_spec s, const void* codes, const float* meta, int64_t n, float* out) {
    switch (s.codec) {
        case C_FP32: memcpy(out, codes, (size_t)n * 4); return 0;
        case C_AL8: return orc_al_dequantize(8, codes, meta, n, s.block, out);
        case C_AL16: return orc_al_dequantize(16, codes, meta, n, s.block, out);
        case C_UF8: return orc_uf8_dequantize((const int8_t*)codes, meta, n, s.block, out);
    }
    return -1;
}

int orc_state_encode(orc_spec s, const float* x, int64_t n, void* codes, float* meta, double* y) {
    switch (s.codec) {
        case C_FP32:
            memcpy(codes, x, (size_t)n * 4);
            if (y)
                for (int64_t i = 0; i < n; i++) y[i] = NAN;
            return 0;
        case C_AL8: return orc_al_quantize(8, x, n, s.block, s.log_floor, codes, meta, y);
        case C_AL16: return orc_al_quantize(16, x, n, s.block, s.log_floor, codes, meta, y);
        case C_UF8: return orc_uf8_quantize(x, n, s.block, (int8_t*)codes, meta, y);
    }
    return -1;
}

static float* fbuf(int64_t n) { return (float*)malloc((size_t)(n > 0 ? n : 1) * sizeof(float)); }
static double* dbuf(int64_t n) { return (double*)malloc((size_t)(n > 0 ? n : 1) * sizeof(double)); }

/* ------------------------------------------------------------------------ */
/* AdamW (dense M, V; section 3.1 Eq. adam_update, with PyTorch AdamW's     */
/* decoupled weight decay and bias corrections, which the paper's reference  */
/* path aligns to).                                                          */
/* ------------------------------------------------------------------------ */
int orc_adamw_step(int64_t n, float* p, const void* g, int32_t g_bf16,
                   double lr, double beta1, double beta2, double eps, double wd, int64_t t,
                   orc_spec ms, void* m, float* m_meta, orc_spec vs, void* v, float* v_meta,
                   double* ym, double* yv) {
    if (n < 0 || t < 1) return -1;
    if (ms.codec != C_FP32 && ms.codec != C_UF8) return -1;
    if (vs.codec != C_FP32 && vs.codec != C_AL8 && vs.codec != C_AL16) return -1;
    float* mh = fbuf(n);
    float* vh = fbuf(n);
    if (orc_state_decode(ms, m, m_meta, n, mh) || orc_state_decode(vs, v, v_meta, n, vh)) {
        free(mh);
        free(vh);
        return -1;
    }
    const double bc1 = 1.0 - pow(beta1, (double)t);
    const double bc2 = 1.0 - pow(beta2, (double)t);
    const double step_size = lr / bc1;
    const double sqrt_bc2 = sqrt(bc2);
    const double decay = 1.0 - lr * wd;
    for (int64_t i = 0; i < n; i++) {
        double gi = grad_at(g, g_bf16, i);
        float m_new = (float)(beta1 * (double)mh[i] + (1.0 - beta1) * gi);
        float v_new = (float)(beta2 * (double)vh[i] + (1.0 - beta2) * (gi * gi));
        double pd = (double)p[i] * decay;
        pd = pd - step_size * (double)m_new / (sqrt((double)v_new) / sqrt_bc2 + eps);
        p[i] = (float)pd;
        mh[i] = m_new;
        vh[i] = v_new;
    }
    int rc = orc_state_encode(ms, mh, n, m, m_meta, ym);
    rc |= orc_state_encode(vs, vh, n, v, v_meta, yv);
    free(mh);
    free(vh);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Factored second moment (Adafactor's row/column statistics, section 3.1). */
/* rowmean_i = exact mean over j of G2_ij; colmean_j = exact mean over i.    */
/* ------------------------------------------------------------------------ */
static void row_col_means(int64_t rows, int64_t cols, const double* a, double* rmean,
                          double* cmean) {
    xsum_t s;
    for (int64_t i = 0; i < rows; i++) {
        xsum_init(&s);
        for (int64_t j = 0; j < cols; j++) xsum_add(&s, a[i * cols + j]);
        rmean[i] = xsum_round(&s) / (double)cols;
    }
    for (int64_t j = 0; j < cols; j++) {
        xsum_init(&s);
        for (int64_t i = 0; i < rows; i++) xsum_add(&s, a[i * cols + j]);
        cmean[j] = xsum_round(&s) / (double)rows;
    }
}

static double mean_f32(const float* x, int64_t n) {
    xsum_t s;
    xsum_init(&s);
    for (int64_t i = 0; i < n; i++) xsum_add(&s, (double)x[i]);
    return xsum_round(&s) / (double)n;
}

/* EMA of a stored vector state: x = fl32(beta * decoded + (1 - beta) * obs). */
static int ema_state(orc_spec s, void* codes, float* meta, int64_t n, const double* obs,
                     double beta, float* out) {
    if (orc_state_decode(s, codes, meta, n, out)) return -1;
    for (int64_t i = 0; i < n; i++) out[i] = (float)(beta * (double)out[i] + (1.0 - beta) * obs[i]);
    return 0;
}

/* RMS of an array (exact sum of squares). */
static double rms_of(const double* u, int64_t n) {
    xsum_t s;
    xsum_init(&s);
    for (int64_t i = 0; i < n; i++) xsum_add(&s, u[i] * u[i]);
    return sqrt(xsum_round(&s) / (double)n);
}

/* Adafactor (Shazeer & Stern) with the Hugging Face option set the paper's
 * reference path aligns to: relative_step off, parameter scaling off, no
 * first moment. beta2_t = 1 - t^decay_rate. Factored when rows > 1. */
int orc_adafactor_step(int64_t rows, int64_t cols, float* p, const void* g, int32_t g_bf16,
                       double lr, double eps1, double clip_d, double decay_rate, double wd,
                       int64_t t, orc_spec vs,
                       void* vr, float* vr_meta, void* vc, float* vc_meta,
                       void* v, float* v_meta,
                       double* yr, double* yc, double* yv) {
    if (rows < 1 || cols < 1 || t < 1) return -1;
    if (vs.codec != C_FP32 && vs.codec != C_AL8 && vs.codec != C_AL16) return -1;
    const int64_t n = rows * cols;
    const double beta2t = 1.0 - pow((double)t, decay_rate);
    const double decay = 1.0 - lr * wd;
    double* g2 = dbuf(n);
    double* u = dbuf(n);
    for (int64_t i = 0; i < n; i++) {
        double gi = grad_at(g, g_bf16, i);
        g2[i] = gi * gi + eps1;
    }
    int rc = 0;
    if (rows > 1) {
        double* rmean = dbuf(rows);
        double* cmean = dbuf(cols);
        float* R = fbuf(rows);
        float* C = fbuf(cols);
        row_col_means(rows, cols, g2, rmean, cmean);
        rc |= ema_state(vs, vr, vr_meta, rows, rmean, beta2t, R);
        rc |= ema_state(vs, vc, vc_meta, cols, cmean, beta2t, C);
        double meanR = mean_f32(R, rows);
        for (int64_t i = 0; i < rows; i++) {
            double ri = 1.0 / sqrt((double)R[i] / meanR);
            for (int64_t j = 0; j < cols; j++) {
                double cj = 1.0 / sqrt((double)C[j]);
                u[i * cols + j] = (ri * cj) * grad_at(g, g_bf16, i * cols + j);
            }
        }
        rc |= orc_state_encode(vs, R, rows, vr, vr_meta, yr);
        rc |= orc_state_encode(vs, C, cols, vc, vc_meta, yc);
        free(rmean);
        free(cmean);
        free(R);
        free(C);
    } else {
        float* V = fbuf(n);
        rc |= ema_state(vs, v, v_meta, n, g2, beta2t, V);
        for (int64_t i = 0; i < n; i++) u[i] = (1.0 / sqrt((double)V[i])) * grad_at(g, g_bf16, i);
        rc |= orc_state_encode(vs, V, n, v, v_meta, yv);
        free(V);
    }
    double rms = rms_of(u, n);
    double clip = rms / clip_d > 1.0 ? rms / clip_d : 1.0;
    for (int64_t i = 0; i < n; i++) {
        double pd = (double)p[i] * decay;
        pd = pd - lr * (u[i] / clip);
        p[i] = (float)pd;
    }
    free(g2);
    free(u);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* CAME (Luo et al.): Adafactor-style factored V, clipped update, momentum,  */
/* and factored confidence statistics of the squared residual between the    */
/* update and the momentum, which scale the momentum (section 3.1). No bias  */
/* correction. 1-D tensors: unfactored V, update = momentum.                 */
/* ------------------------------------------------------------------------ */
int orc_came_step(int64_t rows, int64_t cols, float* p, const void* g, int32_t g_bf16,
                  double lr, double beta1, double beta2, double beta3, double eps1, double eps2,
                  double clip_d, double wd, int64_t t,
                  orc_spec ms, orc_spec vs, orc_spec cs,
                  void* m, float* m_meta,
                  void* vr, float* vr_meta, void* vc, float* vc_meta,
                  void* v, float* v_meta,
                  void* cr, float* cr_meta, void* cc, float* cc_meta,
                  double* ym, double* yr, double* yc, double* yv, double* ycr, double* ycc) {
    if (rows < 1 || cols < 1 || t < 1) return -1;
    if (ms.codec != C_FP32 && ms.codec != C_UF8) return -1;
    if (vs.codec == C_UF8 || cs.codec == C_UF8) return -1;
    const int64_t n = rows * cols;
    const double decay = 1.0 - lr * wd;
    double* g2 = dbuf(n);
    double* u = dbuf(n);
    float* M = fbuf(n);
    for (int64_t i = 0; i < n; i++) {
        double gi = grad_at(g, g_bf16, i);
        g2[i] = gi * gi + eps1;
    }
    int rc = orc_state_decode(ms, m, m_meta, n, M);
    if (rows > 1) {
        double* rmean = dbuf(rows);
        double* cmean = dbuf(cols);
        float* R = fbuf(rows);
        float* C = fbuf(cols);
        row_col_means(rows, cols, g2, rmean, cmean);
        rc |= ema_state(vs, vr, vr_meta, rows, rmean, beta2, R);
        rc |= ema_state(vs, vc, vc_meta, cols, cmean, beta2, C);
        double meanR = mean_f32(R, rows);
        for (int64_t i = 0; i < rows; i++) {
            double ri = 1.0 / sqrt((double)R[i] / meanR);
            for (int64_t j = 0; j < cols; j++) {
                double cj = 1.0 / sqrt((double)C[j]);
                u[i * cols + j] = (ri * cj) * grad_at(g, g_bf16, i * cols + j);
            }
        }
        rc |= orc_state_encode(vs, R, rows, vr, vr_meta, yr);
        rc |= orc_state_encode(vs, C, cols, vc, vc_meta, yc);
        double rms = rms_of(u, n);
        double clip = rms / clip_d > 1.0 ? rms / clip_d : 1.0;
        double* res = dbuf(n);
        for (int64_t i = 0; i < n; i++) {
            float uh = (float)(u[i] / clip); /* the clipped update, an fp32 tensor */
            M[i] = (float)(beta1 * (double)M[i] + (1.0 - beta1) * (double)uh);
            double d = (double)uh - (double)M[i];
            res[i] = d * d + eps2;
        }
        float* Rc = fbuf(rows);
        float* Cc = fbuf(cols);
        row_col_means(rows, cols, res, rmean, cmean);
        rc |= ema_state(cs, cr, cr_meta, rows, rmean, beta3, Rc);
        rc |= ema_state(cs, cc, cc_meta, cols, cmean, beta3, Cc);
        double meanRc = mean_f32(Rc, rows);
        for (int64_t i = 0; i < rows; i++) {
            double si = 1.0 / sqrt((double)Rc[i] / meanRc);
            for (int64_t j = 0; j < cols; j++) {
                double sj = 1.0 / sqrt((double)Cc[j]);
                double upd = (si * sj) * (double)M[i * cols + j];
                double pd = (double)p[i * cols + j] * decay;
                p[i * cols + j] = (float)(pd - lr * upd);
            }
        }
        rc |= orc_state_encode(cs, Rc, rows, cr, cr_meta, ycr);
        rc |= orc_state_encode(cs, Cc, cols, cc, cc_meta, ycc);
        free(res);
        free(Rc);
        free(Cc);
        free(rmean);
        free(cmean);
        free(R);
        free(C);
    } else {
        float* V = fbuf(n);
        rc |= ema_state(vs, v, v_meta, n, g2, beta2, V);
        for (int64_t i = 0; i < n; i++) u[i] = (1.0 / sqrt((double)V[i])) * grad_at(g, g_bf16, i);
        rc |= orc_state_encode(vs, V, n, v, v_meta, yv);
        double rms = rms_of(u, n);
        double clip = rms / clip_d > 1.0 ? rms / clip_d : 1.0;
        for (int64_t i = 0; i < n; i++) {
            float uh = (float)(u[i] / clip);
            M[i] = (float)(beta1 * (double)M[i] + (1.0 - beta1) * (double)uh);
            double pd = (double)p[i] * decay;
            p[i] = (float)(pd - lr * (double)M[i]);
        }
        free(V);
    }
    rc |= orc_state_encode(ms, M, n, m, m_meta, ym);
    free(g2);
    free(u);
    free(M);
    return rc;
}
