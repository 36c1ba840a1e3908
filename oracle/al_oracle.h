/*
 * al_oracle.h -- TEST INFRASTRUCTURE. Not part of the product path.
 *
 * Declarations of the plain, slow, single-threaded binary64 CPU reference
 * ("oracle") for the Adaptive Log-Space (AL) codec, the uniform signed 8-bit
 * momentum code (UF8) and the AdamW / Adafactor / CAME quantized optimizer
 * steps. Only the test suite, the smoke check and the benchmark's CPU
 * baseline load it. It shares no code, header or constant with the HIP
 * library.
 *
 * All functions return 0 on success and a negative value on a bad argument.
 * Arrays are plain host memory. A state is stored under a spec:
 *   codec 0 = FP32  (float array of n, no metadata)
 *   codec 1 = AL8   (uint8 codes, ceil(n/B)*B of them; 2 floats per block)
 *   codec 2 = AL16  (uint16 codes, ceil(n/B)*B; 2 floats per block)
 *   codec 3 = UF8   (int8 codes, ceil(n/B)*B; 1 float per block)
 * Padded code positions beyond n are written as 0.
 * Optional `y` outputs (may be NULL) receive each element's pre-rounding code
 * position (NaN where no rounding decision is taken).
 */
#ifndef AL_ORACLE_H
#define AL_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int32_t codec;
    int32_t block;
    float log_floor;
} orc_spec;

double orc_exact_sum(const double* x, int64_t n);

int orc_al_quantize(int32_t bits, const float* x, int64_t n, int32_t block, float log_floor,
                    void* codes, float* meta, double* y);
int orc_al_dequantize(int32_t bits, const void* codes, const float* meta, int64_t n,
                      int32_t block, float* out);
int orc_uf8_quantize(const float* x, int64_t n, int32_t block, int8_t* codes, float* meta,
                     double* y);
int orc_uf8_dequantize(const int8_t* codes, const float* meta, int64_t n, int32_t block,
                       float* out);
int orc_state_decode(orc_spec s, const void* codes, const float* meta, int64_t n, float* out);
int orc_state_encode(orc_spec s, const float* x, int64_t n, void* codes, float* meta, double* y);

int orc_adamw_step(int64_t n, float* p, const void* g, int32_t g_bf16,
                   double lr, double beta1, double beta2, double eps, double wd, int64_t t,
                   orc_spec ms, void* m, float* m_meta, orc_spec vs, void* v, float* v_meta,
                   double* ym, double* yv);

int orc_adafactor_step(int64_t rows, int64_t cols, float* p, const void* g, int32_t g_bf16,
                       double lr, double eps1, double clip_d, double decay_rate, double wd,
                       int64_t t, orc_spec vs,
                       void* vr, float* vr_meta, void* vc, float* vc_meta,
                       void* v, float* v_meta,
                       double* yr, double* yc, double* yv);

int orc_came_step(int64_t rows, int64_t cols, float* p, const void* g, int32_t g_bf16,
                  double lr, double beta1, double beta2, double beta3, double eps1, double eps2,
                  double clip_d, double wd, int64_t t,
                  orc_spec ms, orc_spec vs, orc_spec cs,
                  void* m, float* m_meta,
                  void* vr, float* vr_meta, void* vc, float* vc_meta,
                  void* v, float* v_meta,
                  void* cr, float* cr_meta, void* cc, float* cc_meta,
                  double* ym, double* yr, double* yc, double* yv, double* ycr, double* ycc);

#ifdef __cplusplus
}
#endif
#endif
