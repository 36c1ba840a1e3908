/*
 * al_synth.h -- seeded synthetic-input fill (part of libal.so).
 *
 * Not part of the optimizer: it only writes benchmark and test inputs into
 * device memory, with the same counter-based definition as the host
 * generator paper_2608_22322_amd/synth.py, so any element can be regenerated
 * on the host bit for bit:
 *
 *   w_k = mix64(key + (3e + k + 1) * 0x9E3779B97F4A7C15), k = 0, 1, 2 (mod 2^64)
 *   S   = sum of the twelve 16-bit fields of w_0, w_1, w_2
 *   v   = fl32(fl32(S - 393210) * scale)
 *   v   = 0 if mix64(mask_key + (e + 1) * 0x9E3779B97F4A7C15) < mask_threshold
 *   out = v (AL_DTYPE_F32) or v rounded to bfloat16, nearest even (AL_DTYPE_BF16)
 *
 * mix64 is the SplitMix64 output function. S - 393210 is a centred
 * Irwin-Hall(12) variate of standard deviation sqrt(65536^2 - 1), so
 * scale = sigma / sqrt(65536^2 - 1) gives an approximately N(0, sigma^2) draw.
 */
#ifndef AL_SYNTH_H
#define AL_SYNTH_H

#include <stdint.h>

#include "al.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Fill out[0..n) (device memory, 16-byte aligned) on `stream`.
 * out_dtype: AL_DTYPE_F32 or AL_DTYPE_BF16. mask_threshold 0 disables the
 * zero mask. Returns AL_EINVAL / AL_EALIGN / AL_EHIP like the other calls. */
al_status al_synth_normal(void* out, int32_t out_dtype, int64_t n, uint64_t key, float scale, uint64_t mask_key,
                          uint64_t mask_threshold, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* AL_SYNTH_H */
