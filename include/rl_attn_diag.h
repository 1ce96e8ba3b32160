/*
 * rl_attn_diag.h -- measurement aids for benchmark reports (gfx950).
 *
 * Not part of the attention operation: these calls measure, on the running
 * device, the ceilings that the attention kernels are reported against (the
 * attainable HBM read bandwidth and the bf16 matrix-core rate). Both
 * synchronise `stream` (a hipStream_t; NULL =
 * default stream), allocate a few bytes of device memory for the duration of
 * the call, and return RL_OK or a negative RL_ERR_* code (rl_attn.h), with
 * rl_attn_last_error() describing a failure.
 */
#ifndef RL_ATTN_DIAG_H
#define RL_ATTN_DIAG_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Streams `bytes` of the device buffer `buf` (16-byte aligned, bytes a
 * positive multiple of 16) through 16-byte loads `reps` times after one
 * warm-up pass, and writes the read rate in GB/s (1e9 bytes per second) to
 * *gb_per_s. The buffer's contents are not used. */
int rl_attn_diag_read_bandwidth(const void* buf, int64_t bytes, int32_t reps, double* gb_per_s, void* stream);

/* Runs `iters` rounds of 32 32x32x16 bf16 MFMAs (four accumulator chains)
 * per wave, two waves per SIMD on every CU, operands in registers, and
 * writes the rate in TFLOP/s (2 flops per multiply-add) to *tflop_per_s.
 * iters must be in [1, 2^24]. */
int rl_attn_diag_mfma_bf16(int64_t iters, double* tflop_per_s, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RL_ATTN_DIAG_H */
