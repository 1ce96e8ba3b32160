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

/* Workspace capacities a decode call would be given (host arithmetic only, no
 * HIP call), for tests of the sizing argument: the device planners must never
 * need more than these. Sizes as for rl_attn_decode_workspace_size, with the
 * device's compute units `cus` and private-pass workers per CU `workers_per_cu`
 * given explicitly. Writes out[0..6] = shared-item capacity, partial-slot
 * capacity, private-pass workers, members per trajectory sub-group (0 = no
 * prefix sharing), the shared-split item target, the group-prefix grid, and
 * the workspace bytes. Returns RL_OK or RL_ERR_INVALID_ARG. */
int rl_attn_diag_decode_capacity(int64_t batch, int64_t num_q_heads, int64_t num_kv_heads, int64_t max_pages,
                                 int64_t page_size, int64_t query_tokens, int32_t split_tokens, int32_t prefix_share,
                                 int32_t cus, int32_t workers_per_cu, int64_t* out);

/* Extend (and deterministic decode) work-unit capacity (host arithmetic only):
 * out[0..3] = unit capacity, query heads per unit, chunk tokens per unit, head
 * blocks per KV head. Returns RL_OK or RL_ERR_INVALID_ARG. */
int rl_attn_diag_extend_capacity(int64_t batch, int64_t total_q, int64_t num_q_heads, int64_t num_kv_heads,
                                 int64_t* out);

#ifdef __cplusplus
}
#endif

#endif /* RL_ATTN_DIAG_H */
