/*
 * rl_attn.h -- paged-KV grouped-query attention for rollout engines (gfx950).
 *
 * The operation: the rollout engines of an RL post-training loop spend most
 * of their time generating (paper, section "Rollout", opening paragraph), and
 * each turn of an agentic session reuses the cached context of earlier turns,
 * so a turn only prefills its newly appended suffix (section "Fast Agentic
 * Rollout with SGLang"). That gives two attention calls over a paged KV cache:
 *
 *   decode : one query token per sequence attends to its whole context;
 *   extend : a chunk of appended tokens attends to the cached prefix and,
 *            causally, to itself.
 *
 * Trajectories of one group (G attempts at the same prompt, section "The
 * Miles RL Loop") reference the same physical pages for the prompt, and the
 * library reads such shared pages once per group.
 *
 * Math (scaled dot-product attention with grouped-query heads):
 *   R = Hq / Hkv, query head h reads KV head g = h / R;
 *   s_t = scale * dot(q[h], K[t, g]);  out[h] = sum_t softmax(s)_t V[t, g];
 *   lse[h] = ln sum_t exp(s_t)  (natural log, scale included).
 * Logical token t of sequence b lives in page block_table[b][t / P], slot t % P.
 * Decode: t < seq_lens[b]. Extend: sequence b owns query rows
 * qo_indptr[b] .. qo_indptr[b+1]-1 (n_b rows); its pages hold kv_lens[b]
 * tokens, the last n_b of which are the chunk itself (already written);
 * row i attends to t <= kv_lens[b] - n_b + i (bottom-right causal mask).
 * An empty key range gives out = 0 and lse = -inf.
 *
 * Tensors: every argument is a non-owning view. dtype/ndim/shape are checked
 * on the host; strides are in elements and free except that the last (head
 * dimension) stride must be 1 (page strides below 2^32 elements, slot strides
 * and block-table column strides below 2^24). All pointers are device pointers on the
 * current HIP device. The library only reads q, pages, tables and lengths and
 * only writes out / lse_out. Head dimension must be 128; Hq % Hkv == 0;
 * page size P must be a power of two in [8, 128]. Sizes: B <= 2^22,
 * Hq <= 4096, B * n * Hq < 2^31 for decode (n query tokens per sequence),
 * total_q < 2^30 for extend, num_pages and max_pages * P below 2^31
 * (RL_ERR_UNSUPPORTED otherwise).
 *
 * Errors: every call returns RL_OK (0) or a negative RL_ERR_* code, and
 * rl_attn_last_error() returns a thread-local message for the last failure on
 * the calling thread. Host-side validation happens before any HIP call.
 * Calls are asynchronous on `stream` (a hipStream_t; NULL = default stream);
 * a launch failure returns RL_ERR_HIP. Calls on distinct streams are
 * thread-safe. Page ids and lengths read on the device are clamped into the
 * valid ranges, so no input can make a kernel read outside the given buffers;
 * out-of-range values are counted in a device error word that
 * rl_attn_check_device_errors() reports (as are invalid FP8 dequantisation scales).
 *
 * Memory: the library owns one workspace per (device, stream), grown with
 * hipMalloc on demand (or ahead of time with rl_attn_reserve_workspace) and
 * never grown while the stream is being captured (RL_ERR_WORKSPACE instead).
 * A graph captured on a stream uses that stream's workspace when replayed:
 * replay it on the capture stream (or ordered with it), since calls that share
 * a workspace must not overlap. Once a call was captured on a stream, a later
 * growth of its workspace keeps the old buffer allocated, so graphs captured
 * before stay valid; rl_attn_release() frees it, after which such graphs must
 * not be replayed.
 */
#ifndef RL_ATTN_H
#define RL_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* RL_FP8_E4M3: one byte per element, the OCP 8-bit E4M3 format (exponent bias
 * 7, no infinities, 0x7F/0xFF are NaN, largest finite magnitude 448). */
enum rl_dtype { RL_BF16 = 1, RL_F32 = 2, RL_I32 = 3, RL_FP8_E4M3 = 4 };

enum rl_status {
  RL_OK = 0,
  RL_ERR_INVALID_ARG = -1,  /* null pointer, negative size, bad option value   */
  RL_ERR_SHAPE = -2,        /* shapes inconsistent with each other             */
  RL_ERR_DTYPE = -3,        /* wrong element type                              */
  RL_ERR_UNSUPPORTED = -4,  /* head_dim != 128, page size, non-unit last stride */
  RL_ERR_WORKSPACE = -5,    /* workspace cannot be allocated (or capture)      */
  RL_ERR_HIP = -6,          /* a HIP runtime call or kernel launch failed      */
  RL_ERR_DEVICE = -7        /* device-side data errors were detected           */
};

/* Non-owning tensor view (DLPack-like). shape/strides beyond ndim are ignored. */
typedef struct {
  void* data;          /* device pointer (host pointers are never dereferenced) */
  int32_t dtype;       /* enum rl_dtype                                         */
  int32_t ndim;        /* 1..4                                                  */
  int64_t shape[4];
  int64_t strides[4];  /* in elements                                           */
} rl_tensor;

enum rl_prefix_mode { RL_PREFIX_AUTO = 0, RL_PREFIX_OFF = 1 };

/* Options for the _ex calls. A NULL pointer means all defaults (zeros). */
typedef struct {
  int32_t split_tokens;  /* decode: keys per split-KV partial (private keys: per
                            worker share; group-shared keys: per shared split);
                            0 = automatic, otherwise a multiple of 64
                            (RL_ERR_INVALID_ARG if not)                          */
  int32_t prefix_share;  /* enum rl_prefix_mode: read group-shared prefix pages once
                            (AUTO) or treat every sequence independently (OFF).
                            With automatic splits and more than one query token
                            per sequence (q, out and lse with batch stride =
                            tokens x token stride), decode runs as in the
                            deterministic mode (one extend unit per sequence and
                            KV head, no split of the keys; faster when no pages
                            are shared, and batch-invariant): with OFF always;
                            with AUTO and bf16 pages when the device finds no
                            shared prefix page in the batch (both passes are
                            queued, the one not needed does no work)            */
  int32_t validate;      /* accepted for compatibility, no effect: every page id a
                            kernel reads is range-checked on every call           */
  int32_t deterministic; /* decode: 1 = batch-invariant and equal to extend. Each
                            sequence is computed by the extend kernel as one query
                            row, with no split of its keys, so its out and lse do
                            not depend on the other sequences of the batch (their
                            number, order or lengths) and are bitwise equal to
                            rl_attn_extend_ex of that token (paper: section
                            "True-On-Policy Alignment" asks for prefill and decode
                            paths that agree bitwise, and for batch invariance).
                            Slower on long contexts (no key split). Extend rows
                            are always invariant in this sense: a row's result
                            does not depend on the other rows of its chunk, the
                            chunk's length or the batch, so a prefill of a whole
                            chunk and its tokens appended one at a time agree
                            bitwise. 0 = default split-KV decode (results depend
                            on the batch within the stated tolerance)            */
  int32_t reserved[4];   /* must be zero                                          */
} rl_attn_opts;

/* Batched decode (paper: batched generation by the rollout engines).
 *   q           [B, Hq, 128] bf16, or [B, n, Hq, 128] for n query tokens per
 *               sequence (1 <= n <= 64; multi-token decode, e.g. verifying the
 *               draft tokens of multi-token prediction, which the case study's
 *               rollout engines use: section "Case Study", subsection
 *               "Configuration"). The n tokens are the last n of the sequence
 *               (their K/V already in the pages) and token i sees keys
 *               t <= seq_lens[b] - n + i; out is [B, n, Hq, 128] and lse_out
 *               [B, n, Hq]. The _fp8 call accepts the same shapes.
 *   k_pages     [num_pages, P, Hkv, 128] bf16
 *   v_pages     same shape and dtype as k_pages
 *   block_table [B, max_pages] int32 (entries past ceil(seq_lens[b]/P) are never read)
 *   seq_lens    [B] int32, 0 <= seq_lens[b] <= max_pages * P
 *   scale       softmax scale (e.g. 1/sqrt(128)); must be positive and finite
 *   out         [B, Hq, 128] bf16 (f32 also accepted), written
 * Returns RL_OK or an RL_ERR_* code. */
int rl_attn_decode(const rl_tensor* q, const rl_tensor* k_pages, const rl_tensor* v_pages,
                   const rl_tensor* block_table, const rl_tensor* seq_lens, float scale,
                   rl_tensor* out, void* stream);

/* Causal extend of appended chunks (paper: each turn prefills only its suffix).
 *   q           [total_q, Hq, 128] bf16
 *   qo_indptr   [B+1] int32, qo_indptr[0] = 0, non-decreasing, qo_indptr[B] = total_q
 *   k_pages, v_pages, block_table as for decode
 *   kv_lens     [B] int32, kv_lens[b] >= n_b (prefix + chunk)
 *   out         [total_q, Hq, 128] bf16 (f32 also accepted), written */
int rl_attn_extend(const rl_tensor* q, const rl_tensor* qo_indptr, const rl_tensor* k_pages,
                   const rl_tensor* v_pages, const rl_tensor* block_table, const rl_tensor* kv_lens,
                   float scale, rl_tensor* out, void* stream);

/* Same as rl_attn_decode, plus an optional log-sum-exp output lse_out
 * ([B, Hq] f32, natural log; NULL = not written) and options (NULL = defaults). */
int rl_attn_decode_ex(const rl_tensor* q, const rl_tensor* k_pages, const rl_tensor* v_pages,
                      const rl_tensor* block_table, const rl_tensor* seq_lens, float scale,
                      rl_tensor* out, rl_tensor* lse_out, const rl_attn_opts* opts, void* stream);

/* Same as rl_attn_extend, plus lse_out ([total_q, Hq] f32, nullable) and options. */
int rl_attn_extend_ex(const rl_tensor* q, const rl_tensor* qo_indptr, const rl_tensor* k_pages,
                      const rl_tensor* v_pages, const rl_tensor* block_table, const rl_tensor* kv_lens,
                      float scale, rl_tensor* out, rl_tensor* lse_out, const rl_attn_opts* opts,
                      void* stream);

/* Allocation-free decode, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc). Arguments, results and options are those of rl_attn_decode_ex
 * (bf16 pages), and it runs the same kernels; its workspace is instead a
 * statically allocated array of 160 MiB per device (its first 256 bytes are an
 * error word), held by every device the library runs on until the process ends.
 * The call makes no hipMalloc, hipFree or other allocating call.
 * Limit: a call whose workspace would exceed 160 MiB - 256 B is rejected with
 * RL_ERR_WORKSPACE before any launch (the workspace grows with the batch, the
 * query heads and query tokens per sequence, and, with a forced split, with
 * max_pages * page_size / split_tokens; e.g. batch 128 with 96 query heads, one
 * token, automatic split, fits). Every call on a device shares that device's
 * array, which keeps the last call's contents: calls that overlap on one
 * device (e.g. on two streams) race; order them on one stream. Device-side
 * input errors of these calls go to the array's error word, which
 * rl_attn_check_device_errors reports on any stream of the device (after
 * synchronising only the stream it is given). */
int rl_attn_decode_noalloc(const rl_tensor* q, const rl_tensor* k_pages, const rl_tensor* v_pages,
                           const rl_tensor* block_table, const rl_tensor* seq_lens, float scale,
                           rl_tensor* out, rl_tensor* lse_out, const rl_attn_opts* opts, void* stream);

/* FP8 KV pages (paper: the rollout engine of the case study, section "Case
 * Study", subsection "Configuration" and its configuration table, serves with
 * an FP8 key-value cache; section "Low-Precision Training" describes the
 * "BF16 train, FP8 serve" arrangement). The paper gives no KV cache format,
 * so the cache here holds E4M3 codes with one fp32 dequantisation scale per
 * KV head. Key t of head g has the value k_scale[g] * E4M3(k_pages[..]), value
 * rows v_scale[g] * E4M3(v_pages[..]); the attention is otherwise exactly
 * rl_attn_decode_ex / rl_attn_extend_ex on those values.
 *   k_pages, v_pages  [num_pages, P, Hkv, 128] RL_FP8_E4M3 (strides as for bf16,
 *                     but multiples of 16 elements)
 *   k_scale, v_scale  [Hkv] f32, device pointers; each entry must be positive
 *                     and finite (checked on the device: a bad scale is
 *                     reported by rl_attn_check_device_errors and its head's
 *                     output is not meaningful)
 * Codes are converted exactly to bf16 for the matrix products. Pages must
 * hold no NaN codes (0x7F, 0xFF) in the rows a call reads: the outputs of a
 * KV head that reads one are unspecified. Everything else (q, out, lse_out, opts, errors) is as for the
 * bf16 calls. */
int rl_attn_decode_fp8(const rl_tensor* q, const rl_tensor* k_pages, const rl_tensor* v_pages,
                       const rl_tensor* k_scale, const rl_tensor* v_scale, const rl_tensor* block_table,
                       const rl_tensor* seq_lens, float scale, rl_tensor* out, rl_tensor* lse_out,
                       const rl_attn_opts* opts, void* stream);

int rl_attn_extend_fp8(const rl_tensor* q, const rl_tensor* qo_indptr, const rl_tensor* k_pages,
                       const rl_tensor* v_pages, const rl_tensor* k_scale, const rl_tensor* v_scale,
                       const rl_tensor* block_table, const rl_tensor* kv_lens, float scale, rl_tensor* out,
                       rl_tensor* lse_out, const rl_attn_opts* opts, void* stream);

/* KV append (paper: each agentic turn prefills only its newly appended
 * suffix, section "Fast Agentic Rollout with SGLang", and every decode step
 * adds one token): writes the new tokens' K and V rows into their pages, in
 * the addressing the attention calls use.
 *   k_new, v_new [total_new, Hkv, 128] bf16: rows qo_indptr[b] .. qo_indptr[b+1]-1
 *                are sequence b's new tokens, in order
 *   qo_indptr    [B+1] int32, non-decreasing from 0 to total_new
 *   block_table  [B, max_pages] int32 (the pages of the new positions must be assigned)
 *   kv_lens      [B] int32: tokens of sequence b after the append (>= n_b); new
 *                row i of sequence b goes to logical position kv_lens[b] - n_b + i
 *   k_pages, v_pages [num_pages, P, Hkv, 128]: only the new positions are written
 * The bf16 call copies the rows. The FP8 call takes E4M3 pages and the
 * per-KV-head scales of rl_attn_decode_fp8 and writes, for each element x of
 * KV head g, the E4M3 code nearest to the float32 quotient x / scale[g] (ties
 * to the even code; magnitudes above 448 saturate to 448). A row whose page id,
 * length or indptr is out of range (or whose scale is not positive and finite)
 * is not written and is reported by rl_attn_check_device_errors(); rows that
 * map to the same position race. Asynchronous on `stream`; allocates nothing
 * beyond the library's per-stream error word. */
int rl_attn_append_kv(const rl_tensor* k_new, const rl_tensor* v_new, const rl_tensor* qo_indptr,
                      const rl_tensor* block_table, const rl_tensor* kv_lens, rl_tensor* k_pages,
                      rl_tensor* v_pages, void* stream);

int rl_attn_append_kv_fp8(const rl_tensor* k_new, const rl_tensor* v_new, const rl_tensor* qo_indptr,
                          const rl_tensor* block_table, const rl_tensor* kv_lens, rl_tensor* k_pages,
                          rl_tensor* v_pages, const rl_tensor* k_scale, const rl_tensor* v_scale,
                          void* stream);

/* Log-sum-exp merge of partial attention results over disjoint key ranges
 * (the split-KV combine, exposed for testing and for callers that split work
 * themselves):
 *   o_parts   [N, S, H, 128] f32     lse_parts [N, S, H] f32 (natural log)
 *   num_parts [N] int32, 0 <= num_parts[n] <= S (only the first num_parts[n] count)
 *   out       [N, H, 128] bf16 or f32    lse_out [N, H] f32 (nullable)
 * With M = max_s lse_s, w_s = exp(lse_s - M): out = sum w_s o_s / sum w_s,
 * lse = M + ln sum w_s; parts with lse = -inf carry no weight; if all do,
 * out = 0 and lse = -inf. */
int rl_attn_merge(const rl_tensor* o_parts, const rl_tensor* lse_parts, const rl_tensor* num_parts,
                  rl_tensor* out, rl_tensor* lse_out, void* stream);

/* Thread-local message describing the last non-OK return on this thread. */
const char* rl_attn_last_error(void);

/* Synchronises `stream`, then returns RL_ERR_DEVICE if any call on this
 * (device, stream) since the last check met an out-of-range page id, length
 * or indptr on the device (those values were clamped), an invalid FP8 scale,
 * or work beyond its workspace's capacity, RL_OK otherwise, and clears the
 * error word. Errors of rl_attn_decode_noalloc calls on this device are
 * included, whatever their stream. Allocates nothing. */
int rl_attn_check_device_errors(void* stream);

/* Grows this (device, stream)'s workspace to at least `bytes` now, so later
 * calls (e.g. under stream capture) need no allocation. */
int rl_attn_reserve_workspace(size_t bytes, void* stream);

/* Workspace bytes a decode / extend call with these sizes may need on the
 * current device, for rl_attn_reserve_workspace ahead of stream capture.
 * Decode: query_tokens query tokens per sequence (1 for a 3-D q, n for q
 * [B, n, Hq, 128]) and split_tokens the opts.split_tokens the call will pass
 * (0 = automatic); the size covers bf16 and FP8 pages, prefix sharing on or off
 * and the deterministic mode. Returns 0 for sizes a call would reject. */
size_t rl_attn_decode_workspace_size(int64_t batch, int64_t num_q_heads, int64_t num_kv_heads,
                                     int64_t max_pages, int64_t page_size, int64_t query_tokens,
                                     int32_t split_tokens);
size_t rl_attn_extend_workspace_size(int64_t batch, int64_t total_q, int64_t num_q_heads,
                                     int64_t num_kv_heads, int64_t max_pages, int64_t page_size);

/* Kernel timing for benchmarks and profiling tools. While enabled, each
 * decode / extend / append call brackets its main kernel with a pair of HIP
 * events on the call's stream (the planner and combine kernels are outside
 * the pair). rl_attn_profile_read() waits for the recorded events and returns
 * the number of timed launches and their mean duration in milliseconds per
 * kind (kind 0 = decode attention kernel, 1 = extend attention kernel, 2 =
 * KV append kernel; a deterministic decode counts as kind 0), then forgets
 * them. Disabled by default; enabling costs two event records per call. */
int rl_attn_profile_enable(int on);
int rl_attn_profile_read(int kind, int* launches, double* mean_ms);

/* Frees every workspace the library holds (synchronises the device first),
 * including buffers kept for graphs captured earlier: replaying such a graph
 * afterwards is an error. */
void rl_attn_release(void);

#ifdef __cplusplus
}
#endif

#endif /* RL_ATTN_H */
