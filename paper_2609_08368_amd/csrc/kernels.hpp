// Kernel argument blocks and launchers (host-visible; no torch types anywhere).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rl {

// Error bits accumulated in the device error word.
enum DeviceError : int {
  kErrLen = 1,       // a length outside [0, max_pages * P] (clamped)
  kErrPage = 2,      // a page id outside [0, num_pages) (clamped)
  kErrIndptr = 4,    // qo_indptr not non-decreasing within [0, total_q] (clamped)
  kErrKvShort = 8,   // kv_lens[b] < chunk length (clamped up)
  kErrScale = 16,    // an FP8 dequantisation scale that is not positive and finite
  kErrCapacity = 32, // the work of a call exceeded its workspace's capacity (affected
                     // outputs are NaN or left unwritten; the host sizing rules out this case)
};

// Slot markers of a decode piece: its result goes straight to out/lse, or
// nowhere (its sequence's partial slots did not fit the workspace).
constexpr int kSlotDirect = -1;
constexpr int kSlotDropped = -2;

// Paged KV cache + block table, shared by decode and extend.
struct PagedKV {
  const void* k;          // [num_pages, P, Hkv, 128] bf16
  const void* v;
  int64_t sp, ss, sh;     // page / slot / head strides (elements), identical for K and V
  int64_t v_sp, v_ss, v_sh;
  const int* bt;          // [B, max_pages] int32
  int64_t bt_sb, bt_sj;
  int num_pages, page_size, log2_page, max_pages;
  // FP8 E4M3 pages: one dequantisation scale per KV head ([Hkv] fp32, strides
  // in elements); null for bf16 pages
  const float* k_scale;
  const float* v_scale;
  int64_t ks_s, vs_s;
};

// Levels of nested shared prefix pages the decode planner detects: the prefix a
// trajectory group shares, then prefixes shared by subsets of it (sessions
// that branch after a common turn).
constexpr int kPrefixLevels = 3;

// Workspace carve-up of one decode call. Private keys: sequence b owns
// [pref[b], pref[b+1]) of the concatenation of all sequences' private key
// ranges (its keys S_b .. L_b - 1), and worker w of n takes the equal share
// [w W / n, (w+1) W / n) of it, cut at sequence boundaries into pieces.
// Shared items cover the prefix pages a node of trajectory-group members
// shares (see the planner) and serve every member of one sub-group (at most
// 128 query rows). Partial results
// live in "slots"; sequence b owns slots base[b] .. base[b] + nparts[b] - 1:
// its shared splits, then its private pieces in key order (nparts[b] == 0:
// one piece, written directly, or every row left to the extend pass a
// multi-token call queued; -1: an empty sequence, written by the combine;
// -2: its slots did not fit, so the combine writes NaN and the error word
// records kErrCapacity).
struct DecodePlanWs {
  int* hdr;        // [0] split tokens C of shared keys, [1] workers, [2] shared items, [3] sub-groups
  int* nparts;     // [B]
  int* base;       // [B]
  long long* pref; // [B + 1] prefix sums of private keys
  int4* seqs;      // [B] (shared keys S, slot of the first private piece, kSlotDirect or kSlotDropped, L,
                   //      1 if the sequence's slots fit the workspace)
  int4* sitems;    // [max_items] (sub-group, first key, end key, slot offset in each member's slots)
  int4* sgroups;   // [kPrefixLevels * B] (sequence whose block table is read, members, end key, splits)
  int2* sg_range;  // [kPrefixLevels * B] (first key, slot offset of the first split)
  int* sg_members; // [kPrefixLevels * B * group_cap] member sequences of each sub-group
  float* part_o;   // [max_slots, Hq, 128]
  float* part_lse; // [max_slots, Hq]
  int* err;        // device error word (persistent)
};

struct DecodeArgs {
  PagedKV kv;
  const void* q;
  int64_t q_sb, q_sh;
  // query tokens per sequence (multi-token decode: the sequence's last n_tok
  // keys are these tokens and token i sees keys t <= L - n_tok + i); token
  // strides of q, out and lse (unused when n_tok == 1)
  int n_tok;
  int64_t q_st, out_st, lse_st;
  // rows of the partial buffers and of the combine per sequence: n_tok * Hq,
  // row i * Hq + h for token i, query head h
  int Hv;
  const int* lens;
  int64_t lens_s;
  int B, Hq, Hkv, R;
  float scale;
  void* out;
  int out_f32;
  int64_t out_sb, out_sh;
  float* lse;             // nullable
  int64_t lse_sb, lse_sh;
  int forced_split;       // 0 = choose on device
  int target_items;       // shared splits the device planner aims for
  int max_items;          // capacity of the shared item list
  int max_workers;        // workers the private pass may use (its grid / workgroups per worker)
  int max_slots;          // capacity of the partial buffers
  int group_cap;          // members per sub-group (128 query rows / (n_tok * R)), 0 = no prefix sharing
  int prefix_grid;        // workgroups of the group-prefix pass (grid-stride over its work)
  int item_waves;         // waves per decode workgroup: a divisor of Hkv * ceil(R / 16), at most 8
  // multi-token decode with an extend pass queued behind it: when the planner
  // finds no shared prefix page, the split passes get no work (no workers, no
  // parts to combine) and the extend pass, gated on the sub-group count in
  // ws.hdr[3], computes every row
  int route_extend;
  DecodePlanWs ws;
};

struct ExtendPlanWs {
  int* hdr;        // [0] number of work units
  int4* items;     // [max_items] (sequence, first chunk row, chunk rows, KV head | head block << 16)
  int* err;
};

struct ExtendArgs {
  PagedKV kv;
  const void* q;
  int64_t q_st, q_sh;
  const int* qo_indptr;
  const int* kv_lens;
  int64_t kv_lens_s, indptr_s;
  int B, total_q, Hq, Hkv, R;
  int rows_head;          // query heads per tile (<= 64)
  int tile_tokens;        // chunk tokens per tile
  int head_blocks;        // ceil(R / rows_head)
  float scale;
  void* out;
  int out_f32;
  int64_t out_st, out_sh;
  float* lse;
  int64_t lse_st, lse_sh;
  int max_items;
  // n > 0: decode through the extend kernel: sequence b owns query rows
  // b n .. b n + n - 1, its last n keys (none if kv_lens[b] == 0; qo_indptr is
  // not read), and the rows of empty sequences are written as zeros with
  // lse = -inf
  int decode_rows;
  // nonzero: bf16 pages take the 64-key register-staged steps as FP8 pages do
  // (a multi-token decode routed through extend units, which owes extend no
  // bitwise agreement and streams its rows faster that way); zero: pages of
  // at least 64 keys take 128-key steps, as every extend and deterministic
  // decode does
  int staged;
  // nullable: the extend planner queues no unit (and writes nothing) when
  // *gate != 0, i.e. when the decode planner that runs before it found shared
  // prefix pages and the split passes compute the rows
  const int* gate;
  ExtendPlanWs ws;
};

struct MergeArgs {
  const float* o;        // [N, S, H, 128]
  int64_t o_sn, o_ss, o_sh;
  const float* lse;      // [N, S, H]
  int64_t l_sn, l_ss, l_sh;
  const int* num;        // [N]
  int64_t num_s;
  int N, S, H;
  void* out;
  int out_f32;
  int64_t out_sn, out_sh;
  float* lse_out;
  int64_t lo_sn, lo_sh;
};

// KV append: new rows [total_new, Hkv, 128] bf16 into their pages.
struct AppendArgs {
  const void* k_new;
  const void* v_new;
  int64_t kn_st, kn_sh, vn_st, vn_sh;
  void* k;                // pages, written
  void* v;
  int64_t sp, ss, sh, v_sp, v_ss, v_sh;
  const float* k_scale;   // FP8 pages: [Hkv] scales (null for bf16)
  const float* v_scale;
  int64_t ks_s, vs_s;
  const int* bt;
  int64_t bt_sb, bt_sj;
  const int* qo_indptr;
  int64_t indptr_s;
  const int* kv_lens;
  int64_t kv_lens_s;
  int B, total_new, Hkv, num_pages, page_size, log2_page, max_pages;
  int* err;
};

// Optional events around the main attention kernel (benchmark timing).
struct KernelTimer {
  hipEvent_t start = nullptr, stop = nullptr;
};

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream, KernelTimer* timer);

// Statically allocated device scratch of the allocation-free decode entry point:
// kScratchBytes per device; the first kScratchErrBytes hold its error word, the
// rest its workspace. scratch_address() returns the current device's copy (its
// address is looked up once per device, and the error word cleared then unless
// `stream` is being captured); scratch_address_if_set_up() returns it only if
// an earlier call already looked it up.
constexpr size_t kScratchBytes = size_t(160) << 20;
constexpr size_t kScratchErrBytes = 256;
hipError_t scratch_address(hipStream_t stream, void** ptr);
bool scratch_address_if_set_up(void** ptr);
// Measurement aids (see rl_attn_diag.h): a grid-stride read of `bytes` and a
// register-only bf16 MFMA loop.
hipError_t launch_diag_read(const void* buf, size_t bytes, unsigned* sink, int cus, hipStream_t stream);
hipError_t launch_diag_mfma(int iters, float* sink, int cus, hipStream_t stream);
double diag_mfma_flops(int iters, int cus);

// Workers of the private decode pass that are resident on one CU at a time
// (from the kernel's occupancy; a worker is one workgroup per wave group).
int decode_workers_per_cu(int R, int Hkv, int item_waves, bool fp8, int n_tok);
hipError_t launch_extend(const ExtendArgs& a, hipStream_t stream, KernelTimer* timer);
hipError_t launch_merge(const MergeArgs& a, hipStream_t stream);
hipError_t launch_append(const AppendArgs& a, hipStream_t stream, KernelTimer* timer);

}  // namespace rl
