// Host side of the C-ABI: argument validation, per-(device, stream)
// workspaces, error reporting and kernel dispatch. Every check that can fail
// on the host runs before the first HIP runtime call.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <tuple>
#include <utility>
#include <vector>

#include "kernels.hpp"
#include "rl_attn.h"
#include "rl_attn_diag.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(RL_ERR_HIP, "%s failed: %s", what, hipGetErrorString(e));
}

// ------------------------------------------------------------------ options
struct EnvDefaults {
  int split_tokens = 0;
  int prefix_share = RL_PREFIX_AUTO;
  int deterministic = 0;
  int target_wgs_per_cu = 64;
  int workers_per_cu = 0;   // 0: as many as are resident at once
  bool fail_alloc = false;
};

const EnvDefaults& env() {
  static EnvDefaults d = [] {
    EnvDefaults e;
    if (const char* s = std::getenv("RL_ATTN_SPLIT_TOKENS")) e.split_tokens = std::atoi(s);
    if (const char* s = std::getenv("RL_ATTN_PREFIX_SHARE")) e.prefix_share = std::strcmp(s, "off") == 0;
    if (const char* s = std::getenv("RL_ATTN_DETERMINISTIC")) e.deterministic = std::atoi(s) != 0;
    if (const char* s = std::getenv("RL_ATTN_TARGET_WGS_PER_CU")) e.target_wgs_per_cu = std::max(1, std::atoi(s));
    if (const char* s = std::getenv("RL_ATTN_WORKERS_PER_CU")) e.workers_per_cu = std::max(0, std::atoi(s));
    if (const char* s = std::getenv("RL_ATTN_TEST_FAIL_ALLOC")) e.fail_alloc = std::atoi(s) != 0;
    return e;
  }();
  return d;
}

struct Opts {
  int split_tokens, prefix_share, deterministic;
};

int read_opts(const rl_attn_opts* o, Opts* out) {
  const EnvDefaults& e = env();
  *out = {e.split_tokens, e.prefix_share, e.deterministic};
  if (!o) return RL_OK;
  for (int i = 0; i < 4; ++i)
    if (o->reserved[i] != 0) return fail(RL_ERR_INVALID_ARG, "opts.reserved[%d] must be zero", i);
  if (o->split_tokens < 0 || o->split_tokens % 64 != 0)
    return fail(RL_ERR_INVALID_ARG, "opts.split_tokens must be 0 or a positive multiple of 64 (got %d)",
                o->split_tokens);
  if (o->prefix_share != RL_PREFIX_AUTO && o->prefix_share != RL_PREFIX_OFF)
    return fail(RL_ERR_INVALID_ARG, "opts.prefix_share must be RL_PREFIX_AUTO or RL_PREFIX_OFF");
  // validate: kept in the struct; page ids are always checked where read
  if (o->validate != 0 && o->validate != 1) return fail(RL_ERR_INVALID_ARG, "opts.validate must be 0 or 1");
  if (o->deterministic != 0 && o->deterministic != 1)
    return fail(RL_ERR_INVALID_ARG, "opts.deterministic must be 0 or 1");
  if (o->split_tokens) out->split_tokens = o->split_tokens;
  out->prefix_share = o->prefix_share;
  out->deterministic = o->deterministic || e.deterministic;
  return RL_OK;
}

// --------------------------------------------------------------- validation
const char* dtype_name(int d) {
  switch (d) {
    case RL_BF16: return "bf16";
    case RL_F32: return "f32";
    case RL_I32: return "int32";
    case RL_FP8_E4M3: return "fp8_e4m3";
    default: return "unknown";
  }
}

int check_view(const rl_tensor* t, const char* name, int ndim) {
  if (!t) return fail(RL_ERR_INVALID_ARG, "%s is NULL", name);
  if (t->ndim != ndim) return fail(RL_ERR_SHAPE, "%s must have %d dimensions (got %d)", name, ndim, t->ndim);
  for (int i = 0; i < ndim; ++i)
    if (t->shape[i] < 0) return fail(RL_ERR_INVALID_ARG, "%s.shape[%d] is negative", name, i);
  return RL_OK;
}

int64_t numel(const rl_tensor* t) {
  int64_t n = 1;
  for (int i = 0; i < t->ndim; ++i) n *= t->shape[i];
  return n;
}

int check_data(const rl_tensor* t, const char* name) {
  if (numel(t) > 0 && !t->data) return fail(RL_ERR_INVALID_ARG, "%s.data is NULL", name);
  return RL_OK;
}

int check_dtype(const rl_tensor* t, const char* name, int dtype) {
  if (t->dtype != dtype)
    return fail(RL_ERR_DTYPE, "%s must be %s (got %s)", name, dtype_name(dtype), dtype_name(t->dtype));
  return RL_OK;
}

// A tensor whose last dimension is the 128-wide head dimension, read or
// written 16 bytes at a time: unit last stride, other strides multiples of
// 8 elements, 16-byte aligned base.
int check_rows128(const rl_tensor* t, const char* name) {
  if (t->shape[t->ndim - 1] != 128)
    return fail(RL_ERR_UNSUPPORTED, "%s: head dimension must be 128 (got %lld)", name,
                (long long)t->shape[t->ndim - 1]);
  if (t->strides[t->ndim - 1] != 1) return fail(RL_ERR_UNSUPPORTED, "%s: last stride must be 1", name);
  for (int i = 0; i < t->ndim - 1; ++i)
    if (t->strides[i] % 8 != 0 || t->strides[i] < 0)
      return fail(RL_ERR_UNSUPPORTED, "%s: stride[%d] must be a non-negative multiple of 8 elements", name, i);
  if (reinterpret_cast<uintptr_t>(t->data) % 16 != 0)
    return fail(RL_ERR_UNSUPPORTED, "%s: data must be 16-byte aligned", name);
  return RL_OK;
}

// The kernels take the row maximum of raw scores and fold the scale into the
// exponent, which needs a positive, finite scale.
int check_scale(float scale) {
  if (!(scale > 0.f) || !std::isfinite(scale))
    return fail(RL_ERR_INVALID_ARG, "scale must be positive and finite (got %g)", (double)scale);
  return RL_OK;
}

#define RL_TRY(x)          \
  do {                     \
    int rc_ = (x);         \
    if (rc_ != RL_OK) return rc_; \
  } while (0)

// ---------------------------------------------------------------- workspace
struct Workspace {
  void* ptr = nullptr;
  size_t size = 0;
  int* err = nullptr;
  // set once a call on this stream was captured into a graph: the graph keeps
  // the buffer's address, so a later growth retires the buffer (freed by
  // rl_attn_release) instead of freeing it
  bool captured = false;
  std::vector<void*> retired;
};

std::mutex g_mu;
std::map<std::pair<int, hipStream_t>, Workspace> g_ws;
std::map<int, int> g_cus;

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int device_cus(int dev) {
  std::lock_guard<std::mutex> lk(g_mu);
  auto it = g_cus.find(dev);
  if (it != g_cus.end()) return it->second;
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
  g_cus[dev] = n;
  return n;
}

int acquire_ws(hipStream_t st, size_t need, Workspace** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> lk(g_mu);
  Workspace& w = g_ws[{dev, st}];
  const bool need_err = w.err == nullptr;
  const bool grow = w.size < need;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  e = hipStreamIsCapturing(st, &cs);
  if (e != hipSuccess) return hip_fail(e, "hipStreamIsCapturing");
  const bool capturing = cs != hipStreamCaptureStatusNone;
  if (need_err || grow) {
    if (capturing)
      return fail(RL_ERR_WORKSPACE,
                  "workspace must grow to %zu bytes while the stream is being captured; call "
                  "rl_attn_reserve_workspace first",
                  need);
    if (env().fail_alloc) return fail(RL_ERR_WORKSPACE, "workspace allocation failed (RL_ATTN_TEST_FAIL_ALLOC)");
  }
  if (need_err) {
    void* p = nullptr;
    e = hipMalloc(&p, 256);
    if (e != hipSuccess) return fail(RL_ERR_WORKSPACE, "hipMalloc(256) for the error word failed: %s", hipGetErrorString(e));
    e = hipMemset(p, 0, 256);
    if (e != hipSuccess) return hip_fail(e, "hipMemset");
    w.err = static_cast<int*>(p);
  }
  if (grow) {
    if (w.ptr) {
      e = hipStreamSynchronize(st);
      if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
      if (w.captured)
        w.retired.push_back(w.ptr);
      else
        (void)hipFree(w.ptr);
      w.ptr = nullptr;
      w.size = 0;
    }
    void* p = nullptr;
    e = hipMalloc(&p, need);
    if (e != hipSuccess) return fail(RL_ERR_WORKSPACE, "hipMalloc(%zu) for the workspace failed: %s", need, hipGetErrorString(e));
    w.ptr = p;
    w.size = need;
  }
  if (capturing) w.captured = true;
  *out = &w;
  return RL_OK;
}

// Where a call's workspace comes from: this (device, stream)'s library
// workspace (grown with hipMalloc), or, for the allocation-free entry point, the
// device's static scratch array (its first bytes are that array's error word).
struct WsView {
  char* ptr;
  int* err;
};

int get_ws(hipStream_t st, size_t need, bool noalloc, WsView* v) {
  if (!noalloc) {
    Workspace* w = nullptr;
    RL_TRY(acquire_ws(st, need, &w));
    v->ptr = static_cast<char*>(w->ptr);
    v->err = w->err;
    return RL_OK;
  }
  const size_t room = rl::kScratchBytes - rl::kScratchErrBytes;
  if (need > room)
    return fail(RL_ERR_WORKSPACE,
                "this call needs %zu bytes of workspace; the allocation-free entry point has %zu "
                "(a smaller batch, or rl_attn_decode_ex, which allocates)",
                need, room);
  void* p = nullptr;
  const hipError_t e = rl::scratch_address(st, &p);
  if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
  v->ptr = static_cast<char*>(p) + rl::kScratchErrBytes;
  v->err = static_cast<int*>(p);
  return RL_OK;
}

// ------------------------------------------------------------ kernel timing
struct Profiler {
  std::mutex mu;
  bool on = false;
  std::vector<rl::KernelTimer> pending[3];   // decode, extend, append
};

Profiler& prof() {
  static Profiler p;
  return p;
}

// Returns a timer to pass to a launch when profiling is on (else nullptr).
rl::KernelTimer* prof_timer(rl::KernelTimer* slot, hipStream_t st) {
  Profiler& p = prof();
  std::lock_guard<std::mutex> lk(p.mu);
  if (!p.on) return nullptr;
  // a call being captured into a graph is not timed (its events would only
  // be recorded at replay)
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(st, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) return nullptr;
  if (hipEventCreate(&slot->start) != hipSuccess) return nullptr;
  if (hipEventCreate(&slot->stop) != hipSuccess) {
    (void)hipEventDestroy(slot->start);
    return nullptr;
  }
  return slot;
}

void prof_commit(int kind, rl::KernelTimer* t) {
  if (!t) return;
  Profiler& p = prof();
  std::lock_guard<std::mutex> lk(p.mu);
  p.pending[kind].push_back(*t);
}

// ------------------------------------------------------------------- decode
constexpr int64_t kMinSplitKeys = 256;   // the planner's smallest automatic split of shared keys

// Capacities (see the planner): with split size C, T = sum(L) / C and D =
// kPrefixLevels (a member's shared keys are cut at most D times by node
// boundaries), private pieces <= workers + B, shared items <= T + D B, partial
// slots <= workers + T + (D + 1) B. An automatic shared split C keeps T at or below the target
// item count, and C >= kMinSplitKeys keeps it at or below
// B * ceil(max_pages * P / kMinSplitKeys); a forced C bounds T by
// B * ceil(max_pages * P / C) and lets the private pass use up to that many
// workers of C keys.
struct DecodeLayout {
  int max_items, max_slots, max_workers, group_cap;
  size_t off_nparts, off_base, off_pref, off_seqs, off_sitems, off_sgroups, off_range, off_members, off_po, off_pl,
      total;
};

int64_t decode_wgs_per_item(int64_t Hq, int64_t Hkv) {
  const int64_t R = Hq / std::max<int64_t>(1, Hkv);
  return Hkv * (R == 1 ? 1 : (R + 15) / 16);
}

// waves of one decode workgroup: the largest divisor of the item's waves (its
// KV heads and 16-head blocks) up to 8, so a workgroup reads whole token rows
int decode_item_waves(int64_t Hq, int64_t Hkv) {
  const int64_t R = Hq / std::max<int64_t>(1, Hkv);
  const int per_item = (int)(Hkv * ((R + 15) / 16));
  for (int w = std::min(per_item, 8); w >= 1; --w)
    if (per_item % w == 0) return w;
  return 1;
}

int target_items_for(int64_t Hq, int64_t Hkv, int cus) {
  return (int)std::max<int64_t>(1, (int64_t)cus * env().target_wgs_per_cu / decode_wgs_per_item(Hq, Hkv));
}

// workers of the private pass resident on one CU (cached per shape)
int workers_per_cu(int64_t Hq, int64_t Hkv, bool fp8, int n_tok) {
  if (env().workers_per_cu > 0) return env().workers_per_cu;
  static std::mutex mu;
  static std::map<std::tuple<int64_t, int64_t, bool, int>, int> cache;
  std::lock_guard<std::mutex> lk(mu);
  auto it = cache.find({Hq, Hkv, fp8, n_tok});
  if (it != cache.end()) return it->second;
  const int R = (int)(Hq / std::max<int64_t>(1, Hkv));
  const int n = rl::decode_workers_per_cu(R, (int)Hkv, decode_item_waves(Hq, Hkv), fp8, n_tok);
  cache[{Hq, Hkv, fp8, n_tok}] = n;
  return n;
}

// Workspace layout of a decode call with n_tok query tokens per sequence (partial
// rows and group sizes count n_tok * Hq rows per sequence) on `cus` compute units
// holding `wpc` private-pass workers each.
DecodeLayout decode_layout_with(int64_t B, int64_t Hq, int64_t Hkv, int64_t max_pages, int64_t P, int split,
                                int cus, int wpc, bool prefix_share, int n_tok) {
  DecodeLayout L{};
  const int64_t R = Hq / std::max<int64_t>(1, Hkv);
  const int64_t rows_kv = R * n_tok;              // query rows of one KV head
  const int64_t Hv = Hq * n_tok;
  const int64_t max_tokens = max_pages * P;
  // an automatic split is at least kMinSplitKeys keys, so a sequence has at most
  // ceil(max_tokens / kMinSplitKeys) shared splits whatever the item target
  const int64_t T = split > 0 ? B * std::max<int64_t>(1, (max_tokens + split - 1) / split)
                              : std::min<int64_t>(target_items_for(Hq, Hkv, cus),
                                                  B * std::max<int64_t>(1, (max_tokens + kMinSplitKeys - 1) /
                                                                               kMinSplitKeys));
  const int64_t workers = split > 0 ? T : (int64_t)cus * wpc;
  const int64_t D = rl::kPrefixLevels;
  L.max_items = (int)std::min<int64_t>(T + D * B, INT32_MAX / 2);
  L.max_workers = (int)std::min<int64_t>(std::max<int64_t>(1, workers), INT32_MAX / 64);
  L.max_slots = (int)std::min<int64_t>(L.max_workers + T + (D + 1) * B, INT32_MAX / 2);
  L.group_cap = (prefix_share && rows_kv <= 64) ? (int)(128 / rows_kv) : 0;
  size_t off = 256;  // header
  L.off_nparts = off;
  off += align256(B * 4);
  L.off_base = off;
  off += align256(B * 4);
  L.off_pref = off;
  off += align256((size_t)(B + 1) * 8);
  L.off_seqs = off;
  off += align256((size_t)B * 16);
  L.off_sitems = off;
  off += align256((size_t)L.max_items * 16);
  L.off_sgroups = off;
  off += align256((size_t)D * B * 16);
  L.off_range = off;
  off += align256((size_t)D * B * 8);
  L.off_members = off;
  off += align256((size_t)D * B * std::max(1, L.group_cap) * 4);
  L.off_po = off;
  off += align256((size_t)L.max_slots * Hv * 128 * 4);
  L.off_pl = off;
  off += align256((size_t)L.max_slots * Hv * 4);
  L.total = off;
  return L;
}

DecodeLayout decode_layout(int64_t B, int64_t Hq, int64_t Hkv, int64_t max_pages, int64_t P, int split, int cus,
                           bool prefix_share, bool fp8, int n_tok) {
  return decode_layout_with(B, Hq, Hkv, max_pages, P, split, cus, workers_per_cu(Hq, Hkv, fp8, n_tok),
                            prefix_share, n_tok);
}

// One dequantisation scale per KV head: [Hkv] f32. The values are checked on
// the device (positive and finite), where they are read.
int check_head_scales(const rl_tensor* t, const char* name, int64_t Hkv) {
  RL_TRY(check_view(t, name, 1));
  RL_TRY(check_dtype(t, name, RL_F32));
  if (t->shape[0] != Hkv)
    return fail(RL_ERR_SHAPE, "%s must have one entry per KV head (%lld, got %lld)", name, (long long)Hkv,
                (long long)t->shape[0]);
  if (t->strides[0] < 0 || t->strides[0] > INT32_MAX)
    return fail(RL_ERR_UNSUPPORTED, "%s: stride must be in [0, 2^31)", name);
  RL_TRY(check_data(t, name));
  return RL_OK;
}

// Paged K/V and block table. kv_dtype is RL_BF16, or RL_FP8_E4M3 with
// per-KV-head scales k_scale and v_scale (both null for bf16).
int fill_paged(const rl_tensor* k, const rl_tensor* v, const rl_tensor* bt, int64_t B, int kv_dtype,
               const rl_tensor* k_scale, const rl_tensor* v_scale, rl::PagedKV* kv) {
  RL_TRY(check_view(k, "k_pages", 4));
  RL_TRY(check_view(v, "v_pages", 4));
  RL_TRY(check_view(bt, "block_table", 2));
  RL_TRY(check_dtype(k, "k_pages", kv_dtype));
  RL_TRY(check_dtype(v, "v_pages", kv_dtype));
  RL_TRY(check_dtype(bt, "block_table", RL_I32));
  for (int i = 0; i < 4; ++i)
    if (k->shape[i] != v->shape[i]) return fail(RL_ERR_SHAPE, "k_pages and v_pages shapes differ (dim %d)", i);
  RL_TRY(check_rows128(k, "k_pages"));
  RL_TRY(check_rows128(v, "v_pages"));
  const int64_t P = k->shape[1];
  if (P < 8 || P > 128 || (P & (P - 1)) != 0)
    return fail(RL_ERR_UNSUPPORTED, "page size must be a power of two in [8, 128] (got %lld)", (long long)P);
  if (bt->shape[0] != B)
    return fail(RL_ERR_SHAPE, "block_table.shape[0] (%lld) != batch (%lld)", (long long)bt->shape[0], (long long)B);
  if (k->shape[0] < 1 && bt->shape[1] > 0) return fail(RL_ERR_SHAPE, "the page pool is empty");
  if (k->shape[0] > INT32_MAX || bt->shape[1] * P > INT32_MAX)
    return fail(RL_ERR_UNSUPPORTED, "page pool or block table too large for 32-bit token indices");
  // index arithmetic on the device: page strides fit 32 bits, slot strides,
  // block-table column strides and page indices fit 24 bits
  const int64_t lim32 = (int64_t)1 << 32, lim24 = (int64_t)1 << 24;
  if (k->strides[0] >= lim32 || v->strides[0] >= lim32 || k->strides[1] >= lim24 || v->strides[1] >= lim24)
    return fail(RL_ERR_UNSUPPORTED, "k_pages/v_pages: page stride must be < 2^32 and slot stride < 2^24 elements");
  if (bt->strides[1] < 0 || bt->strides[1] >= lim24 || bt->shape[1] >= lim24 || bt->strides[0] < 0)
    return fail(RL_ERR_UNSUPPORTED, "block_table: column stride and width must be < 2^24, strides non-negative");
  RL_TRY(check_data(k, "k_pages"));
  RL_TRY(check_data(v, "v_pages"));
  RL_TRY(check_data(bt, "block_table"));
  kv->k = k->data;
  kv->v = v->data;
  kv->sp = k->strides[0];
  kv->ss = k->strides[1];
  kv->sh = k->strides[2];
  kv->v_sp = v->strides[0];
  kv->v_ss = v->strides[1];
  kv->v_sh = v->strides[2];
  kv->bt = static_cast<const int*>(bt->data);
  kv->bt_sb = bt->strides[0];
  kv->bt_sj = bt->strides[1];
  kv->num_pages = (int)k->shape[0];
  kv->page_size = (int)P;
  int lg = 0;
  while ((1 << lg) < P) ++lg;
  kv->log2_page = lg;
  kv->max_pages = (int)bt->shape[1];
  kv->k_scale = kv->v_scale = nullptr;
  kv->ks_s = kv->vs_s = 0;
  if (kv_dtype == RL_FP8_E4M3) {
    // FP8 rows are read 16 bytes (16 elements) at a time
    for (int i = 0; i < 3; ++i)
      if (k->strides[i] % 16 != 0 || v->strides[i] % 16 != 0)
        return fail(RL_ERR_UNSUPPORTED, "k_pages/v_pages (FP8): strides must be multiples of 16 elements");
    RL_TRY(check_head_scales(k_scale, "k_scale", k->shape[2]));
    RL_TRY(check_head_scales(v_scale, "v_scale", k->shape[2]));
    kv->k_scale = static_cast<const float*>(k_scale->data);
    kv->v_scale = static_cast<const float*>(v_scale->data);
    kv->ks_s = k_scale->strides[0];
    kv->vs_s = v_scale->strides[0];
  }
  return RL_OK;
}

int check_out(const rl_tensor* out, const rl_tensor* q, const char* name, int* is_f32) {
  RL_TRY(check_view(out, name, q->ndim));
  if (out->dtype != RL_BF16 && out->dtype != RL_F32)
    return fail(RL_ERR_DTYPE, "%s must be bf16 or f32 (got %s)", name, dtype_name(out->dtype));
  for (int i = 0; i < q->ndim; ++i)
    if (out->shape[i] != q->shape[i]) return fail(RL_ERR_SHAPE, "%s shape must equal q's (dim %d)", name, i);
  RL_TRY(check_rows128(out, name));
  RL_TRY(check_data(out, name));
  *is_f32 = out->dtype == RL_F32;
  return RL_OK;
}

int check_lse(const rl_tensor* lse, int64_t rows, int64_t heads, int64_t tokens = 0) {
  if (!lse) return RL_OK;
  RL_TRY(check_view(lse, "lse_out", tokens ? 3 : 2));
  RL_TRY(check_dtype(lse, "lse_out", RL_F32));
  if (tokens ? (lse->shape[0] != rows || lse->shape[1] != tokens || lse->shape[2] != heads)
             : (lse->shape[0] != rows || lse->shape[1] != heads))
    return fail(RL_ERR_SHAPE, "lse_out shape mismatch");
  RL_TRY(check_data(lse, "lse_out"));
  return RL_OK;
}

// ------------------------------------------------------------------- extend
struct ExtendShape {
  int rows_head, tile_tokens, head_blocks;
};

// query rows per extend work unit: eight waves of 32 rows
constexpr int kExtendRows = 256;

ExtendShape extend_shape(int64_t R) {
  ExtendShape s;
  s.rows_head = (int)std::min<int64_t>(R, kExtendRows);
  s.tile_tokens = std::max(1, kExtendRows / s.rows_head);
  s.head_blocks = (int)((R + s.rows_head - 1) / s.rows_head);
  return s;
}

// Work units are (sequence, KV head, head block, chunk tile): at most
// Hkv * head_blocks * (B + ceil(total_q / tile_tokens)).
size_t extend_ws_bytes(int64_t B, int64_t total_q, int64_t Hkv, int64_t R, int* max_items) {
  const ExtendShape s = extend_shape(R);
  const int64_t items = Hkv * s.head_blocks * (B + (total_q + s.tile_tokens - 1) / s.tile_tokens);
  *max_items = (int)std::min<int64_t>(items, INT32_MAX / 2);
  return 256 + align256((size_t)*max_items * 16);
}

// Work-unit shape, workspace and launch of an extend call whose arguments
// (pages, q, lengths, output) are already filled in. prof_kind: which timing
// slot the attention kernel is counted under; `given`: a workspace already
// carved out of the call's (else the stream's is taken); `timed`: whether the
// kernel timer is recorded around the launch.
int run_extend(rl::ExtendArgs& a, hipStream_t st, int prof_kind, bool noalloc = false, const WsView* given = nullptr,
               bool timed = true) {
  int max_items = 0;
  const size_t bytes = extend_ws_bytes(a.B, a.total_q, a.Hkv, a.R, &max_items);
  WsView w{};
  if (given)
    w = *given;
  else
    RL_TRY(get_ws(st, bytes, noalloc, &w));
  char* base = w.ptr;
  const ExtendShape s = extend_shape(a.R);
  a.rows_head = s.rows_head;
  a.tile_tokens = s.tile_tokens;
  a.head_blocks = s.head_blocks;
  a.max_items = max_items;
  a.ws.hdr = reinterpret_cast<int*>(base);
  a.ws.items = reinterpret_cast<int4*>(base + 256);
  a.ws.err = w.err;
  rl::KernelTimer slot;
  rl::KernelTimer* timer = noalloc || !timed ? nullptr : prof_timer(&slot, st);
  hipError_t e = rl::launch_extend(a, st, timer);
  prof_commit(prof_kind, timer);
  if (e != hipSuccess) return hip_fail(e, "extend kernel launch");
  return RL_OK;
}

int decode_impl(const rl_tensor* q, const rl_tensor* k_pages, const rl_tensor* v_pages, int kv_dtype,
                const rl_tensor* k_scale, const rl_tensor* v_scale, const rl_tensor* block_table,
                const rl_tensor* seq_lens, float scale, rl_tensor* out, rl_tensor* lse_out, const rl_attn_opts* opts,
                void* stream, bool noalloc = false) {
  Opts o;
  RL_TRY(read_opts(opts, &o));
  RL_TRY(check_scale(scale));
  if (!q) return fail(RL_ERR_INVALID_ARG, "q is NULL");
  if (q->ndim != 3 && q->ndim != 4)
    return fail(RL_ERR_SHAPE, "q must have 3 dimensions, or 4 for several query tokens (got %d)", q->ndim);
  RL_TRY(check_view(q, "q", q->ndim));
  RL_TRY(check_dtype(q, "q", RL_BF16));
  RL_TRY(check_rows128(q, "q"));
  const bool multi = q->ndim == 4;
  const int64_t B = q->shape[0], Hq = q->shape[q->ndim - 2];
  const int64_t n_tok = multi ? q->shape[1] : 1;
  if (n_tok < 1 || n_tok > 64) return fail(RL_ERR_UNSUPPORTED, "query tokens per sequence must be in [1, 64]");
  rl::DecodeArgs a{};
  RL_TRY(fill_paged(k_pages, v_pages, block_table, B, kv_dtype, k_scale, v_scale, &a.kv));
  const int64_t Hkv = k_pages->shape[2];
  if (Hkv < 1 || Hq < 1 || Hq % Hkv != 0)
    return fail(RL_ERR_SHAPE, "query heads (%lld) must be a positive multiple of KV heads (%lld)", (long long)Hq,
                (long long)Hkv);
  RL_TRY(check_view(seq_lens, "seq_lens", 1));
  RL_TRY(check_dtype(seq_lens, "seq_lens", RL_I32));
  if (seq_lens->shape[0] != B) return fail(RL_ERR_SHAPE, "seq_lens.shape[0] != batch");
  int is_f32 = 0;
  RL_TRY(check_out(out, q, "out", &is_f32));
  RL_TRY(check_lse(lse_out, B, Hq, multi ? n_tok : 0));
  if (B > (1 << 22) || Hq > 4096 || B * n_tok * Hq > INT32_MAX)
    return fail(RL_ERR_UNSUPPORTED, "batch, query tokens or head count too large");
  RL_TRY(check_data(q, "q"));
  RL_TRY(check_data(seq_lens, "seq_lens"));
  if (B == 0) return RL_OK;
  // token strides (dimension 1 of a 4-D q / out, of a 3-D lse)
  const int64_t q_st = multi ? q->strides[1] : 0, out_st = multi ? out->strides[1] : 0;
  const int64_t lse_st = (multi && lse_out) ? lse_out->strides[1] : 0;
  const int hd = q->ndim - 2;                      // head dimension index of q / out

  hipStream_t st = static_cast<hipStream_t>(stream);
  // extend rows are (sequence, token) pairs in one run: token dimensions must
  // merge with the batch dimension
  const bool rows_merge = !multi || (q->strides[0] == n_tok * q_st && out->strides[0] == n_tok * out_st &&
                                     (!lse_out || lse_out->strides[0] == n_tok * lse_st));
  // Multi-token decode of a batch without shared prefix pages runs through the
  // extend kernel: one unit per (sequence, KV head), longest first, reads every
  // key once with no split and no combine, measured faster than the split path
  // on the ragged 64K batch (n = 2, 4, 8: 1.57, 1.69, 1.90 against 1.72, 1.81,
  // 1.95 ms per call; the split path through the extend kernel's tile routine
  // was no faster, so the difference is the schedule). With prefix sharing off
  // the host takes that route; with sharing on (automatic splits, bf16 pages)
  // both passes are queued and the device decides: the decode planner finds
  // the shared nodes, and with none it gives the split passes no work and the
  // extend planner, gated on its sub-group count, lays out the units. FP8
  // pages keep the split path (n = 4: 1.43 against 1.62 ms through extend).
  auto extend_rows = [&]() {
    rl::ExtendArgs x{};
    x.kv = a.kv;
    x.q = q->data;
    x.q_st = multi ? q_st : q->strides[0];
    x.q_sh = q->strides[hd];
    x.qo_indptr = nullptr;
    x.kv_lens = static_cast<const int*>(seq_lens->data);
    x.kv_lens_s = seq_lens->strides[0];
    x.B = (int)B;
    x.total_q = (int)(B * n_tok);
    x.Hq = (int)Hq;
    x.Hkv = (int)Hkv;
    x.R = (int)(Hq / Hkv);
    x.scale = scale;
    x.out = out->data;
    x.out_f32 = is_f32;
    x.out_st = multi ? out_st : out->strides[0];
    x.out_sh = out->strides[hd];
    x.lse = lse_out ? static_cast<float*>(lse_out->data) : nullptr;
    x.lse_st = lse_out ? (multi ? lse_st : lse_out->strides[0]) : 0;
    x.lse_sh = lse_out ? lse_out->strides[multi ? 2 : 1] : 0;
    x.decode_rows = (int)n_tok;
    return x;
  };
  const bool via_extend =
      o.deterministic || (n_tok > 1 && o.prefix_share == RL_PREFIX_OFF && o.split_tokens == 0 && rows_merge);
  if (via_extend) {
    // one extend row per (sequence, token): the same kernel and per-row
    // arithmetic as extend, with no split of the keys, so the result of a
    // sequence does not depend on the rest of the batch and equals extend's
    // bitwise
    if (!rows_merge)
      return fail(RL_ERR_UNSUPPORTED,
                  "deterministic multi-token decode needs q, out and lse_out with batch stride = tokens x token stride");
    rl::ExtendArgs x = extend_rows();
    x.staged = o.deterministic ? 0 : 1;
    return run_extend(x, st, 0, noalloc);
  }
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  const int cus = device_cus(dev);
  const DecodeLayout lay = decode_layout(B, Hq, Hkv, a.kv.max_pages, a.kv.page_size, o.split_tokens, cus,
                                         o.prefix_share == RL_PREFIX_AUTO, kv_dtype == RL_FP8_E4M3, (int)n_tok);
  // the extend pass's work list follows the decode workspace; the
  // allocation-free entry point keeps the split path alone when both do not
  // fit its static array
  bool route = n_tok > 1 && o.prefix_share == RL_PREFIX_AUTO && o.split_tokens == 0 && rows_merge &&
               kv_dtype != RL_FP8_E4M3;
  const size_t ext_off = align256(lay.total);
  int ext_items = 0;
  size_t need = lay.total;
  if (route) {
    need = ext_off + extend_ws_bytes(B, B * n_tok, Hkv, Hq / Hkv, &ext_items);
    if (noalloc && need > rl::kScratchBytes - rl::kScratchErrBytes) {
      route = false;
      need = lay.total;
    }
  }
  WsView w{};
  RL_TRY(get_ws(st, need, noalloc, &w));
  char* base = w.ptr;
  a.q = q->data;
  a.q_sb = q->strides[0];
  a.q_sh = q->strides[hd];
  a.n_tok = (int)n_tok;
  a.q_st = q_st;
  a.out_st = out_st;
  a.lse_st = lse_st;
  a.Hv = (int)(n_tok * Hq);
  a.lens = static_cast<const int*>(seq_lens->data);
  a.lens_s = seq_lens->strides[0];
  a.B = (int)B;
  a.Hq = (int)Hq;
  a.Hkv = (int)Hkv;
  a.R = (int)(Hq / Hkv);
  a.scale = scale;
  a.out = out->data;
  a.out_f32 = is_f32;
  a.out_sb = out->strides[0];
  a.out_sh = out->strides[hd];
  a.lse = lse_out ? static_cast<float*>(lse_out->data) : nullptr;
  a.lse_sb = lse_out ? lse_out->strides[0] : 0;
  a.lse_sh = lse_out ? lse_out->strides[multi ? 2 : 1] : 0;
  a.forced_split = o.split_tokens;
  a.target_items = target_items_for(Hq, Hkv, cus);
  a.max_items = lay.max_items;
  a.max_slots = lay.max_slots;
  a.max_workers = lay.max_workers;
  a.group_cap = lay.group_cap;
  a.prefix_grid = 2 * cus;
  a.item_waves = decode_item_waves(Hq, Hkv);
  a.ws.hdr = reinterpret_cast<int*>(base);
  a.ws.nparts = reinterpret_cast<int*>(base + lay.off_nparts);
  a.ws.base = reinterpret_cast<int*>(base + lay.off_base);
  a.ws.pref = reinterpret_cast<long long*>(base + lay.off_pref);
  a.ws.seqs = reinterpret_cast<int4*>(base + lay.off_seqs);
  a.ws.sitems = reinterpret_cast<int4*>(base + lay.off_sitems);
  a.ws.sgroups = reinterpret_cast<int4*>(base + lay.off_sgroups);
  a.ws.sg_range = reinterpret_cast<int2*>(base + lay.off_range);
  a.ws.sg_members = reinterpret_cast<int*>(base + lay.off_members);
  a.ws.part_o = reinterpret_cast<float*>(base + lay.off_po);
  a.ws.part_lse = reinterpret_cast<float*>(base + lay.off_pl);
  a.ws.err = w.err;
  a.route_extend = route ? 1 : 0;
  rl::KernelTimer slot;
  rl::KernelTimer* timer = noalloc ? nullptr : prof_timer(&slot, st);
  if (!route) {
    e = rl::launch_decode(a, st, timer);
    prof_commit(0, timer);
    if (e != hipSuccess) return hip_fail(e, "decode kernel launch");
    return RL_OK;
  }
  // both passes: the timer spans them, planners included (either the split
  // passes or the extend pass does the work)
  if (timer) (void)hipEventRecord(timer->start, st);
  e = rl::launch_decode(a, st, nullptr);
  int rc = RL_OK;
  if (e == hipSuccess) {
    rl::ExtendArgs x = extend_rows();
    x.staged = 1;
    x.gate = a.ws.hdr + 3;
    const WsView xw{base + ext_off, w.err};
    rc = run_extend(x, st, 0, noalloc, &xw, false);
  }
  if (timer) (void)hipEventRecord(timer->stop, st);
  prof_commit(0, timer);
  if (e != hipSuccess) return hip_fail(e, "decode kernel launch");
  return rc;
}

int extend_impl(const rl_tensor* q, const rl_tensor* qo_indptr, const rl_tensor* k_pages, const rl_tensor* v_pages,
                int kv_dtype, const rl_tensor* k_scale, const rl_tensor* v_scale, const rl_tensor* block_table,
                const rl_tensor* kv_lens, float scale, rl_tensor* out, rl_tensor* lse_out, const rl_attn_opts* opts,
                void* stream) {
  Opts o;
  RL_TRY(read_opts(opts, &o));
  RL_TRY(check_scale(scale));
  RL_TRY(check_view(q, "q", 3));
  RL_TRY(check_dtype(q, "q", RL_BF16));
  RL_TRY(check_rows128(q, "q"));
  RL_TRY(check_view(kv_lens, "kv_lens", 1));
  RL_TRY(check_dtype(kv_lens, "kv_lens", RL_I32));
  RL_TRY(check_view(qo_indptr, "qo_indptr", 1));
  RL_TRY(check_dtype(qo_indptr, "qo_indptr", RL_I32));
  const int64_t B = kv_lens->shape[0];
  if (qo_indptr->shape[0] != B + 1)
    return fail(RL_ERR_SHAPE, "qo_indptr must have batch + 1 = %lld entries (got %lld)", (long long)(B + 1),
                (long long)qo_indptr->shape[0]);
  const int64_t total_q = q->shape[0], Hq = q->shape[1];
  rl::ExtendArgs a{};
  RL_TRY(fill_paged(k_pages, v_pages, block_table, B, kv_dtype, k_scale, v_scale, &a.kv));
  const int64_t Hkv = k_pages->shape[2];
  if (Hkv < 1 || Hq < 1 || Hq % Hkv != 0)
    return fail(RL_ERR_SHAPE, "query heads (%lld) must be a positive multiple of KV heads (%lld)", (long long)Hq,
                (long long)Hkv);
  int is_f32 = 0;
  RL_TRY(check_out(out, q, "out", &is_f32));
  RL_TRY(check_lse(lse_out, total_q, Hq));
  if (B > (1 << 22) || total_q > INT32_MAX / 2 || Hq > 4096)
    return fail(RL_ERR_UNSUPPORTED, "batch, query rows or head count too large");
  RL_TRY(check_data(q, "q"));
  RL_TRY(check_data(kv_lens, "kv_lens"));
  RL_TRY(check_data(qo_indptr, "qo_indptr"));
  if (B == 0 || total_q == 0) return RL_OK;

  hipStream_t st = static_cast<hipStream_t>(stream);
  a.q = q->data;
  a.q_st = q->strides[0];
  a.q_sh = q->strides[1];
  a.qo_indptr = static_cast<const int*>(qo_indptr->data);
  a.indptr_s = qo_indptr->strides[0];
  a.kv_lens = static_cast<const int*>(kv_lens->data);
  a.kv_lens_s = kv_lens->strides[0];
  a.B = (int)B;
  a.total_q = (int)total_q;
  a.Hq = (int)Hq;
  a.Hkv = (int)Hkv;
  a.R = (int)(Hq / Hkv);
  a.scale = scale;
  a.out = out->data;
  a.out_f32 = is_f32;
  a.out_st = out->strides[0];
  a.out_sh = out->strides[1];
  a.lse = lse_out ? static_cast<float*>(lse_out->data) : nullptr;
  a.lse_st = lse_out ? lse_out->strides[0] : 0;
  a.lse_sh = lse_out ? lse_out->strides[1] : 0;
  return run_extend(a, st, 1);
}

// ------------------------------------------------------------------- append
int append_impl(const rl_tensor* k_new, const rl_tensor* v_new, const rl_tensor* qo_indptr,
                const rl_tensor* block_table, const rl_tensor* kv_lens, rl_tensor* k_pages, rl_tensor* v_pages,
                int kv_dtype, const rl_tensor* k_scale, const rl_tensor* v_scale, void* stream) {
  RL_TRY(check_view(k_new, "k_new", 3));
  RL_TRY(check_view(v_new, "v_new", 3));
  RL_TRY(check_dtype(k_new, "k_new", RL_BF16));
  RL_TRY(check_dtype(v_new, "v_new", RL_BF16));
  for (int i = 0; i < 3; ++i)
    if (k_new->shape[i] != v_new->shape[i]) return fail(RL_ERR_SHAPE, "k_new and v_new shapes differ (dim %d)", i);
  RL_TRY(check_rows128(k_new, "k_new"));
  RL_TRY(check_rows128(v_new, "v_new"));
  RL_TRY(check_view(kv_lens, "kv_lens", 1));
  RL_TRY(check_dtype(kv_lens, "kv_lens", RL_I32));
  RL_TRY(check_view(qo_indptr, "qo_indptr", 1));
  RL_TRY(check_dtype(qo_indptr, "qo_indptr", RL_I32));
  const int64_t B = kv_lens->shape[0];
  if (qo_indptr->shape[0] != B + 1)
    return fail(RL_ERR_SHAPE, "qo_indptr must have batch + 1 = %lld entries (got %lld)", (long long)(B + 1),
                (long long)qo_indptr->shape[0]);
  rl::PagedKV kv{};
  RL_TRY(fill_paged(k_pages, v_pages, block_table, B, kv_dtype, k_scale, v_scale, &kv));
  const int64_t Hkv = k_pages->shape[2];
  if (k_new->shape[1] != Hkv)
    return fail(RL_ERR_SHAPE, "k_new has %lld KV heads, the pages %lld", (long long)k_new->shape[1], (long long)Hkv);
  const int64_t total_new = k_new->shape[0];
  if (B > (1 << 22) || total_new > INT32_MAX / 2 || Hkv > 4096)
    return fail(RL_ERR_UNSUPPORTED, "batch, new rows or head count too large");
  RL_TRY(check_data(k_new, "k_new"));
  RL_TRY(check_data(v_new, "v_new"));
  RL_TRY(check_data(kv_lens, "kv_lens"));
  RL_TRY(check_data(qo_indptr, "qo_indptr"));
  if (B == 0 || total_new == 0) return RL_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  Workspace* w = nullptr;
  RL_TRY(acquire_ws(st, 0, &w));          // the error word only
  rl::AppendArgs a{};
  a.k_new = k_new->data;
  a.v_new = v_new->data;
  a.kn_st = k_new->strides[0];
  a.kn_sh = k_new->strides[1];
  a.vn_st = v_new->strides[0];
  a.vn_sh = v_new->strides[1];
  a.k = k_pages->data;
  a.v = v_pages->data;
  a.sp = kv.sp;
  a.ss = kv.ss;
  a.sh = kv.sh;
  a.v_sp = kv.v_sp;
  a.v_ss = kv.v_ss;
  a.v_sh = kv.v_sh;
  a.k_scale = kv.k_scale;
  a.v_scale = kv.v_scale;
  a.ks_s = kv.ks_s;
  a.vs_s = kv.vs_s;
  a.bt = kv.bt;
  a.bt_sb = kv.bt_sb;
  a.bt_sj = kv.bt_sj;
  a.qo_indptr = static_cast<const int*>(qo_indptr->data);
  a.indptr_s = qo_indptr->strides[0];
  a.kv_lens = static_cast<const int*>(kv_lens->data);
  a.kv_lens_s = kv_lens->strides[0];
  a.B = (int)B;
  a.total_new = (int)total_new;
  a.Hkv = (int)Hkv;
  a.num_pages = kv.num_pages;
  a.page_size = kv.page_size;
  a.log2_page = kv.log2_page;
  a.max_pages = kv.max_pages;
  a.err = w->err;
  rl::KernelTimer slot;
  rl::KernelTimer* timer = prof_timer(&slot, st);
  hipError_t e = rl::launch_append(a, st, timer);
  prof_commit(2, timer);
  if (e != hipSuccess) return hip_fail(e, "append kernel launch");
  return RL_OK;
}

}  // namespace

extern "C" {

int rl_attn_decode(const rl_tensor* q, const rl_tensor* k_pages, const rl_tensor* v_pages,
                   const rl_tensor* block_table, const rl_tensor* seq_lens, float scale, rl_tensor* out,
                   void* stream) {
  return decode_impl(q, k_pages, v_pages, RL_BF16, nullptr, nullptr, block_table, seq_lens, scale, out, nullptr,
                     nullptr, stream);
}

int rl_attn_decode_ex(const rl_tensor* q, const rl_tensor* k_pages, const rl_tensor* v_pages,
                      const rl_tensor* block_table, const rl_tensor* seq_lens, float scale, rl_tensor* out,
                      rl_tensor* lse_out, const rl_attn_opts* opts, void* stream) {
  return decode_impl(q, k_pages, v_pages, RL_BF16, nullptr, nullptr, block_table, seq_lens, scale, out, lse_out,
                     opts, stream);
}

int rl_attn_decode_noalloc(const rl_tensor* q, const rl_tensor* k_pages, const rl_tensor* v_pages,
                           const rl_tensor* block_table, const rl_tensor* seq_lens, float scale, rl_tensor* out,
                           rl_tensor* lse_out, const rl_attn_opts* opts, void* stream) {
  return decode_impl(q, k_pages, v_pages, RL_BF16, nullptr, nullptr, block_table, seq_lens, scale, out, lse_out,
                     opts, stream, true);
}

int rl_attn_decode_fp8(const rl_tensor* q, const rl_tensor* k_pages, const rl_tensor* v_pages,
                       const rl_tensor* k_scale, const rl_tensor* v_scale, const rl_tensor* block_table,
                       const rl_tensor* seq_lens, float scale, rl_tensor* out, rl_tensor* lse_out,
                       const rl_attn_opts* opts, void* stream) {
  return decode_impl(q, k_pages, v_pages, RL_FP8_E4M3, k_scale, v_scale, block_table, seq_lens, scale, out, lse_out,
                     opts, stream);
}

int rl_attn_extend(const rl_tensor* q, const rl_tensor* qo_indptr, const rl_tensor* k_pages,
                   const rl_tensor* v_pages, const rl_tensor* block_table, const rl_tensor* kv_lens, float scale,
                   rl_tensor* out, void* stream) {
  return extend_impl(q, qo_indptr, k_pages, v_pages, RL_BF16, nullptr, nullptr, block_table, kv_lens, scale, out,
                     nullptr, nullptr, stream);
}

int rl_attn_extend_ex(const rl_tensor* q, const rl_tensor* qo_indptr, const rl_tensor* k_pages,
                      const rl_tensor* v_pages, const rl_tensor* block_table, const rl_tensor* kv_lens, float scale,
                      rl_tensor* out, rl_tensor* lse_out, const rl_attn_opts* opts, void* stream) {
  return extend_impl(q, qo_indptr, k_pages, v_pages, RL_BF16, nullptr, nullptr, block_table, kv_lens, scale, out,
                     lse_out, opts, stream);
}

int rl_attn_extend_fp8(const rl_tensor* q, const rl_tensor* qo_indptr, const rl_tensor* k_pages,
                       const rl_tensor* v_pages, const rl_tensor* k_scale, const rl_tensor* v_scale,
                       const rl_tensor* block_table, const rl_tensor* kv_lens, float scale, rl_tensor* out,
                       rl_tensor* lse_out, const rl_attn_opts* opts, void* stream) {
  return extend_impl(q, qo_indptr, k_pages, v_pages, RL_FP8_E4M3, k_scale, v_scale, block_table, kv_lens, scale, out,
                     lse_out, opts, stream);
}

int rl_attn_append_kv(const rl_tensor* k_new, const rl_tensor* v_new, const rl_tensor* qo_indptr,
                      const rl_tensor* block_table, const rl_tensor* kv_lens, rl_tensor* k_pages, rl_tensor* v_pages,
                      void* stream) {
  return append_impl(k_new, v_new, qo_indptr, block_table, kv_lens, k_pages, v_pages, RL_BF16, nullptr, nullptr,
                     stream);
}

int rl_attn_append_kv_fp8(const rl_tensor* k_new, const rl_tensor* v_new, const rl_tensor* qo_indptr,
                          const rl_tensor* block_table, const rl_tensor* kv_lens, rl_tensor* k_pages,
                          rl_tensor* v_pages, const rl_tensor* k_scale, const rl_tensor* v_scale, void* stream) {
  return append_impl(k_new, v_new, qo_indptr, block_table, kv_lens, k_pages, v_pages, RL_FP8_E4M3, k_scale, v_scale,
                     stream);
}

int rl_attn_merge(const rl_tensor* o_parts, const rl_tensor* lse_parts, const rl_tensor* num_parts, rl_tensor* out,
                  rl_tensor* lse_out, void* stream) {
  RL_TRY(check_view(o_parts, "o_parts", 4));
  RL_TRY(check_dtype(o_parts, "o_parts", RL_F32));
  RL_TRY(check_view(lse_parts, "lse_parts", 3));
  RL_TRY(check_dtype(lse_parts, "lse_parts", RL_F32));
  RL_TRY(check_view(num_parts, "num_parts", 1));
  RL_TRY(check_dtype(num_parts, "num_parts", RL_I32));
  RL_TRY(check_view(out, "out", 3));
  if (out->dtype != RL_BF16 && out->dtype != RL_F32) return fail(RL_ERR_DTYPE, "out must be bf16 or f32");
  if (o_parts->shape[3] != 128 || out->shape[2] != 128)
    return fail(RL_ERR_UNSUPPORTED, "head dimension must be 128");
  if (o_parts->strides[3] != 1 || out->strides[2] != 1) return fail(RL_ERR_UNSUPPORTED, "last stride must be 1");
  const int64_t N = o_parts->shape[0], S = o_parts->shape[1], H = o_parts->shape[2];
  if (lse_parts->shape[0] != N || lse_parts->shape[1] != S || lse_parts->shape[2] != H)
    return fail(RL_ERR_SHAPE, "lse_parts shape must be [N, S, H] of o_parts");
  if (num_parts->shape[0] != N) return fail(RL_ERR_SHAPE, "num_parts must have N entries");
  if (out->shape[0] != N || out->shape[1] != H) return fail(RL_ERR_SHAPE, "out shape must be [N, H, 128]");
  RL_TRY(check_lse(lse_out, N, H));
  for (int i = 0; i < 3; ++i)
    if (o_parts->strides[i] % 2 != 0) return fail(RL_ERR_UNSUPPORTED, "o_parts strides must be even");
  if (reinterpret_cast<uintptr_t>(o_parts->data) % 8 != 0) return fail(RL_ERR_UNSUPPORTED, "o_parts must be 8-byte aligned");
  if (N > INT32_MAX / 4096 || H > 4096 || S > INT32_MAX) return fail(RL_ERR_UNSUPPORTED, "merge sizes too large");
  RL_TRY(check_data(o_parts, "o_parts"));
  RL_TRY(check_data(lse_parts, "lse_parts"));
  RL_TRY(check_data(num_parts, "num_parts"));
  RL_TRY(check_data(out, "out"));
  if (N == 0 || H == 0) return RL_OK;
  rl::MergeArgs a{};
  a.o = static_cast<const float*>(o_parts->data);
  a.o_sn = o_parts->strides[0];
  a.o_ss = o_parts->strides[1];
  a.o_sh = o_parts->strides[2];
  a.lse = static_cast<const float*>(lse_parts->data);
  a.l_sn = lse_parts->strides[0];
  a.l_ss = lse_parts->strides[1];
  a.l_sh = lse_parts->strides[2];
  a.num = static_cast<const int*>(num_parts->data);
  a.num_s = num_parts->strides[0];
  a.N = (int)N;
  a.S = (int)S;
  a.H = (int)H;
  a.out = out->data;
  a.out_f32 = out->dtype == RL_F32;
  a.out_sn = out->strides[0];
  a.out_sh = out->strides[1];
  a.lse_out = lse_out ? static_cast<float*>(lse_out->data) : nullptr;
  a.lo_sn = lse_out ? lse_out->strides[0] : 0;
  a.lo_sh = lse_out ? lse_out->strides[1] : 0;
  hipError_t e = rl::launch_merge(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "merge kernel launch");
  return RL_OK;
}

const char* rl_attn_last_error(void) { return g_err.c_str(); }

int rl_attn_check_device_errors(void* stream) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  // the error words to read: this stream's workspace (if a call made one) and
  // the device's scratch array (if an allocation-free call set it up); none is
  // created here
  int* words[2] = {nullptr, nullptr};
  {
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_ws.find({dev, st});
    if (it != g_ws.end()) words[0] = it->second.err;
  }
  void* sp = nullptr;
  if (rl::scratch_address_if_set_up(&sp)) words[1] = static_cast<int*>(sp);
  e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  int word = 0;
  for (int* p : words) {
    if (!p) continue;
    int wv = 0;
    e = hipMemcpy(&wv, p, sizeof(int), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy");
    e = hipMemset(p, 0, sizeof(int));
    if (e != hipSuccess) return hip_fail(e, "hipMemset");
    word |= wv;
  }
  if (word) {
    std::string what;
    if (word & rl::kErrLen) what += " length-out-of-range";
    if (word & rl::kErrPage) what += " page-id-out-of-range";
    if (word & rl::kErrIndptr) what += " qo_indptr-invalid";
    if (word & rl::kErrKvShort) what += " kv_lens-shorter-than-chunk";
    if (word & rl::kErrScale) what += " dequant-scale-invalid";
    if (word & rl::kErrCapacity) what += " workspace-capacity-exceeded";
    return fail(RL_ERR_DEVICE, "device-side input errors (values were clamped):%s", what.c_str());
  }
  return RL_OK;
}

int rl_attn_reserve_workspace(size_t bytes, void* stream) {
  Workspace* w = nullptr;
  return acquire_ws(static_cast<hipStream_t>(stream), bytes, &w);
}

size_t rl_attn_decode_workspace_size(int64_t batch, int64_t num_q_heads, int64_t num_kv_heads, int64_t max_pages,
                                     int64_t page_size, int64_t query_tokens, int32_t split_tokens) {
  if (batch <= 0 || num_q_heads <= 0 || num_kv_heads <= 0 || max_pages < 0 || page_size <= 0) return 0;
  if (query_tokens < 1 || query_tokens > 64 || split_tokens < 0 || split_tokens % 64 != 0) return 0;
  if (batch > (1 << 22) || num_q_heads > 4096 || batch * query_tokens * num_q_heads > INT32_MAX) return 0;
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess) cus = device_cus(dev);
  const int split = split_tokens ? split_tokens : env().split_tokens;
  // bf16 and FP8 pages may keep different numbers of workers resident, a
  // deterministic decode uses the extend work list, and a multi-token decode
  // with prefix sharing on queues both (the extend list after the decode
  // workspace): the largest of these
  int mi = 0;
  const int64_t R = num_q_heads / num_kv_heads;
  const size_t ext = R >= 1 ? extend_ws_bytes(batch, batch * query_tokens, num_kv_heads, R, &mi) : 0;
  size_t total = ext;
  for (bool fp8 : {false, true}) {
    const size_t dec = decode_layout(batch, num_q_heads, num_kv_heads, max_pages, page_size, split, cus, true, fp8,
                                     (int)query_tokens)
                           .total;
    total = std::max(total, query_tokens > 1 ? align256(dec) + ext : dec);
  }
  return total;
}

size_t rl_attn_extend_workspace_size(int64_t batch, int64_t total_q, int64_t num_q_heads, int64_t num_kv_heads,
                                     int64_t max_pages, int64_t page_size) {
  (void)max_pages;
  (void)page_size;
  if (batch <= 0 || num_q_heads <= 0 || num_kv_heads <= 0) return 0;
  int mi = 0;
  return extend_ws_bytes(batch, total_q, num_kv_heads, num_q_heads / num_kv_heads, &mi);
}

// ------------------------------------------------------------ measurement aids
namespace {

// A small device allocation released when the scope ends.
struct DevBuf {
  void* p = nullptr;
  ~DevBuf() {
    if (p) (void)hipFree(p);
  }
};

}  // namespace

int rl_attn_diag_read_bandwidth(const void* buf, int64_t bytes, int32_t reps, double* gb_per_s, void* stream) {
  if (!buf || !gb_per_s) return fail(RL_ERR_INVALID_ARG, "diag_read_bandwidth: null pointer");
  if (bytes <= 0 || bytes % 16 != 0) return fail(RL_ERR_INVALID_ARG, "diag_read_bandwidth: bytes must be a positive multiple of 16");
  if ((reinterpret_cast<uintptr_t>(buf) & 15) != 0) return fail(RL_ERR_INVALID_ARG, "diag_read_bandwidth: buf must be 16-byte aligned");
  if (reps < 1) return fail(RL_ERR_INVALID_ARG, "diag_read_bandwidth: reps must be >= 1");
  hipStream_t st = static_cast<hipStream_t>(stream);
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  const int cus = device_cus(dev);
  DevBuf sink;
  if ((e = hipMalloc(&sink.p, 16)) != hipSuccess) return hip_fail(e, "hipMalloc");
  hipEvent_t a = nullptr, b = nullptr;
  if ((e = hipEventCreate(&a)) != hipSuccess) return hip_fail(e, "hipEventCreate");
  if ((e = hipEventCreate(&b)) != hipSuccess) {
    (void)hipEventDestroy(a);
    return hip_fail(e, "hipEventCreate");
  }
  unsigned* sk = static_cast<unsigned*>(sink.p);
  e = rl::launch_diag_read(buf, (size_t)bytes, sk, cus, st);
  if (e == hipSuccess) e = hipEventRecord(a, st);
  for (int r = 0; r < reps && e == hipSuccess; ++r) e = rl::launch_diag_read(buf, (size_t)bytes, sk, cus, st);
  if (e == hipSuccess) e = hipEventRecord(b, st);
  if (e == hipSuccess) e = hipEventSynchronize(b);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
  (void)hipEventDestroy(a);
  (void)hipEventDestroy(b);
  if (e != hipSuccess) return hip_fail(e, "diag_read_bandwidth");
  *gb_per_s = ms > 0.f ? (double)bytes * reps / (ms * 1e-3) / 1e9 : 0.0;
  return RL_OK;
}

int rl_attn_diag_mfma_bf16(int64_t iters, double* tflop_per_s, void* stream) {
  if (!tflop_per_s) return fail(RL_ERR_INVALID_ARG, "diag_mfma_bf16: null pointer");
  if (iters < 1 || iters > (1 << 24)) return fail(RL_ERR_INVALID_ARG, "diag_mfma_bf16: iters must be in [1, 2^24]");
  hipStream_t st = static_cast<hipStream_t>(stream);
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  const int cus = device_cus(dev);
  DevBuf sink;
  if ((e = hipMalloc(&sink.p, 16)) != hipSuccess) return hip_fail(e, "hipMalloc");
  float* sk = static_cast<float*>(sink.p);
  hipEvent_t a = nullptr, b = nullptr;
  if ((e = hipEventCreate(&a)) != hipSuccess) return hip_fail(e, "hipEventCreate");
  if ((e = hipEventCreate(&b)) != hipSuccess) {
    (void)hipEventDestroy(a);
    return hip_fail(e, "hipEventCreate");
  }
  e = rl::launch_diag_mfma((int)std::min<int64_t>(iters, 64), sk, cus, st);   // warm-up
  if (e == hipSuccess) e = hipEventRecord(a, st);
  if (e == hipSuccess) e = rl::launch_diag_mfma((int)iters, sk, cus, st);
  if (e == hipSuccess) e = hipEventRecord(b, st);
  if (e == hipSuccess) e = hipEventSynchronize(b);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
  (void)hipEventDestroy(a);
  (void)hipEventDestroy(b);
  if (e != hipSuccess) return hip_fail(e, "diag_mfma_bf16");
  *tflop_per_s = ms > 0.f ? rl::diag_mfma_flops((int)iters, cus) / (ms * 1e-3) / 1e12 : 0.0;
  return RL_OK;
}

int rl_attn_diag_decode_capacity(int64_t batch, int64_t num_q_heads, int64_t num_kv_heads, int64_t max_pages,
                                 int64_t page_size, int64_t query_tokens, int32_t split_tokens, int32_t prefix_share,
                                 int32_t cus, int32_t workers_per_cu, int64_t* out) {
  if (!out) return fail(RL_ERR_INVALID_ARG, "diag_decode_capacity: out is NULL");
  if (batch <= 0 || num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads != 0 || max_pages < 0 ||
      page_size <= 0 || query_tokens < 1 || query_tokens > 64 || split_tokens < 0 || split_tokens % 64 != 0 ||
      cus < 1 || workers_per_cu < 1)
    return fail(RL_ERR_INVALID_ARG, "diag_decode_capacity: invalid sizes");
  const DecodeLayout L = decode_layout_with(batch, num_q_heads, num_kv_heads, max_pages, page_size, split_tokens, cus,
                                            workers_per_cu, prefix_share != 0, (int)query_tokens);
  out[0] = L.max_items;
  out[1] = L.max_slots;
  out[2] = L.max_workers;
  out[3] = L.group_cap;
  out[4] = target_items_for(num_q_heads, num_kv_heads, cus);
  out[5] = 2 * (int64_t)cus;
  out[6] = (int64_t)L.total;
  return RL_OK;
}

int rl_attn_diag_extend_capacity(int64_t batch, int64_t total_q, int64_t num_q_heads, int64_t num_kv_heads,
                                 int64_t* out) {
  if (!out) return fail(RL_ERR_INVALID_ARG, "diag_extend_capacity: out is NULL");
  if (batch <= 0 || total_q < 0 || num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads != 0)
    return fail(RL_ERR_INVALID_ARG, "diag_extend_capacity: invalid sizes");
  int mi = 0;
  (void)extend_ws_bytes(batch, total_q, num_kv_heads, num_q_heads / num_kv_heads, &mi);
  const ExtendShape sh = extend_shape(num_q_heads / num_kv_heads);
  out[0] = mi;
  out[1] = sh.rows_head;
  out[2] = sh.tile_tokens;
  out[3] = sh.head_blocks;
  return RL_OK;
}

int rl_attn_profile_enable(int on) {
  Profiler& p = prof();
  std::lock_guard<std::mutex> lk(p.mu);
  p.on = on != 0;
  return RL_OK;
}

int rl_attn_profile_read(int kind, int* launches, double* mean_ms) {
  if (kind < 0 || kind > 2) return fail(RL_ERR_INVALID_ARG, "kind must be 0 (decode), 1 (extend) or 2 (append)");
  if (!launches || !mean_ms) return fail(RL_ERR_INVALID_ARG, "launches and mean_ms must not be NULL");
  std::vector<rl::KernelTimer> ts;
  {
    Profiler& p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    ts.swap(p.pending[kind]);
  }
  double total = 0.0;
  int n = 0;
  int rc = RL_OK;
  for (auto& t : ts) {
    float ms = 0.f;
    if (rc == RL_OK) {
      hipError_t e = hipEventSynchronize(t.stop);
      if (e == hipSuccess) e = hipEventElapsedTime(&ms, t.start, t.stop);
      if (e != hipSuccess) rc = hip_fail(e, "hipEventElapsedTime");
      total += ms;
      ++n;
    }
    (void)hipEventDestroy(t.start);
    (void)hipEventDestroy(t.stop);
  }
  *launches = n;
  *mean_ms = n ? total / n : 0.0;
  return rc;
}

void rl_attn_release(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  (void)hipDeviceSynchronize();
  for (auto& kv : g_ws) {
    if (kv.second.ptr) (void)hipFree(kv.second.ptr);
    for (void* r : kv.second.retired) (void)hipFree(r);
    if (kv.second.err) (void)hipFree(kv.second.err);
  }
  g_ws.clear();
}

}  // extern "C"
