// Causal extend over a paged cache: appended chunk rows attend to the cached
// prefix plus, causally, to the chunk itself (bottom-right mask).
//
// A unit of work is (sequence b, KV head g, block of query heads, run of
// chunk tokens): up to 256 query rows, token-major (row r -> token r / RB,
// head r % RB), all reading the same keys; one workgroup computes it with the
// MFMA tile of tile_attn.hpp. Keys [0, prefix + first token) are visible to
// every row of a unit, so only the last steps of a unit apply the mask.
//
// The planner orders units longest key range first and keeps the units of one
// (sequence, KV head) together on one XCD (workgroups go to the XCDs
// round-robin by index), so they run at the same time and stream the same
// keys through that XCD's L2.
#include "kernels.hpp"
#include "tile_attn.hpp"

namespace rl {

namespace {

constexpr int kSortMax = 1024;          // sequences sorted by key count up to this batch size
constexpr int kXcds = 8;                // workgroups go to the 8 XCDs round-robin by index
constexpr bool kXcdGroups = true;       // keep each (sequence, KV head)'s units on one XCD

struct SeqRange {
  int q0, n, kv;
};

__device__ __forceinline__ SeqRange seq_range(const ExtendArgs& a, int b, int* bad) {
  const int max_tokens = a.kv.max_pages * a.kv.page_size;
  if (a.decode_rows) {
    // decode: sequence b owns rows b * n .. b * n + n - 1, its last n keys
    const int n = a.decode_rows;
    int kv = a.kv_lens[(int64_t)b * a.kv_lens_s];
    if (kv < 0 || kv > max_tokens) {
      *bad |= kErrLen;
      kv = kv < 0 ? 0 : max_tokens;
    }
    if (kv == 0) return {b * n, 0, 0};
    if (kv < n) {
      *bad |= kErrKvShort;
      kv = n <= max_tokens ? n : max_tokens;
    }
    return {b * n, n, kv};
  }
  int q0 = a.qo_indptr[(int64_t)b * a.indptr_s];
  int q1 = a.qo_indptr[(int64_t)(b + 1) * a.indptr_s];
  if (q0 < 0 || q0 > a.total_q || q1 < q0 || q1 > a.total_q) {
    *bad |= kErrIndptr;
    q0 = q0 < 0 ? 0 : (q0 > a.total_q ? a.total_q : q0);
    q1 = q1 < q0 ? q0 : (q1 > a.total_q ? a.total_q : q1);
  }
  int n = q1 - q0;
  int kv = a.kv_lens[(int64_t)b * a.kv_lens_s];
  if (kv < 0 || kv > max_tokens) {
    *bad |= kErrLen;
    kv = kv < 0 ? 0 : max_tokens;
  }
  if (n > kv) {           // the chunk must be inside the cache
    *bad |= kErrKvShort;
    if (n > max_tokens) n = max_tokens;
    kv = n;
  }
  return {q0, n, kv};
}

__global__ __launch_bounds__(1024) void plan_extend_kernel(ExtendArgs a) {
  __shared__ int order[kSortMax];
  __shared__ int keys[kSortMax];
  __shared__ int wave_tot[16];
  const int tid = threadIdx.x;
  int bad = 0;
  if (a.gate && *a.gate != 0) {          // the split decode passes compute the rows
    if (tid == 0) a.ws.hdr[0] = 0;
    return;
  }
  if (a.decode_rows) {
    // decode rows of empty sequences have no work unit: out = 0, lse = -inf.
    // The empty sequences of each pass of blockDim sequences are listed first
    // (one length load per thread), then their rows are written by all threads.
    __shared__ int empties[1024];
    __shared__ int n_empty;
    const int per_seq = a.decode_rows * a.Hq;
    for (int b0 = 0; b0 < a.B; b0 += blockDim.x) {
      if (tid == 0) n_empty = 0;
      __syncthreads();
      const int b = b0 + tid;
      int dummy = 0;
      if (b < a.B && seq_range(a, b, &dummy).n == 0) empties[atomicAdd(&n_empty, 1)] = b;
      __syncthreads();
      const int rows = n_empty * per_seq;
      for (int i = tid; i < rows; i += blockDim.x) {
        const int e = empties[i / per_seq], rest = i % per_seq;
        const int64_t row = (int64_t)e * a.decode_rows + rest / a.Hq;
        const int h = rest % a.Hq;
        if (a.out_f32) {
          float4* op = reinterpret_cast<float4*>((float*)a.out + row * a.out_st + (int64_t)h * a.out_sh);
          for (int c = 0; c < kHeadDim / 4; ++c) op[c] = make_float4(0.f, 0.f, 0.f, 0.f);
        } else {
          uint4* op = reinterpret_cast<uint4*>((__bf16*)a.out + row * a.out_st + (int64_t)h * a.out_sh);
          for (int c = 0; c < kHeadDim / 8; ++c) op[c] = make_uint4(0u, 0u, 0u, 0u);
        }
        if (a.lse) a.lse[row * a.lse_st + (int64_t)h * a.lse_sh] = kNegInf;
      }
      __syncthreads();                   // the list is rebuilt for the next pass
    }
  }
  const bool sorted = a.B <= kSortMax;
  if (sorted) {
    for (int b = tid; b < a.B; b += blockDim.x) keys[b] = seq_range(a, b, &bad).kv;
    __syncthreads();
    for (int b = tid; b < a.B; b += blockDim.x) {
      const int kb = keys[b];
      int rank = 0;
      for (int j = 0; j < a.B; ++j) rank += (keys[j] > kb) || (keys[j] == kb && j < b);
      order[rank] = b;
    }
    __syncthreads();
  }
  const int heads = a.Hkv * a.head_blocks;
  int offset = 0;
  for (int p0 = 0; p0 < a.B; p0 += blockDim.x) {
    const int p = p0 + tid;
    int nt = 0, b = 0;
    SeqRange r{0, 0, 0};
    if (p < a.B) {
      b = sorted ? order[p] : p;
      int dummy = 0;
      r = seq_range(a, b, sorted ? &dummy : &bad);
      nt = (r.n + a.tile_tokens - 1) / a.tile_tokens;
    }
    int tot;
    const int excl = block_exclusive_scan(nt * heads, &tot, wave_tot);
    if (p < a.B) {
      // With a multiple of 8 head groups, group gh of a sequence runs on XCD
      // gh % 8: its units share their keys through that XCD's L2 instead of
      // every XCD streaming every group's keys. Each XCD's units stay in list
      // order (longest first), and every XCD gets the same number of units.
      const bool xcd = kXcdGroups && heads % kXcds == 0;
      for (int gh = 0; gh < heads; ++gh) {
        const int g = gh / a.head_blocks, hb = gh - g * a.head_blocks;
        // last tile first: it has the longest key range of the sequence
        for (int j = 0; j < nt; ++j) {
          int idx = offset + excl + gh * nt + j;
          if (xcd) {
            // position in the XCD's own list: units of the earlier sequences
            // (heads / 8 groups each), then of this sequence's earlier groups
            const int k = (offset + excl) / kXcds + (gh / kXcds) * nt + j;
            idx = k * kXcds + gh % kXcds;
          }
          const int i0 = (nt - 1 - j) * a.tile_tokens;
          const int cnt = min(a.tile_tokens, r.n - i0);
          if (idx < a.max_items)
            a.ws.items[idx] = make_int4(b, i0, cnt, g | (hb << 16));
          else
            bad |= kErrCapacity;     // the host sizing rules this out; reported, never dropped silently
        }
      }
    }
    offset += tot;
  }
  if (tid == 0) a.ws.hdr[0] = offset < a.max_items ? offset : a.max_items;
  if (bad) atomicOr(a.ws.err, bad);
}

constexpr int kExtWaves = 8;            // waves per extend workgroup: 256 query rows per unit

// Page lookups of the tile routine, chosen on the host: one scalar id per
// step (pages of at least 64 keys), one per wave and 32-row set (smaller
// pages), or one per row (in-page offsets past 31 bits). Each is its own
// kernel, so the common case keeps its register allocation. bf16 pages of at
// least 64 keys take 128-key steps with rows loaded straight into LDS
// (kDirectPages).
constexpr int kStepPages = 0, kSetPages = 1, kRowPages = 2, kDirectPages = 3;

template <bool kFp8, int kPages, bool kNt = false>
__global__ __launch_bounds__(kExtWaves * 64, 2) void extend_mfma_kernel(ExtendArgs a) {
  // Units run in list order (longest key range first). Workgroups are handed
  // to the XCDs round-robin, so each XCD takes every eighth entry; the planner
  // lays the list out so those are the units of the (sequence, KV head) groups
  // assigned to that XCD, which then share their keys through its L2.
  const int unit = blockIdx.x;
  if (unit >= a.ws.hdr[0]) return;
  const int4 it = a.ws.items[unit];
  const int b = it.x, i0 = it.y, cnt = it.z, g = it.w & 0xffff, hb = it.w >> 16;
  int bad_seq = 0, bad = 0;               // sequence errors are reported by the planner
  const SeqRange sr = seq_range(a, b, &bad_seq);
  const int prefix = sr.kv - sr.n;
  const int t_end = prefix + i0 + cnt;     // keys [0, t_end) are visible to some row
  const int t_full = prefix + i0;          // keys [0, t_full) are visible to every row

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int RB = a.rows_head;
  // this lane's query row (MFMA column)
  const int r = wave * kWaveRows + (lane & 31);
  const int ti = r / RB, hi = r - ti * RB;
  const bool row_ok = ti < cnt && hb * RB + hi < a.R;
  const int head = g * a.R + hb * RB + (row_ok ? hi : 0);
  const int limit = row_ok ? prefix + i0 + ti : t_end - 1;
  const int64_t qrow = sr.q0 + i0 + (row_ok ? ti : 0);

  bf16x8 qv[8];
  load_q_operand((const __bf16*)a.q + qrow * a.q_st + (int64_t)head * a.q_sh, row_ok, qv);
  f32x16 o[4];
#pragma unroll
  for (int jd = 0; jd < 4; ++jd)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[jd][e] = 0.f;
  float m_run = kNegInf, l_run = 0.f;
  int bad_scale = 0;
  // the K dequantisation scale joins the softmax scale, the V scale the output
  const KvScales dq = kv_scales<kFp8>(a.kv, g, &bad_scale);
  const float scale = a.scale * dq.k;
  const int* bt_row = a.kv.bt + (int64_t)b * a.kv.bt_sb;
  // a wave whose 32 rows are all past the unit's tokens (a short chunk, or
  // the one token of a deterministic decode) only stages
  const bool active = __builtin_amdgcn_ballot_w64(row_ok) != 0;
  if constexpr (kPages == kDirectPages) {
    static_assert(!kFp8, "rows go to LDS as stored: bf16 pages only");
    __shared__ __attribute__((aligned(16))) char kl0[kDlKBytes], kl1[kDlKBytes], vl0[kDlVBytes], vl1[kDlVBytes];
    if (active)
      tile_attend_dl<true, kNt>(a.kv, scale, bt_row, g, t_end, t_full, limit, qv, kl0, kl1, vl0, vl1, o, m_run,
                                l_run, bad);
    else
      tile_attend_dl<false, kNt>(a.kv, scale, bt_row, g, t_end, t_full, limit, qv, kl0, kl1, vl0, vl1, o, m_run,
                                 l_run, bad);
  } else {
    __shared__ TileLds lds;
    auto attend = [&](auto compute_tag) {
      constexpr bool kC = decltype(compute_tag)::value;
      tile_attend_pp<kExtWaves, kPages != kRowPages, kFp8, kC, kPages == kSetPages, kNt>(
          a.kv, scale, bt_row, g, 0, t_end, t_full, limit, qv, lds, o, m_run, l_run, bad);
    };
    if (active)
      attend(std::true_type{});
    else
      attend(std::false_type{});
  }

  const float l_tot = sum_l32(l_run);
  if (row_ok) {
    const float inv = l_tot > 0.f ? dq.v / l_tot : 0.f;
    if (a.out_f32)
      store_o_row((float*)a.out + qrow * a.out_st + (int64_t)head * a.out_sh, o, inv);
    else
      store_o_row((__bf16*)a.out + qrow * a.out_st + (int64_t)head * a.out_sh, o, inv);
    if (a.lse && lane < 32)
      a.lse[qrow * a.lse_st + (int64_t)head * a.lse_sh] =
          l_tot > 0.f ? (m_run + __builtin_amdgcn_logf(l_tot)) * kLn2 : kNegInf;
  }
  if (bad) atomicOr(a.ws.err, kErrPage);
  if (bad_scale) atomicOr(a.ws.err, kErrScale);
}

}  // namespace

hipError_t launch_extend(const ExtendArgs& a, hipStream_t stream, KernelTimer* timer) {
  plan_extend_kernel<<<1, 1024, 0, stream>>>(a);
  const unsigned grid = (unsigned)a.max_items;
  if (timer) (void)hipEventRecord(timer->start, stream);
  const int64_t ss = a.kv.ss > a.kv.v_ss ? a.kv.ss : a.kv.v_ss;
  const bool scalar_ids = ((int64_t)a.kv.page_size * ss + kHeadDim) * 2 < (int64_t(1) << 31);
  const int pages = !scalar_ids ? kRowPages : (a.kv.page_size >= kKeys ? kStepPages : kSetPages);
  // decode through the extend kernel with one unit per (sequence, KV head):
  // every key row is read once, so the rows are loaded non-temporally (pages
  // of at least a step only)
  const bool once = a.decode_rows > 0 && a.head_blocks == 1 && a.decode_rows <= a.tile_tokens;
  auto go = [&](auto fp8_tag) {
    constexpr bool kF = decltype(fp8_tag)::value;
    if constexpr (!kF) {
      if (pages == kStepPages && !a.staged) {
        if (once)
          extend_mfma_kernel<false, kDirectPages, true><<<grid, kExtWaves * 64, 0, stream>>>(a);
        else
          extend_mfma_kernel<false, kDirectPages><<<grid, kExtWaves * 64, 0, stream>>>(a);
        return;
      }
    }
    if (pages == kStepPages && once)
      extend_mfma_kernel<kF, kStepPages, true><<<grid, kExtWaves * 64, 0, stream>>>(a);
    else if (pages == kStepPages)
      extend_mfma_kernel<kF, kStepPages><<<grid, kExtWaves * 64, 0, stream>>>(a);
    else if (pages == kSetPages)
      extend_mfma_kernel<kF, kSetPages><<<grid, kExtWaves * 64, 0, stream>>>(a);
    else
      extend_mfma_kernel<kF, kRowPages><<<grid, kExtWaves * 64, 0, stream>>>(a);
  };
  if (a.kv.k_scale)
    go(std::true_type{});
  else
    go(std::false_type{});
  if (timer) (void)hipEventRecord(timer->stop, stream);
  return hipGetLastError();
}

}  // namespace rl
