// Causal extend over a paged cache: appended chunk rows attend to the cached
// prefix plus, causally, to the chunk itself (bottom-right mask).
//
// A tile is (sequence b, a run of chunk tokens, KV head g, block of query
// heads): up to 128 query rows, token-major (row r -> token r / RB, head
// r % RB), which all read the same keys. The planner orders tiles longest key
// range first so the longest tiles start first.
#include "attn_common.hpp"
#include "kernels.hpp"

namespace rl {

namespace {

constexpr int kWaves = 4;          // waves per workgroup
constexpr int kColBlocks = 2;      // 16-row column blocks per wave (128 query rows per tile)
constexpr int kTile = 32;          // keys per iteration
constexpr int kSortMax = 1024;     // sequences sorted by key count up to this batch size

struct SeqRange {
  int q0, n, kv;
};

__device__ __forceinline__ SeqRange seq_range(const ExtendArgs& a, int b, int* bad) {
  const int max_tokens = a.kv.max_pages * a.kv.page_size;
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

__device__ int block_exclusive_scan(int v, int* total) {
  __shared__ int wave_tot[16];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wave_tot[wave] = x;
  __syncthreads();
  int before = 0, all = 0;
  const int nw = blockDim.x >> 6;
  for (int w = 0; w < nw; ++w) {
    int t = wave_tot[w];
    if (w < wave) before += t;
    all += t;
  }
  __syncthreads();
  *total = all;
  return before + x - v;
}

__global__ __launch_bounds__(1024) void plan_extend_kernel(ExtendArgs a) {
  __shared__ int order[kSortMax];
  __shared__ int keys[kSortMax];
  const int tid = threadIdx.x;
  int bad = 0;
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
    const int excl = block_exclusive_scan(nt, &tot);
    if (p < a.B) {
      // last tile first: it has the longest key range of the sequence
      for (int j = 0; j < nt; ++j) {
        const int idx = offset + excl + j;
        const int tile = nt - 1 - j;
        const int i0 = tile * a.tile_tokens;
        const int cnt = min(a.tile_tokens, r.n - i0);
        if (idx < a.max_items) a.ws.items[idx] = make_int4(b, i0, cnt, 0);
      }
    }
    offset += tot;
  }
  if (tid == 0) a.ws.hdr[0] = offset < a.max_items ? offset : a.max_items;
  if (bad) atomicOr(a.ws.err, bad);
}

__global__ __launch_bounds__(256) void extend_mfma_kernel(ExtendArgs a) {
  __shared__ u16 ks[kTile][kHeadDim + 8];
  __shared__ u16 vs[kTile][kHeadDim + 8];

  const int per_item = a.Hkv * a.head_blocks;
  const int item = blockIdx.x / per_item;
  const int rem = blockIdx.x - item * per_item;
  const int g = rem % a.Hkv;
  const int hb = rem / a.Hkv;
  if (item >= a.ws.hdr[0]) return;
  const int4 it = a.ws.items[item];
  const int b = it.x, i0 = it.y, cnt = it.z;
  int bad = 0;
  const SeqRange sr = seq_range(a, b, &bad);
  const int prefix = sr.kv - sr.n;
  const int t_end = prefix + i0 + cnt;    // keys [0, t_end) are visible to some row

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int col = lane & 15, grp = lane >> 4;
  const int RB = a.rows_head;
  const int head0 = hb * RB;

  bf16x8 qv[kColBlocks][4];
  int limit[kColBlocks];
  int row_tok[kColBlocks], row_head[kColBlocks];
  bool row_ok[kColBlocks];
#pragma unroll
  for (int cb = 0; cb < kColBlocks; ++cb) {
    const int r = (wave * kColBlocks + cb) * 16 + col;
    const int ti = r / RB, hi = r - (r / RB) * RB;
    const bool ok = ti < cnt && head0 + hi < a.R;
    row_ok[cb] = ok;
    row_tok[cb] = ti;
    row_head[cb] = g * a.R + head0 + hi;
    limit[cb] = ok ? prefix + i0 + ti : t_end - 1;
    const __bf16* qp = (const __bf16*)a.q + (int64_t)(sr.q0 + i0 + (ok ? ti : 0)) * a.q_st +
                       (int64_t)(ok ? row_head[cb] : g * a.R) * a.q_sh + grp * 8;
#pragma unroll
    for (int c = 0; c < 4; ++c) qv[cb][c] = ok ? load_bf16x8(qp + c * 32) : zero_bf16x8();
  }

  f32x4 o[kColBlocks][8];
  float m_run[kColBlocks], l_run[kColBlocks];
#pragma unroll
  for (int cb = 0; cb < kColBlocks; ++cb) {
    m_run[cb] = kNegInf;
    l_run[cb] = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) o[cb][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const float sl2 = a.scale * kLog2e;
  const int* bt_row = a.kv.bt + (int64_t)b * a.kv.bt_sb;
  // cooperative loads: thread -> (key row tid/16 (+16), 16-byte chunk tid%16)
  const int ld_row = tid >> 4, ld_chunk = (tid & 15) * 8;
  const __bf16* kbase = (const __bf16*)a.kv.k + (int64_t)g * a.kv.sh + ld_chunk;
  const __bf16* vbase = (const __bf16*)a.kv.v + (int64_t)g * a.kv.v_sh + ld_chunk;
  bf16x8 kr[2], vr[2];
  auto load_tile = [&](int t0) {
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) {
      int t = t0 + ld_row + 16 * rr;
      t = t < t_end ? t : t_end - 1;
      const int64_t pg = page_of(bt_row, a.kv.bt_sj, t, a.kv.log2_page, a.kv.num_pages, &bad);
      const int slot = t & (a.kv.page_size - 1);
      kr[rr] = load_bf16x8(kbase + pg * a.kv.sp + (int64_t)slot * a.kv.ss);
      vr[rr] = load_bf16x8(vbase + pg * a.kv.v_sp + (int64_t)slot * a.kv.v_ss);
    }
  };
  if (t_end > 0) load_tile(0);
  for (int t0 = 0; t0 < t_end; t0 += kTile) {
    __syncthreads();
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) {
      *reinterpret_cast<bf16x8*>(&ks[ld_row + 16 * rr][ld_chunk]) = kr[rr];
      *reinterpret_cast<bf16x8*>(&vs[ld_row + 16 * rr][ld_chunk]) = vr[rr];
    }
    __syncthreads();
    if (t0 + kTile < t_end) load_tile(t0 + kTile);

    bf16x8 ka[2][4];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int c = 0; c < 4; ++c) ka[hh][c] = *reinterpret_cast<const bf16x8*>(&ks[16 * hh + col][c * 32 + grp * 8]);

    bf16x8 pb[kColBlocks];
#pragma unroll
    for (int cb = 0; cb < kColBlocks; ++cb) {
      f32x4 st[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        st[hh] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < 4; ++c) st[hh] = mfma_16x16x32(ka[hh][c], qv[cb][c], st[hh]);
      }
      float sv[8];
      float mt = kNegInf;
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = t0 + 16 * hh + 4 * grp + i;
          const float x = t <= limit[cb] ? st[hh][i] * sl2 : kNegInf;
          sv[hh * 4 + i] = x;
          mt = fmaxf(mt, x);
        }
      mt = group_max(mt);
      const float m_new = fmaxf(m_run[cb], mt);    // finite: key 0 is visible to every row
      const float alpha = exp2_fast(m_run[cb] - m_new);
      float ps = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float p = exp2_fast(sv[e] - m_new);
        ps += p;
        pb[cb][e] = (__bf16)p;
      }
      l_run[cb] = l_run[cb] * alpha + ps;
      m_run[cb] = m_new;
#pragma unroll
      for (int j = 0; j < 8; ++j) o[cb][j] *= alpha;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      bf16x8 va;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int tok = e < 4 ? 4 * grp + e : 16 + 4 * grp + (e - 4);
        va[e] = bits_to_bf16(vs[tok][16 * j + col]);
      }
#pragma unroll
      for (int cb = 0; cb < kColBlocks; ++cb) o[cb][j] = mfma_16x16x32(va, pb[cb], o[cb][j]);
    }
  }

#pragma unroll
  for (int cb = 0; cb < kColBlocks; ++cb) {
    const float l_tot = group_sum(l_run[cb]);
    if (!row_ok[cb]) continue;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const int64_t qrow = sr.q0 + i0 + row_tok[cb];
    const int h = row_head[cb];
    if (a.out_f32) {
      float* op = (float*)a.out + qrow * a.out_st + (int64_t)h * a.out_sh + 4 * grp;
#pragma unroll
      for (int j = 0; j < 8; ++j) *reinterpret_cast<f32x4*>(op + 16 * j) = o[cb][j] * inv;
    } else {
      typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
      __bf16* op = (__bf16*)a.out + qrow * a.out_st + (int64_t)h * a.out_sh + 4 * grp;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        bf16x4 w;
#pragma unroll
        for (int i = 0; i < 4; ++i) w[i] = (__bf16)(o[cb][j][i] * inv);
        *reinterpret_cast<bf16x4*>(op + 16 * j) = w;
      }
    }
    if (a.lse && grp == 0)
      a.lse[qrow * a.lse_st + (int64_t)h * a.lse_sh] =
          l_tot > 0.f ? (m_run[cb] + __builtin_amdgcn_logf(l_tot)) * kLn2 : kNegInf;
  }
  if (bad) atomicOr(a.ws.err, bad & kErrPage ? kErrPage : 0);
}

}  // namespace

hipError_t launch_extend(const ExtendArgs& a, hipStream_t stream, KernelTimer* timer) {
  plan_extend_kernel<<<1, 1024, 0, stream>>>(a);
  const unsigned grid = (unsigned)a.max_items * a.Hkv * a.head_blocks;
  if (timer) (void)hipEventRecord(timer->start, stream);
  extend_mfma_kernel<<<grid, kWaves * 64, 0, stream>>>(a);
  if (timer) (void)hipEventRecord(timer->stop, stream);
  return hipGetLastError();
}

}  // namespace rl
