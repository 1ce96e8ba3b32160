// Batched paged decode: device planner, split-KV attention, log-sum-exp combine.
//
// One work item is (sequence b, split s): keys [s*C, min(L_b, (s+1)*C)) of one
// sequence. The planner runs on the device from the lengths alone, so the host
// never waits for data: it picks C so that the number of work items stays
// near a target, and records, per sequence, how many splits it has.
// A sequence with one split writes its final output directly; longer ones
// write per-split (o, lse) partials that the combine kernel merges
// (flash-decoding; the merge rule is the log-sum-exp identity).
#include "attn_common.hpp"
#include "kernels.hpp"

namespace rl {

namespace {

constexpr int kMinSplit = 256;     // smallest automatic split (tokens)
constexpr int kTile = 32;          // keys per inner iteration

// Exclusive prefix sum over a 1024-thread block; returns the block total in *total.
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

__device__ __forceinline__ int clamp_len(int L, int max_tokens, int* bad) {
  if (L < 0 || L > max_tokens) {
    *bad = 1;
    return L < 0 ? 0 : max_tokens;
  }
  return L;
}

__global__ __launch_bounds__(1024) void plan_decode_kernel(DecodeArgs a) {
  const int tid = threadIdx.x;
  const int max_tokens = a.kv.max_pages * a.kv.page_size;
  int bad = 0;
  long long sum = 0;
  for (int b = tid; b < a.B; b += blockDim.x) sum += clamp_len(a.lens[b * a.lens_s], max_tokens, &bad);
  // block sum of the lengths
  __shared__ long long wsum[16];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o, 64);
  if ((tid & 63) == 0) wsum[tid >> 6] = sum;
  __syncthreads();
  long long total = 0;
  for (int w = 0; w < (int)(blockDim.x >> 6); ++w) total += wsum[w];

  int C = a.forced_split;
  if (C <= 0) {
    long long per = (total + a.target_items - 1) / a.target_items;
    per = (per + 63) & ~63LL;
    C = (int)(per < kMinSplit ? kMinSplit : per);
  }
  int offset = 0;
  for (int b0 = 0; b0 < a.B; b0 += blockDim.x) {
    const int b = b0 + tid;
    int ns = 0;
    if (b < a.B) {
      int dummy = 0;
      const int L = clamp_len(a.lens[b * a.lens_s], max_tokens, &dummy);
      ns = L > 0 ? (L + C - 1) / C : 1;
    }
    int chunk_total;
    const int excl = block_exclusive_scan(ns, &chunk_total);
    if (b < a.B) {
      const int first = offset + excl;
      a.ws.nsplit[b] = ns;
      a.ws.base[b] = first;
      for (int s = 0; s < ns; ++s)
        if (first + s < a.max_items) a.ws.items[first + s] = make_int2(b, s);
    }
    offset += chunk_total;
  }
  if (tid == 0) {
    a.ws.hdr[0] = C;
    a.ws.hdr[1] = offset < a.max_items ? offset : a.max_items;
  }
  if (bad) atomicOr(a.ws.err, kErrLen);
}

// Split-KV decode on MFMA for a packed GQA group of up to 16 query heads.
// One wave per (work item, KV head, 16-head block). Keys are processed 32 at a
// time: K goes straight from HBM into A-operand registers (each lane loads
// 4 x 16 contiguous bytes of one key row), V is staged in LDS and read back
// transposed as the A operand of O^T += V^T P^T.
__global__ __launch_bounds__(64) void decode_mfma_kernel(DecodeArgs a) {
  __shared__ u16 vs[kTile][kHeadDim + 8];

  const int nqb = (a.R + 15) >> 4;
  const int per_item = a.Hkv * nqb;
  const int item = blockIdx.x / per_item;
  const int rem = blockIdx.x - item * per_item;
  const int g = rem % a.Hkv;
  const int qb = rem / a.Hkv;
  if (item >= a.ws.hdr[1]) return;
  const int2 it = a.ws.items[item];
  const int b = it.x, s = it.y;
  const int C = a.ws.hdr[0];
  const int max_tokens = a.kv.max_pages * a.kv.page_size;
  int bad = 0;
  const int L = clamp_len(a.lens[b * a.lens_s], max_tokens, &bad);
  const int t_begin = s * C;
  const int t_end = min(L, t_begin + C);

  const int lane = threadIdx.x;
  const int col = lane & 15, grp = lane >> 4;
  const int row0 = qb * 16;
  const int nrows = min(16, a.R - row0);
  const bool col_ok = col < nrows;
  const int h = g * a.R + row0 + (col_ok ? col : 0);

  bf16x8 qv[4];
  {
    const __bf16* qp = (const __bf16*)a.q + (int64_t)b * a.q_sb + (int64_t)h * a.q_sh + grp * 8;
#pragma unroll
    for (int c = 0; c < 4; ++c) qv[c] = col_ok ? load_bf16x8(qp + c * 32) : zero_bf16x8();
  }

  f32x4 o[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) o[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = kNegInf, l_run = 0.f;
  const float sl2 = a.scale * kLog2e;

  const int* bt_row = a.kv.bt + (int64_t)b * a.kv.bt_sb;
  const __bf16* kbase = (const __bf16*)a.kv.k + (int64_t)g * a.kv.sh + grp * 8;
  const __bf16* vbase = (const __bf16*)a.kv.v + (int64_t)g * a.kv.v_sh + grp * 8;

  if (t_begin < t_end) {
    bf16x8 kc[2][4], vc[2][4];
    auto load_tile = [&](int t0) {
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        int t = t0 + 16 * hh + col;
        t = t < t_end ? t : t_end - 1;
        const int64_t pg = page_of(bt_row, a.kv.bt_sj, t, a.kv.log2_page, a.kv.num_pages, &bad);
        const int slot = t & (a.kv.page_size - 1);
        const __bf16* kp = kbase + pg * a.kv.sp + (int64_t)slot * a.kv.ss;
        const __bf16* vp = vbase + pg * a.kv.v_sp + (int64_t)slot * a.kv.v_ss;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          kc[hh][c] = load_bf16x8(kp + c * 32);
          vc[hh][c] = load_bf16x8(vp + c * 32);
        }
      }
    };
    load_tile(t_begin);
    for (int t0 = t_begin; t0 < t_end; t0 += kTile) {
      __syncthreads();  // previous tile's V reads are done
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int c = 0; c < 4; ++c)
          *reinterpret_cast<bf16x8*>(&vs[16 * hh + col][c * 32 + grp * 8]) = vc[hh][c];
      f32x4 st[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        st[hh] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < 4; ++c) st[hh] = mfma_16x16x32(kc[hh][c], qv[c], st[hh]);
      }
      if (t0 + kTile < t_end) load_tile(t0 + kTile);

      float sv[8];
      float mt = kNegInf;
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = t0 + 16 * hh + 4 * grp + i;
          const float x = t < t_end ? st[hh][i] * sl2 : kNegInf;
          sv[hh * 4 + i] = x;
          mt = fmaxf(mt, x);
        }
      mt = group_max(mt);
      const float m_new = fmaxf(m_run, mt);
      const float alpha = exp2_fast(m_run - m_new);
      float ps = 0.f;
      bf16x8 pb;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float p = exp2_fast(sv[e] - m_new);
        ps += p;
        pb[e] = (__bf16)p;
      }
      l_run = l_run * alpha + ps;
      m_run = m_new;
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] *= alpha;
      __syncthreads();  // V tile visible
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        bf16x8 va;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int tok = e < 4 ? 4 * grp + e : 16 + 4 * grp + (e - 4);
          va[e] = bits_to_bf16(vs[tok][16 * j + col]);
        }
        o[j] = mfma_16x16x32(va, pb, o[j]);
      }
    }
  }

  const float l_tot = group_sum(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse_v = l_tot > 0.f ? (m_run + __builtin_amdgcn_logf(l_tot)) * kLn2 : kNegInf;
  if (col_ok) {
    if (a.ws.nsplit[b] == 1) {
      if (a.out_f32) {
        float* op = (float*)a.out + (int64_t)b * a.out_sb + (int64_t)h * a.out_sh + 4 * grp;
#pragma unroll
        for (int j = 0; j < 8; ++j) *reinterpret_cast<f32x4*>(op + 16 * j) = o[j] * inv;
      } else {
        __bf16* op = (__bf16*)a.out + (int64_t)b * a.out_sb + (int64_t)h * a.out_sh + 4 * grp;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
          bf16x4 w;
#pragma unroll
          for (int i = 0; i < 4; ++i) w[i] = (__bf16)(o[j][i] * inv);
          *reinterpret_cast<bf16x4*>(op + 16 * j) = w;
        }
      }
      if (a.lse && grp == 0) a.lse[(int64_t)b * a.lse_sb + (int64_t)h * a.lse_sh] = lse_v;
    } else {
      float* pp = a.ws.part_o + ((int64_t)item * a.Hq + h) * kHeadDim + 4 * grp;
#pragma unroll
      for (int j = 0; j < 8; ++j) *reinterpret_cast<f32x4*>(pp + 16 * j) = o[j] * inv;
      if (grp == 0) a.ws.part_lse[(int64_t)item * a.Hq + h] = lse_v;
    }
  }
  if (bad) atomicOr(a.ws.err, kErrPage);
}

// Single-query decode (one query head per KV head) on the vector ALUs: each
// 16-lane group takes one key per step (a whole 256-byte row per load), keeps
// its own online-softmax state, and the four groups are merged at the end.
__global__ __launch_bounds__(64) void decode_valu_kernel(DecodeArgs a) {
  const int item = blockIdx.x / a.Hkv;
  const int g = blockIdx.x - item * a.Hkv;
  if (item >= a.ws.hdr[1]) return;
  const int2 it = a.ws.items[item];
  const int b = it.x, s = it.y;
  const int C = a.ws.hdr[0];
  const int max_tokens = a.kv.max_pages * a.kv.page_size;
  int bad = 0;
  const int L = clamp_len(a.lens[b * a.lens_s], max_tokens, &bad);
  const int t_begin = s * C;
  const int t_end = min(L, t_begin + C);
  const int lane = threadIdx.x;
  const int c16 = lane & 15, grp = lane >> 4;
  const int h = g;  // R == 1

  const float sl2 = a.scale * kLog2e;
  float qf[8];
  {
    const bf16x8 qq = load_bf16x8((const __bf16*)a.q + (int64_t)b * a.q_sb + (int64_t)h * a.q_sh + c16 * 8);
#pragma unroll
    for (int i = 0; i < 8; ++i) qf[i] = (float)qq[i] * sl2;
  }
  float m = kNegInf, l = 0.f, acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  const int* bt_row = a.kv.bt + (int64_t)b * a.kv.bt_sb;
  const __bf16* kbase = (const __bf16*)a.kv.k + (int64_t)g * a.kv.sh + c16 * 8;
  const __bf16* vbase = (const __bf16*)a.kv.v + (int64_t)g * a.kv.v_sh + c16 * 8;
  for (int t0 = t_begin; t0 < t_end; t0 += 4) {
    const int t = t0 + grp;
    const bool valid = t < t_end;
    const int tt = valid ? t : t_end - 1;
    const int64_t pg = page_of(bt_row, a.kv.bt_sj, tt, a.kv.log2_page, a.kv.num_pages, &bad);
    const int slot = tt & (a.kv.page_size - 1);
    const bf16x8 kk = load_bf16x8(kbase + pg * a.kv.sp + (int64_t)slot * a.kv.ss);
    const bf16x8 vv = load_bf16x8(vbase + pg * a.kv.v_sp + (int64_t)slot * a.kv.v_ss);
    float d = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) d += qf[i] * (float)kk[i];
    d = xor_sum(d, 1);
    d = xor_sum(d, 2);
    d = xor_sum(d, 4);
    d = xor_sum(d, 8);
    if (valid) {
      const float m_new = fmaxf(m, d);
      const float alpha = exp2_fast(m - m_new);
      const float p = exp2_fast(d - m_new);
      l = l * alpha + p;
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] = acc[i] * alpha + p * (float)vv[i];
      m = m_new;
    }
  }
  const float M = group_max(m);
  const float w = m == kNegInf ? 0.f : exp2_fast(m - M);
  const float l_tot = group_sum(l * w);
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = group_sum(acc[i] * w);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse_v = l_tot > 0.f ? (M + __builtin_amdgcn_logf(l_tot)) * kLn2 : kNegInf;
  if (grp == 0) {
    if (a.ws.nsplit[b] == 1) {
      if (a.out_f32) {
        float* op = (float*)a.out + (int64_t)b * a.out_sb + (int64_t)h * a.out_sh + c16 * 8;
#pragma unroll
        for (int i = 0; i < 8; ++i) op[i] = acc[i] * inv;
      } else {
        bf16x8 w8;
#pragma unroll
        for (int i = 0; i < 8; ++i) w8[i] = (__bf16)(acc[i] * inv);
        *reinterpret_cast<bf16x8*>((__bf16*)a.out + (int64_t)b * a.out_sb + (int64_t)h * a.out_sh + c16 * 8) = w8;
      }
      if (a.lse && c16 == 0) a.lse[(int64_t)b * a.lse_sb + (int64_t)h * a.lse_sh] = lse_v;
    } else {
      float* pp = a.ws.part_o + ((int64_t)item * a.Hq + h) * kHeadDim + c16 * 8;
#pragma unroll
      for (int i = 0; i < 8; ++i) pp[i] = acc[i] * inv;
      if (c16 == 0) a.ws.part_lse[(int64_t)item * a.Hq + h] = lse_v;
    }
  }
  if (bad) atomicOr(a.ws.err, kErrPage);
}

// Merge the split partials of one (sequence, query head): one wave, two
// output elements per lane.
__device__ __forceinline__ void merge_parts(const float* o_base, int64_t o_step, const float* l_base, int64_t l_step,
                                            int n, float* out2, float* lse_out) {
  const int lane = threadIdx.x;
  float M = kNegInf;
  for (int s = 0; s < n; ++s) M = fmaxf(M, l_base[s * l_step]);
  float z = 0.f, a0 = 0.f, a1 = 0.f;
  if (M != kNegInf) {
    for (int s = 0; s < n; ++s) {
      const float ls = l_base[s * l_step];
      const float w = exp2_fast((ls - M) * kLog2e);
      const float2 v = *reinterpret_cast<const float2*>(o_base + s * o_step + 2 * lane);
      z += w;
      a0 += w * v.x;
      a1 += w * v.y;
    }
  }
  const float inv = z > 0.f ? 1.f / z : 0.f;
  out2[0] = a0 * inv;
  out2[1] = a1 * inv;
  *lse_out = z > 0.f ? M + __builtin_amdgcn_logf(z) * kLn2 : kNegInf;
}

__global__ __launch_bounds__(64) void combine_kernel(DecodeArgs a) {
  const int b = blockIdx.x / a.Hq;
  const int h = blockIdx.x - b * a.Hq;
  const int ns = a.ws.nsplit[b];
  if (ns <= 1) return;
  const int base = a.ws.base[b];
  if (base + ns > a.max_items) return;  // cannot happen for consistent plans
  float r[2], lse_v;
  merge_parts(a.ws.part_o + ((int64_t)base * a.Hq + h) * kHeadDim, (int64_t)a.Hq * kHeadDim,
              a.ws.part_lse + (int64_t)base * a.Hq + h, a.Hq, ns, r, &lse_v);
  const int lane = threadIdx.x;
  if (a.out_f32) {
    float* op = (float*)a.out + (int64_t)b * a.out_sb + (int64_t)h * a.out_sh + 2 * lane;
    op[0] = r[0];
    op[1] = r[1];
  } else {
    __bf16* op = (__bf16*)a.out + (int64_t)b * a.out_sb + (int64_t)h * a.out_sh + 2 * lane;
    op[0] = (__bf16)r[0];
    op[1] = (__bf16)r[1];
  }
  if (a.lse && lane == 0) a.lse[(int64_t)b * a.lse_sb + (int64_t)h * a.lse_sh] = lse_v;
}

__global__ __launch_bounds__(64) void merge_kernel(MergeArgs a) {
  const int n = blockIdx.x / a.H;
  const int h = blockIdx.x - n * a.H;
  int cnt = a.num[(int64_t)n * a.num_s];
  cnt = cnt < 0 ? 0 : (cnt > a.S ? a.S : cnt);
  float r[2], lse_v;
  merge_parts(a.o + (int64_t)n * a.o_sn + (int64_t)h * a.o_sh, a.o_ss, a.lse + (int64_t)n * a.l_sn + (int64_t)h * a.l_sh,
              a.l_ss, cnt, r, &lse_v);
  const int lane = threadIdx.x;
  if (a.out_f32) {
    float* op = (float*)a.out + (int64_t)n * a.out_sn + (int64_t)h * a.out_sh + 2 * lane;
    op[0] = r[0];
    op[1] = r[1];
  } else {
    __bf16* op = (__bf16*)a.out + (int64_t)n * a.out_sn + (int64_t)h * a.out_sh + 2 * lane;
    op[0] = (__bf16)r[0];
    op[1] = (__bf16)r[1];
  }
  if (a.lse_out && lane == 0) a.lse_out[(int64_t)n * a.lo_sn + (int64_t)h * a.lo_sh] = lse_v;
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream, KernelTimer* timer) {
  plan_decode_kernel<<<1, 1024, 0, stream>>>(a);
  const unsigned per_item = a.R == 1 ? a.Hkv : a.Hkv * ((a.R + 15) / 16);
  const unsigned grid = (unsigned)a.max_items * per_item;
  if (timer) (void)hipEventRecord(timer->start, stream);
  if (a.R == 1)
    decode_valu_kernel<<<grid, 64, 0, stream>>>(a);
  else
    decode_mfma_kernel<<<grid, 64, 0, stream>>>(a);
  if (timer) (void)hipEventRecord(timer->stop, stream);
  combine_kernel<<<(unsigned)(a.B * a.Hq), 64, 0, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_merge(const MergeArgs& a, hipStream_t stream) {
  merge_kernel<<<(unsigned)(a.N * a.H), 64, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace rl
