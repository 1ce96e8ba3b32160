// KV append: the new tokens' K and V rows (an appended turn's suffix, or one
// decode step's token) are written into their pages before attention reads
// them. Sequence b owns new rows qo_indptr[b] .. qo_indptr[b+1]-1 and holds
// kv_lens[b] tokens after the append, so new row i goes to logical position
// kv_lens[b] - n_b + i. FP8 pages receive the E4M3 code of the row divided
// by the KV head's scale.
//
// A thread moves one 8-element column of up to 8 KV heads of one new row: the
// 16 threads of a head row read and write 256 contiguous bytes (128 for FP8),
// and each thread has 16 row loads in flight before it looks up the page. The
// work is a copy: HBM-bound at 4 (bf16) or 3 (FP8) bytes moved per element.
#include "attn_common.hpp"
#include "kernels.hpp"

namespace rl {

namespace {

constexpr int kAppendThreads = 256;
constexpr int kGroup = 8;               // KV heads per thread (same column of each head row)
// FP8 appends whose 8-head grid would not give every CU a workgroup (a decode
// step's rows) take one head per thread: eight times the threads, each with an
// eighth of the serial quantisation work (a 128-row step: 11.7 -> 6.5 us; bf16
// rows, which are only copied, measured 5% slower that way and keep 8 heads)

// OCP E4M3 code of a float32 value, from the format's bit layout: nearest
// value, ties to the even code; magnitudes of 448 and above (infinity
// included) saturate to 448; NaN gives the NaN code. The sign is kept.
__device__ __forceinline__ uint32_t e4m3_from_f32(float f) {
  const uint32_t u = __float_as_uint(f);
  const uint32_t sign = (u >> 24) & 0x80u;
  const uint32_t a = u & 0x7FFFFFFFu;
  uint32_t code;
  if (a > 0x7F800000u) {
    code = 0x7Fu;                                   // NaN
  } else if (a >= 0x43E00000u) {
    code = 0x7Eu;                                   // >= 448: saturate
  } else if (a < 0x3C800000u) {
    // below 2^-6: the subnormal step is 2^-9, so the code is the value in
    // steps, rounded to nearest even (8 is the smallest normal, code 0x08)
    code = (uint32_t)__builtin_rintf(__uint_as_float(a) * 512.f);
  } else {
    const uint32_t e = (a >> 23) - 127u + 7u;       // biased E4M3 exponent, 1..15
    uint32_t r = (a >> 20) & 7u;                    // top three mantissa bits
    const uint32_t rest = a & 0xFFFFFu;
    if (rest > 0x80000u || (rest == 0x80000u && (r & 1u))) ++r;
    code = (e << 3) + r;                            // r == 8 carries into the exponent
    if (code > 0x7Eu) code = 0x7Eu;
  }
  return code | sign;
}

// E4M3 codes of eight bf16 values divided by the positive scale s (inv: the
// correctly rounded 1/s), four per word. The code is the E4M3 value nearest
// to the correctly rounded float32 quotient. Fast path: q0 = x * inv, then
// one residual correction q0 + (x - q0 s) inv, which is the correctly rounded
// quotient for normal results (Markstein's theorem: the residual is exact in
// an FMA and the reciprocal is correctly rounded); subnormal quotients, where
// it may be off, all encode to zero, and the sign is taken from x so that -0
// stays -0. The clamped value is then converted by the hardware E4M3
// conversion (round to nearest even), which matches the format's definition
// on every input in that range. Non-finite inputs, or a product that
// overflows, take the IEEE division and the bit-level encoder instead.
__device__ __forceinline__ uint2 e4m3_pack8(const bf16x8& x, float s, float inv) {
  float q[8];
  bool special = false;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float xf = (float)x[e];
    const float q0 = xf * inv;
    const float r = __builtin_fmaf(-q0, s, xf);
    q[e] = __builtin_copysignf(__builtin_fmaf(r, inv, q0), xf);
    special |= (__float_as_uint(q0) & 0x7F800000u) == 0x7F800000u;
  }
  uint2 w;
  if (!special) {
    auto c = [&](int e) { return __builtin_amdgcn_fmed3f(q[e], -448.f, 448.f); };
    w.x = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(c(0), c(1), 0, false);
    w.x = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(c(2), c(3), (int)w.x, true);
    w.y = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(c(4), c(5), 0, false);
    w.y = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(c(6), c(7), (int)w.y, true);
  } else {
    w.x = w.y = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t code = e4m3_from_f32((float)x[e] / s);
      if (e < 4) w.x |= code << (8 * e); else w.y |= code << (8 * (e - 4));
    }
  }
  return w;
}

template <bool kFp8, int kG>
__global__ __launch_bounds__(kAppendThreads) void append_kernel(AppendArgs a) {
  // thread -> (new row r, group of up to kG KV heads, 8-element column c)
  const int groups = (a.Hkv + kG - 1) / kG;
  const int per_row = groups * (kHeadDim / 8);
  const int64_t n_items = (int64_t)a.total_new * per_row;
  const int64_t i_raw = (int64_t)blockIdx.x * kAppendThreads + threadIdx.x;
  // FP8: every lane takes part in the wave's owner search below, so a lane
  // past the last item takes the last item and stores nothing
  if (!kFp8 && i_raw >= n_items) return;
  const bool valid = i_raw < n_items;
  const int64_t i = valid ? i_raw : n_items - 1;
  const int r = (int)(i / per_row);
  const int rem = (int)(i - (int64_t)r * per_row);
  const int g0 = (rem / (kHeadDim / 8)) * kG, c = rem % (kHeadDim / 8);
  const int gn = min(kG, a.Hkv - g0);
  // the new rows are read first (always in bounds), so their latency overlaps
  // the lookups below; into bf16 pages they are read non-temporally (the
  // multi-turn batch's 36,098 chunk rows: 54 -> 50 us; into FP8 pages the same
  // loads measured 4% slower, and non-temporal page stores gained nothing)
  bf16x8 kx[kG], vx[kG];
#pragma unroll
  for (int j = 0; j < kG; ++j) {
    const int g = g0 + (j < gn ? j : 0);
    const __bf16* kp = (const __bf16*)a.k_new + r * a.kn_st + g * a.kn_sh + 8 * c;
    const __bf16* vp = (const __bf16*)a.v_new + r * a.vn_st + g * a.vn_sh + 8 * c;
    if constexpr (kFp8) {
      kx[j] = *reinterpret_cast<const bf16x8*>(kp);
      vx[j] = *reinterpret_cast<const bf16x8*>(vp);
    } else {
      kx[j] = load_nt<bf16x8>(kp);
      vx[j] = load_nt<bf16x8>(vp);
    }
  }
  // FP8: the heads' scales are read with the rows (one round trip for both)
  float ksc[kG], vsc[kG];
  if constexpr (kFp8) {
#pragma unroll
    for (int j = 0; j < kG; ++j) {
      const int g = g0 + (j < gn ? j : 0);
      ksc[j] = a.k_scale[g * a.ks_s];
      vsc[j] = a.v_scale[g * a.vs_s];
    }
  }
  // owning sequence b: the last with qo_indptr[b] <= r; q0, q1 its rows' bounds
  int b, q0, q1, kv;
  if (kFp8 && a.B < 64) {
    // FP8 (the quantisation leaves less room to hide the lookups): one round
    // trip for the whole wave. Lane l holds qo_indptr[l] and kv_lens[l]
    // (loaded with the rows); a ballot per distinct row of the wave (at most
    // five: a row has at least 16 items) counts the sequences starting at or
    // before it, and shuffles hand out the owner's bounds and length. The
    // multi-turn batch's chunk rows: 53.0 -> 49.0 us; the same search took
    // the bf16 append 49.9 -> 50.8 us, which keeps the binary search.
    const int lane = threadIdx.x & 63;
    const int x = lane <= a.B ? a.qo_indptr[(int64_t)lane * a.indptr_s] : 0x7fffffff;
    const int y = lane < a.B ? a.kv_lens[(int64_t)lane * a.kv_lens_s] : 0;
    const int r_lo = __builtin_amdgcn_readlane(r, 0), r_hi = __builtin_amdgcn_readlane(r, 63);
    b = 0;
    for (int rr = r_lo; rr <= r_hi; ++rr) {
      const int cnt = __popcll(__builtin_amdgcn_ballot_w64(x <= rr));
      if (r == rr) b = cnt - 1;
    }
    b = min(max(b, 0), a.B - 1);
    q0 = __shfl(x, b);
    q1 = __shfl(x, b + 1);
    kv = __shfl(y, b);
  } else {
    int lo = 0, hi = a.B - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (a.qo_indptr[(int64_t)mid * a.indptr_s] <= r) lo = mid; else hi = mid - 1;
    }
    b = lo;
    q0 = a.qo_indptr[(int64_t)b * a.indptr_s];
    q1 = a.qo_indptr[(int64_t)(b + 1) * a.indptr_s];
    kv = a.kv_lens[(int64_t)b * a.kv_lens_s];
  }
  if (!valid) return;
  if (r < q0 || r >= q1) {              // qo_indptr not a partition of the new rows
    atomicOr(a.err, kErrIndptr);
    return;
  }
  const int n = q1 - q0;
  if (kv < n || kv > a.max_pages * a.page_size) {
    atomicOr(a.err, kv < n ? kErrKvShort : kErrLen);
    return;
  }
  const int t = kv - n + (r - q0);
  const int page = a.bt[(int64_t)b * a.bt_sb + (int64_t)(t >> a.log2_page) * a.bt_sj];
  if ((unsigned)page >= (unsigned)a.num_pages) {   // never write outside the pool
    atomicOr(a.err, kErrPage);
    return;
  }
  const int slot = t & (a.page_size - 1);
  const int64_t kbase = (int64_t)page * a.sp + (int64_t)slot * a.ss + 8 * c;
  const int64_t vbase = (int64_t)page * a.v_sp + (int64_t)slot * a.v_ss + 8 * c;
#pragma unroll
  for (int j = 0; j < kG; ++j) {
    if (j >= gn) break;
    const int g = g0 + j;
    const int64_t ko = kbase + (int64_t)g * a.sh, vo = vbase + (int64_t)g * a.v_sh;
    if constexpr (!kFp8) {
      *reinterpret_cast<bf16x8*>((__bf16*)a.k + ko) = kx[j];
      *reinterpret_cast<bf16x8*>((__bf16*)a.v + vo) = vx[j];
    } else {
      const float ks = ksc[j], vs = vsc[j];
      if (!scale_ok(ks) || !scale_ok(vs)) {
        atomicOr(a.err, kErrScale);
        continue;
      }
      *reinterpret_cast<uint2*>((uint8_t*)a.k + ko) = e4m3_pack8(kx[j], ks, 1.0f / ks);
      *reinterpret_cast<uint2*>((uint8_t*)a.v + vo) = e4m3_pack8(vx[j], vs, 1.0f / vs);
    }
  }
}

}  // namespace

hipError_t launch_append(const AppendArgs& a, hipStream_t stream, KernelTimer* timer) {
  auto grid_of = [&](int g) {
    const int64_t threads = (int64_t)a.total_new * ((a.Hkv + g - 1) / g) * (kHeadDim / 8);
    return (unsigned)((threads + kAppendThreads - 1) / kAppendThreads);
  };
  const bool one = a.k_scale != nullptr && grid_of(kGroup) < 256u;
  const unsigned grid = grid_of(one ? 1 : kGroup);
  if (timer) (void)hipEventRecord(timer->start, stream);
  if (a.k_scale) {
    if (one)
      append_kernel<true, 1><<<grid, kAppendThreads, 0, stream>>>(a);
    else
      append_kernel<true, kGroup><<<grid, kAppendThreads, 0, stream>>>(a);
  } else {
    append_kernel<false, kGroup><<<grid, kAppendThreads, 0, stream>>>(a);
  }
  if (timer) (void)hipEventRecord(timer->stop, stream);
  return hipGetLastError();
}

}  // namespace rl
