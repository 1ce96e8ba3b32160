// Device-side building blocks shared by the decode and extend kernels (gfx950).
//
// MFMA conventions used throughout (v_mfma_f32_16x16x32_bf16, wave64):
//   A operand (16 x 32): lane l holds row (l % 16) and 8 consecutive k values
//                        selected by the lane group (l / 16);
//   B operand (32 x 16): lane l holds column (l % 16), k values as for A;
//   C/D (16 x 16, f32):  lane l holds column (l % 16), rows 4*(l/16) + i, i < 4.
// Both operands of one product always place the same contraction index at the
// same (lane group, element) slot, so any bijection between slots and the
// contracted index gives the same dot products; the kernels choose that
// bijection to make loads contiguous.
//
// Attention is computed "transposed": S^T = K Q^T puts keys on MFMA rows and
// query rows on MFMA columns, so a query row's softmax state (running max and
// sum, and its column of O^T = V^T P^T) stays inside the lanes with the same
// l % 16 and the rescale factor never crosses lanes.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.hpp"

namespace rl {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16;

constexpr int kHeadDim = 128;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ f32x4 mfma_16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// Cross-lane exchanges that stay in the VALU (no LDS round trip). Inside a
// 16-lane row DPP permutes operands: quad_perm [1,0,3,2] and [2,3,0,1] pair
// lane l with l^1 and l^2, half_mirror pairs l with 7-l inside 8 lanes and
// mirror pairs l with 15-l. Across rows and halves, the gfx950 lane swaps
// exchange rows 2i and 2i+1 (permlane16) or lanes l and l+32 (permlane32);
// each returns both swapped registers, and as the two hold, in every lane, the
// lane's own value and its partner's, their max or sum is the pair's.
template <int kCtrl>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), kCtrl, 0xf, 0xf, false));
}
constexpr int kDppXor1 = 0xb1;         // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4e;         // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;  // l -> 7 - l within 8 lanes
constexpr int kDppMirror = 0x140;      // l -> 15 - l within 16 lanes

__device__ __forceinline__ float max_l16(float v) {   // max over lanes l, l^16
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_l16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float max_l32(float v) {   // max over lanes l, l^32
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_l32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// Sum over the 16 lanes of a row; every lane of the row receives it.
__device__ __forceinline__ float row_sum16(float v) {
  v += dpp<kDppXor1>(v);
  v += dpp<kDppXor2>(v);
  v += dpp<kDppHalfMirror>(v);
  return v + dpp<kDppMirror>(v);
}
// Max / sum over the four lane groups (lanes l, l^16, l^32, l^48).
__device__ __forceinline__ float group_max(float v) { return max_l32(max_l16(v)); }
__device__ __forceinline__ float group_sum(float v) { return sum_l32(sum_l16(v)); }
// Max / sum over all 64 lanes; every lane receives it.
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp<kDppXor1>(v));
  v = fmaxf(v, dpp<kDppXor2>(v));
  v = fmaxf(v, dpp<kDppHalfMirror>(v));
  v = fmaxf(v, dpp<kDppMirror>(v));
  return group_max(v);
}
__device__ __forceinline__ float wave_sum(float v) { return group_sum(row_sum16(v)); }

__device__ __forceinline__ bf16x8 zero_bf16x8() {
  bf16x8 z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = (__bf16)0.0f;
  return z;
}

__device__ __forceinline__ bf16x8 load_bf16x8(const __bf16* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}

__device__ __forceinline__ __bf16 bits_to_bf16(u16 b) { return __builtin_bit_cast(__bf16, b); }

// Bytes per stored KV element: bf16, or an FP8 E4M3 code.
template <bool kFp8>
constexpr int kv_bytes() { return kFp8 ? 1 : 2; }

// Eight consecutive stored KV elements as loaded from memory: a bf16x8, or
// eight FP8 E4M3 codes. Kernels that prefetch keep this raw form in flight and
// convert where the values are used, so a conversion never waits on a load
// that was issued for a later step.
template <bool kFp8>
struct KvRawOf {
  typedef bf16x8 type;
};
template <>
struct KvRawOf<true> {
  typedef uint2 type;
};
template <bool kFp8>
using KvRaw = typename KvRawOf<kFp8>::type;

template <bool kFp8>
__device__ __forceinline__ KvRaw<kFp8> load_kv_raw(const char* p) {
  return *reinterpret_cast<const KvRaw<kFp8>*>(p);
}

// Loads of K/V rows that a pass reads exactly once (single- and multi-token
// decode, the group-prefix pass): non-temporal, so the caches stream them.
// Measured on gfx950 with 256-byte rows 2 KB apart, 16-byte loads: 6.7 TB/s
// when each instruction reads half of one 128-byte line of every row it
// touches (the other half in the next instruction) and 6.9 TB/s for whole
// rows per instruction, against 5.8-6.0 TB/s with ordinary loads; a row read
// in pieces scattered over both of its lines by each of four instructions
// drops to 4.2 TB/s (each piece fetches its lines again). The extend pass
// keeps ordinary loads: its work units of one (sequence, KV head) share keys
// through the L2.
typedef unsigned int nt_u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int nt_u32x2 __attribute__((ext_vector_type(2)));
template <typename T>
__device__ __forceinline__ T load_nt(const void* p) {
  static_assert(sizeof(T) == 16 || sizeof(T) == 8, "16- or 8-byte row loads");
  if constexpr (sizeof(T) == 16)
    return __builtin_bit_cast(T, __builtin_nontemporal_load(static_cast<const nt_u32x4*>(p)));
  else
    return __builtin_bit_cast(T, __builtin_nontemporal_load(static_cast<const nt_u32x2*>(p)));
}
template <bool kFp8>
__device__ __forceinline__ KvRaw<kFp8> load_kv_raw_nt(const char* p) {
  return load_nt<KvRaw<kFp8>>(p);
}

// Raw elements as a bf16x8 MFMA operand: bf16 as stored; FP8 E4M3 codes
// converted by the gfx950 packed conversion, two per instruction, which is
// exact (every E4M3 value, subnormals included, is a bf16 value; the
// conversion's scale is 1).
template <bool kFp8>
__device__ __forceinline__ bf16x8 kv_to_bf16x8(KvRaw<kFp8> w) {
  if constexpr (!kFp8) {
    return w;
  } else {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w.x, 1.0f, false);
    const bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w.x, 1.0f, true);
    const bf16x2 c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w.y, 1.0f, false);
    const bf16x2 d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w.y, 1.0f, true);
    return bf16x8{a.x, a.y, b.x, b.y, c.x, c.y, d.x, d.y};
  }
}

// Load and convert at once (for loads whose values are used right away).
template <bool kFp8>
__device__ __forceinline__ bf16x8 load_kv8(const char* p) {
  return kv_to_bf16x8<kFp8>(load_kv_raw<kFp8>(p));
}
template <bool kFp8>
__device__ __forceinline__ bf16x8 load_kv8_nt(const char* p) {
  return kv_to_bf16x8<kFp8>(load_kv_raw_nt<kFp8>(p));
}

// A dequantisation scale is usable when it is positive, non-zero and finite:
// its bit pattern lies in [1, 0x7f7fffff] (smallest positive subnormal up to
// the largest finite float). Tested on the bits rather than by comparisons,
// since the device code is compiled assuming no NaN operands.
__device__ __forceinline__ bool scale_ok(float s) { return (__float_as_uint(s) - 1u) < 0x7f7fffffu; }

// Dequantisation scales of KV head g (1 for bf16 pages); *bad is set when a
// scale is not positive and finite.
struct KvScales {
  float k, v;
};
template <bool kFp8, typename KV>
__device__ __forceinline__ KvScales kv_scales(const KV& kv, int g, int* bad) {
  if constexpr (!kFp8) {
    return {1.f, 1.f};
  } else {
    const float ks = kv.k_scale[g * kv.ks_s], vs = kv.v_scale[g * kv.vs_s];
    if (!scale_ok(ks) || !scale_ok(vs)) *bad = 1;
    return {ks, vs};
  }
}

// Page id of logical token t, clamped into the pool (a bad id is recorded in
// *bad). The host guarantees that block-table column strides and indices fit
// 24 bits, so the index is a single 24-bit multiply.
__device__ __forceinline__ uint32_t page_of(const int* bt_row, uint32_t bt_sj, int t, int log2p, int num_pages,
                                            int* bad) {
  int pg = bt_row[__umul24((uint32_t)(t >> log2p), bt_sj)];
  if ((unsigned)pg >= (unsigned)num_pages) {
    *bad = 1;
    pg = pg < 0 ? 0 : num_pages - 1;
  }
  return (uint32_t)pg;
}

// Element offset of (page, slot) inside a page pool: the page stride fits 32
// bits and the slot stride 24 bits (host-checked), so this is one 32x32->64
// multiply-add plus one 24-bit multiply.
__device__ __forceinline__ uint64_t row_offset(uint32_t pg, uint32_t sp, int slot, uint32_t ss) {
  return (uint64_t)pg * sp + __umul24((uint32_t)slot, ss);
}

// Inclusive prefix sums over a wave's 64 lanes, without LDS: DPP row shifts
// (row_shr 1, 2, 4, 8; lanes shifted in from outside the 16-lane row read 0)
// scan each row, then each row adds the totals of the rows below it, read from
// lanes 15, 31 and 47. Every lane of the wave must be active.
template <int kCtrl>
__device__ __forceinline__ int dpp_shr(int v) {
  return __builtin_amdgcn_update_dpp(0, v, kCtrl, 0xf, 0xf, true);
}
__device__ __forceinline__ int wave_inclusive_scan(int x) {
  x += dpp_shr<0x111>(x);
  x += dpp_shr<0x112>(x);
  x += dpp_shr<0x114>(x);
  x += dpp_shr<0x118>(x);
  const int r0 = __builtin_amdgcn_readlane(x, 15), r1 = __builtin_amdgcn_readlane(x, 31);
  const int r2 = __builtin_amdgcn_readlane(x, 47);
  const int row = (threadIdx.x & 63) >> 4;
  return x + (row >= 1 ? r0 : 0) + (row >= 2 ? r1 : 0) + (row >= 3 ? r2 : 0);
}
template <int kCtrl>
__device__ __forceinline__ long long dpp_shr64(long long v) {
  const uint32_t lo = (uint32_t)dpp_shr<kCtrl>((int)(uint32_t)v);
  const uint32_t hi = (uint32_t)dpp_shr<kCtrl>((int)(uint32_t)((unsigned long long)v >> 32));
  return (long long)(((unsigned long long)hi << 32) | lo);
}
__device__ __forceinline__ long long readlane64(long long v, int lane) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((unsigned long long)v >> 32), lane);
  return (long long)(((unsigned long long)hi << 32) | lo);
}
__device__ __forceinline__ long long wave_inclusive_scan64(long long x) {
  x += dpp_shr64<0x111>(x);
  x += dpp_shr64<0x112>(x);
  x += dpp_shr64<0x114>(x);
  x += dpp_shr64<0x118>(x);
  const long long r0 = readlane64(x, 15), r1 = readlane64(x, 31), r2 = readlane64(x, 47);
  const int row = (threadIdx.x & 63) >> 4;
  return x + (row >= 1 ? r0 : 0) + (row >= 2 ? r1 : 0) + (row >= 3 ? r2 : 0);
}

// Exclusive prefix sum over the calling block (all threads must call it);
// wave_tot is a 16-int LDS scratch array. Returns this thread's exclusive sum
// and the block total in *total.
__device__ __forceinline__ int block_exclusive_scan(int v, int* total, int* wave_tot) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int x = wave_inclusive_scan(v);
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

// 64-bit version of block_exclusive_scan (wave_tot: 16 slots).
__device__ __forceinline__ long long block_exclusive_scan64(long long v, long long* total, long long* wave_tot) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const long long x = wave_inclusive_scan64(v);
  if (lane == 63) wave_tot[wave] = x;
  __syncthreads();
  long long before = 0, all = 0;
  const int nw = blockDim.x >> 6;
  for (int w = 0; w < nw; ++w) {
    const long long t = wave_tot[w];
    if (w < wave) before += t;
    all += t;
  }
  __syncthreads();
  *total = all;
  return before + x - v;
}

}  // namespace rl
