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

__device__ __forceinline__ float xor_max(float v, int mask) { return fmaxf(v, __shfl_xor(v, mask, 64)); }
__device__ __forceinline__ float xor_sum(float v, int mask) { return v + __shfl_xor(v, mask, 64); }

// Max / sum over the four lane groups (lanes l, l^16, l^32, l^48).
__device__ __forceinline__ float group_max(float v) { return xor_max(xor_max(v, 16), 32); }
__device__ __forceinline__ float group_sum(float v) { return xor_sum(xor_sum(v, 16), 32); }

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

// Exclusive prefix sum over the calling block (all threads must call it);
// wave_tot is a 16-int LDS scratch array. Returns this thread's exclusive sum
// and the block total in *total.
__device__ __forceinline__ int block_exclusive_scan(int v, int* total, int* wave_tot) {
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

}  // namespace rl
