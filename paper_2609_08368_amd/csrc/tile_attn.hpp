// Multi-row attention tile on MFMA 32x32x16, shared by the extend kernel
// (rows = chunk tokens x query heads) and the group-prefix kernel (rows =
// trajectory-group members x query heads). A workgroup of kWaves waves owns up
// to 32 * kWaves query rows that all read the same keys of one KV head; each
// wave owns 32 rows, i.e. one 32-wide MFMA column block.
//
// Per 64-key step the workgroup stages K and V of the step in LDS (double
// buffered: the rows of a later step are fetched into registers while the
// current step computes -- one step ahead, or two with kDeep -- and page ids
// one step before the rows they address), then every wave computes
//   S^T = K Q^T            (A = K rows from LDS, B = Q held in registers),
//   P^T = exp2(S^T - m)    (per query column, in registers),
//   O^T += V^T P^T         (A = V^T read with the LDS transpose load),
// so a query row's softmax state stays in the two lanes that hold its column.
// The running maximum is only raised when a step's maximum exceeds it by more
// than 2^8 (lazy rescaling): until then exp2 arguments stay below 8, which
// fp32 sums and bf16 probabilities hold as well as values below 1, and the
// O^T rescale (64 multiplies per lane) is skipped on almost every step.
#pragma once

#include "attn_common.hpp"

namespace rl {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kWaveRows = 32;              // query rows per wave
constexpr int kKeys = 64;                  // keys per step
constexpr int kKStride = kHeadDim + 8;     // LDS row pitch of K (u16): 272 B
constexpr int kVStride = kHeadDim + 32;    // LDS row pitch of V (u16): 320 B, spreads transpose loads over banks
constexpr float kLazy = 8.0f;              // log2 headroom before the running max is raised

struct TileLds {
  u16 ks[2][kKeys][kKStride];
  u16 vs[2][kKeys][kVStride];
};

__device__ __forceinline__ f32x16 mfma_32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Loads this lane's query row as the B operand of S^T = K Q^T: chunk c holds
// elements 16c + 8*(lane/32) .. +8 (the same k order as the K operand below).
__device__ __forceinline__ void load_q_operand(const __bf16* row, bool ok, bf16x8 (&qv)[8]) {
  const int kg = (threadIdx.x & 63) >> 5;
#pragma unroll
  for (int c = 0; c < 8; ++c) qv[c] = ok ? load_bf16x8(row + 16 * c + 8 * kg) : zero_bf16x8();
}

// Attention of this lane's query column over keys [t_lo, t_hi) of one KV head
// g of the sequence whose block-table row is bt_row. Keys above `limit` are
// masked for this column; keys below t_full are visible to every column of the
// workgroup (no mask work for those steps). t_lo must be a multiple of kKeys.
// Accumulates into o (O^T, 4 blocks of 32 dims), m_run (log2 units) and l_run
// (this lane's half of the row sum; add lane ^ 32's for the total).
template <int kWaves, bool kDeep>
__device__ __forceinline__ void tile_attend(const PagedKV& kv, float scale, const int* bt_row, int g, int t_lo,
                                            int t_hi, int t_full, int limit, const bf16x8 (&qv)[8], TileLds& lds,
                                            f32x16 (&o)[4], float& m_run, float& l_run, int& bad) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int col = lane & 31, kg = lane >> 5;
  const float sl2 = scale * kLog2e;

  // cooperative staging: thread -> (key rows tid/16 + kRowStep i, 16-byte chunk tid % 16)
  constexpr int kRowStep = kWaves * 4;              // key rows covered by one pass of the workgroup
  constexpr int kStageRows = kKeys / kRowStep;      // key rows each thread stages per step
  const uint32_t bt_sj = (uint32_t)kv.bt_sj;
  const int ld_row = tid >> 4, ld_chunk = (tid & 15) * 8;
  const __bf16* kbase = (const __bf16*)kv.k + (int64_t)g * kv.sh + ld_chunk;
  const __bf16* vbase = (const __bf16*)kv.v + (int64_t)g * kv.v_sh + ld_chunk;
  const uint32_t ksp = (uint32_t)kv.sp, kss = (uint32_t)kv.ss;
  const uint32_t vsp = (uint32_t)kv.v_sp, vss = (uint32_t)kv.v_ss;
  const int pmask = kv.page_size - 1;
  // A page of at least one step holds all keys of an aligned step: one lookup
  // per step. Page ids are loaded one step ahead of the K/V rows they address,
  // so a step's row loads never wait for a block-table load.
  const bool page_holds_step = kv.page_size >= kKeys;
  int praw[kStageRows];
  auto fetch_pages = [&](int t0) {
#pragma unroll
    for (int i = 0; i < kStageRows; ++i) {
      int t = t0 + (page_holds_step ? 0 : ld_row + kRowStep * i);
      t = t < t_hi ? t : t_hi - 1;
      praw[i] = (page_holds_step && i) ? 0 : bt_row[__umul24((uint32_t)(t >> kv.log2_page), bt_sj)];
    }
  };
  typedef bf16x8 Rows[kStageRows];
  auto fetch_rows = [&](int t0, Rows& kr, Rows& vr) {
#pragma unroll
    for (int i = 0; i < kStageRows; ++i) {
      int t = t0 + ld_row + kRowStep * i;
      t = t < t_hi ? t : t_hi - 1;
      int pg = praw[page_holds_step ? 0 : i];
      if ((unsigned)pg >= (unsigned)kv.num_pages) {
        bad = 1;
        pg = pg < 0 ? 0 : kv.num_pages - 1;
      }
      kr[i] = load_bf16x8(kbase + row_offset((uint32_t)pg, ksp, t & pmask, kss));
      vr[i] = load_bf16x8(vbase + row_offset((uint32_t)pg, vsp, t & pmask, vss));
    }
  };
  auto stage = [&](int buf, const Rows& kr, const Rows& vr) {
#pragma unroll
    for (int i = 0; i < kStageRows; ++i) {
      *reinterpret_cast<bf16x8*>(&lds.ks[buf][ld_row + kRowStep * i][ld_chunk]) = kr[i];
      *reinterpret_cast<bf16x8*>(&lds.vs[buf][ld_row + kRowStep * i][ld_chunk]) = vr[i];
    }
  };

  // Transpose-load addressing for the V^T operand. In a 16-lane block, lane i
  // receives element i % 4 of the 8 bytes addressed by lane 4e + i / 4 as its
  // element e. Lane l therefore addresses key row 4*(l/32) + (l%16)/4 (plus 8
  // for the second load) and columns 16*((l/16)%2) + 4*(l%4) of a 16-key,
  // 32-column block, and receives V[keys][its own column] in the k order of
  // the P^T operand (key 8*(e/4) + 4*(l/32) + e%4 of the 16-key group).
  const int tr_row = 4 * kg + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  if (t_lo >= t_hi) return;
  const int nsteps = (t_hi - t_lo + kKeys - 1) / kKeys;

  // one step: prefetch, S^T, softmax, PV, then stage the next step's rows
  auto step = [&](int j, Rows& k_next, Rows& v_next, Rows& k_free, Rows& v_free) {
    const int t0 = t_lo + j * kKeys;
    const int buf = j & 1;
    if constexpr (kDeep) {
      // rows of step j+2 go into the set staged at the end of step j-1
      if (j + 2 < nsteps) {
        fetch_rows(t0 + 2 * kKeys, k_free, v_free);
        if (j + 3 < nsteps) fetch_pages(t0 + 3 * kKeys);
      }
    } else {
      if (j + 1 < nsteps) {
        fetch_rows(t0 + kKeys, k_next, v_next);
        if (j + 2 < nsteps) fetch_pages(t0 + 2 * kKeys);
      }
    }

    // S^T for the two 32-key blocks of this step; the two accumulation chains
    // are interleaved so each MFMA's predecessor in its chain has retired
    f32x16 sc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[kb][e] = 0.f;
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8 kop = *reinterpret_cast<const bf16x8*>(&lds.ks[buf][32 * kb + col][16 * c + 8 * kg]);
        sc[kb] = mfma_32x32x16(kop, qv[c], sc[kb]);
      }

    // Row max of the raw scores (the positive scale commutes with max and is
    // folded into the exponent below); the mask only where some column cannot
    // see all of the step's keys. Keys at or beyond t_hi are masked as well.
    float mt = kNegInf;
    if (t0 + kKeys > t_full) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = t0 + 32 * kb + 8 * (e >> 2) + 4 * kg + (e & 3);
          if (key > limit || key >= t_hi) sc[kb][e] = kNegInf;
        }
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; e += 2) mt = fmaxf(mt, fmaxf(sc[kb][e], sc[kb][e + 1]));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64)) * sl2;
    // lazy rescale: raise the running max only when the step's max exceeds it by 2^8
    const bool raise = mt > m_run + kLazy;
    if (__builtin_amdgcn_ballot_w64(raise) != 0) {
      const float m_new = raise ? mt : m_run;
      const float alpha = exp2_fast(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int jd = 0; jd < 4; ++jd) o[jd] *= alpha;
      m_run = m_new;
    }

    // p = exp2(scale * log2(e) * s - m), rounded to bf16 for the PV product; the
    // row sum keeps the fp32 values (four independent partial sums)
    bf16x8 pb[4];
    const float neg_m = -m_run;
    float ps[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int h = 0; h < 4; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float p = exp2_fast(fmaf(sc[h >> 1][8 * (h & 1) + e], sl2, neg_m));
        ps[e & 3] += p;
        pb[h][e] = (__bf16)p;
      }
    l_run += (ps[0] + ps[1]) + (ps[2] + ps[3]);

    // O^T += V^T P^T over the step's four 16-key groups
#pragma unroll
    for (int h = 0; h < 4; ++h) {
#pragma unroll
      for (int jd = 0; jd < 4; ++jd) {
        const u16* vp = &lds.vs[buf][16 * h + tr_row][32 * jd + tr_col];
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)vp);
        const i16x4 up = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vp + 8 * kVStride));
        const i16x8 v8 = __builtin_shufflevector(lo, up, 0, 1, 2, 3, 4, 5, 6, 7);
        o[jd] = mfma_32x32x16(__builtin_bit_cast(bf16x8, v8), pb[h], o[jd]);
      }
    }
    if (j + 1 < nsteps) {
      stage(buf ^ 1, k_next, v_next);
      __syncthreads();
    }
  };

  Rows ka, va, kb2, vb2;
  fetch_pages(t_lo);
  fetch_rows(t_lo, ka, va);
  stage(0, ka, va);
  if (nsteps > 1) fetch_pages(t_lo + kKeys);
  if constexpr (kDeep) {
    // two steps in flight: rows of step 1 load now, page ids of step 2 too
    if (nsteps > 1) {
      fetch_rows(t_lo + kKeys, kb2, vb2);
      if (nsteps > 2) fetch_pages(t_lo + 2 * kKeys);
    }
    __syncthreads();
    for (int j = 0; j < nsteps; j += 2) {
      step(j, kb2, vb2, ka, va);
      if (j + 1 < nsteps) step(j + 1, ka, va, kb2, vb2);
    }
  } else {
    __syncthreads();
    for (int j = 0; j < nsteps; ++j) step(j, ka, va, ka, va);
  }
}

// Normalised output row of this lane's column: element (jd, q, i) of o holds
// dimension 32 jd + 8 q + 4 (lane/32) + i.
template <typename T>
__device__ __forceinline__ void store_o_row(T* row, const f32x16 (&o)[4], float inv) {
  const int kg = (threadIdx.x & 63) >> 5;
  typedef T t4 __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int jd = 0; jd < 4; ++jd)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      t4 w;
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = (T)(o[jd][4 * q + i] * inv);
      *reinterpret_cast<t4*>(row + 32 * jd + 8 * q + 4 * kg) = w;
    }
}

}  // namespace rl
