// Multi-row attention tile on MFMA 32x32x16, shared by the extend kernel
// (rows = chunk tokens x query heads; tile_attend_pp, and tile_attend_dl with
// 128-key steps for bf16 pages of at least 64 keys), the group-prefix kernel
// (rows = trajectory-group members x query heads) and the multi-token decode
// kernel (rows = query tokens x query heads; both tile_attend). A workgroup of
// kWaves waves owns up to 32 * kWaves query rows that all read the same keys
// of one KV head; each wave owns 32 rows, i.e. one 32-wide MFMA column block.
//
// Per 64-key step the workgroup stages K and V of the step in LDS (double
// buffered: the rows of the next step are fetched into registers while the
// current step computes, and page ids one step before the rows they
// address), then every wave computes
//   S^T = K Q^T            (A = K rows from LDS, B = Q held in registers),
//   P^T = exp2(S^T - m)    (per query column, in registers),
//   O^T += V^T P^T         (A = V^T read with the LDS transpose load),
// so a query row's softmax state stays in the two lanes that hold its column.
// The running maximum is only raised when a step's maximum exceeds it by more
// than 2^8 (lazy rescaling): until then exp2 arguments stay below 8, which
// fp32 sums and bf16 probabilities hold as well as values below 1, and the
// O^T rescale (64 multiplies per lane) is skipped on almost every step.
#pragma once

#include <type_traits>

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
// g of the sequence whose block-table row is bt_row. Keys above `limit` and
// keys below t_min are masked for this column; keys in [t_min, t_full) are
// visible to every column of the workgroup (no mask work for those steps).
// t_lo must be a multiple of kKeys. A column that sees no key keeps m_run =
// -inf and l_run = 0. Accumulates into o (O^T, 4 blocks of 32 dims), m_run
// (log2 units) and l_run (this lane's half of the row sum; add lane ^ 32's
// for the total). A wave that holds no query row passes active = false: it
// still stages its share of the rows and meets every barrier, but issues no
// MFMA and no softmax work.
template <int kWaves, bool kFp8 = false>
__device__ __forceinline__ void tile_attend(const PagedKV& kv, float scale, const int* bt_row, int g, int t_lo,
                                            int t_hi, int t_full, int limit, const bf16x8 (&qv)[8], TileLds& lds,
                                            f32x16 (&o)[4], float& m_run, float& l_run, int& bad,
                                            int t_min = -1, bool active = true) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int col = lane & 31, kg = lane >> 5;
  const float sl2 = scale * kLog2e;

  // cooperative staging: thread -> (key rows tid/16 + kRowStep i, 16-byte chunk tid % 16)
  constexpr int kRowStep = kWaves * 4;              // key rows covered by one pass of the workgroup
  constexpr int kStageRows = kKeys / kRowStep;      // key rows each thread stages per step
  const uint32_t bt_sj = (uint32_t)kv.bt_sj;
  const int ld_row = tid >> 4, ld_chunk = (tid & 15) * 8;
  constexpr int ES = kv_bytes<kFp8>();
  const char* kbase = (const char*)kv.k + ES * ((int64_t)g * kv.sh + ld_chunk);
  const char* vbase = (const char*)kv.v + ES * ((int64_t)g * kv.v_sh + ld_chunk);
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
  typedef KvRaw<kFp8> Rows[kStageRows];      // raw rows in flight, converted when staged
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
      kr[i] = load_kv_raw_nt<kFp8>(kbase + ES * row_offset((uint32_t)pg, ksp, t & pmask, kss));
      vr[i] = load_kv_raw_nt<kFp8>(vbase + ES * row_offset((uint32_t)pg, vsp, t & pmask, vss));
    }
  };
  auto stage = [&](int buf, const Rows& kr, const Rows& vr) {
#pragma unroll
    for (int i = 0; i < kStageRows; ++i) {
      *reinterpret_cast<bf16x8*>(&lds.ks[buf][ld_row + kRowStep * i][ld_chunk]) = kv_to_bf16x8<kFp8>(kr[i]);
      *reinterpret_cast<bf16x8*>(&lds.vs[buf][ld_row + kRowStep * i][ld_chunk]) = kv_to_bf16x8<kFp8>(vr[i]);
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
  auto step = [&](int j, Rows& k_next, Rows& v_next) {
    const int t0 = t_lo + j * kKeys;
    const int buf = j & 1;
    if (j + 1 < nsteps) {
      fetch_rows(t0 + kKeys, k_next, v_next);
      if (j + 2 < nsteps) fetch_pages(t0 + 2 * kKeys);
    }

    if (active) {
      // S^T for the two 32-key blocks of this step; the two accumulation chains
      // are interleaved so each MFMA's predecessor in its chain has retired
      // K operands are read two 16-dimension slices ahead of their MFMAs; the
      // scheduling fences keep the compiler from moving each read next to its
      // use, which would leave one LDS read in flight per wave
      f32x16 sc[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) sc[kb][e] = 0.f;
      bf16x8 kop[3][2];
      auto read_k = [&](int c, bf16x8 (&dst)[2]) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
          dst[kb] = *reinterpret_cast<const bf16x8*>(&lds.ks[buf][32 * kb + col][16 * c + 8 * kg]);
      };
      read_k(0, kop[0]);
      read_k(1, kop[1]);
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        if (c + 2 < 8) read_k(c + 2, kop[(c + 2) % 3]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) sc[kb] = mfma_32x32x16(kop[c % 3][kb], qv[c], sc[kb]);
        __builtin_amdgcn_sched_barrier(0);
      }

      // Row max of the raw scores (the positive scale commutes with max and is
      // folded into the exponent below); the mask only where some column cannot
      // see all of the step's keys. Keys at or beyond t_hi are masked as well.
      float mt = kNegInf;
      if (t0 + kKeys > t_full || t0 < t_min) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int key = t0 + 32 * kb + 8 * (e >> 2) + 4 * kg + (e & 3);
            if (key > limit || key >= t_hi || key < t_min) sc[kb][e] = kNegInf;
          }
      }
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; e += 2) mt = fmaxf(mt, fmaxf(sc[kb][e], sc[kb][e + 1]));
      mt = max_l32(mt) * sl2;
      // lazy rescale: raise the running max only when the step's max exceeds it by 2^8
      const bool raise = mt > m_run + kLazy;
      if (__builtin_amdgcn_ballot_w64(raise) != 0) {
        // a column that does not raise keeps its state (alpha = 1, also when it
        // has seen no key yet and m_run - m_run would be -inf + inf)
        const float alpha = raise ? exp2_fast(m_run - mt) : 1.f;
        l_run *= alpha;
#pragma unroll
        for (int jd = 0; jd < 4; ++jd) o[jd] *= alpha;
        m_run = raise ? mt : m_run;
      }

      // p = exp2(scale * log2(e) * s - m), rounded to bf16 for the PV product; the
      // row sum keeps the fp32 values (four independent partial sums)
      bf16x8 pb[4];
      const float neg_m = m_run == kNegInf ? 0.f : -m_run;    // no key seen yet: p = exp2(-inf) = 0
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
    }
    if (j + 1 < nsteps) {
      stage(buf ^ 1, k_next, v_next);
      __syncthreads();
    }
  };

  Rows ka, va;
  fetch_pages(t_lo);
  fetch_rows(t_lo, ka, va);
  stage(0, ka, va);
  if (nsteps > 1) fetch_pages(t_lo + kKeys);
  __syncthreads();
  for (int j = 0; j < nsteps; ++j) step(j, ka, va);
}

// The same attention with a ping-pong schedule for eight waves (two per SIMD).
// Waves 0-3 and 4-7 form two groups that each hold one wave of every SIMD. A
// step is split into an MFMA phase (S^T of this step, then O^T += V^T P^T of
// the previous step) and a softmax phase, separated by workgroup barriers; the
// second group starts one barrier late, so on every SIMD one wave issues MFMAs
// while the other runs the softmax, and they swap at every barrier.
// K is staged one step ahead of V: in its MFMA phase of step j each wave writes
// its rows of K(j+1) and V(j), which are read only after the barrier that ends
// the second group's MFMA phase of step j; the buffers they overwrite (K(j-1),
// V(j-2)) were last read before the barrier that ended that group's MFMA phase
// of step j-1, and every write happens after it. Both groups pass the same
// number of barriers. The LDS buffers are still being read when the first
// group returns: a caller that reuses them must synchronise the workgroup.
// A wave that holds no query row runs the kCompute = false instance: it
// stages its rows and meets every barrier but issues no MFMA and no softmax
// work (the two instances keep the same barrier sequence).
//
// kUniformPages: in-page byte offsets fit 31 bits. A wave stages four
// consecutive key rows of each 32-row set of a step, and pages hold at least
// eight keys, so each set's page id is the same for the whole wave (kSetPages,
// for pages of fewer than 64 keys; otherwise one id serves the whole step and
// workgroup): it is read with a scalar load
// (through the constant address space; the block table is not written while
// the kernel runs), the page base is formed on the scalar unit, and a thread's
// in-page row offsets are fixed except for the clamp to the last key in the
// sequence's final step, which stays in the page of its set. Otherwise every
// thread looks up the page of each row it stages.
template <int kWaves, bool kUniformPages, bool kFp8 = false, bool kCompute = true, bool kSetPages = false,
          bool kNt = false>
__device__ __forceinline__ void tile_attend_pp(const PagedKV& kv, float scale, const int* bt_row, int g, int t_lo,
                                               int t_hi, int t_full, int limit, const bf16x8 (&qv)[8], TileLds& lds,
                                               f32x16 (&o)[4], float& m_run, float& l_run, int& bad) {
  static_assert(kWaves == 8, "the ping-pong schedule pairs two waves on each SIMD");
  constexpr int kAhead = 3;                       // LDS operand reads in flight ahead of the MFMAs
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int col = lane & 31, kg = lane >> 5;
  const bool late = (tid >> 6) >= 4;
  const float sl2 = scale * kLog2e;

  constexpr int kRowStep = kWaves * 4;
  constexpr int kStageRows = kKeys / kRowStep;
  typedef KvRaw<kFp8> Rows[kStageRows];      // raw rows in flight, converted when put into LDS
  const uint32_t bt_sj = (uint32_t)kv.bt_sj;
  const int ld_row = tid >> 4, ld_chunk = (tid & 15) * 8;
  const int pmask = kv.page_size - 1;
  auto put_k = [&](int buf, const Rows& r) {
#pragma unroll
    for (int i = 0; i < kStageRows; ++i)
      *reinterpret_cast<bf16x8*>(&lds.ks[buf][ld_row + kRowStep * i][ld_chunk]) = kv_to_bf16x8<kFp8>(r[i]);
  };
  auto put_v = [&](int buf, const Rows& r) {
#pragma unroll
    for (int i = 0; i < kStageRows; ++i)
      *reinterpret_cast<bf16x8*>(&lds.vs[buf][ld_row + kRowStep * i][ld_chunk]) = kv_to_bf16x8<kFp8>(r[i]);
  };
  const int tr_row = 4 * kg + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  if (t_lo >= t_hi) return;
  const int nsteps = (t_hi - t_lo + kKeys - 1) / kKeys;
  const int t_last = t_lo + (nsteps - 1) * kKeys;     // first key of the final step

  // ---- row fetch, per-row page lookups --------------------------------------
  typedef int Ids[kStageRows];
  constexpr int ES = kv_bytes<kFp8>();
  const char* kbase = (const char*)kv.k + ES * ((int64_t)g * kv.sh + ld_chunk);
  const char* vbase = (const char*)kv.v + ES * ((int64_t)g * kv.v_sh + ld_chunk);
  const uint32_t ksp = (uint32_t)kv.sp, kss = (uint32_t)kv.ss;
  const uint32_t vsp = (uint32_t)kv.v_sp, vss = (uint32_t)kv.v_ss;
  const bool page_holds_step = kv.page_size >= kKeys;
  // kNt: rows that no other work unit reads (decode through this routine)
  // are loaded non-temporally; units that share keys through the L2 keep
  // ordinary loads
  auto load_row = [&](const char* p) { return kNt ? load_kv_raw_nt<kFp8>(p) : load_kv_raw<kFp8>(p); };
  auto load_ids = [&](int t0, Ids& ids) {
#pragma unroll
    for (int i = 0; i < kStageRows; ++i) {
      int t = t0 + (page_holds_step ? 0 : ld_row + kRowStep * i);
      t = t < t_hi ? t : t_hi - 1;
      ids[i] = (page_holds_step && i) ? 0 : bt_row[__umul24((uint32_t)(t >> kv.log2_page), bt_sj)];
    }
  };
  auto fetch = [&](int t0, const Ids& ids, const char* base, uint32_t sp, uint32_t ss, Rows& r) {
#pragma unroll
    for (int i = 0; i < kStageRows; ++i) {
      int t = t0 + ld_row + kRowStep * i;
      t = t < t_hi ? t : t_hi - 1;
      int pg = ids[page_holds_step ? 0 : i];
      if ((unsigned)pg >= (unsigned)kv.num_pages) {
        bad = 1;
        pg = pg < 0 ? 0 : kv.num_pages - 1;
      }
      r[i] = load_row(base + ES * row_offset((uint32_t)pg, sp, t & pmask, ss));
    }
  };

  // ---- row fetch, one scalar page lookup per step ----------------------------
  typedef __attribute__((address_space(4))) const int ConstInt;
  const ConstInt* bt_c = (const ConstInt*)bt_row;
  const char* kbase_u = (const char*)kv.k + ES * ((int64_t)g * kv.sh);
  const char* vbase_u = (const char*)kv.v + ES * ((int64_t)g * kv.v_sh);
  // byte offsets of this thread's rows in their pages (for a page of at least
  // a step, relative to the step's first key)
  uint32_t koff[kStageRows], voff[kStageRows];
#pragma unroll
  for (int i = 0; i < kStageRows; ++i) {
    koff[i] = ES * (ld_chunk + ((uint32_t)(ld_row + kRowStep * i) & (uint32_t)pmask) * kss);
    voff[i] = ES * (ld_chunk + ((uint32_t)(ld_row + kRowStep * i) & (uint32_t)pmask) * vss);
  }
  const int wave_row = __builtin_amdgcn_readfirstlane(4 * (tid >> 6));   // the wave's first row of a set
  typedef int Pids[kStageRows];
  // page ids of the wave's row sets of the step starting at t0 (one page for
  // the whole step unless kSetPages)
  auto page_ids = [&](int t0, Pids& p) {
    const int tc = t0 < t_last ? t0 : t_last;
#pragma unroll
    for (int i = 0; i < kStageRows; ++i) {
      if (!kSetPages && i > 0) {
        p[i] = p[0];
        continue;
      }
      int t = kSetPages ? tc + wave_row + kRowStep * i : tc;
      t = t < t_hi ? t : t_hi - 1;
      int pg = bt_c[__umul24((uint32_t)(t >> kv.log2_page), bt_sj)];
      if ((unsigned)pg >= (unsigned)kv.num_pages) {
        bad = 1;
        pg = pg < 0 ? 0 : kv.num_pages - 1;
      }
      p[i] = pg;
    }
  };
  auto fetch_u = [&](int t0, const Pids& p, const char* base, int64_t sp, uint32_t ss,
                     const uint32_t (&off)[kStageRows], Rows& r) {
    const int tc = t0 < t_last ? t0 : t_last;
    const uint32_t step_off = ES * ((uint32_t)(tc & pmask) * ss);   // zero when a page holds at most a step
    if (tc + kKeys <= t_hi) {
#pragma unroll
      for (int i = 0; i < kStageRows; ++i)
        r[i] = load_row(base + ES * ((int64_t)p[i] * sp) + step_off + off[i]);
    } else {
      const int last = t_hi - 1 - tc;
#pragma unroll
      for (int i = 0; i < kStageRows; ++i) {
        const int rr = min(ld_row + kRowStep * i, last);
        r[i] = load_row(base + ES * ((int64_t)p[i] * sp) +
                                 ES * (ld_chunk + ((uint32_t)(tc + rr) & (uint32_t)pmask) * ss));
      }
    }
  };

  f32x16 sc[2];
  bf16x8 pb[4];

  // MFMA phase: operands are read kAhead MFMAs ahead; the fences keep each
  // read ahead of the MFMAs that do not need it
  auto mfma_phase = [&](auto pv_tag, auto s_tag, int vbuf, int kbuf) {
    if constexpr (!kCompute) return;
    constexpr bool kPV = decltype(pv_tag)::value, kS = decltype(s_tag)::value;
    constexpr int i0 = kPV ? 0 : 16, i1 = kS ? 32 : 16;
    if constexpr (kS) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) sc[kb][e] = 0.f;
    }
    auto read = [&](int i) -> bf16x8 {
      if (i < 16) {
        const u16* vp = &lds.vs[vbuf][16 * (i >> 2) + tr_row][32 * (i & 3) + tr_col];
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)vp);
        const i16x4 up = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vp + 8 * kVStride));
        return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, up, 0, 1, 2, 3, 4, 5, 6, 7));
      }
      const int c = (i - 16) >> 1, kb = (i - 16) & 1;
      return *reinterpret_cast<const bf16x8*>(&lds.ks[kbuf][32 * kb + col][16 * c + 8 * kg]);
    };
    bf16x8 ring[kAhead + 1];
    // the S^T MFMAs of this step go first, then the PV MFMAs of the previous
    // one (independent chains; measured 2% faster with FP8 pages, the same
    // with bf16)
    auto at = [&](int ii) { return (kPV && kS) ? (ii < 16 ? ii + 16 : ii - 16) : i0 + ii; };
    constexpr int n = i1 - i0;
#pragma unroll
    for (int ii = 0; ii < kAhead; ++ii) ring[ii % (kAhead + 1)] = read(at(ii));
#pragma unroll
    for (int ii = 0; ii < n; ++ii) {
      const int i = at(ii);
      if (ii + kAhead < n) ring[(ii + kAhead) % (kAhead + 1)] = read(at(ii + kAhead));
      __builtin_amdgcn_sched_barrier(0);
      if (i < 16)
        o[i & 3] = mfma_32x32x16(ring[ii % (kAhead + 1)], pb[i >> 2], o[i & 3]);
      else
        sc[(i - 16) & 1] = mfma_32x32x16(ring[ii % (kAhead + 1)], qv[(i - 16) >> 1], sc[(i - 16) & 1]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // softmax phase of the step starting at key t0: S^T -> P^T (bf16), running max and sum
  auto softmax_phase = [&](int t0) {
    if constexpr (!kCompute) return;
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
    mt = max_l32(mt) * sl2;
    const bool raise = mt > m_run + kLazy;
    if (__builtin_amdgcn_ballot_w64(raise) != 0) {
      const float m_new = raise ? mt : m_run;
      const float alpha = exp2_fast(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int jd = 0; jd < 4; ++jd) o[jd] *= alpha;
      m_run = m_new;
    }
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
  };

  // Row fetches past the final step read that step again: the loads stay
  // unconditional, so no register copy has to wait for them.
  // Invariant at the top of step j: kr = rows of K(j+1), vr = rows of V(j);
  // ids (or scalar page ids) of steps j+1 and j+2 are at hand.
  Rows kr, vr;
  Ids id_k, id_v;
  Pids pid_1 = {}, pid_2 = {};
  if constexpr (kUniformPages) {
    Pids p0;
    page_ids(t_lo, p0);
    fetch_u(t_lo, p0, kbase_u, kv.sp, kss, koff, kr);
    fetch_u(t_lo, p0, vbase_u, kv.v_sp, vss, voff, vr);
    put_k(0, kr);
    page_ids(t_lo + kKeys, pid_1);
    fetch_u(t_lo + kKeys, pid_1, kbase_u, kv.sp, kss, koff, kr);
    page_ids(t_lo + 2 * kKeys, pid_2);
  } else {
    load_ids(t_lo, id_k);
    fetch(t_lo, id_k, kbase, ksp, kss, kr);
    fetch(t_lo, id_k, vbase, vsp, vss, vr);
    put_k(0, kr);
    load_ids(t_lo + kKeys, id_v);
    fetch(t_lo + kKeys, id_v, kbase, ksp, kss, kr);
    load_ids(t_lo + 2 * kKeys, id_k);
  }
  __syncthreads();
  if (late) __syncthreads();

  // LDS writes of the rows at hand (MFMA phase of step j)
  auto stage = [&](int j) {
    if (j + 1 < nsteps) put_k((j + 1) & 1, kr);
    put_v(j & 1, vr);
  };
  // loads of the rows of V(j+1) and K(j+2) (softmax phase of step j)
  auto fetch_next = [&](int j) {
    const int t0 = t_lo + j * kKeys;
    if constexpr (kUniformPages) {
      fetch_u(t0 + kKeys, pid_1, vbase_u, kv.v_sp, vss, voff, vr);
      fetch_u(t0 + 2 * kKeys, pid_2, kbase_u, kv.sp, kss, koff, kr);
#pragma unroll
      for (int i = 0; i < kStageRows; ++i) pid_1[i] = pid_2[i];
    } else {
      fetch(t0 + kKeys, id_v, vbase, vsp, vss, vr);
      fetch(t0 + 2 * kKeys, id_k, kbase, ksp, kss, kr);
#pragma unroll
      for (int i = 0; i < kStageRows; ++i) id_v[i] = id_k[i];
      load_ids(t0 + 3 * kKeys, id_k);
    }
  };
  // the scalar page id of step j+3 is read at the end of step j's softmax
  // phase, so the barrier's wait covers its latency
  auto next_page = [&](int j) {
    if constexpr (kUniformPages) page_ids(t_lo + (j + 3) * kKeys, pid_2);
  };
  const std::true_type yes{};
  const std::false_type no{};
  // The LDS writes of a step follow its MFMAs (the MFMAs start as soon as the
  // barrier opens); the global loads of the next rows open the softmax phase,
  // whose VALU work leaves the vector memory path idle, and have the rest of
  // that phase and the next MFMA phase to arrive (loads issued in the MFMA
  // phase, after its MFMAs, measured 4% slower with bf16 pages).
  mfma_phase(no, yes, 0, 0);
  stage(0);
  __syncthreads();
  fetch_next(0);
  softmax_phase(t_lo);
  next_page(0);
  __syncthreads();
  for (int j = 1; j < nsteps; ++j) {
    mfma_phase(yes, yes, (j - 1) & 1, j & 1);
    stage(j);
    __syncthreads();
    fetch_next(j);
    softmax_phase(t_lo + j * kKeys);
    next_page(j);
    __syncthreads();
  }
  mfma_phase(yes, no, (nsteps - 1) & 1, 0);
  if (!late) __syncthreads();
}

// ---- 128-key steps, rows loaded straight into LDS ---------------------------
// The ping-pong schedule above with steps of 128 keys (one MFMA phase holds the
// 32 S^T MFMAs of a step and the 32 PV MFMAs of the one before, so barriers and
// phase switches per flop are halved) and bf16 rows moved from global memory
// into LDS by the load itself (global_load_lds_dwordx4): no row passes through
// registers and no wave writes LDS, which leaves room for the doubled score and
// probability tiles.
//
// LDS layout of a step's K (and V): 32 blocks of four 256-byte rows, padded to
// kDlKPitch (kDlVPitch) bytes. Row r of the step sits in block r % 16 + 16 (r / 64)
// at slot (r / 16) % 4, so
//  * one load instruction fills one block (lane l -> slot l / 16, 16-byte chunk
//    l % 16), and a block's rows lie in one 64-key half of the step, i.e. in
//    one page: the wave's address is a scalar page base plus a lane offset;
//  * the K operand read (32 consecutive rows, one 16-byte chunk each) and the
//    transposed V read are a per-lane base plus compile-time offsets;
//  * 16 consecutive K rows fall in 16 blocks whose padding puts them on
//    distinct 4-bank groups, and the four rows each 32-lane group of the
//    transposed V read touches sit 16 banks apart (no bank conflicts).
// Each of the two K and two V buffers is its own LDS array, and the step loop
// is unrolled by two, so every operand read names its buffer and adds a
// compile-time offset.
constexpr int kDlKeys = 128;
constexpr int kDlKPitch = 1024 + 16;
constexpr int kDlVPitch = 1024 + 64;
constexpr int kDlKBytes = 32 * kDlKPitch;
constexpr int kDlVBytes = 32 * kDlVPitch;

// Attention of this lane's query column over keys [0, t_hi) of KV head g, as
// tile_attend_pp (same arguments and results) for bf16 pages of at least 64
// keys whose in-page offsets fit 31 bits. Its rounding differs from the
// 64-key routines (the running max and the sums advance per 128 keys).
// Schedule: the rows of K(j+1) and V(j) are requested after the barrier that
// ends the second group's MFMA phase of step j-1 (the last reads of the
// buffers they fill): by the first group between the first eight MFMAs of its
// phase j, by the second group at the start of its softmax phase j-1. Each
// wave waits for its own loads before the barrier after which they are first
// read, one MFMA phase and one softmax phase later.
template <bool kCompute, bool kNt>
__device__ __forceinline__ void tile_attend_dl(const PagedKV& kv, float scale, const int* bt_row, int g, int t_hi,
                                               int t_full, int limit, const bf16x8 (&qv)[8], char* kl0, char* kl1,
                                               char* vl0, char* vl1, f32x16 (&o)[4], float& m_run, float& l_run,
                                               int& bad) {
  constexpr int kAhead = 3;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int col = lane & 31, kg = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool late = wave >= 4;
  const float sl2 = scale * kLog2e;
  if (t_hi <= 0) return;
  const int nsteps = (t_hi + kDlKeys - 1) / kDlKeys;
  const int pmask = kv.page_size - 1;

  // loads: wave w fills blocks w + 8 i (i = 0..3) of K and of V; block b holds
  // rows b % 16 + 16 s (s = lane / 16) of half b / 16, chunk lane % 16
  typedef __attribute__((address_space(4))) const int ConstInt;
  const ConstInt* bt_c = (const ConstInt*)bt_row;
  const char* kbase = (const char*)kv.k + 2 * ((int64_t)g * kv.sh);
  const char* vbase = (const char*)kv.v + 2 * ((int64_t)g * kv.v_sh);
  const uint32_t kss = (uint32_t)kv.ss, vss = (uint32_t)kv.v_ss;
  // row of this lane's slot within its half of the step, for blocks w and
  // w + 16 (blocks w + 8 and w + 24 hold the rows 8 further)
  const int lrow = wave + 16 * (lane >> 4);
  const uint32_t lchunk = 16u * (uint32_t)(lane & 15);
  // page ids of the two halves of step j (scalar loads; a half past the last
  // key takes the first half's page)
  auto page_pair = [&](int j, int (&p)[2]) {
    const int t0 = j * kDlKeys;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int t = (t0 + 64 * h < t_hi) ? t0 + 64 * h : t0;
      int pg = bt_c[__umul24((uint32_t)(t >> kv.log2_page), (uint32_t)kv.bt_sj)];
      if ((unsigned)pg >= (unsigned)kv.num_pages) {
        bad = 1;
        pg = pg < 0 ? 0 : kv.num_pages - 1;
      }
      p[h] = pg;
    }
  };
  // block w + 8 i of step j's rows into one buffer; rows past the last key
  // load that key again
  auto dma_block = [&](int j, const int (&p)[2], const char* base, int64_t sp, uint32_t ss, char* dst, int pitch,
                       int i) {
    const int t0 = j * kDlKeys;
    const int h = i >> 1;
    const int hh = (t0 + 64 * h < t_hi) ? h : 0;      // the half whose page this block reads
    const int last = min(63, t_hi - 1 - t0 - 64 * hh);
    const int row = min(lrow + 8 * (i & 1), last);
    const char* sbase = base + 2 * ((int64_t)p[h] * sp + (int64_t)((t0 + 64 * hh) & pmask) * ss);
    const uint32_t voff = 2u * (uint32_t)row * ss + lchunk;
    const uint32_t lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)(dst + (wave + 8 * i) * pitch);
    // Issued as assembly: the compiler would otherwise wait for every row load
    // in flight before LDS reads it cannot tell apart from the loads'
    // destinations (the transposed V reads), stalling the MFMA phase. The
    // rows' readers are ordered by wait_loads and the barriers instead; a wait
    // the compiler counts for its own loads can only be lengthened by these
    // (loads complete in order).
    // (m0 holds the LDS address: an input operand, so the compiler sets it)
    if constexpr (kNt)
      asm volatile("global_load_lds_dwordx4 %0, %1 nt" ::"v"(voff), "s"(sbase), "{m0}"(lds) : "memory");
    else
      asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "{m0}"(lds) : "memory");
  };
  auto dma = [&](int j, const int (&p)[2], const char* base, int64_t sp, uint32_t ss, char* dst, int pitch) {
#pragma unroll
    for (int i = 0; i < 4; ++i) dma_block(j, p, base, sp, ss, dst, pitch, i);
  };
  auto wait_loads = [&]() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); };
  // A workgroup barrier without the memory fence of __syncthreads: the row
  // loads are ordered explicitly instead. A wave waits for its own row loads
  // (wait_loads) before the barrier after which they are read, and every LDS
  // operand read of a phase is consumed by that phase's MFMAs before the
  // barrier that ends it. The empty asm statements keep the compiler from
  // moving LDS accesses across the barrier.
  auto barrier = [&]() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  // operand reads: per-lane bases (see the layout above)
  const int kread = (col & 15) * kDlKPitch + (col >> 4) * 256 + 16 * kg;
  const int tr_row = 4 * kg + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const int vread = tr_row * kDlVPitch + 2 * tr_col;

  f32x16 sc[4];
  bf16x8 pb[8];

  // hook(ii) runs after the ii-th MFMA of the phase, ii < 8 (the first
  // group's row loads, spread between MFMAs so their address arithmetic
  // issues while the MFMAs run)
  auto mfma_phase = [&](auto pv_tag, auto s_tag, const char* vbuf, const char* kbuf, auto&& hook) {
    if constexpr (!kCompute) {
#pragma unroll
      for (int ii = 0; ii < 8; ++ii) hook(ii);
      return;
    }
    constexpr bool kPV = decltype(pv_tag)::value, kS = decltype(s_tag)::value;
    constexpr int i0 = kPV ? 0 : 32, i1 = kS ? 64 : 32;
    const f32x16 zero = {};
    auto read = [&](int i) -> bf16x8 {
      if (i < 32) {
        const int h = i >> 2, jd = i & 3;
        const char* vp = vbuf + vread + 16 * (h >> 2) * kDlVPitch + 256 * (h & 3) + 64 * jd;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)vp);
        const i16x4 up = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vp + 8 * kDlVPitch));
        return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, up, 0, 1, 2, 3, 4, 5, 6, 7));
      }
      const int c = (i - 32) >> 2, kb = (i - 32) & 3;
      return *reinterpret_cast<const bf16x8*>(kbuf + kread + 16 * (kb >> 1) * kDlKPitch + 512 * (kb & 1) + 32 * c);
    };
    // the PV MFMAs of the previous step go first: P^T is dead before the
    // scores of this step are born (the first MFMA of each score chain takes a
    // zero accumulator), which keeps the phase within the register file
    bf16x8 ring[kAhead + 1];
    auto at = [&](int ii) { return i0 + ii; };
    constexpr int n = i1 - i0;
#pragma unroll
    for (int ii = 0; ii < kAhead; ++ii) ring[ii % (kAhead + 1)] = read(at(ii));
#pragma unroll
    for (int ii = 0; ii < n; ++ii) {
      const int i = at(ii);
      if (ii + kAhead < n) ring[(ii + kAhead) % (kAhead + 1)] = read(at(ii + kAhead));
      __builtin_amdgcn_sched_barrier(0);
      if (i < 32)
        o[i & 3] = mfma_32x32x16(ring[ii % (kAhead + 1)], pb[i >> 2], o[i & 3]);
      else
        sc[(i - 32) & 3] =
            mfma_32x32x16(ring[ii % (kAhead + 1)], qv[(i - 32) >> 2], i < 36 ? zero : sc[(i - 32) & 3]);
      __builtin_amdgcn_sched_barrier(0);
      if (ii < 8) {
        hook(ii);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };

  auto softmax_phase = [&](int t0) {
    if constexpr (!kCompute) return;
    float mt = kNegInf;
    if (t0 + kDlKeys > t_full) {
      // a key is visible when it is at most this lane's last visible key; the
      // fences keep each compare next to its select (hoisted, the 64 compare
      // masks would not fit the scalar registers)
      const int d = min(limit, t_hi - 1) - t0 - 4 * kg;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          if (32 * kb + 8 * (e >> 2) + (e & 3) > d) sc[kb][e] = kNegInf;
          if ((e & 3) == 3) __builtin_amdgcn_sched_barrier(0);
        }
    }
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 16; e += 2) mt = fmaxf(mt, fmaxf(sc[kb][e], sc[kb][e + 1]));
    mt = max_l32(mt) * sl2;
    const bool raise = mt > m_run + kLazy;
    if (__builtin_amdgcn_ballot_w64(raise) != 0) {
      const float m_new = raise ? mt : m_run;
      const float alpha = exp2_fast(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int jd = 0; jd < 4; ++jd) o[jd] *= alpha;
      m_run = m_new;
    }
    const float neg_m = -m_run;
    float ps[4] = {0.f, 0.f, 0.f, 0.f};
    // one 16-key group at a time (fenced), so the scores die as their
    // probabilities are packed
#pragma unroll
    for (int h = 0; h < 8; ++h) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float p = exp2_fast(fmaf(sc[h >> 1][8 * (h & 1) + e], sl2, neg_m));
        ps[e & 3] += p;
        pb[h][e] = (__bf16)p;
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    l_run += (ps[0] + ps[1]) + (ps[2] + ps[3]);
    // P^T and the row sum are formed here, in the softmax phase: without
    // these pins the compiler sinks the exponentials (or the sum's additions)
    // past the barrier into the next MFMA phase, where their 64 fp32 values
    // would sit beside the new scores
#pragma unroll
    for (int h = 0; h < 8; ++h) asm volatile("" : "+v"(pb[h]));
    asm volatile("" : "+v"(l_run));
  };

  const std::true_type yes{};
  const std::false_type no{};
  // page ids of steps j (pv, for V) and j+1 (pk, for K) at each issue; the ids
  // of the step after are read at the end of a softmax phase, where the
  // barrier's wait covers the scalar load (an outstanding scalar load would
  // make the MFMA phase's LDS reads wait for it too)
  int pv[2], pk[2];
  int pid_next = 2;                                  // step whose ids the next read fetches
  page_pair(0, pv);
  dma(0, pv, kbase, kv.sp, kss, kl0, kDlKPitch);
  if (nsteps > 1) page_pair(1, pk);
  wait_loads();
  barrier();
  auto next_pages = [&]() {
    if (pid_next < nsteps) page_pair(pid_next, pk);
  };
  // the two groups run the same steps with their loads, waits and barriers
  // placed as described above; kLate is the second group
  auto run = [&](auto late_tag) {
    constexpr bool kLate = decltype(late_tag)::value;
    // loads of K(j+1) and V(j), block by block (ii = 0..7); buffers by the
    // parity of j
    auto issue_block = [&](int j, auto par, int ii) {
      constexpr int P = decltype(par)::value;
      if (ii < 4) {
        if (j + 1 < nsteps) dma_block(j + 1, pk, kbase, kv.sp, kss, P ? kl0 : kl1, kDlKPitch, ii);
      } else {
        dma_block(j, pv, vbase, kv.v_sp, vss, P ? vl1 : vl0, kDlVPitch, ii - 4);
      }
    };
    auto issue_done = [&](int j) {
      pv[0] = pk[0];
      pv[1] = pk[1];
      pid_next = j + 2;
    };
    auto issue = [&](int j, auto par) {
#pragma unroll
      for (int ii = 0; ii < 8; ++ii) issue_block(j, par, ii);
      issue_done(j);
    };
    const auto none = [](int) {};
    if constexpr (kLate) {
      issue(0, std::integral_constant<int, 0>{});
      next_pages();
      barrier();
    }
    // step j: K(j) in buffer j % 2, V(j-1) in buffer (j-1) % 2
    auto body = [&](int j, auto par, auto first) {
      constexpr int P = decltype(par)::value;
      char* kcur = P ? kl1 : kl0;
      char* vprev = P ? vl0 : vl1;
      auto hook = [&](int ii) {
        if constexpr (!kLate) issue_block(j, par, ii);
      };
      if constexpr (decltype(first)::value)
        mfma_phase(no, yes, vprev, kcur, hook);
      else
        mfma_phase(yes, yes, vprev, kcur, hook);
      if constexpr (!kLate) issue_done(j);
      if constexpr (kLate) wait_loads();
      barrier();
      if constexpr (kLate) {
        if (j + 1 < nsteps) issue(j + 1, std::integral_constant<int, 1 - P>{});
      }
      softmax_phase(j * kDlKeys);
      next_pages();
      if constexpr (!kLate) wait_loads();
      barrier();
    };
    const std::integral_constant<int, 0> even{};
    const std::integral_constant<int, 1> odd{};
    body(0, even, yes);
    int j = 1;
    for (; j + 1 < nsteps; j += 2) {
      body(j, odd, no);
      body(j + 1, even, no);
    }
    if (j < nsteps) body(j, odd, no);
    // PV of the final step: V(n-1) in buffer (n-1) % 2
    if ((nsteps - 1) & 1)
      mfma_phase(yes, no, vl1, kl0, none);
    else
      mfma_phase(yes, no, vl0, kl0, none);
    if constexpr (!kLate) barrier();
  };
  if (late)
    run(std::true_type{});
  else
    run(std::false_type{});
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
