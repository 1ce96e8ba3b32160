// Multi-row attention tile on MFMA 32x32x16, shared by the extend kernel
// (rows = chunk tokens x query heads; tile_attend_pp), the group-prefix kernel
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
