// Batched paged decode: device planner, split-KV attention, trajectory-group
// prefix pass, log-sum-exp combine.
//
// The planner runs on the device from the lengths and the block table, so the
// host never waits for data. It
//   * picks the split size C (a multiple of 64 keys) so that the number of
//     work items stays near a target;
//   * finds trajectory groups: sequences whose block tables start with the
//     same page id form a group with its lowest-indexed member as leader, and
//     share the leading full pages they have in common with the leader (the
//     minimum over the group). The G attempts at one prompt are scheduled
//     together and reuse the prompt's cached prefix (paper, sections "The
//     Miles RL Loop" and "Fast Agentic Rollout with SGLang"), so their block
//     tables point at the same physical pages;
//   * emits shared items (a split of a group's shared keys, computed once for
//     up to 128 query rows of every member) and private items (a split of the
//     rest of one sequence).
// A sequence whose whole context is one private item writes its output
// directly; otherwise every item writes an (o, lse) partial into a slot of the
// sequence and the combine kernel merges them (flash-decoding; the merge is the
// log-sum-exp identity). A multi-token call may queue an extend pass behind
// these (route_extend): when the planner finds no shared prefix page it hands
// every row to that pass and gives the split passes no work.
#include <type_traits>

#include "kernels.hpp"
#include "tile_attn.hpp"

namespace rl {

namespace {

constexpr int kMinSplit = 256;     // smallest automatic split of shared keys
constexpr int kMinWorkerKeys = 64; // fewest keys per private-pass worker (automatic)
constexpr int kTile = 32;          // keys per inner iteration of the private kernel
constexpr int kGroupMax = 1024;    // batches up to this size get trajectory-group detection
constexpr int kIntMax = 0x7fffffff;
constexpr int kHashBits = 11;     // planner hash table: 2048 slots for up to kGroupMax (parent, page) keys
constexpr int kCmpUnroll = 8;     // block-table entries a lane compares per round
static_assert(kPrefixLevels * 16 <= 62, "per-level sub-group counts are packed in 16-bit fields");

__device__ __forceinline__ int clamp_len(int L, int max_tokens, int* bad) {
  if (L < 0 || L > max_tokens) {
    *bad = 1;
    return L < 0 ? 0 : max_tokens;
  }
  return L;
}

__device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Exclusive scan of v over the workgroup, with the totals of v and of w, in
// one pair of barriers (wave_tot: 32 slots).
__device__ __forceinline__ long long block_scan_sum64(long long v, long long w, long long* tot_v, long long* tot_w,
                                                      long long* wave_tot) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const long long x = wave_inclusive_scan64(v);
  w = wave_inclusive_scan64(w);
  if (lane == 63) {
    wave_tot[wave] = x;
    wave_tot[16 + wave] = w;
  }
  __syncthreads();
  long long before = 0, all = 0, all_w = 0;
  const int nw = blockDim.x >> 6;
  for (int i = 0; i < nw; ++i) {
    const long long t = wave_tot[i];
    if (i < wave) before += t;
    all += t;
    all_w += wave_tot[16 + i];
  }
  __syncthreads();
  *tot_v = all;
  *tot_w = all_w;
  return before + x - v;
}

// Key of the planner's hash table: (parent node leader + 1, page id); ~0 = empty.
__device__ __forceinline__ unsigned long long node_key(int parent, int page) {
  return ((unsigned long long)(uint32_t)(parent + 1) << 32) | (uint32_t)page;
}
__device__ __forceinline__ int key_hash(unsigned long long key) {
  return (int)((((uint32_t)key ^ (uint32_t)(key >> 32) * 0x9e3779b1u) * 2654435761u) >> (32 - kHashBits));
}

__global__ __launch_bounds__(1024) void plan_decode_kernel(DecodeArgs a) {
  // per sequence (small batches): length; per level: the leader of its shared
  // node (-1: none) and the end of its shared keys after that level; per node
  // (indexed by its leader): members and first sub-group
  __shared__ int sL[kGroupMax];
  __shared__ int sLead[kPrefixLevels][kGroupMax], sEnd[kPrefixLevels][kGroupMax];
  __shared__ int sNum[kPrefixLevels][kGroupMax], sSg[kPrefixLevels][kGroupMax];
  __shared__ int sKmin[kGroupMax], sCnt[kGroupMax];
  __shared__ unsigned long long hKey[1 << kHashBits];
  __shared__ int hMin[1 << kHashBits];
  __shared__ int wave_tot[16];
  __shared__ long long wsum[32];
  // small batches: the private prefix sums, and per sub-group (first key,
  // first slot offset, end key, splits), kept here for the later phases
  __shared__ long long sPref[kGroupMax + 1];
  __shared__ int4 sSgInfo[kPrefixLevels * kGroupMax];
  const int tid = threadIdx.x, nthr = blockDim.x, lane = tid & 63, wave = tid >> 6, nwaves = nthr >> 6;
  const int lg = a.kv.log2_page, P = a.kv.page_size;
  const int max_tokens = a.kv.max_pages * P;
  // small batches (one sequence per thread) keep per-sequence state in LDS
  // and get trajectory-group detection
  const bool small = a.B <= kGroupMax;
  // grouping: the batch is searched for shared prefix pages; it stays on only
  // if a node is found
  bool grouping = a.group_cap >= 2 && small;
  const uint32_t bt_sj = (uint32_t)a.kv.bt_sj;
  int bad = 0, cap_bad = 0;

  // the first page id of every sequence (the key of level 0 of the search
  // below) is read with the lengths, so the two loads share one wait
  const int page0 = grouping && tid < a.B && a.kv.max_pages > 0 ? a.kv.bt[(int64_t)tid * a.kv.bt_sb] : 0;

  // lengths and their sum
  long long sum = 0;
  for (int b = tid; b < a.B; b += nthr) {
    const int L = clamp_len(a.lens[b * a.lens_s], max_tokens, &bad);
    sum += L;
    if (small) sL[b] = L;
  }
  sum = wave_inclusive_scan64(sum);
  if (lane == 63) wsum[wave] = sum;
  __syncthreads();
  long long total = 0;
  for (int w = 0; w < nwaves; ++w) total += wsum[w];

  int C = a.forced_split;
  if (C <= 0) {
    long long per = (total + a.target_items - 1) / a.target_items;
    per = (per + 63) & ~63LL;
    C = (int)(per < kMinSplit ? kMinSplit : per);
  }

  // Shared prefix pages as a tree of nodes, level by level. At level 0 the
  // sequences whose block tables start with the same page id form a node (the
  // trajectory group: G attempts at one prompt share its cached prefix); at
  // level v > 0 the members of a level v-1 node are split by the page id that
  // follows the node's shared range (sessions that branch after a common turn).
  // A node's leader is its lowest-indexed member; the node shares the leading
  // full pages that every member has in common with the leader (from the
  // parent's end on), and is kept if it has another member and at least one
  // such page. Its keys [parent end, node end) are then read once for all its
  // members by the group-prefix pass.
  if (grouping) {
    // lanes per member in the comparisons: the most (up to a wave) that still
    // cover the whole batch with the workgroup's threads
    int lpm_log = 6;
    while (lpm_log > 0 && (a.B << lpm_log) > nthr) --lpm_log;
    const int lpm = 1 << lpm_log;
    for (int v = 0; v < kPrefixLevels; ++v) {
      for (int i = tid; i < (1 << kHashBits); i += nthr) {
        hKey[i] = ~0ull;
        hMin[i] = kIntMax;
      }
      for (int i = tid; i < a.B; i += nthr) {
        sKmin[i] = kIntMax;
        sCnt[i] = 0;
      }
      __syncthreads();
      const int b = tid;
      const int parent = (b < a.B && v > 0) ? sLead[v - 1][b] : -1;
      const int start = (b < a.B && v > 0) ? sEnd[v - 1][b] : 0;
      // takes part: in a node at the previous level (or at level 0), with a
      // full page at the position that follows the shared range
      const bool part = b < a.B && (v == 0 || parent >= 0) && (sL[b] >> lg) > (start >> lg);
      const int page = !part ? 0
                       : v == 0 ? page0
                                : a.kv.bt[(int64_t)b * a.kv.bt_sb + (int64_t)__umul24((uint32_t)(start >> lg), bt_sj)];
      const unsigned long long key = node_key(parent, page);
      if (part) {
        int h = key_hash(key);
        for (;;) {
          const unsigned long long prev = atomicCAS(&hKey[h], ~0ull, key);
          if (prev == ~0ull || prev == key) {
            atomicMin(&hMin[h], b);
            break;
          }
          h = (h + 1) & ((1 << kHashBits) - 1);
        }
      }
      __syncthreads();
      if (b < a.B) {
        int lead = -1;
        if (part) {
          int h = key_hash(key);
          while (hKey[h] != key) h = (h + 1) & ((1 << kHashBits) - 1);
          lead = hMin[h];
        }
        sLead[v][b] = lead;
      }
      __syncthreads();
      // leading full pages each member shares with its leader from the parent's
      // end on; the node shares the minimum. All members are compared at once:
      // an aligned group of lpm lanes per member, each lane checking
      // kCmpUnroll entries per round (lane s: entries c + s + lpm u), so a
      // round covers lpm * kCmpUnroll pages of every member and costs one
      // round trip to the block table
      for (int m0 = 0; m0 < a.B; m0 += nthr >> lpm_log) {
        const int m = m0 + (tid >> lpm_log), sub = tid & (lpm - 1);
        const int lead = m < a.B ? sLead[v][m] : -1;
        const bool member = lead >= 0 && lead != m;
        const int p0 = member ? (v == 0 ? 0 : sEnd[v - 1][m]) >> lg : 0;
        // both rows hold full pages at p0 (they took part), so lim > p0; the
        // test keeps every index read below in [p0, lim) regardless
        const int lim = member ? min(sL[m], sL[lead]) >> lg : 0;
        bool active = member && lim > p0;
        const int* rb = a.kv.bt + (int64_t)(member ? m : 0) * a.kv.bt_sb;
        const int* rl = a.kv.bt + (int64_t)(member ? lead : 0) * a.kv.bt_sb;
        int k = lim;
        for (int c = p0; __builtin_amdgcn_ballot_w64(active) != 0; c += lpm * kCmpUnroll) {
          int found = kIntMax;
          if (active) {
            int x[kCmpUnroll], y[kCmpUnroll];
#pragma unroll
            for (int u = 0; u < kCmpUnroll; ++u) {
              const int kk = min(c + sub + lpm * u, lim - 1);
              x[u] = rb[__umul24((uint32_t)kk, bt_sj)];
              y[u] = rl[__umul24((uint32_t)kk, bt_sj)];
            }
#pragma unroll
            for (int u = 0; u < kCmpUnroll; ++u) {
              const int kk = c + sub + lpm * u;
              if (kk < lim && x[u] != y[u]) found = min(found, kk);
            }
          }
          for (int o = 1; o < lpm; o <<= 1) found = min(found, __shfl_xor(found, o, 64));
          if (active) {
            if (found != kIntMax) {
              k = found;
              active = false;
            } else if (c + lpm * kCmpUnroll >= lim) {
              active = false;
            }
          }
        }
        if (member && sub == 0) {
          atomicMin(&sKmin[lead], k);
          atomicAdd(&sCnt[lead], 1);
        }
      }
      __syncthreads();
      bool kept = false;
      if (b < a.B) {
        const int lead = sLead[v][b];
        kept = lead >= 0 && sCnt[lead] >= 1 && sKmin[lead] > (start >> lg);
        sLead[v][b] = kept ? lead : -1;
        sEnd[v][b] = kept ? sKmin[lead] * P : start;
        sNum[v][b] = (kept && lead == b) ? sCnt[b] + 1 : 0;
      }
      // no node at this level: none below it either (and with none at the
      // first level the batch has no shared pages at all)
      if (!__syncthreads_or(kept)) {
        if (v == 0) {
          grouping = false;
          break;
        }
        for (int w = v + 1; w < kPrefixLevels; ++w)
          if (b < a.B) {
            sLead[w][b] = -1;
            sEnd[w][b] = sEnd[v][b];
            sNum[w][b] = 0;
          }
        __syncthreads();
        break;
      }
    }
  }
  // keys [*t0, *t1) of sequence b shared at level v, if b is in a node there
  auto level_range = [&](int v, int b, int* t0, int* t1) -> bool {
    *t0 = v == 0 ? 0 : sEnd[v - 1][b];
    *t1 = sEnd[v][b];
    return sLead[v][b] >= 0;
  };
  // all shared keys of sequence b: its private keys start there
  auto shared_keys = [&](int b) -> int { return grouping ? sEnd[kPrefixLevels - 1][b] : 0; };
  const int cap = a.group_cap;

  // sub-groups of at most `cap` members: bases by exclusive scans over the
  // nodes' leaders, level after level
  int n_sg = 0;
  if (grouping) {
    // one scan for all levels: the per-level counts of a leader are packed in
    // 16-bit fields (a level's total is at most B <= kGroupMax, so no field
    // carries into the next), beside the sum of shared keys times sub-groups
    const int b = tid;
    long long packed = 0, keys = 0;
    for (int v = 0; v < kPrefixLevels; ++v) {
      int t0 = 0, t1 = 0;
      if (b < a.B && level_range(v, b, &t0, &t1) && sLead[v][b] == b) {
        const int nsub = ceil_div(sNum[v][b], cap);
        packed += (long long)nsub << (16 * v);
        keys += (long long)nsub * (t1 - t0);
      }
    }
    long long tot_packed, tot_sh;
    const long long excl = block_scan_sum64(packed, keys, &tot_packed, &tot_sh, wsum);
    for (int v = 0; v < kPrefixLevels; ++v) {
      if (b < a.B) sSg[v][b] = n_sg + (int)((excl >> (16 * v)) & 0xFFFF);
      n_sg += (int)((tot_packed >> (16 * v)) & 0xFFFF);
    }
    // Split of the shared keys: at least C, and large enough that the shared
    // items of all sub-groups times the KV heads fit the group-prefix grid in
    // one round (its workgroups are all resident; a second, partly filled
    // round would double the pass's time)
    if (a.forced_split <= 0 && tot_sh > 0) {
      long long per = (tot_sh * a.Hkv + a.prefix_grid - 1) / a.prefix_grid;
      per = (per + 63) & ~63LL;
      if (per > C) C = (int)per;
    }
  }
  // shared splits of sequence b over all levels
  auto shared_splits = [&](int b) -> int {
    int n = 0;
    if (grouping)
      for (int v = 0; v < kPrefixLevels; ++v) {
        int t0, t1;
        if (level_range(v, b, &t0, &t1)) n += ceil_div(t1 - t0, C);
      }
    return n;
  };

  // Private keys, counted in tiles of kTile keys (each sequence's range is
  // rounded up to whole tiles, so every piece starts on a tile boundary):
  // prefix sums per sequence, then the number of workers (a worker takes W / n
  // tiles, at least kMinWorkerKeys keys or the forced split, and at most
  // max_workers of them run)
  __syncthreads();   // the sums' per-wave totals are read before they are reused
  long long poff = 0;
  for (int b0 = 0; b0 < a.B; b0 += nthr) {
    const int b = b0 + tid;
    long long priv = 0;
    if (b < a.B) {
      int dummy = 0;
      const int L = small ? sL[b] : clamp_len(a.lens[b * a.lens_s], max_tokens, &dummy);
      priv = ceil_div(L - shared_keys(b), kTile);
    }
    long long tot;
    const long long ex = poff + block_exclusive_scan64(priv, &tot, wsum);
    if (b < a.B) {
      a.ws.pref[b] = ex;
      if (small) sPref[b] = ex;
    }
    poff += tot;
  }
  const long long W = poff;
  int nwork = 1;
  if (W > 0) {
    const long long per = (a.forced_split > 0 ? a.forced_split : kMinWorkerKeys) / kTile;
    const long long n = (W + per - 1) / per;
    nwork = (int)(n < a.max_workers ? n : a.max_workers);
  }
  if (tid == 0) {
    a.ws.pref[a.B] = W;
    if (small) sPref[a.B] = W;
  }
  __syncthreads();   // prefix sums visible to the workgroup
  // workers whose share starts before tile y of the concatenation (0 < y <= W)
  auto starts_before = [&](long long y) -> long long { return (y * nwork + W - 1) / W; };

  // Multi-token decode with no shared prefix page and an extend pass queued
  // behind this one: that pass computes every row (one unit per sequence and
  // KV head, longest first), and the split passes get no work.
  const bool handoff = a.route_extend && n_sg == 0;

  // Per sequence: its shared splits (level by level), then one private piece
  // per worker share it overlaps (a worker start strictly inside the range
  // begins a new piece)
  int slot_off = 0;
  for (int b0 = 0; b0 < a.B; b0 += nthr) {
    const int b = b0 + tid;
    int L = 0, S = 0, nsh = 0, npriv = 0, nslots = 0;
    bool direct = false, empty = false;
    if (b < a.B) {
      int dummy = 0;
      L = small ? sL[b] : clamp_len(a.lens[b * a.lens_s], max_tokens, &dummy);
      S = shared_keys(b);
      nsh = shared_splits(b);
      const long long p0 = small ? sPref[b] : a.ws.pref[b], p1 = small ? sPref[b + 1] : a.ws.pref[b + 1];
      npriv = p1 > p0 ? (int)(1 + starts_before(p1) - starts_before(p0 + 1)) : 0;
      empty = L == 0;
      direct = S == 0 && npriv == 1;
      nslots = direct || empty ? 0 : nsh + npriv;
    }
    int slot_tot;
    const int slot_base = slot_off + block_exclusive_scan(nslots, &slot_tot, wave_tot);
    if (b < a.B) {
      // a sequence whose slots do not fit writes nothing (the host sizes the
      // workspace so that this never happens; it is reported, not raced)
      const bool fits = slot_base + nslots <= a.max_slots;
      if (!fits && !handoff) cap_bad = 1;
      a.ws.nparts[b] = handoff ? 0 : (empty ? -1 : (fits ? nslots : -2));
      a.ws.base[b] = slot_base;
      a.ws.seqs[b] = make_int4(S, !fits ? kSlotDropped : (direct ? kSlotDirect : slot_base + nsh), L, fits ? 1 : 0);
      // its place in the sub-groups of every node it belongs to; a node's
      // splits take the member's slots after those of its ancestors
      int off = 0;
      for (int v = 0; v < kPrefixLevels && S > 0; ++v) {
        int t0, t1;
        if (!level_range(v, b, &t0, &t1)) continue;
        const int lead = sLead[v][b];
        int rank = 0;
        for (int j = lead + 1; j <= b; ++j) rank += sLead[v][j] == lead;
        const int sg = sSg[v][lead] + rank / cap, pos = rank % cap;
        const int n_split = ceil_div(t1 - t0, C);
        a.ws.sg_members[sg * cap + pos] = b;
        if (pos == 0) {
          a.ws.sgroups[sg] = make_int4(b, min(cap, sNum[v][lead] - (rank / cap) * cap), t1, n_split);
          a.ws.sg_range[sg] = make_int2(t0, off);
          sSgInfo[sg] = make_int4(t0, off, t1, n_split);
        }
        off += n_split;
      }
    }
    slot_off += slot_tot;
  }
  __syncthreads();

  // shared items: the splits of each sub-group's shared keys
  int sitem_off = 0;
  for (int g0 = 0; g0 < n_sg; g0 += nthr) {
    const int sg = g0 + tid;
    // (first key, first slot offset, end key, splits)
    const int4 info = sg < n_sg ? sSgInfo[sg] : make_int4(0, 0, 0, 0);
    int tot;
    const int base = sitem_off + block_exclusive_scan(info.w, &tot, wave_tot);
    for (int s = 0; s < info.w; ++s) {
      if (base + s < a.max_items)
        a.ws.sitems[base + s] = make_int4(sg, info.x + s * C, min(info.z, info.x + (s + 1) * C), info.y + s);
      else
        cap_bad = 1;
    }
    sitem_off += tot;
  }
  if (tid == 0) {
    a.ws.hdr[0] = C;
    a.ws.hdr[1] = handoff ? 0 : nwork;
    a.ws.hdr[2] = min(sitem_off, a.max_items);
    a.ws.hdr[3] = n_sg;
  }
  if (bad) atomicOr(a.ws.err, kErrLen);
  if (cap_bad) atomicOr(a.ws.err, kErrCapacity);
}

// Writes a finished (o, l, m) for one query head: directly to out/lse, or as
// a normalised partial into a slot.
struct HeadResult {
  float inv, lse;
};

__device__ __forceinline__ HeadResult finish(float m_log2, float l) {
  HeadResult r;
  r.inv = l > 0.f ? 1.f / l : 0.f;
  r.lse = l > 0.f ? (m_log2 + __builtin_amdgcn_logf(l)) * kLn2 : kNegInf;
  return r;
}

// Calls f(b, first key, end key, slot) for each piece of worker w's share of
// the concatenated private key ranges (see the planner): the share is cut at
// sequence boundaries; a piece that starts at a worker boundary inside a
// sequence is that sequence's k-th private piece, k counting the worker
// starts inside its range up to this one.
template <typename F>
__device__ __forceinline__ void for_each_piece(const DecodeArgs& a, int w, F&& f) {
  const int n = a.ws.hdr[1];
  if (w >= n) return;
  const long long W = a.ws.pref[a.B];
  long long x = (long long)w * W / n;
  const long long x_end = (long long)(w + 1) * W / n;
  if (x >= x_end) return;
  int lo = 0, hi = a.B - 1;   // first sequence whose range ends after x
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (a.ws.pref[mid + 1] > x) hi = mid; else lo = mid + 1;
  }
  for (int b = lo; x < x_end; ++b) {
    const long long p0 = a.ws.pref[b], p1 = a.ws.pref[b + 1];
    if (p1 <= x) continue;
    const long long e = p1 < x_end ? p1 : x_end;
    const int4 sq = a.ws.seqs[b];   // (S, first private slot or a slot marker, L, slots fit)
    int slot = sq.y;
    if (slot >= 0 && x > p0) slot += w - (int)(((p0 + 1) * n + W - 1) / W) + 1;
    const int t_end = sq.x + (int)((e - p0) * kTile);
    f(b, sq.x + (int)((x - p0) * kTile), t_end < sq.z ? t_end : sq.z, slot);
    x = e;
  }
}

// A lane's share of one key row of one KV head, as four 8-element chunks of
// the head dimension: chunk c of lane group grp holds elements d0 = 32 grp +
// 8 c .. d0 + 7, so a lane's chunks are contiguous (64 bytes of bf16, or 32
// bytes of FP8 codes: two 16-byte loads rather than four 8-byte ones, which
// would move half the bytes per load instruction). The scores only need Q and
// K in the same order, and V is staged into LDS by position. Rows are kept as
// loaded and converted where they are used.
template <bool kFp8>
struct RowPart;
template <>
struct RowPart<false> {
  bf16x8 r[4];
  __device__ static int d0(int c, int grp) { return 32 * grp + 8 * c; }
  __device__ void load(const char* row, int grp) {
#pragma unroll
    for (int c = 0; c < 4; ++c) r[c] = *reinterpret_cast<const bf16x8*>(row + 2 * d0(c, grp));
  }
  __device__ bf16x8 chunk(int c) const { return r[c]; }
};
template <>
struct RowPart<true> {
  uint4 r[2];
  __device__ static int d0(int c, int grp) { return 32 * grp + 8 * c; }
  __device__ void load(const char* row, int grp) {
    r[0] = *reinterpret_cast<const uint4*>(row + 32 * grp);
    r[1] = *reinterpret_cast<const uint4*>(row + 32 * grp + 16);
  }
  __device__ bf16x8 chunk(int c) const {
    const uint4 w = r[c >> 1];
    return kv_to_bf16x8<true>((c & 1) ? make_uint2(w.z, w.w) : make_uint2(w.x, w.y));
  }
};

// Split-KV decode on MFMA for a packed GQA group of up to 16 query heads.
// One wave per (private item, KV head, 16-head block). Keys are processed 32
// at a time. With pages of at least 32 keys, K and V rows are loaded whole
// (every instruction reads whole rows) with non-temporal loads and staged in
// the wave's own LDS tiles; K is read back as the A operand of S^T = K Q^T
// and V transposed as the A operand of O^T += V^T P^T. Measured on the ragged
// 64K batch: 1.50-1.56 ms per kernel (6.7-6.9 TB/s) against 1.68-1.69 ms with
// K loaded straight into A-operand registers (each lane its RowPart of a row,
// so an instruction reads 64-byte pieces of 16 rows, which non-temporal
// loads fetch again per piece) and V staged the same way; FP8 pages 0.84
// against 0.89 ms (with 8-byte loads, 16 lanes per row, 0.93 ms). Pages of
// fewer than 32 keys keep the RowPart path. Rows are fetched one tile ahead
// (bf16) or two (FP8), and page ids one tile ahead of the rows they address.
template <bool kFp8>
__global__ __launch_bounds__(512) void decode_mfma_kernel(DecodeArgs a) {
  // dynamic LDS: per wave a V tile and a K tile (32 keys x 272 B each)
  extern __shared__ u16 vs_dyn[];
  typedef u16 VTile[kTile][kHeadDim + 8];

  const int nqb = (a.R + 15) >> 4;
  const int per_item = a.Hkv * nqb;
  const int wpg = a.item_waves;             // waves per workgroup; divides per_item
  const int nch = per_item / wpg;
  // workgroup -> (worker, wave group); a worker's wave groups take the same keys
  const int worker = blockIdx.x / nch;
  const int wave = threadIdx.x >> 6;
  const int rem = (blockIdx.x - worker * nch) * wpg + wave;
  // the wave's V tile and K tile (K is staged only when a page holds a tile)
  VTile& vs = reinterpret_cast<VTile*>(vs_dyn)[2 * wave];
  VTile& ks = reinterpret_cast<VTile*>(vs_dyn)[2 * wave + 1];
  const int g = rem % a.Hkv;
  const int qb = rem / a.Hkv;
  int bad = 0;

  const int lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int row0 = qb * 16;
  const int nrows = min(16, a.R - row0);
  const bool col_ok = col < nrows;
  const int h = g * a.R + row0 + (col_ok ? col : 0);
  int bad_scale = 0;
  const KvScales dq = kv_scales<kFp8>(a.kv, g, &bad_scale);
  const float sl2 = a.scale * dq.k * kLog2e;   // the K dequantisation scale joins the softmax scale

  for_each_piece(a, worker, [&](int b, int t_begin, int t_end, int slot) {
  bf16x8 qv[4];
  {
    const __bf16* qp = (const __bf16*)a.q + (int64_t)b * a.q_sb + (int64_t)h * a.q_sh;
#pragma unroll
    for (int c = 0; c < 4; ++c) qv[c] = col_ok ? load_bf16x8(qp + RowPart<kFp8>::d0(c, grp)) : zero_bf16x8();
  }

  f32x4 o[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) o[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = kNegInf, l_run = 0.f;

  const int* bt_row = a.kv.bt + (int64_t)b * a.kv.bt_sb;
  const uint32_t bt_sj = (uint32_t)a.kv.bt_sj;
  constexpr int ES = kv_bytes<kFp8>();
  const char* kbase = (const char*)a.kv.k + ES * (int64_t)g * a.kv.sh;
  const char* vbase = (const char*)a.kv.v + ES * (int64_t)g * a.kv.v_sh;
  const uint32_t ksp = (uint32_t)a.kv.sp, kss = (uint32_t)a.kv.ss;
  const uint32_t vsp = (uint32_t)a.kv.v_sp, vss = (uint32_t)a.kv.v_ss;
  const int pmask = a.kv.page_size - 1;
  // tiles start at multiples of 32 keys, so a page of >= 32 keys holds a whole tile
  const bool page_holds_tile = a.kv.page_size >= kTile && (t_begin & (kTile - 1)) == 0;

  // The two ways of finding a tile's pages are separate code paths, so the
  // scalar page ids of the first never merge with the vector ones of the other.
  auto run = [&](auto holds_tag) {
    constexpr bool kHolds = decltype(holds_tag)::value;
    // Rows of the next kDepth tiles are in flight while a tile is computed.
    // FP8 rows are half the bytes, so they go two tiles ahead (the same bytes
    // and registers in flight as one bf16 tile).
    constexpr int kDepth = kFp8 ? 2 : 1;
    // Rows in flight. kWhole (one page per tile): whole rows, loaded
    // non-temporally 16 bytes per lane and staged in LDS; bf16: 16 lanes per
    // 256-byte row (lane l: elements 8 (l % 16) .. + 7 of rows 4 i + l / 16),
    // FP8: 8 lanes per 128-byte row (lane l: codes 16 (l % 8) .. + 15 of rows
    // 8 i + l / 8). Otherwise each lane's RowPart of keys 16 hh + col, K kept
    // in registers.
    constexpr bool kWhole = kHolds;
    typedef std::conditional_t<kFp8, uint4, bf16x8> Piece;
    struct WholeRows {
      Piece r[kFp8 ? 4 : 8];
    };
    typedef std::conditional_t<kWhole, WholeRows, RowPart<kFp8>[2]> Rows;
    Rows kc0, kc1, vc0, vc1;
    int praw[2];                        // page ids of the next tile to fetch
    // When a page holds the whole tile its id is the same for the wave and is
    // read through the scalar unit (the block table is not written while the
    // kernel runs). Its wait then does not include the vector loads of rows
    // issued before it, which retire in order.
    typedef __attribute__((address_space(4))) const int ConstInt;
    const ConstInt* bt_c = (const ConstInt*)bt_row;
    auto fetch_pages = [&](int t0) {
      if constexpr (kHolds) {
        const int t = __builtin_amdgcn_readfirstlane(t0 < t_end ? t0 : t_end - 1);
        praw[0] = bt_c[__umul24((uint32_t)(t >> a.kv.log2_page), bt_sj)];
        praw[1] = 0;
      } else {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          int t = t0 + 16 * hh + col;
          t = t < t_end ? t : t_end - 1;
          praw[hh] = bt_row[__umul24((uint32_t)(t >> a.kv.log2_page), bt_sj)];
        }
      }
    };
    auto fetch_rows = [&](int t0, Rows& kc, Rows& vc) {
      if constexpr (kWhole) {
        int pg = praw[0];
        if ((unsigned)pg >= (unsigned)a.kv.num_pages) {
          bad = 1;
          pg = pg < 0 ? 0 : a.kv.num_pages - 1;
        }
        constexpr int kRowsPer = kFp8 ? 8 : 4, kLanesPerRow = 64 / kRowsPer, kN = kFp8 ? 4 : 8;
        const int piece = (kFp8 ? 16 : 8) * (lane & (kLanesPerRow - 1));
#pragma unroll
        for (int i = 0; i < kN; ++i) {
          int t = t0 + kRowsPer * i + lane / kLanesPerRow;
          t = t < t_end ? t : t_end - 1;
          kc.r[i] = load_nt<Piece>(kbase + ES * (row_offset((uint32_t)pg, ksp, t & pmask, kss) + piece));
          vc.r[i] = load_nt<Piece>(vbase + ES * (row_offset((uint32_t)pg, vsp, t & pmask, vss) + piece));
        }
      } else {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          int t = t0 + 16 * hh + col;
          t = t < t_end ? t : t_end - 1;
          int pg = praw[kHolds ? 0 : hh];
          if ((unsigned)pg >= (unsigned)a.kv.num_pages) {
            bad = 1;
            pg = pg < 0 ? 0 : a.kv.num_pages - 1;
          }
          kc[hh].load(kbase + ES * row_offset((uint32_t)pg, ksp, t & pmask, kss), grp);
          vc[hh].load(vbase + ES * row_offset((uint32_t)pg, vsp, t & pmask, vss), grp);
        }
      }
    };
    // one tile of keys [t0, t0 + 32) from the rows in (kc, vc), which then take
    // the rows kDepth tiles ahead. Prefetches past the piece are clamped to its
    // last key (in bounds, and never used): unconditional loads keep the number
    // of loads in flight the same on every path, so each wait covers only the
    // tile it needs.
    auto tile = [&](int t0, Rows& kc, Rows& vc) {
      __syncthreads();  // previous tile's K and V reads are done
      const int tn = t0 + kDepth * kTile;
      if constexpr (kWhole) {
        // stage both tiles, then the rows kDepth tiles ahead take the
        // registers at once
        if constexpr (kFp8) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int row = 8 * i + (lane >> 3), e0 = 16 * (lane & 7);
            const uint4 kw = kc.r[i], vw = vc.r[i];
            *reinterpret_cast<bf16x8*>(&vs[row][e0]) = kv_to_bf16x8<true>(make_uint2(vw.x, vw.y));
            *reinterpret_cast<bf16x8*>(&vs[row][e0 + 8]) = kv_to_bf16x8<true>(make_uint2(vw.z, vw.w));
            *reinterpret_cast<bf16x8*>(&ks[row][e0]) = kv_to_bf16x8<true>(make_uint2(kw.x, kw.y));
            *reinterpret_cast<bf16x8*>(&ks[row][e0 + 8]) = kv_to_bf16x8<true>(make_uint2(kw.z, kw.w));
          }
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            *reinterpret_cast<bf16x8*>(&vs[4 * i + (lane >> 4)][8 * (lane & 15)]) = kv_to_bf16x8<kFp8>(vc.r[i]);
            *reinterpret_cast<bf16x8*>(&ks[4 * i + (lane >> 4)][8 * (lane & 15)]) = kv_to_bf16x8<kFp8>(kc.r[i]);
          }
        }
        fetch_rows(tn, kc, vc);
        fetch_pages(tn + kTile);
        // the wave reads the K rows its other lanes wrote
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      } else {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int c = 0; c < 4; ++c)
            *reinterpret_cast<bf16x8*>(&vs[16 * hh + col][RowPart<kFp8>::d0(c, grp)]) = vc[hh].chunk(c);
      }
      f32x4 st[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) st[hh] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          bf16x8 ka;
          if constexpr (kWhole)
            ka = *reinterpret_cast<const bf16x8*>(&ks[16 * hh + col][RowPart<kFp8>::d0(c, grp)]);
          else
            ka = kc[hh].chunk(c);
          st[hh] = mfma_16x16x32(ka, qv[c], st[hh]);
        }
      if constexpr (!kWhole) {
        fetch_rows(tn, kc, vc);
        fetch_pages(tn + kTile);
      }

      float mt = kNegInf;
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = t0 + 16 * hh + 4 * grp + i;
          if (t >= t_end) st[hh][i] = kNegInf;
          mt = fmaxf(mt, st[hh][i]);
        }
      mt = group_max(mt) * sl2;
      const float m_new = fmaxf(m_run, mt);
      const float alpha = exp2_fast(m_run - m_new);
      const float neg_m = -m_new;
      float ps = 0.f;
      bf16x8 pb;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float p = exp2_fast(fmaf(st[e >> 2][e & 3], sl2, neg_m));
        ps += p;
        pb[e] = (__bf16)p;
      }
      l_run = l_run * alpha + ps;
      m_run = m_new;
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] *= alpha;
      __syncthreads();  // V tile visible
      // V^T operand: element e of lane (grp, col) is V[tok(e)][16 j + col], tok(e) =
      // 4 grp + e (e < 4) or 16 + 4 grp + e - 4 (the keys of pb). With FP8 pages
      // two transposed reads per MFMA give it: lane 4e + q of a 16-lane block
      // addresses row 4 grp + e (then 16 rows further), columns 16 j + 4 q ..
      // + 3, and the read hands lane i element i % 4 of lane 4e + i / 4's chunk
      // as its element e (FP8 decode 0.834 -> 0.816 ms on the ragged batch).
      // bf16 keeps eight 16-bit reads: the transposed form measured 0.5-0.9%
      // slower there, its registers allocated differently.
      const int tr_row = 4 * grp + ((lane & 15) >> 2), tr_col = 4 * (lane & 3);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        bf16x8 va;
        if constexpr (kFp8) {
          const u16* vp = &vs[tr_row][16 * j + tr_col];
          const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)vp);
          const i16x4 up = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vp + 16 * (kHeadDim + 8)));
          va = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, up, 0, 1, 2, 3, 4, 5, 6, 7));
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int tok = e < 4 ? 4 * grp + e : 16 + 4 * grp + (e - 4);
            va[e] = bits_to_bf16(vs[tok][16 * j + col]);
          }
        }
        o[j] = mfma_16x16x32(va, pb, o[j]);
      }
    };
    fetch_pages(t_begin);
    fetch_rows(t_begin, kc0, vc0);
    if constexpr (kDepth == 2) {
      fetch_pages(t_begin + kTile);
      fetch_rows(t_begin + kTile, kc1, vc1);
    }
    fetch_pages(t_begin + kDepth * kTile);
    if constexpr (kDepth == 1) {
      for (int t0 = t_begin; t0 < t_end; t0 += kTile) tile(t0, kc0, vc0);
    } else {
      // Tiles go in pairs, one per buffer, with no branch between them: the
      // second tile of the last pair may lie past the piece, where every key is
      // masked (p = 0, alpha = 1), which leaves o, m and l exactly unchanged.
      for (int t0 = t_begin; t0 < t_end; t0 += 2 * kTile) {
        tile(t0, kc0, vc0);
        tile(t0 + kTile, kc1, vc1);
      }
    }
  };
  if (t_begin < t_end) {
    if (page_holds_tile)
      run(std::true_type{});
    else
      run(std::false_type{});
  }

  const HeadResult res = finish(m_run, group_sum(l_run));
  const float inv = res.inv * dq.v;            // the V dequantisation scale
  if (col_ok && slot != kSlotDropped) {
    if (slot == kSlotDirect) {
      if (a.out_f32) {
        float* op = (float*)a.out + (int64_t)b * a.out_sb + (int64_t)h * a.out_sh + 4 * grp;
#pragma unroll
        for (int j = 0; j < 8; ++j) *reinterpret_cast<f32x4*>(op + 16 * j) = o[j] * inv;
      } else {
        typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
        __bf16* op = (__bf16*)a.out + (int64_t)b * a.out_sb + (int64_t)h * a.out_sh + 4 * grp;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          bf16x4 w;
#pragma unroll
          for (int i = 0; i < 4; ++i) w[i] = (__bf16)(o[j][i] * inv);
          *reinterpret_cast<bf16x4*>(op + 16 * j) = w;
        }
      }
      if (a.lse && grp == 0) a.lse[(int64_t)b * a.lse_sb + (int64_t)h * a.lse_sh] = res.lse;
    } else {
      float* pp = a.ws.part_o + ((int64_t)slot * a.Hv + h) * kHeadDim + 4 * grp;
#pragma unroll
      for (int j = 0; j < 8; ++j) *reinterpret_cast<f32x4*>(pp + 16 * j) = o[j] * inv;
      if (grp == 0) a.ws.part_lse[(int64_t)slot * a.Hv + h] = res.lse;
    }
  }
  });
  if (bad) atomicOr(a.ws.err, kErrPage);
  if (bad_scale) atomicOr(a.ws.err, kErrScale);
}

// Single-query decode (one query head per KV head) on the vector ALUs: each
// 16-lane group takes one key per step (a whole 256-byte row per load), keeps
// its own online-softmax state, and the four groups are merged at the end.
template <bool kFp8>
__global__ __launch_bounds__(64) void decode_valu_kernel(DecodeArgs a) {
  const int worker = blockIdx.x / a.Hkv;
  const int g = blockIdx.x - worker * a.Hkv;
  int bad = 0, bad_scale = 0;
  const int lane = threadIdx.x;
  const int c16 = lane & 15, grp = lane >> 4;
  const int h = g;  // R == 1
  const KvScales dq = kv_scales<kFp8>(a.kv, g, &bad_scale);
  const float sl2 = a.scale * dq.k * kLog2e;

  for_each_piece(a, worker, [&](int b, int t_begin, int t_end, int slot) {
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
  const uint32_t bt_sj = (uint32_t)a.kv.bt_sj;
  constexpr int ES = kv_bytes<kFp8>();
  const char* kbase = (const char*)a.kv.k + ES * ((int64_t)g * a.kv.sh + c16 * 8);
  const char* vbase = (const char*)a.kv.v + ES * ((int64_t)g * a.kv.v_sh + c16 * 8);
  // kU keys per group per round (keys t0 + 4 u + grp): the round's page ids
  // are loaded together, then its rows, so a round waits for two round trips
  // instead of 2 kU; the keys are then taken in the same order as one at a time
  constexpr int kU = 4;
  for (int t0 = t_begin; t0 < t_end; t0 += 4 * kU) {
    uint32_t pg[kU];
    int slot_t[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int t = t0 + 4 * u + grp;
      const int tt = t < t_end ? t : t_end - 1;
      pg[u] = page_of(bt_row, bt_sj, tt, a.kv.log2_page, a.kv.num_pages, &bad);
      slot_t[u] = tt & (a.kv.page_size - 1);
    }
    KvRaw<kFp8> kr[kU], vr[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      kr[u] = load_kv_raw_nt<kFp8>(kbase + ES * row_offset(pg[u], (uint32_t)a.kv.sp, slot_t[u], (uint32_t)a.kv.ss));
      vr[u] = load_kv_raw_nt<kFp8>(vbase + ES * row_offset(pg[u], (uint32_t)a.kv.v_sp, slot_t[u], (uint32_t)a.kv.v_ss));
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const bool valid = t0 + 4 * u + grp < t_end;
      const bf16x8 kk = kv_to_bf16x8<kFp8>(kr[u]);
      float d = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) d += qf[i] * (float)kk[i];
      d = row_sum16(d);
      if (valid) {
        const bf16x8 vv = kv_to_bf16x8<kFp8>(vr[u]);
        const float m_new = fmaxf(m, d);
        const float alpha = exp2_fast(m - m_new);
        const float p = exp2_fast(d - m_new);
        l = l * alpha + p;
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = acc[i] * alpha + p * (float)vv[i];
        m = m_new;
      }
    }
  }
  const float M = group_max(m);
  const float w = m == kNegInf ? 0.f : exp2_fast(m - M);
  const float l_tot = group_sum(l * w);
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = group_sum(acc[i] * w);
  const HeadResult res = finish(M, l_tot);
  const float inv = res.inv * dq.v;
  if (grp == 0 && slot != kSlotDropped) {
    if (slot == kSlotDirect) {
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
      if (a.lse && c16 == 0) a.lse[(int64_t)b * a.lse_sb + (int64_t)h * a.lse_sh] = res.lse;
    } else {
      float* pp = a.ws.part_o + ((int64_t)slot * a.Hv + h) * kHeadDim + c16 * 8;
#pragma unroll
      for (int i = 0; i < 8; ++i) pp[i] = acc[i] * inv;
      if (c16 == 0) a.ws.part_lse[(int64_t)slot * a.Hv + h] = res.lse;
    }
  }
  });
  if (bad) atomicOr(a.ws.err, kErrPage);
  if (bad_scale) atomicOr(a.ws.err, kErrScale);
}

// Multi-token decode (n_tok > 1, e.g. verifying multi-token-prediction
// drafts): the n_tok * R rows (query token, query head) of one KV head share
// every key, so one workgroup computes up to 128 of them with the LDS-staged
// tile routine (K and V read once per workgroup), over the same equal-work
// pieces as single-token decode. Token i of a sequence of length L sees keys
// t <= L - n_tok + i. Pieces start on 32-key tiles; the routine's steps start
// on 64-key boundaries, so a piece's first step masks the keys before it.
constexpr int kMultiWaves = 4;          // waves per multi-token workgroup: 128 rows
constexpr int kXcds = 8;                // XCDs of the device; workgroup i runs on XCD i % 8
constexpr bool kMultiXcd = true;        // a worker's workgroups on one XCD

template <bool kFp8>
__global__ __launch_bounds__(kMultiWaves * 64, 2) void decode_multi_kernel(DecodeArgs a) {
  __shared__ TileLds lds;
  const int rows = a.n_tok * a.R;
  const int nrb = (rows + kMultiWaves * kWaveRows - 1) / (kMultiWaves * kWaveRows);
  const int nch = a.Hkv * nrb;                  // workgroups per worker
  // Workgroups are dealt to the XCDs round-robin by index; when the workers
  // divide evenly, worker w's workgroups (its KV heads, which read the
  // interleaved head rows of the same tokens) are numbered so that all of
  // them land on XCD w % 8, one after another.
  int worker, rem;
  if (kMultiXcd && a.max_workers % kXcds == 0) {
    const int x = blockIdx.x % kXcds, k = blockIdx.x / kXcds;
    const int m = k / nch;
    rem = k - m * nch;
    worker = x + kXcds * m;
  } else {
    worker = blockIdx.x / nch;
    rem = blockIdx.x - worker * nch;
  }
  const int g = rem % a.Hkv, rb = rem / a.Hkv;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rr = rb * kMultiWaves * kWaveRows + wave * kWaveRows + (lane & 31);
  const bool row_ok = rr < rows;
  const int tok = row_ok ? rr / a.R : 0;
  const int head = g * a.R + (row_ok ? rr - tok * a.R : 0);
  int bad = 0, bad_short = 0, bad_scale = 0;
  const KvScales dq = kv_scales<kFp8>(a.kv, g, &bad_scale);
  const float scale = a.scale * dq.k;

  for_each_piece(a, worker, [&](int b, int t_begin, int t_end, int slot) {
    const int L = a.ws.seqs[b].z;
    if (L < a.n_tok) bad_short = 1;          // the query tokens must be in the cache
    const int limit = L - a.n_tok + tok;
    bf16x8 qv[8];
    load_q_operand((const __bf16*)a.q + (int64_t)b * a.q_sb + (int64_t)tok * a.q_st + (int64_t)head * a.q_sh, row_ok,
                   qv);
    f32x16 o[4];
#pragma unroll
    for (int jd = 0; jd < 4; ++jd)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[jd][e] = 0.f;
    float m_run = kNegInf, l_run = 0.f;
    const int t_lo = t_begin & ~(kKeys - 1);
    // keys below L - n + 1 are visible to every token (t_full may not pass the
    // piece's end: the routine masks keys at or past t_hi only from t_full on)
    const int t_full = min(L - a.n_tok + 1, t_end);
    tile_attend<kMultiWaves, kFp8>(a.kv, scale, a.kv.bt + (int64_t)b * a.kv.bt_sb, g, t_lo, t_end, t_full,
                                          limit, qv, lds, o, m_run, l_run, bad, t_begin,
                                          rb * kMultiWaves * kWaveRows + wave * kWaveRows < rows);
    const HeadResult res = finish(m_run, sum_l32(l_run));
    if (row_ok && slot != kSlotDropped) {
      const float inv = res.inv * dq.v;
      if (slot == kSlotDirect) {
        const int64_t oo = (int64_t)b * a.out_sb + (int64_t)tok * a.out_st + (int64_t)head * a.out_sh;
        if (a.out_f32)
          store_o_row((float*)a.out + oo, o, inv);
        else
          store_o_row((__bf16*)a.out + oo, o, inv);
        if (a.lse && lane < 32)
          a.lse[(int64_t)b * a.lse_sb + (int64_t)tok * a.lse_st + (int64_t)head * a.lse_sh] = res.lse;
      } else {
        const int64_t row = (int64_t)slot * a.Hv + (int64_t)tok * a.Hq + head;
        store_o_row(a.ws.part_o + row * kHeadDim, o, inv);
        if (lane < 32) a.ws.part_lse[row] = res.lse;
      }
    }
    __syncthreads();  // the LDS tiles are reused by the next piece
  });
  if (bad) atomicOr(a.ws.err, kErrPage);
  if (bad_short) atomicOr(a.ws.err, kErrKvShort);
  if (bad_scale) atomicOr(a.ws.err, kErrScale);
}

// Group-prefix pass: one workgroup per (shared item, KV head) computes a split
// of a node's shared keys once for all the query rows of one of its sub-groups
// (row r -> member r / (n R), then query token, then query head), reading each
// shared page once per sub-group, and writes one partial per member into that
// member's slot for this split.
constexpr int kPrefixWaves = 4;         // waves per group-prefix workgroup: 128 member rows

template <bool kFp8>
__global__ __launch_bounds__(kPrefixWaves * 64, 2) void prefix_kernel(DecodeArgs a) {
  __shared__ TileLds lds;
  // grid-stride over (shared item, KV head): a batch without trajectory groups
  // costs one small launch that exits at once
  const int n_work = a.ws.hdr[2] * a.Hkv;
  for (int wi = blockIdx.x; wi < n_work; wi += gridDim.x) {
    const int item = wi / a.Hkv;
    const int g = wi - item * a.Hkv;
    const int4 it = a.ws.sitems[item];
    const int sg = it.x, t0 = it.y, t1 = it.z, split = it.w;   // split: slot offset in each member's slots
    const int4 info = a.ws.sgroups[sg];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = wave * kWaveRows + (lane & 31);
    const int rows_m = a.n_tok * a.R;               // rows of one member
    const int member = r / rows_m, rm = r - member * rows_m;
    const int tok = rm / a.R, hi = rm - tok * a.R;
    const bool row_ok = member < info.y;
    const int b = a.ws.sg_members[sg * a.group_cap + (row_ok ? member : 0)];
    const int head = g * a.R + hi;
    // token tok of a member of length L sees keys t <= L - n + tok (with one
    // token the shared keys are all visible)
    const int limit = a.n_tok == 1 ? t1 - 1 : a.ws.seqs[b].z - a.n_tok + tok;

    bf16x8 qv[8];
    load_q_operand((const __bf16*)a.q + (int64_t)b * a.q_sb + (int64_t)tok * a.q_st + (int64_t)head * a.q_sh, row_ok,
                   qv);
    f32x16 o[4];
#pragma unroll
    for (int jd = 0; jd < 4; ++jd)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[jd][e] = 0.f;
    float m_run = kNegInf, l_run = 0.f;
    int bad = 0, bad_scale = 0;
    const KvScales dq = kv_scales<kFp8>(a.kv, g, &bad_scale);
    // a node below the first level starts where its parent ends, a page
    // boundary that need not be a step boundary: keys below t0 are masked
    tile_attend<kPrefixWaves, kFp8>(a.kv, a.scale * dq.k, a.kv.bt + (int64_t)info.x * a.kv.bt_sb, g,
                                           t0 & ~(kKeys - 1), t1, a.n_tok == 1 ? t1 : t0, limit, qv, lds, o, m_run,
                                           l_run, bad, t0, wave * kWaveRows / rows_m < info.y);
    const HeadResult res = finish(m_run, sum_l32(l_run));
    if (row_ok) {
      const int slot = a.ws.base[b] + split;
      if (a.ws.seqs[b].w) {                        // the member's slots fit the workspace
        const int64_t row = (int64_t)slot * a.Hv + (int64_t)tok * a.Hq + head;
        store_o_row(a.ws.part_o + row * kHeadDim, o, res.inv * dq.v);
        if (lane < 32) a.ws.part_lse[row] = res.lse;
      }
    }
    if (bad) atomicOr(a.ws.err, kErrPage);
    if (bad_scale) atomicOr(a.ws.err, kErrScale);
    __syncthreads();  // the LDS tiles are reused by the next work unit
  }
}

// Merge the partials of one (sequence, query head): one wave, two output
// elements per lane. The lanes load the parts' log-sum-exps in parallel and
// reduce them with cross-lane operations; the weighted sum over parts then
// streams the partial outputs with independent loads.
__device__ __forceinline__ void merge_parts(const float* o_base, int64_t o_step, const float* l_base, int64_t l_step,
                                            int n, float* out2, float* lse_out) {
  const int lane = threadIdx.x & 63;
  // The o rows of the first kPre parts are loaded together with the lse
  // values, so a row of at most kPre parts (the usual case) waits for one
  // round trip instead of two.
  constexpr int kPre = 4;
  float2 pre[kPre];
#pragma unroll
  for (int u = 0; u < kPre; ++u)
    pre[u] = u < n ? *reinterpret_cast<const float2*>(o_base + (int64_t)u * o_step + 2 * lane) : make_float2(0.f, 0.f);
  const float l0 = lane < n ? l_base[(int64_t)lane * l_step] : kNegInf;
  float M = l0;
  for (int s0 = 64; s0 < n; s0 += 64)
    if (s0 + lane < n) M = fmaxf(M, l_base[(int64_t)(s0 + lane) * l_step]);
  M = wave_max(M);
  float z = 0.f, a0 = 0.f, a1 = 0.f;
  if (M != kNegInf) {
    for (int s0 = 0; s0 < n; s0 += 64) {
      const float lv = s0 == 0 ? l0 : (s0 + lane < n ? l_base[(int64_t)(s0 + lane) * l_step] : kNegInf);
      const float my_w = s0 + lane < n ? exp2_fast((lv - M) * kLog2e) : 0.f;
      z += my_w;
      const int cnt = min(64, n - s0);
      int s = 0;
      if (s0 == 0) {
#pragma unroll
        for (int u = 0; u < kPre; ++u)
          if (u < cnt) {
            const float w = __shfl(my_w, u, 64);
            a0 += w * pre[u].x;
            a1 += w * pre[u].y;
          }
        s = min(cnt, kPre);
      }
      for (; s + 4 <= cnt; s += 4) {
        float2 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
          v[u] = *reinterpret_cast<const float2*>(o_base + (int64_t)(s0 + s + u) * o_step + 2 * lane);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float w = __shfl(my_w, s + u, 64);
          a0 += w * v[u].x;
          a1 += w * v[u].y;
        }
      }
      for (; s < cnt; ++s) {
        const float2 v = *reinterpret_cast<const float2*>(o_base + (int64_t)(s0 + s) * o_step + 2 * lane);
        const float w = __shfl(my_w, s, 64);
        a0 += w * v.x;
        a1 += w * v.y;
      }
    }
    z = wave_sum(z);
  }
  const float inv = z > 0.f ? 1.f / z : 0.f;
  out2[0] = a0 * inv;
  out2[1] = a1 * inv;
  *lse_out = z > 0.f ? M + __builtin_amdgcn_logf(z) * kLn2 : kNegInf;
}

// One (sequence, row) per wave, kCombineRows rows of one sequence per
// workgroup (row hv = token * Hq + query head): a sequence without parts to
// merge costs one workgroup per kCombineRows rows rather than one per row
// (at 8 tokens of 96 heads, 98K single-wave workgroups took 25 us to launch
// and return).
constexpr int kCombineRows = 8;

__global__ __launch_bounds__(kCombineRows * 64) void combine_kernel(DecodeArgs a) {
  const int nblk = (a.Hv + kCombineRows - 1) / kCombineRows;
  const int b = blockIdx.x / nblk;
  const int hv = (blockIdx.x - b * nblk) * kCombineRows + (threadIdx.x >> 6);
  // the planner writes both for every sequence; they are read together
  const int n = a.ws.nparts[b];
  const int base = a.ws.base[b];
  if (n == 0 || hv >= a.Hv) return;     // n == 0: written directly by its only piece
  const int tok = hv / a.Hq, h = hv - tok * a.Hq;
  float r[2] = {0.f, 0.f}, lse_v = kNegInf;   // an empty sequence (n == -1): zeros, -inf
  if (n == -2) {          // its slots did not fit the workspace (reported as kErrCapacity)
    r[0] = r[1] = lse_v = __uint_as_float(0x7fc00000u);   // a quiet NaN
  } else if (n > 0) {
    merge_parts(a.ws.part_o + ((int64_t)base * a.Hv + hv) * kHeadDim, (int64_t)a.Hv * kHeadDim,
                a.ws.part_lse + (int64_t)base * a.Hv + hv, a.Hv, n, r, &lse_v);
  }
  const int lane = threadIdx.x & 63;
  const int64_t oo = (int64_t)b * a.out_sb + (int64_t)tok * a.out_st + (int64_t)h * a.out_sh + 2 * lane;
  if (a.out_f32) {
    float* op = (float*)a.out + oo;
    op[0] = r[0];
    op[1] = r[1];
  } else {
    __bf16* op = (__bf16*)a.out + oo;
    op[0] = (__bf16)r[0];
    op[1] = (__bf16)r[1];
  }
  if (a.lse && lane == 0) a.lse[(int64_t)b * a.lse_sb + (int64_t)tok * a.lse_st + (int64_t)h * a.lse_sh] = lse_v;
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

template <bool kFp8>
void launch_decode_kernels(const DecodeArgs& a, hipStream_t stream, KernelTimer* timer) {
  const unsigned per_item = a.R == 1 ? a.Hkv : a.Hkv * ((a.R + 15) / 16);
  if (a.group_cap >= 2) prefix_kernel<kFp8><<<(unsigned)a.prefix_grid, kPrefixWaves * 64, 0, stream>>>(a);
  if (timer) (void)hipEventRecord(timer->start, stream);
  if (a.n_tok > 1) {
    const int rows = a.n_tok * a.R;
    const int64_t nch = (int64_t)a.Hkv * ((rows + kMultiWaves * kWaveRows - 1) / (kMultiWaves * kWaveRows));
    decode_multi_kernel<kFp8><<<(unsigned)(a.max_workers * nch), kMultiWaves * 64, 0, stream>>>(a);
  } else if (a.R == 1) {
    decode_valu_kernel<kFp8><<<(unsigned)a.max_workers * per_item, 64, 0, stream>>>(a);
  } else {
    const unsigned nch = per_item / a.item_waves;
    const unsigned grid = (unsigned)((int64_t)a.max_workers * nch);
    const size_t lds = (size_t)2 * a.item_waves * kTile * (kHeadDim + 8) * sizeof(u16);
    decode_mfma_kernel<kFp8><<<grid, 64 * a.item_waves, lds, stream>>>(a);
  }
  if (timer) (void)hipEventRecord(timer->stop, stream);
}

template <bool kFp8>
int workers_per_cu_of(int R, int Hkv, int item_waves, int n_tok) {
  int blocks = 0;
  // multi-token decode: one worker per CU; a worker's Hkv x row-block
  // workgroups then run in equal rounds
  if (n_tok > 1) return 1;
  if (R == 1) {
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, decode_valu_kernel<kFp8>, 64, 0) != hipSuccess) blocks = 0;
    return blocks / Hkv > 1 ? blocks / Hkv : 1;
  }
  const size_t lds = (size_t)2 * item_waves * kTile * (kHeadDim + 8) * sizeof(u16);
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, decode_mfma_kernel<kFp8>, 64 * item_waves, lds) != hipSuccess)
    blocks = 0;
  const int nch = Hkv * ((R + 15) / 16) / item_waves;
  return blocks / nch > 1 ? blocks / nch : 1;
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream, KernelTimer* timer) {
  plan_decode_kernel<<<1, 1024, 0, stream>>>(a);
  if (a.kv.k_scale)
    launch_decode_kernels<true>(a, stream, timer);
  else
    launch_decode_kernels<false>(a, stream, timer);
  combine_kernel<<<(unsigned)((int64_t)a.B * ((a.Hv + kCombineRows - 1) / kCombineRows)), kCombineRows * 64, 0,
                   stream>>>(a);
  return hipGetLastError();
}

int decode_workers_per_cu(int R, int Hkv, int item_waves, bool fp8, int n_tok) {
  return fp8 ? workers_per_cu_of<true>(R, Hkv, item_waves, n_tok) : workers_per_cu_of<false>(R, Hkv, item_waves, n_tok);
}

hipError_t launch_merge(const MergeArgs& a, hipStream_t stream) {
  merge_kernel<<<(unsigned)(a.N * a.H), 64, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace rl
