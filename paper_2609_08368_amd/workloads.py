"""Seeded synthetic rollout-attention workloads (inputs only, no attention math).

Both the HIP path (tests, bench) and the CPU oracle consume what this module
builds; it holds no part of the attention computation. Shapes follow the
rollout engines of the paper: trajectory groups of G = 8 attempts per prompt
(section "The Miles RL Loop" and the case-study table), sessions capped at
65,536 tokens (case-study table), batches of many concurrent requests
(case-study results), and turns that append a chunk of tokens to a long cached
prefix (section "Fast Agentic Rollout with SGLang"). Paging, page sizes, head
counts and length distributions are synthetic stand-ins; the recipe is:

* metadata (lengths, page permutation, per-KV-head scales) from
  ``numpy.random.default_rng(seed)``;
* bulk values from ``torch.Generator(device).manual_seed(seed * 16 + tensor)``
  with tensor ids q=1, k=2, v=3: standard normal float32, multiplied by the
  per-KV-head scale where the workload has one, rounded to bf16
  (round-to-nearest-even, torch's cast);
* physical page ids are a seeded permutation of the pool; pages no sequence
  references, slots past a sequence's length in its last page and block-table
  entries past the last used page are "poison" (NaN pages / a NaN page id) in
  correctness runs, so a stray read shows up as NaN in the output.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

HEAD_DIM = 128


@dataclasses.dataclass
class Paged:
    """Metadata of a paged KV cache plus its queries (numpy, host side)."""

    name: str
    kind: str                     # "decode" or "extend"
    seed: int
    hq: int
    hkv: int
    page_size: int
    num_pages: int
    block_table: np.ndarray       # [B, max_pages] int32
    kv_lens: np.ndarray           # [B] int32: tokens in the cache (decode: seq_lens)
    q_lens: np.ndarray            # [B] int32: query rows per sequence (decode: 1)
    poison_page: int              # a page id no sequence references (-1 if none)
    kv_head_scale: Optional[np.ndarray] = None   # [Hkv] float32 multipliers for K and V
    shared_prefix_pages: int = 0  # leading pages shared inside each group (group prefix workloads)
    group_size: int = 1

    @property
    def batch(self) -> int:
        return int(self.kv_lens.shape[0])

    @property
    def qo_indptr(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.q_lens)]).astype(np.int32)

    @property
    def total_q(self) -> int:
        return int(self.q_lens.sum())

    def kv_bytes(self, unique: bool = False) -> int:
        """K and V bytes the attention reads (bf16, all KV heads)."""
        per_token = self.hkv * HEAD_DIM * 2 * 2
        if not unique:
            return int(self.kv_lens.astype(np.int64).sum()) * per_token
        pages = set()
        for b in range(self.batch):
            used = -(-int(self.kv_lens[b]) // self.page_size)
            for j in range(used):
                pages.add((int(self.block_table[b, j]), min(self.page_size, int(self.kv_lens[b]) - j * self.page_size)))
        # a page shared by several sequences is counted once, with its largest use
        best = {}
        for p, n in pages:
            best[p] = max(best.get(p, 0), n)
        return int(sum(best.values())) * per_token

    def flops(self) -> float:
        """Multiply-adds x 2 over unmasked (query row, key) pairs, QK^T and PV."""
        n = self.q_lens.astype(np.float64)
        kv = self.kv_lens.astype(np.float64)
        pairs = n * (kv - n) + n * (n + 1) / 2      # decode: n = 1 -> kv pairs
        return float(4.0 * self.hq * HEAD_DIM * pairs.sum())


def _assign_pages(rng, lens, page_size, pool_pages=None, group_size=1, shared_tokens=0):
    """Give each sequence physical pages from a seeded permutation of the pool.

    Members of a group (consecutive ``group_size`` sequences) reference the
    same physical ids for their first ``shared_tokens // page_size`` pages.
    Returns (block_table, num_pages, poison_page).
    """
    b_count = len(lens)
    used = [-(-int(l) // page_size) for l in lens]
    shared = shared_tokens // page_size
    need = 0
    for b in range(b_count):
        own = used[b] - (shared if shared and b % group_size else 0)
        need += own
    pool = pool_pages if pool_pages is not None else need + 1
    if pool < need + 1:
        raise ValueError("pool too small")
    perm = rng.permutation(pool).astype(np.int32)
    max_pages = max(1, max(used))
    poison = int(perm[need])
    table = np.full((b_count, max_pages), poison, dtype=np.int32)
    nxt = 0
    for b in range(b_count):
        start = 0
        if shared and b % group_size:
            leader = b - b % group_size
            table[b, :shared] = table[leader, :shared]
            start = shared
        for j in range(start, used[b]):
            table[b, j] = perm[nxt]
            nxt += 1
    return table, pool, poison


def _assign_tree_pages(rng, lens, page_size, levels):
    """Pages for branching sessions: ``levels`` = [(block size, tokens), ...] with
    each block size dividing the one before. Consecutive members in blocks of the
    level-k size reference the same physical pages for that level's tokens,
    which follow the previous levels' tokens (all token counts multiples of the
    page size); the rest of each sequence has pages of its own. Page ids are a
    seeded permutation of the pool. Returns (block_table, num_pages, poison_page).
    """
    b_count = len(lens)
    used = [-(-int(l) // page_size) for l in lens]
    bounds, t = [], 0
    for size, tokens in levels:
        if tokens % page_size:
            raise ValueError("level tokens must be whole pages")
        bounds.append((size, t // page_size, (t + tokens) // page_size))
        t += tokens
    need = 0
    for b in range(b_count):
        for size, p0, p1 in bounds:
            if b % size == 0:
                need += max(0, min(used[b], p1) - p0)
        need += max(0, used[b] - bounds[-1][2])
    pool = need + 1
    perm = rng.permutation(pool).astype(np.int32)
    poison = int(perm[need])
    table = np.full((b_count, max(1, max(used))), poison, dtype=np.int32)
    nxt = 0
    for b in range(b_count):
        for size, p0, p1 in bounds:
            first = b - b % size
            for j in range(p0, min(used[b], p1)):
                if b == first:
                    table[b, j] = perm[nxt]
                    nxt += 1
                else:
                    table[b, j] = table[first, j]
        for j in range(bounds[-1][2], used[b]):
            table[b, j] = perm[nxt]
            nxt += 1
    return table, pool, poison


def decode_tiny(seed: int = 1001) -> Paged:
    """Batch 4, 8 query / 2 KV heads, contexts 128/256/384/512, page 16, pool of 256 pages."""
    rng = np.random.default_rng(seed)
    lens = np.array([128, 256, 384, 512], dtype=np.int32)
    table, pool, poison = _assign_pages(rng, lens, 16, pool_pages=256)
    return Paged("decode_tiny_b4_h8kv2_l128-512_p16", "decode", seed, 8, 2, 16, pool, table,
                 lens, np.ones(4, np.int32), poison)


def decode_uniform(seed: int = 1002) -> Paged:
    """Batch 64, 64 query / 8 KV heads, every context 8192 tokens, page 64, shuffled pool."""
    rng = np.random.default_rng(seed)
    lens = np.full(64, 8192, dtype=np.int32)
    table, pool, poison = _assign_pages(rng, lens, 64)
    return Paged("decode_uniform_b64_h64kv8_l8192_p64", "decode", seed, 64, 8, 64, pool, table,
                 lens, np.ones(64, np.int32), poison)


def decode_ragged(seed: int = 1003, sigma: float = 1.0) -> Paged:
    """Batch 128, 96 query / 8 KV heads, lognormal contexts (median 16K, sigma 1) clipped to [1K, 64K].

    K and V of KV head h are multiplied by s_h ~ U(0.5, 2) before rounding.
    """
    rng = np.random.default_rng(seed)
    x = rng.lognormal(mean=math.log(16384.0), sigma=sigma, size=128)
    lens = np.clip(np.rint(x), 1024, 65536).astype(np.int32)
    scales = rng.uniform(0.5, 2.0, size=8).astype(np.float32)
    table, pool, poison = _assign_pages(rng, lens, 64)
    return Paged("decode_ragged_b128_h96kv8_lognormal16k_1k-64k_p64", "decode", seed, 96, 8, 64, pool,
                 table, lens, np.ones(128, np.int32), poison, kv_head_scale=scales)


def decode_group_prefix(seed: int = 1004, shuffle: bool = False) -> Paged:
    """16 prompts x G=8 trajectories: a shared 4096-token prefix (same page ids per group)
    plus private continuations U{512..16384}; 64 query / 8 KV heads, page 64.

    ``shuffle`` permutes the batch order (a correctness variant; groups are then
    no longer contiguous in the batch).
    """
    rng = np.random.default_rng(seed)
    groups, g_size, shared = 16, 8, 4096
    priv = rng.integers(512, 16384, size=groups * g_size, endpoint=True)
    lens = (shared + priv).astype(np.int32)
    table, pool, poison = _assign_pages(rng, lens, 64, group_size=g_size, shared_tokens=shared)
    if shuffle:
        order = rng.permutation(len(lens))
        lens, table = lens[order], table[order]
    return Paged("decode_group_prefix_16x8_h64kv8_shared4096_priv512-16k_p64", "decode", seed, 64, 8,
                 64, pool, table, lens, np.ones(len(lens), np.int32), poison,
                 shared_prefix_pages=shared // 64, group_size=g_size)


def extend_multiturn(seed: int = 1005) -> Paged:
    """Batch 32, cached prefix U{8192..65536}, appended chunk U{64..2048}, 64 query / 8 KV heads, page 64."""
    rng = np.random.default_rng(seed)
    prefix = rng.integers(8192, 65536, size=32, endpoint=True)
    chunk = rng.integers(64, 2048, size=32, endpoint=True)
    kv = (prefix + chunk).astype(np.int32)
    table, pool, poison = _assign_pages(rng, kv, 64)
    return Paged("extend_multiturn_b32_h64kv8_prefix8k-64k_chunk64-2048_p64", "extend", seed, 64, 8, 64,
                 pool, table, kv, chunk.astype(np.int32), poison)


def decode_group_long_prefix(seed: int = 1006) -> Paged:
    """The group-prefix batch with long prompts: 16 prompts x G=8, shared prefix of 32768 tokens
    (far more than the GPU's last-level cache), private continuations U{512..4096}, 64/8 heads, page 64."""
    rng = np.random.default_rng(seed)
    shared = 32768
    lens = (shared + rng.integers(512, 4096, size=128, endpoint=True)).astype(np.int32)
    table, pool, poison = _assign_pages(rng, lens, 64, group_size=8, shared_tokens=shared)
    return Paged("decode_group_long_prefix_16x8_shared32768_h64kv8_p64", "decode", seed, 64, 8, 64, pool,
                 table, lens, np.ones(128, np.int32), poison, shared_prefix_pages=shared // 64, group_size=8)


def decode_branching(seed: int = 1007, shuffle: bool = False) -> Paged:
    """Branching sessions: 16 prompts x G=8 trajectories sharing a 4096-token prompt;
    each group branches into 2 subsets of 4 sharing the next 2048 tokens (a common
    turn), each of those into pairs sharing 1024 more; then private continuations
    U{512..4096}. 64 query / 8 KV heads, page 64. ``shuffle`` permutes the batch."""
    rng = np.random.default_rng(seed)
    levels = [(8, 4096), (4, 2048), (2, 1024)]
    priv = rng.integers(512, 4096, size=128, endpoint=True)
    lens = (4096 + 2048 + 1024 + priv).astype(np.int32)
    table, pool, poison = _assign_tree_pages(rng, lens, 64, levels)
    if shuffle:
        order = rng.permutation(len(lens))
        lens, table = lens[order], table[order]
    return Paged("decode_branching_16x8_tree4096-2048-1024_h64kv8_p64", "decode", seed, 64, 8, 64, pool,
                 table, lens, np.ones(len(lens), np.int32), poison, shared_prefix_pages=64, group_size=8)


def custom(seed: int, kind: str, kv_lens, q_lens=None, hq: int = 8, hkv: int = 2, page_size: int = 16,
           pool_extra: int = 3, group_size: int = 1, shared_tokens: int = 0, kv_head_scale=None,
           branches=None) -> Paged:
    """A small workload of any shape (tests). ``branches``: [(block size, tokens), ...]
    gives tree-shaped sharing (see _assign_tree_pages) instead of ``group_size`` /
    ``shared_tokens``."""
    rng = np.random.default_rng(seed)
    lens = np.asarray(kv_lens, dtype=np.int32)
    ql = np.ones(len(lens), np.int32) if q_lens is None else np.asarray(q_lens, dtype=np.int32)
    used = [-(-int(l) // page_size) for l in lens]
    need = sum(used) + 1
    if branches:
        table, pool, poison = _assign_tree_pages(rng, lens, page_size, branches)
        group_size, shared_tokens = branches[0]
    else:
        table, pool, poison = _assign_pages(rng, lens, page_size, pool_pages=need + pool_extra,
                                            group_size=group_size, shared_tokens=shared_tokens)
    scales = None if kv_head_scale is None else np.asarray(kv_head_scale, np.float32)
    return Paged(f"custom_{kind}_{seed}", kind, seed, hq, hkv, page_size, pool, table, lens, ql, poison,
                 kv_head_scale=scales, shared_prefix_pages=shared_tokens // page_size, group_size=group_size)


WORKLOADS = {
    "decode_tiny": decode_tiny,
    "decode_uniform": decode_uniform,
    "decode_ragged": decode_ragged,
    "decode_group_prefix": decode_group_prefix,
    "extend_multiturn": extend_multiturn,
}


def materialize(w: Paged, device="cpu", poison: bool = True, chunk_pages: int = 2048):
    """Build the tensors of a workload on ``device`` (torch).

    Returns a dict with q (bf16), k_pages, v_pages (bf16 ``[num_pages, P, Hkv, 128]``),
    block_table, kv_lens (int32), qo_indptr (int32, extend) and scale (float).
    """
    import torch

    dev = torch.device(device)

    def gen(tid):
        g = torch.Generator(device=dev)
        g.manual_seed(w.seed * 16 + tid)
        return g

    q_rows = w.batch if w.kind == "decode" else w.total_q
    q = torch.randn((q_rows, w.hq, HEAD_DIM), generator=gen(1), device=dev,
                    dtype=torch.float32).to(torch.bfloat16)
    pools = []
    head_scale = None
    if w.kv_head_scale is not None:
        head_scale = torch.tensor(w.kv_head_scale, device=dev, dtype=torch.float32).view(1, 1, -1, 1)
    for tid in (2, 3):
        g = gen(tid)
        pool = torch.empty((w.num_pages, w.page_size, w.hkv, HEAD_DIM), device=dev, dtype=torch.bfloat16)
        for p0 in range(0, w.num_pages, chunk_pages):
            p1 = min(w.num_pages, p0 + chunk_pages)
            x = torch.randn((p1 - p0, w.page_size, w.hkv, HEAD_DIM), generator=g, device=dev,
                            dtype=torch.float32)
            if head_scale is not None:
                x.mul_(head_scale)
            pool[p0:p1] = x.to(torch.bfloat16)
            del x
        pools.append(pool)
    k_pages, v_pages = pools
    if poison:
        poison_pages(w, k_pages, v_pages)
    out = {
        "q": q,
        "k_pages": k_pages,
        "v_pages": v_pages,
        "block_table": torch.from_numpy(w.block_table.copy()).to(dev),
        "kv_lens": torch.from_numpy(w.kv_lens.copy()).to(dev),
        "scale": float(np.float32(1.0 / math.sqrt(HEAD_DIM))),
    }
    if w.kind == "extend":
        out["qo_indptr"] = torch.from_numpy(w.qo_indptr.copy()).to(dev)
    return out


FP8_E4M3_MAX = 448.0


def materialize_fp8(w: Paged, device="cpu", poison: bool = True, chunk_pages: int = 2048):
    """Build a workload with FP8 E4M3 KV pages and per-KV-head scales.

    The bf16 pages of ``materialize`` (same seed, same values) are divided by
    a per-KV-head scale, amax over that head's pool / 448 (computed in float32),
    and cast to ``torch.float8_e4m3fn`` (torch's round-to-nearest-even cast);
    the returned ``k_scale`` / ``v_scale`` are those ``[Hkv]`` float32 scales.
    Poisoned rows hold the NaN code 0x7F. The bf16 pages are not returned.
    """
    import torch

    t = materialize(w, device, poison=False, chunk_pages=chunk_pages)
    for name in ("k_pages", "v_pages"):
        src = t.pop(name)
        amax = torch.zeros(w.hkv, device=src.device, dtype=torch.float32)
        for p0 in range(0, w.num_pages, chunk_pages):
            blk = src[p0:p0 + chunk_pages].float().abs()
            amax = torch.maximum(amax, blk.amax(dim=(0, 1, 3)))
            del blk
        scale = torch.where(amax > 0, amax / FP8_E4M3_MAX, torch.ones_like(amax))
        dst = torch.empty(src.shape, device=src.device, dtype=torch.float8_e4m3fn)
        inv = scale.view(1, 1, -1, 1)
        for p0 in range(0, w.num_pages, chunk_pages):
            x = src[p0:p0 + chunk_pages].float() / inv
            dst[p0:p0 + chunk_pages] = x.clamp_(-FP8_E4M3_MAX, FP8_E4M3_MAX).to(torch.float8_e4m3fn)
            del x
        del src
        t[name] = dst
        t[name.replace("pages", "scale")] = scale
    if poison:
        poison_pages(w, t["k_pages"].view(torch.uint8), t["v_pages"].view(torch.uint8), fill=0x7F)
    return t


def referenced_pages(w: Paged) -> np.ndarray:
    ids = set()
    for b in range(w.batch):
        used = -(-int(w.kv_lens[b]) // w.page_size)
        ids.update(int(x) for x in w.block_table[b, :used])
    return np.array(sorted(ids), dtype=np.int64)


def poison_pages(w: Paged, k_pages, v_pages, fill=float("nan")):
    """Fill unreferenced pages and the unused tail slots of last pages with NaN
    (``fill``: the value written, e.g. the E4M3 NaN code on a uint8 view)."""
    import torch

    dev = k_pages.device
    used = np.zeros(w.num_pages, dtype=bool)
    used[referenced_pages(w)] = True
    unused = torch.from_numpy(np.nonzero(~used)[0]).to(dev)
    nan = fill
    if unused.numel():
        k_pages.index_fill_(0, unused, nan)
        v_pages.index_fill_(0, unused, nan)
    # tail slots: a page is "full" for the purpose of poisoning only if every sequence
    # referencing it uses all of it; pages shared by several sequences are always full
    fill = {}
    for b in range(w.batch):
        l = int(w.kv_lens[b])
        used_pages = -(-l // w.page_size)
        for j in range(used_pages):
            n = min(w.page_size, l - j * w.page_size)
            pid = int(w.block_table[b, j])
            fill[pid] = max(fill.get(pid, 0), n)
    for pid, n in fill.items():
        if n < w.page_size:
            k_pages[pid, n:] = nan
            v_pages[pid, n:] = nan


def to_numpy_bits(t) -> np.ndarray:
    """bf16 torch tensor (any device) -> numpy uint16 bit patterns on the host."""
    import torch

    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


def compact_subset(w: Paged, tensors: dict, rows):
    """Host copy of the sequences ``rows`` of a workload with a compacted page pool.

    Used to check sampled sequences of full-size workloads against the oracle
    without copying the whole pool: the selected sequences' pages are copied
    (in block-table order) into a small pool and the block table is rewritten.
    Returns a dict of numpy arrays (bf16 as uint16 bits, FP8 E4M3 as uint8 codes).
    """
    import torch

    rows = [int(r) for r in rows]
    page_ids = []
    table = []
    index = {}
    for b in rows:
        used = -(-int(w.kv_lens[b]) // w.page_size)
        row = []
        for pid in w.block_table[b, :used]:
            pid = int(pid)
            if pid not in index:
                index[pid] = len(page_ids)
                page_ids.append(pid)
            row.append(index[pid])
        table.append(row)
    width = max(1, max(len(r) for r in table))
    bt = np.zeros((len(rows), width), dtype=np.int32)
    for i, r in enumerate(table):
        bt[i, :len(r)] = r
    ids = torch.tensor(page_ids if page_ids else [0], dtype=torch.long, device=tensors["k_pages"].device)
    def page_bits(t):
        if t.dtype == torch.float8_e4m3fn:
            return t.view(torch.uint8).index_select(0, ids).cpu().numpy()
        return to_numpy_bits(t.index_select(0, ids))

    k = page_bits(tensors["k_pages"])
    v = page_bits(tensors["v_pages"])
    res = {"k_pages": k, "v_pages": v, "block_table": bt,
           "kv_lens": w.kv_lens[rows].copy(), "q_lens": w.q_lens[rows].copy()}
    if w.kind == "decode":
        res["q"] = to_numpy_bits(tensors["q"][torch.tensor(rows, device=tensors["q"].device)])
    else:
        indptr = w.qo_indptr
        q_rows = np.concatenate([np.arange(indptr[b], indptr[b + 1]) for b in rows]).astype(np.int64)
        res["q"] = to_numpy_bits(tensors["q"][torch.from_numpy(q_rows).to(tensors["q"].device)])
        res["qo_indptr"] = np.concatenate([[0], np.cumsum(w.q_lens[rows])]).astype(np.int32)
        res["q_rows"] = q_rows
    return res
