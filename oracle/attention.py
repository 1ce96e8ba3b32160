"""Plain float64 softmax attention over a paged KV cache (test infrastructure).

Every function here is the textbook definition written out with numpy; there is
no tiling, splitting, fusion or reordering beyond what the definition states.
Matrix products over one (sequence, KV head) use numpy's matmul as a library
step. The paper only describes the workload this serves (see the package
docstring); the formulas are scaled dot-product attention (Vaswani et al.,
2017) with grouped-query head sharing.

Conventions (readings where the paper is silent):

* bf16 tensors arrive as ``uint16`` bit patterns and are widened exactly to
  float64; float arrays are taken as given. An FP8 KV cache arrives as
  ``uint8`` OCP E4M3 codes with one dequantisation scale per KV head (the
  case-study rollout engines serve an FP8 key-value cache, section "Case
  Study", subsection "Configuration", and its configuration table); the
  oracle decodes the codes exactly and multiplies by the scale.
* Query head ``h`` of ``Hq`` reads KV head ``h // (Hq // Hkv)``.
* Scores are ``scale * (q . k)`` with ``scale`` first rounded to float32 (the
  ABI passes a float32); the log-sum-exp is in natural log and includes the
  scale.
* Logical token ``t`` of sequence ``b`` lives in physical page
  ``block_table[b, t // P]`` at slot ``t % P``; tokens are gathered in logical
  order, so the result does not depend on the page size or the physical order
  of pages.
* Extend: row ``i`` of a chunk of ``n`` tokens whose sequence holds ``kv``
  tokens in total (prefix ``p = kv - n`` plus the chunk, whose K/V are already
  in the pages) attends to tokens ``t <= p + i`` (bottom-right causal mask).
* An empty key range yields output 0 and log-sum-exp ``-inf``.
"""

from __future__ import annotations

import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) to float64 exactly; pass floats through."""
    a = np.asarray(bits)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if a.dtype == np.int16:
        return bf16_bits_to_f64(a.view(np.uint16))
    return a.astype(np.float64)


def fp8_e4m3_to_f64(bits: np.ndarray) -> np.ndarray:
    """Decode OCP FP8 E4M3 codes (uint8) to float64, from the format's definition.

    A code is ``s eeee mmm`` with exponent bias 7: ``e == 0`` encodes the
    subnormals ``(-1)^s * 2^-6 * m/8``; ``e == 15, m == 7`` encodes NaN (the
    format has no infinities); every other code is ``(-1)^s * 2^(e-7) * (1 + m/8)``
    (largest finite magnitude 448).
    """
    b = np.asarray(bits, dtype=np.uint8).astype(np.int64)
    sign = np.where(b & 0x80, -1.0, 1.0)
    e = (b >> 3) & 0xF
    m = (b & 0x7).astype(np.float64)
    normal = np.ldexp(1.0 + m / 8.0, (e - 7).astype(np.int64))
    sub = np.ldexp(m / 8.0, -6)
    val = np.where(e == 0, sub, normal)
    val = np.where((e == 15) & (b & 0x7 == 7), np.nan, val)
    return sign * val


def kv_to_f64(x: np.ndarray) -> np.ndarray:
    """KV elements to float64: uint8 arrays are FP8 E4M3 codes, anything else goes to bf16_bits_to_f64."""
    a = np.asarray(x)
    if a.dtype == np.uint8:
        return fp8_e4m3_to_f64(a)
    return bf16_bits_to_f64(a)


def gather_head(pages: np.ndarray, block_row: np.ndarray, length: int, g: int, head_scale=None) -> np.ndarray:
    """Rows ``0..length-1`` of KV head ``g`` of one sequence, in logical order.

    ``pages`` is ``[num_pages, P, Hkv, D]`` (bf16 bit patterns, or FP8 E4M3
    codes as uint8); ``block_row`` is the sequence's block-table row. Token
    ``t`` comes from page ``block_row[t // P]``, slot ``t % P``. With
    ``head_scale`` (one dequantisation scale per KV head) an element stands
    for its decoded value times ``head_scale[g]``. Returns float64 ``[length, D]``.
    """
    page_size = pages.shape[1]
    d = pages.shape[3]
    out = np.empty((length, d), dtype=np.float64)
    for t in range(0, length, page_size):
        page = int(block_row[t // page_size])
        take = min(page_size, length - t)
        out[t:t + take] = kv_to_f64(pages[page, :take, g, :])
    if head_scale is not None:
        out *= np.float64(head_scale[g])
    return out


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float):
    """softmax(scale * q k^T) v for query rows ``q [R, D]`` over keys ``k, v [L, D]``.

    Returns ``(o [R, D], lse [R])`` in float64. ``L == 0`` gives ``o = 0`` and
    ``lse = -inf``.
    """
    q = np.atleast_2d(np.asarray(q, dtype=np.float64))
    rows, d = q.shape
    if k.shape[0] == 0:
        return np.zeros((rows, d)), np.full(rows, -np.inf)
    s = np.float64(np.float32(scale)) * (q @ k.T)          # [R, L]
    m = s.max(axis=1, keepdims=True)
    w = np.exp(s - m)
    z = w.sum(axis=1)
    o = (w @ v) / z[:, None]
    lse = m[:, 0] + np.log(z)
    return o, lse


def attend_range(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float, t0: int, t1: int):
    """Attention restricted to keys ``t0 <= t < t1`` (one split-KV partial)."""
    return attend(q, k[t0:t1], v[t0:t1], scale)


def _masked_attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float, limits: np.ndarray):
    """Row ``r`` of ``q`` attends to keys ``t <= limits[r]`` (limits >= 0)."""
    s = np.float64(np.float32(scale)) * (q @ k.T)
    t = np.arange(k.shape[0])
    s = np.where(t[None, :] <= limits[:, None], s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    w = np.exp(s - m)
    z = w.sum(axis=1)
    o = (w @ v) / z[:, None]
    lse = m[:, 0] + np.log(z)
    return o, lse


def decode(q, k_pages, v_pages, block_table, seq_lens, scale, k_scale=None, v_scale=None):
    """Batched decode: ``out[b, h] = softmax_t(scale q[b,h] . K_b[t, g]) V_b[t, g]``, t < L_b.

    q ``[B, Hq, D]``; k_pages/v_pages ``[num_pages, P, Hkv, D]`` (bf16, or FP8
    E4M3 codes with per-KV-head dequantisation scales ``k_scale``/``v_scale``
    of shape ``[Hkv]``); block_table ``[B, max_pages]``; seq_lens ``[B]``.
    Returns ``(out [B, Hq, D], lse [B, Hq])`` float64.
    """
    qf = bf16_bits_to_f64(q)
    b_count, hq, d = qf.shape
    hkv = k_pages.shape[2]
    r = hq // hkv
    out = np.zeros((b_count, hq, d))
    lse = np.full((b_count, hq), -np.inf)
    for b in range(b_count):
        length = int(seq_lens[b])
        for g in range(hkv):
            k = gather_head(k_pages, block_table[b], length, g, k_scale)
            v = gather_head(v_pages, block_table[b], length, g, v_scale)
            o, l = attend(qf[b, g * r:(g + 1) * r], k, v, scale)
            out[b, g * r:(g + 1) * r] = o
            lse[b, g * r:(g + 1) * r] = l
    return out, lse


def extend(q, qo_indptr, k_pages, v_pages, block_table, kv_lens, scale, row_block: int = 32, k_scale=None,
           v_scale=None):
    """Causal extend over a paged cache (pages and scales as in ``decode``).

    q ``[total_q, Hq, D]``; sequence ``b`` owns query rows
    ``qo_indptr[b] .. qo_indptr[b+1]-1`` (n_b of them) and holds ``kv_lens[b]``
    tokens in its pages, the last n_b of which are the chunk itself. Chunk row
    ``i`` attends to tokens ``t <= kv_b - n_b + i``. ``row_block`` only bounds
    memory (chunk rows are independent of each other).
    Returns ``(out [total_q, Hq, D], lse [total_q, Hq])`` float64.
    """
    qf = bf16_bits_to_f64(q)
    total_q, hq, d = qf.shape
    hkv = k_pages.shape[2]
    r = hq // hkv
    out = np.zeros((total_q, hq, d))
    lse = np.full((total_q, hq), -np.inf)
    for b in range(len(kv_lens)):
        q0, q1 = int(qo_indptr[b]), int(qo_indptr[b + 1])
        n = q1 - q0
        if n <= 0:
            continue
        kv = int(kv_lens[b])
        prefix = kv - n
        for g in range(hkv):
            k = gather_head(k_pages, block_table[b], kv, g, k_scale)
            v = gather_head(v_pages, block_table[b], kv, g, v_scale)
            for i0 in range(0, n, row_block):
                i1 = min(n, i0 + row_block)
                rows = qf[q0 + i0:q0 + i1, g * r:(g + 1) * r].reshape(-1, d)   # token-major
                limits = np.repeat(prefix + np.arange(i0, i1), r)
                reach = prefix + i1            # keys beyond the last row's limit are unused
                o, l = _masked_attend(rows, k[:reach], v[:reach], scale, limits)
                out[q0 + i0:q0 + i1, g * r:(g + 1) * r] = o.reshape(i1 - i0, r, d)
                lse[q0 + i0:q0 + i1, g * r:(g + 1) * r] = l.reshape(i1 - i0, r)
    return out, lse


def merge(o_parts, lse_parts, num_parts):
    """Log-sum-exp merge of attention results over disjoint key ranges.

    o_parts ``[N, S, H, D]``, lse_parts ``[N, S, H]``, num_parts ``[N]`` (only
    the first ``num_parts[n]`` parts of row n count). With
    ``M = max_s lse_s`` and ``w_s = exp(lse_s - M)``:
    ``out = sum_s w_s o_s / sum_s w_s`` and ``lse = M + log sum_s w_s``.
    Parts with ``lse = -inf`` carry no weight; if every part is empty the
    result is ``out = 0``, ``lse = -inf``.
    """
    o_parts = np.asarray(o_parts, dtype=np.float64)
    lse_parts = np.asarray(lse_parts, dtype=np.float64)
    n_rows, _, h, d = o_parts.shape
    out = np.zeros((n_rows, h, d))
    lse = np.full((n_rows, h), -np.inf)
    for n in range(n_rows):
        s_count = int(num_parts[n])
        for hh in range(h):
            ls = lse_parts[n, :s_count, hh]
            if s_count == 0 or not np.any(ls > -np.inf):
                continue
            m = ls.max()
            w = np.exp(ls - m)
            z = w.sum()
            out[n, hh] = (w[:, None] * o_parts[n, :s_count, hh]).sum(axis=0) / z
            lse[n, hh] = m + np.log(z)
    return out, lse
