"""KV append, written out plainly (test infrastructure).

Each agentic turn prefills only its newly appended suffix and every decode
step adds one token (paper, section "Fast Agentic Rollout with SGLang"), so
before attention reads them the new tokens' K and V rows are written into
their pages. Addressing follows the attention calls: sequence b owns the new
rows ``qo_indptr[b] .. qo_indptr[b+1]-1`` (n_b rows, in order) and holds
``kv_lens[b]`` tokens after the append, so new row i goes to logical position
``kv_lens[b] - n_b + i``, i.e. page ``block_table[b, t // P]``, slot ``t % P``.

bf16 pages receive the rows unchanged. FP8 pages (the case study's FP8 KV
cache, section "Case Study", subsection "Configuration"; format and scaling
are a reading, the paper gives neither) receive OCP E4M3 codes: the quotient
``x / scale[g]`` is formed in float32 (the precision in which the kernel
takes the same integer decision), then rounded to the nearest E4M3 value,
ties to the even code, magnitudes above 448 saturating to 448 and NaN giving
the NaN code with the input's sign.
"""

from __future__ import annotations

import numpy as np

from .attention import fp8_e4m3_to_f64

# the finite non-negative E4M3 values in code order 0x00 .. 0x7E (increasing)
_FINITE = fp8_e4m3_to_f64(np.arange(0x7F, dtype=np.uint8))


def fp8_e4m3_encode(x) -> np.ndarray:
    """Nearest OCP E4M3 code of each float32 value (ties to the even code), by
    search over the format's value table; saturating at 448."""
    x = np.asarray(x, dtype=np.float32)
    a = np.abs(x.astype(np.float64)).ravel()
    nan = np.isnan(a)
    a = np.where(nan, 0.0, np.minimum(a, 448.0))
    hi = np.searchsorted(_FINITE, a, side="left")       # first value >= a
    hi = np.minimum(hi, len(_FINITE) - 1)
    lo = np.maximum(hi - 1, 0)
    d_lo = a - _FINITE[lo]
    d_hi = _FINITE[hi] - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    code = np.where(pick_hi, hi, lo).astype(np.uint8)
    code = np.where(nan, np.uint8(0x7F), code)
    sign = np.signbit(x.ravel()).astype(np.uint8) << 7
    return (code | sign).astype(np.uint8).reshape(x.shape)


def quantize_rows(rows_bits: np.ndarray, head_scale) -> np.ndarray:
    """bf16 rows ``[..., Hkv, D]`` (uint16 bits) -> E4M3 codes of ``x / scale[g]`` (quotient in float32)."""
    x = (np.asarray(rows_bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)
    s = np.asarray(head_scale, dtype=np.float32).reshape((1,) * (x.ndim - 2) + (-1, 1))
    q = (x / s).astype(np.float32)                       # float32 division, correctly rounded
    return fp8_e4m3_encode(q)


def append_kv(k_pages, v_pages, block_table, kv_lens, qo_indptr, k_new, v_new, k_scale=None, v_scale=None):
    """Return copies of the pages with the new rows written.

    ``k_pages``/``v_pages``: ``[num_pages, P, Hkv, D]`` uint16 (bf16 bits) or
    uint8 (E4M3 codes, then ``k_scale``/``v_scale`` give the per-KV-head
    scales); ``k_new``/``v_new``: ``[total_new, Hkv, D]`` uint16 (bf16 bits).
    """
    kp = np.array(k_pages, copy=True)
    vp = np.array(v_pages, copy=True)
    fp8 = kp.dtype == np.uint8
    if fp8:
        k_rows = quantize_rows(k_new, k_scale)
        v_rows = quantize_rows(v_new, v_scale)
    else:
        k_rows, v_rows = np.asarray(k_new), np.asarray(v_new)
    page_size = kp.shape[1]
    for b in range(len(kv_lens)):
        q0, q1 = int(qo_indptr[b]), int(qo_indptr[b + 1])
        n = q1 - q0
        for i in range(n):
            t = int(kv_lens[b]) - n + i
            page = int(block_table[b, t // page_size])
            kp[page, t % page_size] = k_rows[q0 + i]
            vp[page, t % page_size] = v_rows[q0 + i]
    return kp, vp
