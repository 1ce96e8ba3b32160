"""Randomised properties of the oracle (CPU only, hypothesis): over drawn batch
sizes, GQA shapes, page sizes, physical page orders and lengths (empty
sequences and empty chunks included), the paged oracle equals textbook dense
attention computed independently with scipy on unpaged tensors, decode and
extend alike."""

import numpy as np
import scipy.special
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle
from tests.oracle_pins import D, from_bits, pack_pages, to_bf16_bits

GQA = [(1, 1), (2, 1), (4, 2), (6, 3), (8, 2), (8, 8), (12, 4)]


def _pack_v(v, lens, bt, kp_shape, ps):
    vp = np.full(kp_shape, 0x7FC0, dtype=np.uint16)
    for b in range(len(lens)):
        for j in range(-(-int(lens[b]) // ps)):
            take = min(ps, int(lens[b]) - j * ps)
            vp[bt[b, j], :take] = v[b, j * ps:j * ps + take]
    return vp


def _dense_rows(q_rows, k, v, limits, scale):
    """Rows of q [n, Hq, D] (floats) over dense k/v [L, Hkv, D]; row i sees keys t <= limits[i]."""
    n, hq, _ = q_rows.shape
    r = hq // k.shape[1]
    kk = np.repeat(k, r, axis=1)
    vv = np.repeat(v, r, axis=1)
    out = np.zeros((n, hq, D))
    lse = np.full((n, hq), -np.inf)
    for i in range(n):
        m = int(limits[i]) + 1
        if m <= 0:
            continue
        s = np.einsum("hd,thd->ht", q_rows[i], kk[:m]) * float(np.float32(scale))
        out[i] = np.einsum("ht,thd->hd", scipy.special.softmax(s, axis=1), vv[:m])
        lse[i] = scipy.special.logsumexp(s, axis=1)
    return out, lse


def _close(a, b, tol=1e-11):
    return np.max(np.abs(a - b), initial=0.0) <= tol * max(1.0, np.max(np.abs(b), initial=0.0))


@settings(max_examples=30, deadline=None)
@given(seed=st.integers(0, 2**31 - 1), gqa=st.sampled_from(GQA), ps=st.sampled_from([1, 4, 8, 16, 64]),
       lens=st.lists(st.integers(0, 80), min_size=1, max_size=4), scale=st.floats(0.01, 0.5))
def test_decode_equals_dense_attention(seed, gqa, ps, lens, scale):
    rng = np.random.default_rng(seed)
    hq, hkv = gqa
    lens = np.array(lens, dtype=np.int32)
    lmax = max(1, int(lens.max()))
    q = to_bf16_bits(rng.standard_normal((len(lens), hq, D)))
    k = to_bf16_bits(rng.standard_normal((len(lens), lmax, hkv, D)))
    v = to_bf16_bits(rng.standard_normal((len(lens), lmax, hkv, D)))
    kp, bt = pack_pages(k, lens, ps, rng, extra_pages=int(rng.integers(1, 4)))
    vp = _pack_v(v, lens, bt, kp.shape, ps)
    out, lse = oracle.decode(q, kp, vp, bt, lens, scale)
    for b in range(len(lens)):
        ref_o, ref_l = _dense_rows(from_bits(q[b:b + 1]), from_bits(k[b]), from_bits(v[b]),
                                   np.array([int(lens[b]) - 1]), scale)
        assert _close(out[b], ref_o[0]), f"decode of sequence {b} != dense attention"
        assert np.array_equal(np.isneginf(lse[b]), np.isneginf(ref_l[0]))
        fin = np.isfinite(ref_l[0])
        assert _close(lse[b][fin], ref_l[0][fin]), f"lse of sequence {b} != scipy logsumexp"


@settings(max_examples=30, deadline=None)
@given(seed=st.integers(0, 2**31 - 1), gqa=st.sampled_from(GQA), ps=st.sampled_from([1, 8, 16]),
       shape=st.lists(st.tuples(st.integers(0, 40), st.integers(0, 12)), min_size=1, max_size=3),
       row_block=st.sampled_from([1, 3, 32]))
def test_extend_equals_dense_causal_attention(seed, gqa, ps, shape, row_block):
    rng = np.random.default_rng(seed)
    hq, hkv = gqa
    prefix = np.array([p for p, _ in shape], dtype=np.int32)
    n = np.array([c for _, c in shape], dtype=np.int32)
    kv = prefix + n
    indptr = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    lmax = max(1, int(kv.max()))
    q = to_bf16_bits(rng.standard_normal((int(n.sum()), hq, D)))
    k = to_bf16_bits(rng.standard_normal((len(shape), lmax, hkv, D)))
    v = to_bf16_bits(rng.standard_normal((len(shape), lmax, hkv, D)))
    kp, bt = pack_pages(k, kv, ps, rng)
    vp = _pack_v(v, kv, bt, kp.shape, ps)
    out, lse = oracle.extend(q, indptr, kp, vp, bt, kv, 0.0883883, row_block=row_block)
    for b in range(len(shape)):
        rows = slice(int(indptr[b]), int(indptr[b + 1]))
        limits = int(prefix[b]) + np.arange(int(n[b]))          # bottom-right causal
        ref_o, ref_l = _dense_rows(from_bits(q[rows]), from_bits(k[b]), from_bits(v[b]), limits, 0.0883883)
        assert _close(out[rows], ref_o), f"extend of sequence {b} != dense causal attention"
        assert _close(lse[rows], ref_l), f"extend lse of sequence {b} != scipy logsumexp"
