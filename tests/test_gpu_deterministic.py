"""Deterministic decode and the invariance of extend rows (through the C-ABI).

The paper's true-on-policy alignment (section "True-On-Policy Alignment")
needs attention whose prefill and decode paths agree bitwise and whose results
do not depend on the batch. Checked here: deterministic decode equals extend
of the same token bitwise; its result for a sequence is the same in any batch;
an extend row gives the same bits whether its chunk is prefilled at once or
appended one token at a time; and the results match the oracle.
"""

import numpy as np
import pytest
import torch

from paper_2609_08368_amd import rl_attn as ra
from paper_2609_08368_amd import workloads as wl
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def det_decode(t, rows=None, fp8=False, out_dtype=torch.bfloat16):
    """Deterministic decode of all sequences (or of the batch made of ``rows``)."""
    q, bt, lens = t["q"], t["block_table"], t["kv_lens"]
    if rows is not None:
        idx = torch.tensor(rows, device=DEV)
        q, bt, lens = q[idx].contiguous(), bt[idx].contiguous(), lens[idx].contiguous()
    out = H.poison_like(torch.empty(q.shape, dtype=out_dtype, device=DEV))
    lse = H.poison_like(torch.empty(q.shape[:2], dtype=torch.float32, device=DEV))
    if fp8:
        ra.decode_fp8(q, t["k_pages"], t["v_pages"], t["k_scale"], t["v_scale"], bt, lens, t["scale"], out=out,
                      lse=lse, deterministic=True)
    else:
        ra.decode(q, t["k_pages"], t["v_pages"], bt, lens, t["scale"], out=out, lse=lse, deterministic=True)
    torch.cuda.synchronize()
    return out, lse


def one_row_extend(t, fp8=False):
    """Extend with one chunk token per sequence (kv_lens = decode lengths)."""
    q = t["q"]
    B = q.shape[0]
    e = dict(t)
    e["qo_indptr"] = torch.arange(B + 1, dtype=torch.int32, device=DEV)
    lens = t["kv_lens"]
    # sequences with no keys have no chunk token (an empty chunk)
    if bool((lens == 0).any()):
        keep = (lens > 0).to(torch.int32)
        e["qo_indptr"] = torch.cat([torch.zeros(1, dtype=torch.int32, device=DEV), keep.cumsum(0).to(torch.int32)])
        e["q"] = q[lens > 0].contiguous()
    out = H.poison_like(torch.empty(e["q"].shape, dtype=torch.bfloat16, device=DEV))
    lse = H.poison_like(torch.empty(e["q"].shape[:2], dtype=torch.float32, device=DEV))
    if fp8:
        ra.extend_fp8(e["q"], e["qo_indptr"], t["k_pages"], t["v_pages"], t["k_scale"], t["v_scale"],
                      t["block_table"], lens, t["scale"], out=out, lse=lse)
    else:
        ra.extend(e["q"], e["qo_indptr"], t["k_pages"], t["v_pages"], t["block_table"], lens, t["scale"], out=out,
                  lse=lse)
    torch.cuda.synchronize()
    return out, lse, lens > 0


def bits_equal(a, b):
    if a.dtype == torch.bfloat16:
        return torch.equal(a.view(torch.int16), b.view(torch.int16))
    return torch.equal(a.view(torch.int32), b.view(torch.int32))


CASES = [
    # (page_size, Hq, Hkv, lens)
    (16, 8, 2, [1, 15, 16, 17, 100, 300, 0]),
    (64, 96, 8, [63, 64, 65, 700, 1]),
    (32, 2, 2, [1, 31, 33, 250]),              # one query head per KV head
    (128, 40, 2, [129, 5, 400]),               # 20 query heads per KV head
    (8, 12, 3, [7, 8, 9, 200]),
]


@pytest.mark.parametrize("fp8", [False, True])
@pytest.mark.parametrize("case", CASES, ids=[f"P{c[0]}_h{c[1]}kv{c[2]}" for c in CASES])
def test_deterministic_decode_matches_oracle_and_extend(case, fp8):
    ps, hq, hkv, lens = case
    w = wl.custom(120 + hq, "decode", lens, hq=hq, hkv=hkv, page_size=ps)
    H.say(f"deterministic decode {case} fp8={fp8}")
    t = (wl.materialize_fp8 if fp8 else wl.materialize)(w, DEV)
    out, lse = det_decode(t, fp8=fp8)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what=f"deterministic {case}")
    eo, el, nonempty = one_row_extend(t, fp8=fp8)
    assert bits_equal(out[nonempty], eo), "deterministic decode != extend of the same token"
    assert bits_equal(lse[nonempty], el), "deterministic decode lse != extend lse"
    empty = ~nonempty
    assert torch.all(out[empty] == 0) and torch.all(torch.isneginf(lse[empty]))


def test_deterministic_decode_f32_output():
    w = wl.custom(131, "decode", [90, 0, 513], hq=16, hkv=4, page_size=16)
    H.say("deterministic decode, f32 out")
    t = wl.materialize(w, DEV)
    out, lse = det_decode(t, out_dtype=torch.float32)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what="deterministic f32")
    assert torch.all(out[1] == 0)


def test_deterministic_decode_is_batch_invariant():
    """A sequence's bits do not depend on the batch it is decoded in (size, order, partners)."""
    rng = np.random.default_rng(5)
    lens = rng.integers(1, 3000, size=24).tolist()
    w = wl.custom(132, "decode", lens, hq=32, hkv=4, page_size=64)
    H.say("batch invariance")
    t = wl.materialize(w, DEV)
    full_o, full_l = det_decode(t)
    for rows in ([5], [23, 0, 5, 7], list(range(23, -1, -1)), [5, 5, 11], list(range(0, 24, 3))):
        o, l = det_decode(t, rows=rows)
        idx = torch.tensor(rows, device=DEV)
        assert bits_equal(o, full_o[idx]), f"rows {rows}: outputs depend on the batch"
        assert bits_equal(l, full_l[idx]), f"rows {rows}: lse depends on the batch"
    # the default split-KV decode agrees within the path's tolerance
    d_o, d_l = H.run_decode(w, t)
    H.compare(full_o, H.f64(d_o), max_abs=2e-2, rel_rms=5e-3, what="deterministic vs split decode")


@pytest.mark.parametrize("ps", [16, 64])
def test_extend_prefill_equals_token_by_token(ps):
    """True-on-policy rescoring: prefilling a chunk gives each row the bits that appending
    its tokens one at a time (extend with one token, and deterministic decode) gives."""
    prefix, n = 700, 300
    w = wl.custom(133, "extend", [prefix + n, 90 + 40], q_lens=[n, 40], hq=24, hkv=2, page_size=ps)
    H.say(f"prefill vs token-by-token P={ps}")
    t = wl.materialize(w, DEV)
    out, lse = H.run_extend(w, t)
    indptr = w.qo_indptr
    for b in range(w.batch):
        nb, kv = int(w.q_lens[b]), int(w.kv_lens[b])
        rows = torch.arange(int(indptr[b]), int(indptr[b + 1]), device=DEV)
        q_b = t["q"][rows].contiguous()
        # each token appended on its own: kv length prefix + i + 1
        lens_i = torch.arange(kv - nb + 1, kv + 1, dtype=torch.int32, device=DEV)
        bt_i = t["block_table"][b:b + 1].expand(nb, -1).contiguous()
        step = {"q": q_b, "k_pages": t["k_pages"], "v_pages": t["v_pages"], "block_table": bt_i,
                "kv_lens": lens_i, "scale": t["scale"]}
        dec_o, dec_l = det_decode(step)
        assert bits_equal(dec_o, out[rows]), f"seq {b}: prefill rows != token-by-token decode"
        assert bits_equal(dec_l, lse[rows]), f"seq {b}: prefill lse != token-by-token decode"
        # and a chunk split in two extend calls
        half = nb // 2
        for lo, hi in ((0, half), (half, nb)):
            if hi == lo:
                continue
            ext = {"q": q_b[lo:hi].contiguous(), "qo_indptr": torch.tensor([0, hi - lo], dtype=torch.int32, device=DEV),
                   "k_pages": t["k_pages"], "v_pages": t["v_pages"], "block_table": t["block_table"][b:b + 1].contiguous(),
                   "kv_lens": torch.tensor([kv - nb + hi], dtype=torch.int32, device=DEV), "scale": t["scale"]}
            eo, el = H.run_extend(None, ext)
            assert bits_equal(eo, out[rows[lo:hi]]), f"seq {b}: chunk split changes the bits"
            assert bits_equal(el, lse[rows[lo:hi]])
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what="prefill")


def test_deterministic_decode_full_size_sampled():
    """The ragged 64K batch in deterministic mode: sampled sequences vs the oracle."""
    w = wl.decode_ragged()
    H.say(f"deterministic full size: B={w.batch} sum(L)={int(w.kv_lens.sum())}")
    t = wl.materialize(w, DEV)
    out, lse = det_decode(t)
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
    order = np.argsort(w.kv_lens, kind="stable")
    rows = sorted({int(order[0]), int(order[-1]), int(order[len(order) // 2]), 3})
    ref_o, ref_l = H.oracle_decode_rows(w, t, rows)
    sel = torch.tensor(rows, device=DEV)
    res = H.compare(out[sel], ref_o, lse[sel], ref_l, what="deterministic ragged")
    H.say(f"  rows={rows} {res}")
    # batch invariance at full size: the longest sequence alone
    lo, ll = det_decode(t, rows=[int(order[-1])])
    assert bits_equal(lo[0], out[int(order[-1])]) and bits_equal(ll[0], lse[int(order[-1])])
    del t
    torch.cuda.empty_cache()
