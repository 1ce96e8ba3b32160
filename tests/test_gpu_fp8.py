"""FP8 E4M3 KV pages on the GPU (through the C-ABI) against the float64 oracle.

The oracle decodes each code exactly and multiplies by its KV head's scale;
the kernels convert codes exactly to bf16 and fold the K scale into the
softmax scale and the V scale into the output, so the path's error is the
same as with bf16 pages and the same tolerances apply.
"""

import numpy as np
import pytest
import torch

from paper_2609_08368_amd import rl_attn as ra
from paper_2609_08368_amd import workloads as wl
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

DECODE_CASES = [
    # (page_size, Hq, Hkv, lens, split)
    (16, 8, 2, [1, 15, 16, 17, 100, 300], 0),
    (16, 8, 2, [1, 15, 16, 17, 100, 300], 64),
    (8, 12, 1, [7, 8, 9, 64, 65, 129], 64),
    (64, 64, 8, [63, 64, 65, 200, 1], 0),
    (128, 16, 1, [127, 128, 129, 400], 128),
    (32, 2, 2, [1, 31, 33, 250], 64),        # one query head per KV head: vector-ALU path
    (16, 40, 2, [50, 190], 64),              # two 16-head blocks
    (16, 8, 2, [0, 20, 0, 1], 0),            # empty sequences
    (32, 24, 2, [31, 32, 33, 97, 600], 64),  # pages of exactly one 32-key tile: whole-row loads
    (64, 96, 8, [5, 130, 257, 2000], 0),     # the agentic head shape
]


@pytest.mark.parametrize("case", DECODE_CASES, ids=[f"P{c[0]}_h{c[1]}kv{c[2]}_s{c[4]}_{i}"
                                                    for i, c in enumerate(DECODE_CASES)])
def test_fp8_decode_shapes(case):
    ps, hq, hkv, lens, split = case
    w = wl.custom(61 + len(lens), "decode", lens, hq=hq, hkv=hkv, page_size=ps)
    H.say(f"fp8 decode case {case}")
    t = wl.materialize_fp8(w, DEV)
    out, lse = H.run_decode(w, t, split_tokens=split)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what=f"fp8 {case}")


PREFIX_CASES = [
    # (page_size, Hq, Hkv, group_size, groups, shared_tokens, private lens, split)
    (64, 64, 8, 8, 2, 4096, [512, 700, 1000, 64, 3, 200, 900, 513], 0),
    (16, 8, 2, 4, 2, 60, [1, 30, 70, 2], 64),
    (16, 2, 2, 3, 2, 48, [10, 0, 5], 0),
]


@pytest.mark.parametrize("case", PREFIX_CASES, ids=[f"P{c[0]}_h{c[1]}kv{c[2]}_G{c[3]}" for c in PREFIX_CASES])
@pytest.mark.parametrize("share", [True, False])
def test_fp8_decode_group_prefix(case, share):
    ps, hq, hkv, gs, ng, shared, priv, split = case
    lens = [shared + priv[j % len(priv)] + 7 * g for g in range(ng) for j in range(gs)]
    w = wl.custom(70 + gs, "decode", lens, hq=hq, hkv=hkv, page_size=ps, group_size=gs, shared_tokens=shared)
    H.say(f"fp8 prefix case {case} share={share}")
    t = wl.materialize_fp8(w, DEV)
    out, lse = H.run_decode(w, t, split_tokens=split, prefix_share=share)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what=f"fp8 {case} share={share}")


EXTEND_CASES = [
    # (page_size, Hq, Hkv, kv_lens, q_lens)
    (16, 8, 2, [300, 129, 64], [129, 100, 16]),      # per-row page lookups
    (64, 64, 8, [500, 70], [33, 70]),                # one scalar page lookup per step
    (128, 8, 1, [600], [257]),
    (32, 16, 16, [200, 50], [150, 7]),               # one query head per KV head
    (16, 8, 2, [30, 0, 12], [0, 0, 12]),             # empty chunks
    (8, 12, 3, [90, 13, 200], [20, 13, 70]),         # pages of 8 keys: eight pages per 64-key step
]


@pytest.mark.parametrize("case", EXTEND_CASES, ids=[f"P{c[0]}_h{c[1]}kv{c[2]}_{i}" for i, c in enumerate(EXTEND_CASES)])
def test_fp8_extend_shapes(case):
    ps, hq, hkv, kv, ql = case
    w = wl.custom(81 + sum(ql), "extend", kv, q_lens=ql, hq=hq, hkv=hkv, page_size=ps)
    H.say(f"fp8 extend case {case}")
    t = wl.materialize_fp8(w, DEV)
    out, lse = H.run_extend(w, t)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what=f"fp8 {case}")


def _pow2_pair(w, seed_scale=True):
    """FP8 tensors with power-of-two scales, and bf16 pages holding exactly the same values."""
    t = wl.materialize_fp8(w, DEV)
    for k in ("k_scale", "v_scale"):
        t[k] = torch.exp2(torch.round(torch.log2(t[k])))
    b = dict(t)
    for name, sk in (("k_pages", "k_scale"), ("v_pages", "v_scale")):
        b[name] = (t[name].float() * t[sk].view(1, 1, -1, 1)).to(torch.bfloat16)
    del b["k_scale"], b["v_scale"]
    return t, b


def test_fp8_decode_equals_bf16_bitwise_at_power_of_two_scales():
    """With power-of-two scales the folded scales are exact: FP8 pages give the same bits
    as bf16 pages holding the dequantised values (same split, same summation order)."""
    lens = [1, 33, 64, 700, 2000, 5]
    for hq, hkv, ps in ((32, 4, 16), (2, 2, 32), (64, 8, 64)):
        w = wl.custom(90 + hq, "decode", lens, hq=hq, hkv=hkv, page_size=ps)
        H.say(f"fp8 == bf16 decode h{hq}kv{hkv} P{ps}")
        t8, tb = _pow2_pair(w)
        o8, l8 = H.run_decode(w, t8, split_tokens=128)
        ob, lb = H.run_decode(w, tb, split_tokens=128)
        assert torch.equal(o8.view(torch.int16), ob.view(torch.int16)), "decode outputs differ"
        assert torch.equal(l8, lb), "decode lse differ"


def test_fp8_group_prefix_equals_bf16_bitwise_at_power_of_two_scales():
    lens = [4096 + x for x in (512, 700, 1000, 64, 3, 200, 900, 513)]
    w = wl.custom(95, "decode", lens, hq=64, hkv=8, page_size=64, group_size=8, shared_tokens=4096)
    H.say("fp8 == bf16 group prefix")
    t8, tb = _pow2_pair(w)
    o8, l8 = H.run_decode(w, t8, split_tokens=1024)
    ob, lb = H.run_decode(w, tb, split_tokens=1024)
    assert torch.equal(o8.view(torch.int16), ob.view(torch.int16)), "group-prefix outputs differ"
    assert torch.equal(l8, lb), "group-prefix lse differ"


def test_fp8_extend_equals_bf16_bitwise_at_power_of_two_scales():
    """FP8 extend advances 64 keys per step at every page size, as bf16 extend does
    with pages of fewer than 64 keys (bf16 pages of 64 keys and more take 128-key steps
    and round differently), so the bf16 side holds the same keys in pages of 32."""
    for ps in (16, 64):
        w = wl.custom(96, "extend", [700, 250, 90], q_lens=[300, 250, 1], hq=16, hkv=2, page_size=ps)
        H.say(f"fp8 == bf16 extend P={ps}")
        t8, tb = _pow2_pair(w)
        tb = H.pages_below(tb, 64)
        o8, l8 = H.run_extend(w, t8)
        ob, lb = H.run_extend(w, tb)
        assert torch.equal(o8.view(torch.int16), ob.view(torch.int16)), "extend outputs differ"
        assert torch.equal(l8, lb), "extend lse differ"


def test_fp8_decode_full_size_sampled():
    """The 128-sequence agentic decode workload (up to 64K tokens) with FP8 pages, in the
    benchmark's launch configuration; sampled sequences vs the oracle."""
    w = wl.decode_ragged()
    H.say(f"fp8 full size decode: B={w.batch} sum(L)={int(w.kv_lens.sum())}")
    t = wl.materialize_fp8(w, DEV)
    out, lse = H.run_decode(w, t)
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
    order = np.argsort(w.kv_lens, kind="stable")
    rows = sorted({int(order[0]), int(order[-1]), int(order[len(order) // 2]), 7, 90})
    ref_o, ref_l = H.oracle_decode_rows(w, t, rows)
    sel = torch.tensor(rows, device=DEV)
    res = H.compare(out[sel], ref_o, lse[sel], ref_l, what="fp8 decode_ragged")
    H.say(f"  rows={rows} {res}")
    del t
    torch.cuda.empty_cache()


def test_fp8_extend_full_size_sampled():
    w = wl.extend_multiturn()
    H.say(f"fp8 full size extend: B={w.batch} total_q={w.total_q}")
    t = wl.materialize_fp8(w, DEV)
    out, lse = H.run_extend(w, t)
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
    order = np.argsort(w.kv_lens, kind="stable")
    indptr = w.qo_indptr
    for seq in (int(order[-1]), int(order[0])):
        n = int(w.q_lens[seq])
        rows = sorted({0, n // 2, n - 1, min(n - 1, 128)})
        ref_o, ref_l = H.oracle_extend_rows(w, t, seq, rows)
        sel = torch.tensor([int(indptr[seq]) + i for i in rows], device=DEV)
        res = H.compare(out[sel], ref_o, lse[sel], ref_l, what=f"fp8 extend seq {seq}")
        H.say(f"  seq {seq} rows={rows} {res}")
    del t
    torch.cuda.empty_cache()


BAD_SCALES = [-1.0, 0.0, -0.0, float("inf"), float("-inf"), float("nan"), -float("nan")]
SCALE_CALLS = ["decode", "decode_multi_token", "decode_deterministic", "decode_group_prefix", "extend", "append"]


@pytest.mark.parametrize("call", SCALE_CALLS)
@pytest.mark.parametrize("bad", BAD_SCALES, ids=[repr(b) for b in BAD_SCALES])
def test_fp8_invalid_scale_is_reported(call, bad):
    """A scale that is not positive and finite (NaN of either sign included) is flagged in
    the device error word by every kernel that reads one, whatever the compiler assumes about
    NaN operands; a valid scale raises no error."""
    if call in ("decode", "decode_deterministic", "append"):
        w = wl.custom(97, "decode", [40, 70], hq=8, hkv=2, page_size=16)
    elif call == "decode_group_prefix":
        w = wl.custom(98, "decode", [64 + 5, 64 + 9, 64 + 30], hq=8, hkv=2, page_size=16, group_size=3,
                      shared_tokens=64)
    else:
        w = wl.custom(99, "extend", [40, 70], q_lens=[3, 3], hq=8, hkv=2, page_size=16)
    H.say(f"fp8 bad scale {bad} {call}")
    t = wl.materialize_fp8(w, DEV)

    def go():
        if call == "decode":
            H.run_decode(w, t)
        elif call == "decode_deterministic":
            H.run_decode(w, t, deterministic=True)
        elif call == "decode_group_prefix":
            H.run_decode(w, t, split_tokens=64)
        elif call == "decode_multi_token":
            q = t["q"].view(w.batch, 3, w.hq, 128)
            ra.decode_fp8(q, t["k_pages"], t["v_pages"], t["k_scale"], t["v_scale"], t["block_table"],
                          t["kv_lens"], t["scale"], out=torch.empty_like(q))
        elif call == "extend":
            H.run_extend(w, t)
        else:
            rows = torch.randn((w.batch, w.hkv, 128), device=DEV).to(torch.bfloat16)
            ra.append_kv_fp8(rows, rows, torch.arange(w.batch + 1, dtype=torch.int32, device=DEV),
                             t["block_table"], t["kv_lens"], t["k_pages"], t["v_pages"], t["k_scale"], t["v_scale"])

    ra.check_device_errors()
    go()
    ra.check_device_errors()    # valid scales: no error
    which = "k_scale" if call in ("extend", "decode_group_prefix") else "v_scale"
    t[which][1] = bad
    go()
    with pytest.raises(ra.RlAttnError) as e:
        ra.check_device_errors()
    assert e.value.status == "RL_ERR_DEVICE" and "dequant-scale-invalid" in str(e.value)
    ra.check_device_errors()    # cleared
