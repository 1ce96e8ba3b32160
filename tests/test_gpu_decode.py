"""Decode on the GPU (through the C-ABI) against the float64 oracle."""

import numpy as np
import pytest
import torch

from paper_2609_08368_amd import rl_attn as ra
from paper_2609_08368_amd import workloads as wl
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.mark.parametrize("out_dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("split", [0, 64, 128])
def test_decode_tiny_full(out_dtype, split):
    w = wl.decode_tiny()
    H.say(f"decode_tiny out={out_dtype} split={split}")
    t = wl.materialize(w, DEV)
    out, lse = H.run_decode(w, t, out_dtype=out_dtype, split_tokens=split)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what=f"decode_tiny split={split}")


CASES = [
    # (page_size, Hq, Hkv, lens, split)
    (16, 8, 2, [1, 15, 16, 17, 100, 300], 0),
    (16, 8, 2, [1, 15, 16, 17, 100, 300], 64),
    (8, 12, 1, [7, 8, 9, 64, 65, 129], 64),
    (64, 64, 8, [63, 64, 65, 200, 1], 0),
    (64, 96, 8, [5, 130, 257], 64),
    (128, 16, 1, [127, 128, 129, 400], 128),
    (32, 2, 2, [1, 31, 33, 250], 64),        # one query head per KV head: vector-ALU path
    (16, 3, 3, [40, 1, 77], 0),
    (16, 6, 3, [40, 1, 77], 64),             # GQA 2
    (16, 40, 2, [50, 190], 64),              # GQA 20: two 16-head blocks
    (64, 32, 1, [1000, 3], 256),
    (32, 24, 2, [31, 32, 33, 97, 600], 0),   # pages of exactly one 32-key tile: whole-row loads
    (32, 24, 2, [31, 32, 33, 97, 600], 64),
    (16, 40, 2, [300, 17], 0),               # pages below a tile: each lane loads its share of a row
]


@pytest.mark.parametrize("case", CASES, ids=[f"P{c[0]}_h{c[1]}kv{c[2]}_s{c[4]}" for c in CASES])
def test_decode_shapes(case):
    ps, hq, hkv, lens, split = case
    w = wl.custom(11 + len(lens), "decode", lens, hq=hq, hkv=hkv, page_size=ps)
    H.say(f"decode case {case}")
    t = wl.materialize(w, DEV)
    out, lse = H.run_decode(w, t, split_tokens=split)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what=str(case))


def test_decode_single_key_is_exact():
    w = wl.custom(5, "decode", [1, 1, 1], hq=8, hkv=2, page_size=16)
    H.say("single key")
    t = wl.materialize(w, DEV)
    out, lse = H.run_decode(w, t)
    ref_o, ref_l = H.oracle_full(w, t)
    for b in range(3):
        pg = int(w.block_table[b, 0])
        for h in range(8):
            v = t["v_pages"][pg, 0, h // 4]
            assert torch.equal(out[b, h].view(torch.int16), v.view(torch.int16)), "single key: out != V bitwise"
    H.compare(out, ref_o, lse, ref_l, lse_rel=1e-6, what="single key")


def test_decode_empty_sequence():
    w = wl.custom(6, "decode", [0, 20, 0, 1], hq=8, hkv=2, page_size=16)
    H.say("empty sequences")
    t = wl.materialize(w, DEV)
    out, lse = H.run_decode(w, t)
    assert torch.all(out[0] == 0) and torch.all(out[2] == 0)
    assert torch.all(torch.isneginf(lse[0])) and torch.all(torch.isneginf(lse[2]))
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what="empty")


def test_decode_plain_signature_and_determinism():
    w = wl.custom(7, "decode", [300, 5, 1000, 64], hq=32, hkv=4, page_size=16)
    H.say("plain signature / determinism")
    t = wl.materialize(w, DEV)
    outs = []
    for _ in range(3):
        out = torch.full_like(t["q"], float("nan"))
        ra.decode_plain(t["q"], t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], out=out)
        torch.cuda.synchronize()
        outs.append(out)
    for o in outs[1:]:
        assert torch.equal(o.view(torch.int16), outs[0].view(torch.int16)), "run-to-run results differ"
    ref_o, _ = H.oracle_full(w, t)
    H.compare(outs[0], ref_o, what="plain")


def test_decode_strided_views():
    """Non-contiguous q/out/pages (views into larger buffers) are honoured."""
    w = wl.custom(8, "decode", [70, 129], hq=8, hkv=2, page_size=16)
    H.say("strided views")
    t = wl.materialize(w, DEV)
    big_q = torch.zeros((2, 12, 136), dtype=torch.bfloat16, device=DEV)
    big_q[:, 2:10, :128] = t["q"]
    q = big_q[:, 2:10, :128]
    big_k = torch.zeros((w.num_pages, 16, 3, 128), dtype=torch.bfloat16, device=DEV)
    big_v = torch.zeros_like(big_k)
    big_k[:, :, 1:3] = t["k_pages"]
    big_v[:, :, 0:2] = t["v_pages"]
    big_out = torch.full((2, 8, 256), float("nan"), dtype=torch.float32, device=DEV)
    out = big_out[:, :, 64:192]
    mp = t["block_table"].shape[1]
    bt = torch.zeros((2, 4 * mp), dtype=torch.int32, device=DEV)
    bt[:, ::4] = t["block_table"]
    ra.decode(q, big_k[:, :, 1:3], big_v[:, :, 0:2], bt[:, ::4], t["kv_lens"], t["scale"], out=out,
              split_tokens=64)
    torch.cuda.synchronize()
    ref_o, _ = H.oracle_full(w, t)
    H.compare(out, ref_o, what="strided")
    assert torch.isnan(big_out[:, :, :64]).all() and torch.isnan(big_out[:, :, 192:]).all()


@pytest.mark.parametrize("name", ["decode_uniform", "decode_ragged", "decode_group_prefix", "decode_group_long_prefix"])
def test_decode_full_size_sampled(name):
    """Full-size workloads in the benchmark's launch configuration; sampled sequences vs the oracle."""
    w = wl.WORKLOADS[name]() if name in wl.WORKLOADS else getattr(wl, name)()
    H.say(f"full size {name}: B={w.batch} sum(L)={int(w.kv_lens.sum())}")
    t = wl.materialize(w, DEV)
    out, lse = H.run_decode(w, t)
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
    order = np.argsort(w.kv_lens, kind="stable")
    rng = np.random.default_rng(0)
    rows = sorted({int(order[0]), int(order[-1]), int(order[len(order) // 2]),
                   *rng.choice(w.batch, size=3, replace=False).tolist()})
    ref_o, ref_l = H.oracle_decode_rows(w, t, rows)
    sel = torch.tensor(rows, device=DEV)
    res = H.compare(out[sel], ref_o, lse[sel], ref_l, what=name)
    H.say(f"  {name} rows={rows} {res}")
    del t
    torch.cuda.empty_cache()


PREFIX_CASES = [
    # (page_size, Hq, Hkv, group_size, groups, shared_tokens, private lens, split)
    (16, 8, 2, 4, 3, 64, [5, 40, 0, 17], 0),            # a member with no private keys
    (16, 8, 2, 4, 2, 60, [1, 30, 70, 2], 64),           # shared prefix not page aligned: 3 full pages
    (64, 64, 8, 8, 2, 4096, [512, 700, 1000, 64, 3, 200, 900, 513], 0),
    (64, 64, 8, 8, 2, 4096, [512, 700, 1000, 64, 3, 200, 900, 513], 1024),
    (32, 16, 1, 20, 1, 256, list(range(1, 21)), 128),   # 20 members x 16 rows: two sub-groups
    (16, 2, 2, 3, 2, 48, [10, 0, 5], 0),                 # one query head per KV head
]


@pytest.mark.parametrize("case", PREFIX_CASES, ids=[f"P{c[0]}_h{c[1]}kv{c[2]}_G{c[3]}_s{c[7]}" for c in PREFIX_CASES])
@pytest.mark.parametrize("share", [True, False])
def test_decode_group_prefix_sharing(case, share):
    ps, hq, hkv, gs, ng, shared, priv, split = case
    lens = [shared + priv[j % len(priv)] + 7 * g for g in range(ng) for j in range(gs)]
    w = wl.custom(50 + gs, "decode", lens, hq=hq, hkv=hkv, page_size=ps, group_size=gs, shared_tokens=shared)
    H.say(f"prefix case {case} share={share}")
    t = wl.materialize(w, DEV)
    out, lse = H.run_decode(w, t, split_tokens=split, prefix_share=share)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what=f"{case} share={share}")


def test_decode_group_prefix_shuffled_batch():
    """Groups scattered over the batch (shuffled order) are still found; results match the oracle."""
    w = wl.decode_group_prefix(shuffle=True)
    H.say("group prefix, shuffled batch")
    t = wl.materialize(w, DEV)
    out, lse = H.run_decode(w, t)
    out_off, lse_off = H.run_decode(w, t, prefix_share=False)
    assert torch.isfinite(out.float()).all()
    rows = [0, 1, 17, 64, 127]
    ref_o, ref_l = H.oracle_decode_rows(w, t, rows)
    sel = torch.tensor(rows, device=DEV)
    H.compare(out[sel], ref_o, lse[sel], ref_l, what="shuffled shared")
    H.compare(out_off[sel], ref_o, lse_off[sel], ref_l, what="shuffled unshared")
    # both runs agree with each other everywhere at the path's tolerance (each is a
    # bf16-rounded result, so they differ by up to twice the per-side error)
    H.compare(out, H.f64(out_off), what="shared vs unshared")


def test_decode_many_sequences():
    """More sequences than the planner keeps in LDS (1,500 > 1,024): per-sequence state
    goes through chunked scans, with no group detection."""
    rng = np.random.default_rng(21)
    lens = rng.integers(0, 200, size=1500).tolist()
    w = wl.custom(21, "decode", lens, hq=8, hkv=2, page_size=16)
    H.say("1500 sequences")
    t = wl.materialize(w, DEV)
    for split in (0, 64):
        out, lse = H.run_decode(w, t, split_tokens=split)
        ref_o, ref_l = H.oracle_full(w, t)
        H.compare(out, ref_o, lse, ref_l, what=f"1500 sequences split={split}")


@pytest.mark.parametrize("split", [64, 128, 256])
def test_decode_worker_shares_span_sequences(split):
    """Worker shares that start and end inside sequences and cover many short ones."""
    lens = [1] * 40 + [1000] + [33, 31, 32, 64, 65, 0, 5] * 6 + [700]
    w = wl.custom(22, "decode", lens, hq=16, hkv=2, page_size=32)
    H.say(f"worker shares split={split}")
    t = wl.materialize(w, DEV)
    out, lse = H.run_decode(w, t, split_tokens=split)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what=f"worker shares split={split}")
