"""Extend on the GPU (through the C-ABI) against the float64 oracle."""

import numpy as np
import pytest
import torch

from paper_2609_08368_amd import rl_attn as ra
from paper_2609_08368_amd import workloads as wl
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

CASES = [
    # (page_size, Hq, Hkv, kv_lens, q_lens)
    (16, 8, 2, [40, 17, 100], [5, 17, 1]),          # second: empty prefix
    (16, 8, 2, [300, 129, 64], [129, 100, 16]),
    (64, 64, 8, [500, 70], [33, 70]),
    (8, 12, 3, [90, 13], [20, 13]),                  # GQA 4
    (32, 16, 16, [200, 50], [150, 7]),               # one query head per KV head
    (16, 24, 2, [80, 33], [17, 33]),                 # GQA 12: 10 tokens per tile
    (16, 256, 1, [40, 9], [3, 2]),                   # GQA 256: two 128-head blocks
    (128, 8, 1, [600], [257]),
    # 128-key steps (bf16 pages of at least 64 keys): one step, a step whose second
    # 64-key half lies past the last key, exact multiples of 128, both halves of a step
    # in one page (the second starting inside it), a short second sequence
    (64, 16, 2, [1, 64, 65, 128, 129, 192, 193, 256], [1, 64, 1, 128, 3, 64, 100, 256]),
    (128, 8, 2, [1000, 255, 256, 257], [300, 255, 1, 257]),
    (128, 32, 4, [130, 380], [130, 60]),
    (16, 8, 2, [30, 0, 12], [0, 0, 12]),             # empty chunks
]


@pytest.mark.parametrize("case", CASES, ids=[f"P{c[0]}_h{c[1]}kv{c[2]}_{i}" for i, c in enumerate(CASES)])
def test_extend_shapes(case):
    ps, hq, hkv, kv, ql = case
    w = wl.custom(21 + sum(ql), "extend", kv, q_lens=ql, hq=hq, hkv=hkv, page_size=ps)
    H.say(f"extend case {case}")
    t = wl.materialize(w, DEV)
    if w.total_q == 0:
        return
    out, lse = H.run_extend(w, t)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what=str(case))


def test_extend_f32_out_and_plain_signature():
    w = wl.custom(31, "extend", [100, 60], q_lens=[40, 60], hq=16, hkv=2, page_size=16)
    H.say("extend f32 / plain")
    t = wl.materialize(w, DEV)
    out, lse = H.run_extend(w, t, out_dtype=torch.float32)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what="f32")
    out2 = torch.full_like(t["q"], float("nan"))
    ra.extend_plain(t["q"], t["qo_indptr"], t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"],
                    t["scale"], out=out2)
    torch.cuda.synchronize()
    H.compare(out2, ref_o, what="plain")
    out3 = torch.full_like(t["q"], float("nan"))
    ra.extend_plain(t["q"], t["qo_indptr"], t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"],
                    t["scale"], out=out3)
    torch.cuda.synchronize()
    assert torch.equal(out2.view(torch.int16), out3.view(torch.int16)), "run-to-run results differ"


def test_extend_one_query_matches_decode():
    w = wl.custom(41, "extend", [77, 300, 16], q_lens=[1, 1, 1], hq=32, hkv=4, page_size=16)
    H.say("extend n=1 vs decode")
    t = wl.materialize(w, DEV)
    out_e, lse_e = H.run_extend(w, t)
    out_d, lse_d = H.run_decode(w, t)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out_e, ref_o, lse_e, ref_l, what="extend n=1")
    H.compare(out_d, ref_o, lse_d, ref_l, what="decode")


def test_extend_full_size_sampled():
    """The multi-turn extend workload at full size; sampled rows vs the oracle."""
    w = wl.extend_multiturn()
    H.say(f"full size extend: B={w.batch} total_q={w.total_q} flops={w.flops():.3e}")
    t = wl.materialize(w, DEV)
    out, lse = H.run_extend(w, t)
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
    order = np.argsort(w.kv_lens, kind="stable")
    indptr = w.qo_indptr
    for seq in (int(order[-1]), int(order[0]), int(order[len(order) // 2])):
        n = int(w.q_lens[seq])
        rows = sorted({0, 1, n // 2, n - 2, n - 1, min(n - 1, 127), min(n - 1, 128)})
        ref_o, ref_l = H.oracle_extend_rows(w, t, seq, rows)
        sel = torch.tensor([int(indptr[seq]) + i for i in rows], device=DEV)
        res = H.compare(out[sel], ref_o, lse[sel], ref_l, what=f"extend seq {seq}")
        H.say(f"  seq {seq} kv={int(w.kv_lens[seq])} n={n} rows={rows} {res}")
    del t
    torch.cuda.empty_cache()


def test_extend_determinism():
    """Run-to-run identical results, on both page-addressing paths."""
    for ps in (16, 64):
        w = wl.custom(23, "extend", [700, 250, 90], q_lens=[300, 250, 1], hq=16, hkv=2, page_size=ps)
        H.say(f"extend determinism P={ps}")
        t = wl.materialize(w, DEV)
        outs = [H.run_extend(w, t)[0] for _ in range(3)]
        for o in outs[1:]:
            assert torch.equal(o.view(torch.int16), outs[0].view(torch.int16)), "run-to-run results differ"
