"""Tree-shaped prefix sharing (branching sessions) on the GPU, against the oracle.

Trajectories of one prompt share the prompt's pages; subsets of them that branch
after a common turn share further pages (the paper's branching sessions, section
"Linear and Branching Sessions"). The decode planner finds these nested shared
ranges (up to three levels) and the group-prefix pass reads each once per
sub-group. Sharing is a performance path only: results with sharing on and off
must both match the oracle, which ignores sharing.
"""

import numpy as np
import pytest
import torch

from paper_2609_08368_amd import rl_attn as ra
from paper_2609_08368_amd import workloads as wl
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

CASES = [
    # (page_size, Hq, Hkv, branches [(block, tokens)], groups, private lens, split, query tokens)
    (16, 8, 2, [(4, 64), (2, 32)], 2, [5, 40, 0, 17], 0, 1),
    (16, 8, 2, [(4, 64), (2, 32)], 2, [5, 40, 0, 17], 64, 1),
    (64, 64, 8, [(8, 1024), (4, 512), (2, 256)], 2, [512, 700, 1000, 64, 3, 200, 900, 513], 0, 1),
    (64, 64, 8, [(8, 1024), (4, 512), (2, 256)], 2, [512, 700, 1000, 64, 3, 200, 900, 513], 256, 1),
    (32, 16, 1, [(6, 96), (3, 64)], 3, [1, 30, 70, 2, 0, 33], 0, 1),       # one KV head, GQA 16
    (16, 2, 2, [(4, 48), (2, 16)], 2, [10, 0, 5, 7], 0, 1),                # one query head per KV head
    (64, 96, 8, [(8, 512), (4, 256), (2, 128)], 1, [300, 10, 64, 700, 5, 90, 128, 1], 0, 1),   # GQA 12
    (64, 24, 2, [(4, 256), (2, 128)], 2, [100, 300, 64, 5], 0, 4),          # 4 query tokens per sequence
    (16, 8, 2, [(8, 32), (4, 16), (2, 16)], 2, [3, 9, 40, 16, 0, 1, 2, 30], 0, 2),
    (8, 12, 3, [(4, 40), (2, 24)], 2, [8, 16, 3, 50], 64, 1),               # pages of 8 keys
]


def branching(case, fp8=False):
    ps, hq, hkv, branches, groups, priv, split, n = case
    G = branches[0][0]
    base = sum(t for _, t in branches)
    lens = [base + priv[j % len(priv)] + 3 * g for g in range(groups) for j in range(G)]
    if n > 1:
        w = wl.custom(900 + len(lens) + ps, "extend", lens, q_lens=[n] * len(lens), hq=hq, hkv=hkv, page_size=ps,
                      branches=branches)
    else:
        w = wl.custom(900 + len(lens) + ps, "decode", lens, hq=hq, hkv=hkv, page_size=ps, branches=branches)
    t = (wl.materialize_fp8 if fp8 else wl.materialize)(w, DEV)
    return w, t


def run(w, t, n, **opts):
    if n == 1:
        return H.run_decode(w, t, **opts)
    q = t["q"].view(w.batch, n, w.hq, 128)
    out = H.poison_like(torch.empty(q.shape, dtype=torch.bfloat16, device=DEV))
    lse = H.poison_like(torch.empty(q.shape[:-1], dtype=torch.float32, device=DEV))
    if H.is_fp8(t):
        ra.decode_fp8(q, t["k_pages"], t["v_pages"], t["k_scale"], t["v_scale"], t["block_table"], t["kv_lens"],
                      t["scale"], out=out, lse=lse, **opts)
    else:
        ra.decode(q, t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], out=out, lse=lse, **opts)
    torch.cuda.synchronize()
    return out.reshape(-1, w.hq, 128), lse.reshape(-1, w.hq)


@pytest.mark.parametrize("share", [True, False])
@pytest.mark.parametrize("case", CASES, ids=[f"P{c[0]}_h{c[1]}kv{c[2]}_L{len(c[3])}_s{c[6]}_n{c[7]}_{i}"
                                             for i, c in enumerate(CASES)])
def test_branching_decode(case, share):
    H.say(f"branching {case} share={share}")
    w, t = branching(case)
    out, lse = run(w, t, case[7], split_tokens=case[6], prefix_share=share)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what=f"branching {case} share={share}")
    ra.check_device_errors()


@pytest.mark.parametrize("case", [CASES[2], CASES[7]], ids=["h64kv8", "n4"])
def test_branching_fp8(case):
    H.say(f"branching fp8 {case}")
    w, t = branching(case, fp8=True)
    out, lse = run(w, t, case[7], split_tokens=case[6])
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what=f"branching fp8 {case}")


def test_branching_shuffled_batch_full_size():
    """The 16 x 8 branching batch in shuffled order: every row against the oracle,
    with sharing on and off."""
    w = wl.decode_branching(shuffle=True)
    H.say(f"branching full size shuffled: B={w.batch} sum(L)={int(w.kv_lens.sum())}")
    t = wl.materialize(w, DEV)
    for share in (True, False):
        out, lse = H.run_decode(w, t, prefix_share=share)
        call = H.HostCall.from_gpu("decode", t, out, lse)
        H.full_parity(call, f"branching shuffled share={share}").check(f"branching shuffled share={share}")
    ra.check_device_errors()


def test_branching_equals_flat_groups_when_one_level():
    """A tree of one level is a plain trajectory group: the same bits either way."""
    lens = [4096 + x for x in (512, 700, 1000, 64, 3, 200, 900, 513)]
    wt = wl.custom(960, "decode", lens, hq=64, hkv=8, page_size=64, branches=[(8, 4096)])
    wg = wl.custom(960, "decode", lens, hq=64, hkv=8, page_size=64, group_size=8, shared_tokens=4096)
    assert np.array_equal(wt.kv_lens, wg.kv_lens)
    for w in (wt, wg):
        t = wl.materialize(w, DEV)
        out, lse = H.run_decode(w, t)
        ref_o, ref_l = H.oracle_full(w, t)
        H.compare(out, ref_o, lse, ref_l, what=w.name)
