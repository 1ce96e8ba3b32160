"""Multi-token decode (q [B, n, Hq, 128], e.g. verifying multi-token-prediction
drafts) on the GPU through the C-ABI, against the oracle.

Token i of a sequence of length L is at position L - n + i and sees keys
t <= L - n + i: the oracle's extend with n-row chunks is exactly that.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2609_08368_amd import rl_attn as ra
from paper_2609_08368_amd import workloads as wl
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def mtp_problem(seed, lens, n, hq, hkv, ps, fp8=False, **kw):
    w = wl.custom(seed, "extend", lens, q_lens=[n] * len(lens), hq=hq, hkv=hkv, page_size=ps, **kw)
    t = (wl.materialize_fp8 if fp8 else wl.materialize)(w, DEV)
    return w, t


def run_mtp(w, t, n, out_dtype=torch.bfloat16, **opts):
    B = w.batch
    q = t["q"].view(B, n, w.hq, 128)
    out = H.poison_like(torch.empty(q.shape, dtype=out_dtype, device=DEV))
    lse = H.poison_like(torch.empty((B, n, w.hq), dtype=torch.float32, device=DEV))
    if H.is_fp8(t):
        ra.decode_fp8(q, t["k_pages"], t["v_pages"], t["k_scale"], t["v_scale"], t["block_table"], t["kv_lens"],
                      t["scale"], out=out, lse=lse, **opts)
    else:
        ra.decode(q, t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], out=out, lse=lse, **opts)
    torch.cuda.synchronize()
    return out, lse


def check(w, t, n, out, lse, what):
    ref_o, ref_l = H.oracle_full(w, t)            # extend with n-row chunks
    B = w.batch
    return H.compare(out.reshape(B * n, w.hq, 128), ref_o, lse.reshape(B * n, w.hq), ref_l, what=what)


CASES = [
    # (page_size, Hq, Hkv, lens, n, split)
    (16, 8, 2, [5, 17, 100, 300], 2, 0),
    (16, 8, 2, [4, 33, 64, 200], 4, 64),
    (64, 96, 8, [63, 700, 1500, 8], 4, 0),       # the agentic shape: 48 rows per KV head
    (64, 64, 8, [400, 9, 2000], 8, 0),
    (32, 2, 2, [31, 250, 3], 3, 64),              # one query head per KV head: rows = tokens
    (128, 40, 2, [129, 600], 4, 128),             # 80 rows per KV head
    (16, 256, 2, [50, 90], 2, 0),                 # 256 rows per KV head: two row blocks
    (8, 12, 3, [8, 9, 200], 8, 64),
    (64, 8, 1, [2048 + 5, 64, 65], 5, 0),
]


@pytest.mark.parametrize("case", CASES, ids=[f"P{c[0]}_h{c[1]}kv{c[2]}_n{c[4]}_s{c[5]}" for c in CASES])
def test_mtp_decode_shapes(case):
    ps, hq, hkv, lens, n, split = case
    w, t = mtp_problem(160 + n + hq, lens, n, hq, hkv, ps)
    H.say(f"mtp {case}")
    out, lse = run_mtp(w, t, n, split_tokens=split)
    check(w, t, n, out, lse, f"mtp {case}")
    ra.check_device_errors()


@pytest.mark.parametrize("n", [2, 4])
def test_mtp_decode_fp8_and_f32_out(n):
    w, t = mtp_problem(170 + n, [70, 700, 1300, n], n, 32, 4, 64, fp8=True)
    H.say(f"mtp fp8 n={n}")
    out, lse = run_mtp(w, t, n, out_dtype=torch.float32)
    check(w, t, n, out, lse, "mtp fp8")


@pytest.mark.parametrize("share", [True, False])
def test_mtp_decode_group_prefix(share):
    gs, shared, n = 8, 4096, 4
    priv = [512, 700, 1000, 64, 4, 200, 900, 513]
    lens = [shared + priv[j] + 7 * g for g in range(2) for j in range(gs)]
    w, t = mtp_problem(175, lens, n, 64, 8, 64, group_size=gs, shared_tokens=shared)
    H.say(f"mtp group prefix share={share}")
    out, lse = run_mtp(w, t, n, prefix_share=share)
    check(w, t, n, out, lse, f"mtp group share={share}")


def test_mtp_single_token_shape_equals_decode():
    """q [B, 1, Hq, 128] is the plain decode, bitwise."""
    w, t = mtp_problem(176, [90, 700, 1], 1, 24, 2, 16)
    H.say("mtp n=1 vs decode")
    o4, l4 = run_mtp(w, t, 1)
    o3 = H.poison_like(torch.empty(t["q"].shape, dtype=torch.bfloat16, device=DEV))
    l3 = H.poison_like(torch.empty(t["q"].shape[:2], dtype=torch.float32, device=DEV))
    ra.decode(t["q"], t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], out=o3, lse=l3)
    torch.cuda.synchronize()
    assert torch.equal(o4[:, 0].view(torch.int16), o3.view(torch.int16)) and torch.equal(l4[:, 0], l3)


@pytest.mark.parametrize("n", [2, 4, 8])
def test_mtp_deterministic_equals_extend(n):
    """Deterministic multi-token decode is extend of the same tokens, bitwise."""
    w, t = mtp_problem(177 + n, [n, 300, 1200, 64 + n], n, 24, 2, 64)
    H.say(f"mtp deterministic n={n}")
    out, lse = run_mtp(w, t, n, deterministic=True)
    eo, el = H.run_extend(w, t)
    assert torch.equal(out.reshape(-1, w.hq, 128).view(torch.int16), eo.view(torch.int16))
    assert torch.equal(lse.reshape(-1, w.hq), el)
    check(w, t, n, out, lse, "mtp deterministic")


@pytest.mark.parametrize("n", [2, 8])
def test_mtp_unshared_runs_as_deterministic(n):
    """With prefix sharing off and automatic splits, multi-token decode runs through
    the extend kernel's 64-key steps: bitwise the deterministic mode over the same keys
    in pages of 32 (which take those steps too), and the oracle's values."""
    w, t = mtp_problem(185 + n, [n, 333, 1500, 64 + n], n, 96, 8, 64)
    H.say(f"mtp unshared n={n}")
    out, lse = run_mtp(w, t, n, prefix_share=False)
    do, dl = run_mtp(w, H.pages_below(t, 64), n, deterministic=True)
    assert torch.equal(out.view(torch.int16), do.view(torch.int16)) and torch.equal(lse, dl)
    check(w, t, n, out, lse, f"mtp unshared n={n}")
    ra.check_device_errors()


def test_mtp_unshared_split_path_cases():
    """Prefix sharing off with a forced split, or with q rows that do not merge with the
    batch dimension, keeps the split path (no error), and matches the oracle."""
    n = 4
    w, t = mtp_problem(190, [70, 900, 2100, 5], n, 96, 8, 64)
    H.say("mtp unshared, forced split")
    out, lse = run_mtp(w, t, n, prefix_share=False, split_tokens=256)
    check(w, t, n, out, lse, "mtp unshared split 256")
    H.say("mtp unshared, q with a padded batch stride")
    B = w.batch
    qpad = torch.zeros((B, n + 1, w.hq, 128), dtype=torch.bfloat16, device=DEV)
    qpad[:, :n] = t["q"].view(B, n, w.hq, 128)
    q = qpad[:, :n]                                   # batch stride (n + 1) x token stride
    out = H.poison_like(torch.empty((B, n, w.hq, 128), dtype=torch.bfloat16, device=DEV))
    lse = H.poison_like(torch.empty((B, n, w.hq), dtype=torch.float32, device=DEV))
    ra.decode(q, t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], out=out, lse=lse,
              prefix_share=False)
    torch.cuda.synchronize()
    check(w, t, n, out, lse, "mtp unshared padded q")
    ra.check_device_errors()


@pytest.mark.parametrize("n", [2, 8])
def test_mtp_route_follows_shared_pages(n):
    """Prefix sharing on, bf16 pages, automatic splits: a batch without shared pages is
    computed by the queued extend pass (bitwise the deterministic mode over the same keys
    in pages of 32: both advance 64 keys per step); a trajectory-group batch by the split
    passes, whose rows the extend pass must leave alone."""
    w, t = mtp_problem(190 + n, [n, 300, 1400, 64 + n], n, 96, 8, 64)
    H.say(f"mtp route without shared pages n={n}")
    out, lse = run_mtp(w, t, n)
    do, dl = run_mtp(w, H.pages_below(t, 64), n, deterministic=True)
    assert torch.equal(out.view(torch.int16), do.view(torch.int16)) and torch.equal(lse, dl)
    check(w, t, n, out, lse, f"mtp route no sharing n={n}")
    gs, shared = 4, 1024
    lens = [shared + 64 + 37 * j + 5 * g for g in range(2) for j in range(gs)]
    w, t = mtp_problem(195 + n, lens, 2, 16, 4, 64, group_size=gs, shared_tokens=shared)
    H.say("mtp route with shared pages n=2")
    out, lse = run_mtp(w, t, 2)
    do, dl = run_mtp(w, t, 2, deterministic=True)
    assert not torch.equal(lse, dl), "the extend pass overwrote the split passes' rows"
    check(w, t, 2, out, lse, "mtp route sharing")
    ra.check_device_errors()


def test_mtp_empty_sequence():
    w, t = mtp_problem(180, [0, 40, 0], 2, 8, 2, 16)
    H.say("mtp empty sequences")
    out, lse = run_mtp(w, t, 2)
    assert torch.all(out[0] == 0) and torch.all(out[2] == 0)
    assert torch.all(torch.isneginf(lse[0])) and torch.all(torch.isneginf(lse[2]))
    sub = wl.compact_subset(w, t, [1])          # the non-empty sequence alone
    ref_o, ref_l = oracle.extend(sub["q"], sub["qo_indptr"], sub["k_pages"], sub["v_pages"], sub["block_table"],
                                 sub["kv_lens"], t["scale"])
    H.compare(out[1], ref_o, lse[1], ref_l, what="mtp non-empty sequence")


def test_mtp_full_size_sampled():
    """The ragged 64K batch with 4 query tokens per sequence, in the benchmark's launch
    configuration; sampled sequences vs the oracle."""
    n = 4
    w = wl.decode_ragged()
    H.say(f"mtp full size: B={w.batch} n={n}")
    t = wl.materialize(w, DEV, poison=False)
    g = torch.Generator(device=DEV)
    g.manual_seed(4242)
    q = torch.randn((w.batch, n, w.hq, 128), generator=g, device=DEV).to(torch.bfloat16)
    out = torch.empty_like(q)
    lse = torch.empty((w.batch, n, w.hq), dtype=torch.float32, device=DEV)
    ra.decode(q, t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], out=out, lse=lse)
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
    order = np.argsort(w.kv_lens, kind="stable")
    rows = sorted({int(order[0]), int(order[-1]), int(order[len(order) // 2]), 5})
    sub = wl.compact_subset(w, t, rows)
    q_sub = H.to_host(q[torch.tensor(rows, device=DEV)].reshape(-1, w.hq, 128).contiguous())
    qo = (np.arange(len(rows) + 1) * n).astype(np.int32)
    ref_o, ref_l = oracle.extend(q_sub, qo, sub["k_pages"], sub["v_pages"], sub["block_table"], sub["kv_lens"],
                                 t["scale"])
    sel = torch.tensor(rows, device=DEV)
    res = H.compare(out[sel].reshape(-1, w.hq, 128), ref_o, lse[sel].reshape(-1, w.hq), ref_l, what="mtp ragged")
    H.say(f"  rows={rows} {res}")
    del t
    torch.cuda.empty_cache()
