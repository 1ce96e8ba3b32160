"""Seeded random configurations through the C-ABI against the oracle.

Each case draws a page size, KV heads, a GQA ratio, a batch of ragged lengths
(empty ones included), the call (decode, multi-token decode or extend), bf16 or
FP8 pages, a forced or automatic split, trajectory groups sharing a prefix, and
the deterministic mode, all from one seed, so a failure names its case.
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


def draw(seed):
    rng = np.random.default_rng(10_000 + seed)
    c = {
        "ps": int(rng.choice([8, 16, 32, 64, 128])),
        "hkv": int(rng.choice([1, 2, 4, 8])),
        "r": int(rng.choice([1, 2, 3, 4, 6, 8, 12, 16, 20])),
        "kind": str(rng.choice(["decode", "decode", "mtp", "extend"])),
        "fp8": bool(rng.random() < 0.35),
        "split": int(rng.choice([0, 0, 64, 128, 256])),
        "det": bool(rng.random() < 0.2),
    }
    c["n"] = int(rng.integers(2, 9)) if c["kind"] == "mtp" else 1
    b = int(rng.integers(1, 11))
    groups = c["kind"] != "extend" and rng.random() < 0.3
    if groups:
        gs = int(rng.integers(2, 6))
        shared = int(rng.integers(1, 5)) * c["ps"] * int(rng.integers(1, 3))
        ng = max(1, b // gs)
        lens = [shared + int(rng.integers(0, 600)) + c["n"] for _ in range(ng * gs)]
        c.update(group_size=gs, shared=shared)
    else:
        lens = [int(x) for x in rng.integers(0, 3000, size=b)]
        lens = [0 if rng.random() < 0.12 else x for x in lens]
        if c["kind"] == "mtp":
            lens = [x if x == 0 else max(x, c["n"]) for x in lens]
        c.update(group_size=1, shared=0)
    c["lens"] = lens
    if c["kind"] == "extend":
        c["q_lens"] = [int(rng.integers(0, min(x, 300) + 1)) for x in lens]
    return c


@pytest.mark.parametrize("seed", range(120))
def test_random_configuration(seed):
    c = draw(seed)
    H.say(f"random case {seed}: {c}")
    hq = c["hkv"] * c["r"]
    kind = "extend" if c["kind"] in ("extend", "mtp") else "decode"
    q_lens = c.get("q_lens") or ([c["n"] if x else 0 for x in c["lens"]] if c["kind"] == "mtp" else None)
    w = wl.custom(20_000 + seed, kind, c["lens"], q_lens=q_lens, hq=hq, hkv=c["hkv"], page_size=c["ps"],
                  group_size=c["group_size"], shared_tokens=c["shared"])
    t = (wl.materialize_fp8 if c["fp8"] else wl.materialize)(w, DEV)
    if c["kind"] == "extend":
        if w.total_q == 0:
            return
        out, lse = H.run_extend(w, t)
        ref_o, ref_l = H.oracle_full(w, t)
        H.compare(out, ref_o, lse, ref_l, what=f"random {seed}")
        ra.check_device_errors()
        return
    if c["kind"] == "decode":
        out, lse = H.run_decode(w, t, split_tokens=c["split"], deterministic=c["det"])
        ref_o, ref_l = H.oracle_full(w, t)
        H.compare(out, ref_o, lse, ref_l, what=f"random {seed}")
        ra.check_device_errors()
        return
    # multi-token decode: every sequence holds n tokens (or none); q [B, n, Hq, 128]
    n, B = c["n"], w.batch
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    q = torch.randn((B, n, hq, 128), generator=g, device=DEV).to(torch.bfloat16)
    out = H.poison_like(torch.empty(q.shape, dtype=torch.bfloat16, device=DEV))
    lse = H.poison_like(torch.empty((B, n, hq), dtype=torch.float32, device=DEV))
    opts = dict(out=out, lse=lse, split_tokens=c["split"], deterministic=c["det"])
    if c["fp8"]:
        ra.decode_fp8(q, t["k_pages"], t["v_pages"], t["k_scale"], t["v_scale"], t["block_table"], t["kv_lens"],
                      t["scale"], **opts)
    else:
        ra.decode(q, t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], **opts)
    torch.cuda.synchronize()
    ra.check_device_errors()
    # the oracle's extend over the non-empty sequences, n rows each
    rows = [b for b in range(B) if w.kv_lens[b] > 0]
    empty = [b for b in range(B) if w.kv_lens[b] == 0]
    if empty:
        sel = torch.tensor(empty, device=DEV)
        assert torch.all(out[sel] == 0) and torch.all(torch.isneginf(lse[sel]))
    if not rows:
        return
    sub = wl.compact_subset(w, t, rows)
    qs = H.to_host(q[torch.tensor(rows, device=DEV)].reshape(-1, hq, 128).contiguous())
    qo = (np.arange(len(rows) + 1) * n).astype(np.int32)
    sc = H.host_scales(t)
    ref_o, ref_l = oracle.extend(qs, qo, sub["k_pages"], sub["v_pages"], sub["block_table"], sub["kv_lens"],
                                 t["scale"], **sc)
    sel = torch.tensor(rows, device=DEV)
    H.compare(out[sel].reshape(-1, hq, 128), ref_o, lse[sel].reshape(-1, hq), ref_l, what=f"random mtp {seed}")
