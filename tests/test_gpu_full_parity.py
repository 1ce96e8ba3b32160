"""Every output row of every full-size workload against the float64 oracle.

The calls run on the GPU through the C-ABI in the benchmark's launch
configuration (default options, the workloads' own seeds and sizes); their
outputs and log-sum-exps are then compared, row by row, with the oracle
evaluated on the host cores (``gpu_helpers.full_parity``: a thread pool over
sequences, or over (sequence, KV head) pairs for extend). The tolerances are
the path's: max-abs 2e-2 and relative RMS 5e-3 over the whole output, lse
within 1e-4 relative. The multi-turn extend batch is checked in parts (each a
share of its (sequence, KV head) pairs, dealt longest first), so no single test
runs for minutes; the last test of each extend set checks the whole output.
"""

import numpy as np
import pytest
import torch

from paper_2609_08368_amd import rl_attn as ra
from paper_2609_08368_amd import workloads as wl
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
EXTEND_PARTS = 6


def decode_call(w, fp8=False, **opts):
    t = (wl.materialize_fp8 if fp8 else wl.materialize)(w, DEV)
    out, lse = H.run_decode(w, t, **opts)
    call = H.HostCall.from_gpu("decode", t, out, lse)
    del t, out, lse
    torch.cuda.empty_cache()
    return call


DECODE = [
    # (workload, FP8 pages, options)
    ("decode_tiny", False, {}),
    ("decode_uniform", False, {}),
    ("decode_ragged", False, {}),
    ("decode_ragged", True, {}),
    ("decode_group_prefix", False, {}),
    ("decode_group_prefix", False, {"prefix_share": False}),
    ("decode_ragged", False, {"deterministic": True}),
]


@pytest.mark.parametrize("case", DECODE, ids=[f"{c[0]}{'_fp8' if c[1] else ''}{''.join('_' + k for k in c[2])}"
                                              for c in DECODE])
def test_full_parity_decode(case):
    name, fp8, opts = case
    w = wl.WORKLOADS[name]()
    what = f"{name}{' fp8' if fp8 else ''} {opts}"
    H.say(f"full-row parity {what}: B={w.batch} sum(L)={int(w.kv_lens.sum())}")
    call = decode_call(w, fp8, **opts)
    H.full_parity(call, what).check(what)


def test_full_parity_multi_token_decode():
    """The ragged batch with 4 query tokens per sequence: every (sequence, token) row
    against the oracle's extend with 4-row chunks."""
    n = 4
    w = wl.decode_ragged()
    H.say(f"full-row parity multi-token decode n={n}: B={w.batch}")
    t = wl.materialize(w, DEV)
    g = torch.Generator(device=DEV)
    g.manual_seed(4242)
    q = torch.randn((w.batch, n, w.hq, 128), generator=g, device=DEV).to(torch.bfloat16)
    out = H.poison_like(torch.empty_like(q))
    lse = H.poison_like(torch.empty((w.batch, n, w.hq), dtype=torch.float32, device=DEV))
    ra.decode(q, t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], out=out, lse=lse)
    torch.cuda.synchronize()
    indptr = (np.arange(w.batch + 1) * n).astype(np.int32)
    call = H.HostCall.from_gpu("extend", t, out.reshape(-1, w.hq, 128), lse.reshape(-1, w.hq),
                               q=q.reshape(-1, w.hq, 128), qo_indptr=indptr)
    del t, q, out, lse
    torch.cuda.empty_cache()
    H.full_parity(call, "multi-token decode n=4").check("multi-token decode n=4")


def extend_call(fp8):
    w = wl.extend_multiturn()
    H.say(f"extend{' fp8' if fp8 else ''} full size: B={w.batch} total_q={w.total_q}")
    t = (wl.materialize_fp8 if fp8 else wl.materialize)(w, DEV)
    out, lse = H.run_extend(w, t)
    call = H.HostCall.from_gpu("extend", t, out, lse)
    del t, out, lse
    torch.cuda.empty_cache()
    return call


@pytest.fixture(scope="module")
def extend_bf16():
    return {"call": extend_call(False), "acc": H.ParityAcc(), "parts": set()}


@pytest.fixture(scope="module")
def extend_fp8():
    return {"call": extend_call(True), "acc": H.ParityAcc(), "parts": set()}


def _part(state, part, what):
    acc = H.full_parity(state["call"], f"{what} part {part}/{EXTEND_PARTS}", part=part, parts=EXTEND_PARTS)
    state["acc"].merge(acc)
    state["parts"].add(part)
    acc.check(f"{what} part {part}")


def _whole(state, what):
    assert state["parts"] == set(range(EXTEND_PARTS)), f"{what}: parts {sorted(state['parts'])} checked"
    r = state["acc"].check(what)
    total_q = state["call"].q.shape[0]
    assert r["rows"] == total_q * state["call"].q.shape[1], f"{what}: {r['rows']} rows checked"
    H.say(f"  {what} whole output: {r}")


@pytest.mark.parametrize("part", range(EXTEND_PARTS))
def test_full_parity_extend(extend_bf16, part):
    _part(extend_bf16, part, "extend_multiturn")


def test_full_parity_extend_whole(extend_bf16):
    _whole(extend_bf16, "extend_multiturn")


@pytest.mark.parametrize("part", range(EXTEND_PARTS))
def test_full_parity_extend_fp8(extend_fp8, part):
    _part(extend_fp8, part, "extend_multiturn fp8")


def test_full_parity_extend_fp8_whole(extend_fp8):
    _whole(extend_fp8, "extend_multiturn fp8")
