"""rl_attn_decode_noalloc: decode whose workspace is the library's static scratch array.

Checked through the C-ABI: its outputs equal rl_attn_decode_ex's bitwise (the same
kernels and plan) and the oracle's within the path's tolerances, on two calls in a
row (the second with a smaller input, so stale scratch contents of the first would
show), with each option the entry point accepts; it needs no reserved workspace
under HIP graph capture; a call whose workspace exceeds the array is refused
before any launch; and a call made while every library allocation is forced to
fail still succeeds (run in a child process, since the forcing switch is read
once per process).
"""

import os
import subprocess
import sys

import pytest
import torch

from paper_2609_08368_amd import rl_attn as ra
from paper_2609_08368_amd import workloads as wl
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def both(w, t, **opts):
    """(no-alloc out, lse), (decode_ex out, lse) of the same call."""
    res = []
    for fn in (ra.decode_noalloc, ra.decode):
        out = H.poison_like(torch.empty_like(t["q"]))
        lse = H.poison_like(torch.empty(t["q"].shape[:-1], dtype=torch.float32, device=DEV))
        fn(t["q"], t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], out=out, lse=lse, **opts)
        torch.cuda.synchronize()
        res.append((out, lse))
    return res


OPTS = [{}, {"split_tokens": 8192}, {"prefix_share": False}, {"deterministic": True}]


@pytest.mark.parametrize("opts", OPTS, ids=["default", "split8192", "no_share", "deterministic"])
def test_noalloc_equals_decode_ex_on_two_calls(opts):
    big = wl.decode_ragged()
    small = wl.custom(811, "decode", [0, 5, 300, 1, 64, 2000, 129], hq=16, hkv=2, page_size=16)
    for w in (big, small):
        H.say(f"no-alloc {w.name} {opts}")
        t = wl.materialize(w, DEV)
        (o_na, l_na), (o_ex, l_ex) = both(w, t, **opts)
        assert torch.equal(o_na.view(torch.int16), o_ex.view(torch.int16)), "out differs from rl_attn_decode_ex"
        assert torch.equal(l_na, l_ex), "lse differs from rl_attn_decode_ex"
        call = H.HostCall.from_gpu("decode", t, o_na, l_na)
        H.full_parity(call, f"no-alloc {w.name}").check(f"no-alloc {w.name}")
        ra.check_device_errors()
        del t
        torch.cuda.empty_cache()


def test_noalloc_group_prefix_and_multi_token():
    """Trajectory groups (the group-prefix pass writes partials into the scratch) and 4
    query tokens per sequence, each followed by a smaller call."""
    wg = wl.custom(812, "decode", [4096 + x for x in (512, 700, 1000, 64, 3, 200, 900, 513)], hq=64, hkv=8,
                   page_size=64, group_size=8, shared_tokens=4096)
    wm = wl.custom(813, "extend", [900, 64, 3000], q_lens=[4, 4, 4], hq=24, hkv=2, page_size=64)
    ws = wl.custom(814, "decode", [10, 90], hq=8, hkv=2, page_size=16)
    for w in (wg, ws, wm, ws):
        H.say(f"no-alloc {w.name}")
        t = wl.materialize(w, DEV)
        if w.kind == "extend":      # multi-token decode: q [B, 4, Hq, 128]
            q = t["q"].view(w.batch, 4, w.hq, 128)
            outs = []
            for fn in (ra.decode_noalloc, ra.decode):
                out = H.poison_like(torch.empty_like(q))
                lse = H.poison_like(torch.empty(q.shape[:-1], dtype=torch.float32, device=DEV))
                fn(q, t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], out=out, lse=lse)
                torch.cuda.synchronize()
                outs.append((out, lse))
            (o_na, l_na), (o_ex, l_ex) = outs
            call = H.HostCall.from_gpu("extend", t, o_na.reshape(-1, w.hq, 128), l_na.reshape(-1, w.hq))
        else:
            (o_na, l_na), (o_ex, l_ex) = both(w, t)
            call = H.HostCall.from_gpu("decode", t, o_na, l_na)
        assert torch.equal(o_na.view(torch.int16), o_ex.view(torch.int16))
        assert torch.equal(l_na, l_ex)
        H.full_parity(call, f"no-alloc {w.name}").check(f"no-alloc {w.name}")


def test_noalloc_captures_without_reserved_workspace():
    """Captured on a fresh stream with nothing reserved; every replay, with new query
    values and eager work between replays, equals the eager rl_attn_decode_ex call."""
    w = wl.custom(815, "decode", [700, 4, 3000, 129, 64], hq=16, hkv=2, page_size=64)
    t = wl.materialize(w, DEV)
    H.say("no-alloc graph capture")
    q_static = torch.empty_like(t["q"])
    out = torch.empty_like(t["q"])
    lse = torch.empty(t["q"].shape[:-1], dtype=torch.float32, device=DEV)
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        ra.decode_noalloc(q_static, t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"],
                          out=out, lse=lse, stream=s)
    torch.cuda.synchronize()
    for rep in range(4):
        gen = torch.Generator(device=DEV)
        gen.manual_seed(900 + rep)
        q_static.copy_(torch.randn(t["q"].shape, generator=gen, device=DEV).to(torch.bfloat16))
        g.replay()
        torch.cuda.synchronize()
        ref_o = torch.empty_like(out)
        ref_l = torch.empty_like(lse)
        ra.decode(q_static.clone(), t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"],
                  out=ref_o, lse=ref_l)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref_o.view(torch.int16)), f"replay {rep}: out differs"
        assert torch.equal(lse, ref_l), f"replay {rep}: lse differs"
    ref_o, ref_l = H.oracle_full(w, dict(t, q=q_static))
    H.compare(out, ref_o, lse, ref_l, what="no-alloc graph")


def test_noalloc_rejects_calls_beyond_the_scratch():
    """8 query tokens x 96 heads of 128 sequences need about 1 GB of partials: refused,
    with the outputs untouched (nothing launched)."""
    w = wl.decode_ragged()
    t = wl.materialize(w, DEV, poison=False)
    q = torch.zeros((w.batch, 8, w.hq, 128), dtype=torch.bfloat16, device=DEV)
    out = torch.full_like(q, 7.0)
    with pytest.raises(ra.RlAttnError) as e:
        ra.decode_noalloc(q, t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], out=out)
    assert e.value.status == "RL_ERR_WORKSPACE" and "allocation-free" in str(e.value)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all()), "a refused call wrote its output"


CHILD = r"""
import sys, torch
sys.path.insert(0, {root!r})
from paper_2609_08368_amd import rl_attn as ra
from paper_2609_08368_amd import workloads as wl
w = wl.custom(816, "decode", [300, 1, 2000], hq=16, hkv=2, page_size=16)
t = wl.materialize(w, "cuda:0")
s = torch.cuda.Stream()
out = torch.empty_like(t["q"])
with torch.cuda.stream(s):
    ra.decode_noalloc(t["q"], t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], out=out,
                      stream=s)
torch.cuda.synchronize()
try:
    ra.decode(t["q"], t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], stream=s)
    print("decode_ex allocated despite the forced failure")
    sys.exit(1)
except ra.RlAttnError as e:
    assert e.status == "RL_ERR_WORKSPACE", e
ra.check_device_errors(stream=s)
print("NOALLOC_CHILD_OK", float(out.float().abs().sum()))
"""


def test_noalloc_never_allocates():
    """With every library allocation forced to fail, the allocation-free call still
    runs (on a fresh stream), while rl_attn_decode_ex on that stream is refused."""
    env = dict(os.environ, RL_ATTN_TEST_FAIL_ALLOC="1")
    H.say("no-alloc under forced allocation failure (child process)")
    r = subprocess.run([sys.executable, "-c", CHILD.format(root=ROOT)], env=env, capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 0 and "NOALLOC_CHILD_OK" in r.stdout, r.stdout + r.stderr
