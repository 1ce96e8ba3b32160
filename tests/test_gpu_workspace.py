"""Workspaces: one per (device, stream). Calls on two streams at once each use
their own; releasing every workspace and calling again gives the same bits; a
failed workspace allocation is reported as RL_ERR_WORKSPACE, not a crash."""

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


def test_two_streams_at_once():
    wd = wl.custom(501, "decode", [900, 3, 2500, 64], hq=16, hkv=2, page_size=64)
    we = wl.custom(502, "extend", [700, 300], q_lens=[200, 300], hq=16, hkv=2, page_size=16)
    td, te = wl.materialize(wd, DEV), wl.materialize(we, DEV)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    torch.cuda.synchronize()
    for _ in range(3):
        od = torch.empty_like(td["q"])
        oe = torch.empty_like(te["q"])
        with torch.cuda.stream(s1):
            ra.decode(td["q"], td["k_pages"], td["v_pages"], td["block_table"], td["kv_lens"], td["scale"], out=od,
                      stream=s1)
        with torch.cuda.stream(s2):
            ra.extend(te["q"], te["qo_indptr"], te["k_pages"], te["v_pages"], te["block_table"], te["kv_lens"],
                      te["scale"], out=oe, stream=s2)
        outs.append((od, oe))
    torch.cuda.synchronize()
    ref_d, _ = H.oracle_full(wd, td)
    ref_e, _ = H.oracle_full(we, te)
    for od, oe in outs:
        H.compare(od, ref_d, what="decode on stream 1")
        H.compare(oe, ref_e, what="extend on stream 2")
        assert torch.equal(od.view(torch.int16), outs[0][0].view(torch.int16))
        assert torch.equal(oe.view(torch.int16), outs[0][1].view(torch.int16))
    ra.check_device_errors(s1)
    ra.check_device_errors(s2)


def test_release_then_call_again():
    w = wl.custom(503, "decode", [1200, 77, 5], hq=8, hkv=2, page_size=32)
    t = wl.materialize(w, DEV)
    first, lse1 = H.run_decode(w, t)
    ra.release()
    second, lse2 = H.run_decode(w, t)
    assert torch.equal(first.view(torch.int16), second.view(torch.int16)) and torch.equal(lse1, lse2)
    ra.check_device_errors()


def test_failed_allocation_is_reported():
    """A process whose workspace allocations fail (forced from the host) gets
    RL_ERR_WORKSPACE from the call, and no kernel runs."""
    code = ("import torch\n"
            "from paper_2609_08368_amd import rl_attn as ra, workloads as wl\n"
            "w = wl.custom(504, 'decode', [100, 40], hq=8, hkv=2, page_size=16)\n"
            "t = wl.materialize(w, 'cuda:0')\n"
            "try:\n"
            "    ra.decode(t['q'], t['k_pages'], t['v_pages'], t['block_table'], t['kv_lens'], t['scale'])\n"
            "except ra.RlAttnError as e:\n"
            "    print('status', e.status, flush=True)\n"
            "    raise SystemExit(0)\n"
            "raise SystemExit(1)\n")
    env = dict(os.environ, RL_ATTN_TEST_FAIL_ALLOC="1")
    H.say("subprocess with forced allocation failure")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True, timeout=200)
    assert r.returncode == 0 and "status RL_ERR_WORKSPACE" in r.stdout, r.stdout + r.stderr


def test_host_tensor_is_refused():
    """A tensor that is not on the current device never reaches the library: the
    binding raises before any call (a host pointer would reach a kernel)."""
    w = wl.custom(505, "decode", [100, 40], hq=8, hkv=2, page_size=16)
    t = wl.materialize(w, DEV)
    for name in ("q", "k_pages", "block_table", "kv_lens"):
        args = dict(t)
        args[name] = t[name].cpu()
        with pytest.raises(ValueError, match="current device"):
            ra.decode(args["q"], args["k_pages"], args["v_pages"], args["block_table"], args["kv_lens"], t["scale"])
    out_host = torch.empty(t["q"].shape, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="current device"):
        ra.decode(t["q"], t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], out=out_host)
    ra.check_device_errors()
