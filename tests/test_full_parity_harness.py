"""The full-row parity harness itself (host only): its per-task oracle calls,
(sequence, KV head) slicing and error accumulation give the same answer as one
oracle call over the whole batch, and a planted error anywhere is caught."""

import numpy as np
import pytest
import torch

from paper_2609_08368_amd import workloads as wl
from tests import gpu_helpers as H


def _call(w, t, ref_o, ref_l, q=None, qo_indptr=None, kind=None):
    sc = H.host_scales(t)
    host = {k: H.to_host(v) for k, v in t.items() if isinstance(v, torch.Tensor) and not k.endswith("_scale")}
    kind = kind or w.kind
    return H.HostCall(kind, host["q"] if q is None else q, host["k_pages"], host["v_pages"], host["block_table"],
                      host["kv_lens"], t["scale"], ref_o.astype(np.float32), ref_l.astype(np.float32),
                      qo_indptr=host.get("qo_indptr") if qo_indptr is None else qo_indptr,
                      k_scale=sc.get("k_scale"), v_scale=sc.get("v_scale"))


@pytest.mark.parametrize("fp8", [False, True])
def test_decode_harness_agrees_with_one_oracle_call(fp8):
    w = wl.custom(301, "decode", [0, 1, 17, 300, 64, 129], hq=12, hkv=3, page_size=16)
    t = (wl.materialize_fp8 if fp8 else wl.materialize)(w, "cpu")
    ref_o, ref_l = H.oracle_full(w, t)
    call = _call(w, t, ref_o, ref_l)
    r = H.full_parity(call, "harness decode", workers=3).check("harness decode")
    assert r["rows"] == w.batch * w.hq
    assert r["max_abs"] < 1e-6 and r["lse_rel"] < 1e-6


@pytest.mark.parametrize("fp8", [False, True])
def test_extend_harness_agrees_with_one_oracle_call(fp8):
    w = wl.custom(302, "extend", [40, 100, 0, 90, 7], q_lens=[5, 100, 0, 33, 7], hq=8, hkv=2, page_size=16)
    t = (wl.materialize_fp8 if fp8 else wl.materialize)(w, "cpu")
    ref_o, ref_l = H.oracle_full(w, t)
    call = _call(w, t, ref_o, ref_l)
    accs = [H.full_parity(call, "harness extend", part=p, parts=3, workers=2) for p in range(3)]
    total = H.ParityAcc()
    for a in accs:
        total.merge(a)
    r = total.check("harness extend")
    assert r["rows"] == w.total_q * w.hq
    assert r["max_abs"] < 1e-6 and r["lse_rel"] < 1e-6


@pytest.mark.parametrize("where", ["decode", "extend"])
def test_harness_catches_planted_errors(where):
    if where == "decode":
        w = wl.custom(303, "decode", [3, 50, 200], hq=8, hkv=2, page_size=16)
    else:
        w = wl.custom(304, "extend", [60, 130], q_lens=[20, 64], hq=8, hkv=2, page_size=16)
    t = wl.materialize(w, "cpu")
    ref_o, ref_l = H.oracle_full(w, t)
    # one element off by 0.05: max-abs
    bad = ref_o.copy()
    bad[-1, 5, 77] += 0.05
    with pytest.raises(AssertionError, match="max-abs"):
        H.full_parity(_call(w, t, bad, ref_l), "planted", workers=2).check("planted")
    # two query heads of one KV head swapped in one row: rel-RMS or max-abs
    bad = ref_o.copy()
    bad[0, [4, 5]] = bad[0, [5, 4]]
    with pytest.raises(AssertionError):
        H.full_parity(_call(w, t, bad, ref_l), "planted", workers=2).check("planted")
    # one lse off by 1e-3 relative
    badl = ref_l.copy()
    badl[-1, 2] *= 1 + 1e-3
    with pytest.raises(AssertionError, match="lse"):
        H.full_parity(_call(w, t, ref_o, badl), "planted", workers=2).check("planted")
    # a NaN output
    bad = ref_o.copy()
    bad[0, 0, 0] = np.nan
    with pytest.raises(AssertionError, match="non-finite"):
        H.full_parity(_call(w, t, bad, ref_l), "planted", workers=2).check("planted")


def test_multi_token_layout_matches_extend_rows():
    """Multi-token decode rows ([B, n] flattened, indptr = n * b) are the extend rows of
    n-token chunks ending at each sequence's last key."""
    n = 3
    w = wl.custom(305, "extend", [10, 70, 3], q_lens=[n] * 3, hq=8, hkv=2, page_size=16)
    t = wl.materialize(w, "cpu")
    ref_o, ref_l = H.oracle_full(w, t)
    call = _call(w, t, ref_o, ref_l, qo_indptr=(np.arange(4) * n).astype(np.int32), kind="extend")
    r = H.full_parity(call, "multi-token layout", workers=2).check("multi-token layout")
    assert r["rows"] == 3 * n * 8
