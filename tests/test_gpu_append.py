"""KV append on the GPU (through the C-ABI) against the oracle, bit for bit.

Integer/byte work: the pools after the append must equal the oracle's pools
exactly (every byte, so nothing outside the new positions is touched); FP8
codes are compared exactly (the kernel and the oracle both decide a code from
the float32 quotient of the row by its KV head's scale).
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


def new_rows(w, seed, spread=1.0):
    """Seeded bf16 rows [total_new, Hkv, 128] for K and V (the chunk tokens of an extend workload)."""
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    shape = (w.total_q, w.hkv, 128)
    k = (torch.randn(shape, generator=g, device=DEV) * spread).to(torch.bfloat16)
    v = (torch.randn(shape, generator=g, device=DEV) * spread).to(torch.bfloat16)
    return k, v


def host(t):
    return H.to_host(t)


def run_append(t, k, v, fp8):
    kp, vp = t["k_pages"].clone(), t["v_pages"].clone()
    if fp8:
        ra.append_kv_fp8(k, v, t["qo_indptr"], t["block_table"], t["kv_lens"], kp, vp, t["k_scale"], t["v_scale"])
    else:
        ra.append_kv(k, v, t["qo_indptr"], t["block_table"], t["kv_lens"], kp, vp)
    torch.cuda.synchronize()
    return kp, vp


def oracle_append(w, t, k, v, fp8):
    sc = {"k_scale": t["k_scale"].cpu().numpy(), "v_scale": t["v_scale"].cpu().numpy()} if fp8 else {}
    return oracle.append_kv(host(t["k_pages"]), host(t["v_pages"]), w.block_table, w.kv_lens, w.qo_indptr,
                            host(k), host(v), **sc)


CASES = [
    # (page_size, Hkv, kv_lens, chunk lengths)
    (16, 2, [40, 17, 100], [5, 17, 1]),          # a chunk that is the whole sequence
    (64, 8, [500, 70, 64], [33, 70, 64]),
    (8, 1, [90, 13, 9], [20, 13, 0]),            # an empty chunk
    (128, 4, [600, 1], [257, 1]),
    (32, 16, [200, 50], [150, 7]),
]


@pytest.mark.parametrize("fp8", [False, True])
@pytest.mark.parametrize("case", CASES, ids=[f"P{c[0]}_kv{c[1]}_{i}" for i, c in enumerate(CASES)])
def test_append_matches_oracle_bitwise(case, fp8):
    ps, hkv, kv, ql = case
    w = wl.custom(140 + sum(ql), "extend", kv, q_lens=ql, hq=hkv, hkv=hkv, page_size=ps)
    H.say(f"append {case} fp8={fp8}")
    t = (wl.materialize_fp8 if fp8 else wl.materialize)(w, DEV)
    k, v = new_rows(w, 7 + sum(ql))
    kp, vp = run_append(t, k, v, fp8)
    ok, ov = oracle_append(w, t, k, v, fp8)
    assert np.array_equal(host(kp), ok), "K pool differs from the oracle's"
    assert np.array_equal(host(vp), ov), "V pool differs from the oracle's"
    ra.check_device_errors()


@pytest.mark.parametrize("fp8", [False, True])
@pytest.mark.parametrize("batch", [64, 128, 255, 256, 300])
def test_append_many_sequences(batch, fp8):
    """Batches past the FP8 owner search's wave-wide form (up to 63 sequences; a binary
    search from 64 on, as for bf16 pages): decode-like steps of zero to two rows per
    sequence, empty ones mixed in, 8 KV heads."""
    rng = np.random.default_rng(160 + batch)
    ql = rng.choice([0, 1, 1, 1, 2], size=batch)
    ql[0], ql[-1] = 0, 1                       # an empty first chunk, a row in the last
    kv = ql + rng.integers(0, 70, size=batch)
    w = wl.custom(160 + batch, "extend", [int(x) for x in kv], q_lens=[int(x) for x in ql], hq=8, hkv=8,
                  page_size=16)
    H.say(f"append {batch} sequences fp8={fp8}")
    t = (wl.materialize_fp8 if fp8 else wl.materialize)(w, DEV)
    k, v = new_rows(w, 9 + batch)
    kp, vp = run_append(t, k, v, fp8)
    ok, ov = oracle_append(w, t, k, v, fp8)
    assert np.array_equal(host(kp), ok), "K pool differs from the oracle's"
    assert np.array_equal(host(vp), ov), "V pool differs from the oracle's"
    ra.check_device_errors()


def test_append_fp8_rounding_and_saturation():
    """Near-ties where the float32 quotient decides the code, values beyond 448 x scale
    (saturate), zeros of both signs, and values in the subnormal range."""
    w = wl.custom(150, "extend", [20], q_lens=[4], hq=2, hkv=2, page_size=16)
    H.say("fp8 append rounding")
    t = wl.materialize_fp8(w, DEV)
    t["k_scale"] = torch.tensor([0.3, 1 / 3], dtype=torch.float32, device=DEV)
    t["v_scale"] = torch.tensor([0.001, 2.0], dtype=torch.float32, device=DEV)
    bits = np.zeros((4, 2, 128), np.uint16)
    bits[0, 0, :2] = [0x3B90, 0x3B60]
    bits[0, 1, :3] = [0x3A80, 0x3BA0, 0x3C10]
    bits[1, :, :4] = [0x8000, 0x0000, 0x4400, 0xC400]          # -0, +0, 512, -512
    rng = np.random.default_rng(3)
    bits[2] = rng.integers(0x3000, 0x3A00, size=(2, 128))        # small values: subnormal codes
    bits[3] = rng.integers(0, 0x10000, size=(2, 128))            # anything, NaN/inf included
    k = torch.from_numpy(bits.view(np.int16)).to(DEV).view(torch.bfloat16)
    v = k.clone()
    kp, vp = run_append(t, k, v, True)
    ok, ov = oracle_append(w, t, k, v, True)
    gk, gv = host(kp), host(vp)
    nan_k = (ok & 0x7F) == 0x7F
    assert np.array_equal((gk & 0x7F) == 0x7F, nan_k)            # NaN inputs give a NaN code
    assert np.array_equal(np.where(nan_k, 0, gk), np.where(nan_k, 0, ok)), "K codes"
    nan_v = (ov & 0x7F) == 0x7F
    assert np.array_equal(np.where(nan_v, 0, gv), np.where(nan_v, 0, ov)), "V codes"


def test_append_then_extend_equals_materialised_pages():
    """Appending a chunk's rows and then attending gives the bits of attending over pages
    that held those rows from the start."""
    w = wl.custom(151, "extend", [700, 250, 90], q_lens=[300, 250, 1], hq=16, hkv=2, page_size=64)
    H.say("append then extend")
    t = wl.materialize(w, DEV)
    # take the chunk rows out of the pages, clear them, append them back
    idx = []
    for b in range(w.batch):
        n, kv = int(w.q_lens[b]), int(w.kv_lens[b])
        idx += [(int(w.block_table[b, tt // 64]), tt % 64) for tt in range(kv - n, kv)]
    pg = torch.tensor([p for p, _ in idx], device=DEV)
    sl = torch.tensor([s for _, s in idx], device=DEV)
    k_rows, v_rows = t["k_pages"][pg, sl].clone(), t["v_pages"][pg, sl].clone()
    cleared = dict(t)
    cleared["k_pages"], cleared["v_pages"] = t["k_pages"].clone(), t["v_pages"].clone()
    cleared["k_pages"][pg, sl] = 0
    cleared["v_pages"][pg, sl] = 0
    kp, vp = run_append(cleared, k_rows, v_rows, False)
    assert torch.equal(kp.view(torch.int16), t["k_pages"].view(torch.int16))
    appended = dict(t)
    appended["k_pages"], appended["v_pages"] = kp, vp
    o1, l1 = H.run_extend(w, appended)
    o2, l2 = H.run_extend(w, t)
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)) and torch.equal(l1, l2)


def test_append_bad_inputs_are_not_written_and_reported():
    w = wl.custom(152, "extend", [40, 30], q_lens=[4, 3], hq=2, hkv=2, page_size=16)
    H.say("append error paths")
    t = wl.materialize(w, DEV)
    k, v = new_rows(w, 9)
    ra.check_device_errors()
    bad = dict(t)
    bad["block_table"] = t["block_table"].clone()
    bad["block_table"][0, 2] = w.num_pages + 5                   # sequence 0's new rows live in page 2
    kp, vp = run_append(bad, k, v, False)
    with pytest.raises(ra.RlAttnError) as e:
        ra.check_device_errors()
    assert "page-id-out-of-range" in str(e.value)
    # sequence 1 is written, sequence 0 is not; nothing else changes
    ref_k, _ = oracle.append_kv(host(t["k_pages"]), host(t["v_pages"]), w.block_table[1:], w.kv_lens[1:],
                                np.array([0, 3], np.int32), host(k)[4:], host(v)[4:])
    assert np.array_equal(host(kp), ref_k), "only the valid sequence is written"
    short = dict(t)
    short["kv_lens"] = torch.tensor([3, 30], dtype=torch.int32, device=DEV)   # 3 < 4 new rows
    run_append(short, k, v, False)
    with pytest.raises(ra.RlAttnError) as e:
        ra.check_device_errors()
    assert "kv_lens-shorter-than-chunk" in str(e.value)


@pytest.mark.parametrize("fp8", [False, True])
def test_append_full_size(fp8):
    """The multi-turn extend batch's chunks (33.8K tokens x 8 KV heads): every new position
    holds the row (bf16) or the oracle's codes (FP8)."""
    w = wl.extend_multiturn()
    H.say(f"append full size fp8={fp8}: {w.total_q} rows")
    t = (wl.materialize_fp8 if fp8 else wl.materialize)(w, DEV, poison=False)
    k, v = new_rows(w, 11)
    kp, vp = t["k_pages"], t["v_pages"]
    if fp8:
        ra.append_kv_fp8(k, v, t["qo_indptr"], t["block_table"], t["kv_lens"], kp, vp, t["k_scale"], t["v_scale"])
    else:
        ra.append_kv(k, v, t["qo_indptr"], t["block_table"], t["kv_lens"], kp, vp)
    torch.cuda.synchronize()
    ra.check_device_errors()
    pos = []
    for b in range(w.batch):
        n, kv = int(w.q_lens[b]), int(w.kv_lens[b])
        pos += [(int(w.block_table[b, tt // w.page_size]), tt % w.page_size) for tt in range(kv - n, kv)]
    pg = torch.tensor([p for p, _ in pos], device=DEV)
    sl = torch.tensor([s for _, s in pos], device=DEV)
    gk, gv = host(kp[pg, sl]), host(vp[pg, sl])
    if fp8:
        want_k = oracle.quantize_rows(host(k), t["k_scale"].cpu().numpy())
        want_v = oracle.quantize_rows(host(v), t["v_scale"].cpu().numpy())
    else:
        want_k, want_v = host(k), host(v)
    assert np.array_equal(gk, want_k) and np.array_equal(gv, want_v)
    del t
    torch.cuda.empty_cache()


@pytest.mark.parametrize("scales", [(0.3, 1 / 3), (0.7, 0.1), (0.013, 0.0125), (1.0, 2.0 ** -20)])
def test_append_fp8_every_bf16_value(scales):
    """All 65,536 bf16 bit patterns appended under two KV-head scales: every code equals the
    oracle's (NaN inputs must give a NaN code)."""
    w = wl.custom(153, "extend", [300], q_lens=[256], hq=2, hkv=2, page_size=16)
    H.say(f"fp8 append, every bf16 value, scales {scales}")
    t = wl.materialize_fp8(w, DEV)
    t["k_scale"] = torch.tensor(scales, dtype=torch.float32, device=DEV)
    t["v_scale"] = torch.tensor(scales[::-1], dtype=torch.float32, device=DEV)
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16).reshape(256, 2, 128)
    k = torch.from_numpy(bits.view(np.int16)).to(DEV).view(torch.bfloat16)
    v = torch.from_numpy(bits[::-1].copy().view(np.int16)).to(DEV).view(torch.bfloat16)
    kp, vp = run_append(t, k, v, True)
    ok, ov = oracle_append(w, t, k, v, True)
    for got, want in ((host(kp), ok), (host(vp), ov)):
        nan = (want & 0x7F) == 0x7F
        assert np.array_equal((got & 0x7F) == 0x7F, nan), "NaN codes"
        assert np.array_equal(np.where(nan, 0, got), np.where(nan, 0, want)), "codes differ from the oracle"
