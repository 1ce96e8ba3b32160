"""Checks that pin the float64 oracle to things other than itself.

Each ``pin_*`` function takes an oracle-like object (the ``oracle`` package, or
a deliberately broken copy of it in the mutation tests) and raises
``AssertionError`` when the oracle disagrees with what mathematics fixes:

* brute-force dense attention through scipy's softmax / logsumexp, on a
  different data layout (dense, GQA expanded with ``np.repeat``);
* a single key (output equals that key's value row exactly);
* identical keys (output equals the mean of the value rows, lse = s + ln L);
* page size and physical page order (bitwise invariance);
* split/merge identity;
* extend versus decode, and extend from an empty prefix versus textbook causal
  attention;
* GQA expansion to multi-head attention;
* scale homogeneity ((2q, scale/2) is bitwise the same problem);
* batch permutation and shared-versus-private prefix pages;
* FP8 E4M3 KV pages: every code against torch's independent float8_e4m3fn
  conversion and the format's closed forms; with unit scales the result equals
  the bf16 oracle on the same values bitwise; per-KV-head power-of-two scales
  equal exactly scaled bf16 pages; arbitrary scales agree with brute force;
* KV append: clearing and re-appending the last rows restores the pages
  bitwise; the E4M3 encoder against torch's float8_e4m3fn cast (values,
  midpoints, both signs), round trips, brute-force nearest values and
  saturation; FP8 append writes torch's cast of the float32 quotient, only at
  the new positions.

The paper prints no attention values, so parity with printed values is
unpinned; the closed-form golden file in ``tests/golden`` stands in for a
worked example.
"""

from __future__ import annotations

import json
import math
import os

import numpy as np
import scipy.special

D = 128
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float -> bf16 bit patterns by truncating float32 (any bit pattern is a valid bf16)."""
    return (np.asarray(x, dtype=np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def from_bits(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def pack_pages(dense_bits, lens, page_size, rng, extra_pages=2):
    """Dense per-sequence rows ``[B, Lmax, Hkv, D]`` -> shuffled page pool + block table.

    Unused pages and tail slots hold NaN (bf16 0x7fc0).
    """
    b_count, _, hkv, d = dense_bits.shape
    used = [-(-int(l) // page_size) for l in lens]
    total = sum(used) + extra_pages
    perm = rng.permutation(total)
    pool = np.full((total, page_size, hkv, d), 0x7FC0, dtype=np.uint16)
    table = np.full((b_count, max(1, max(used))), perm[-1], dtype=np.int32)
    nxt = 0
    for b in range(b_count):
        for j in range(used[b]):
            pid = perm[nxt]
            nxt += 1
            table[b, j] = pid
            take = min(page_size, int(lens[b]) - j * page_size)
            pool[pid, :take] = dense_bits[b, j * page_size:j * page_size + take]
    return pool, table


def dense_reference(q_bits, k_bits, v_bits, lens, scale, causal_limits=None):
    """Textbook attention on dense tensors with scipy (independent formulation).

    q ``[B, Hq, D]`` (decode) ; k/v ``[B, Lmax, Hkv, D]``. GQA is expanded by
    repeating each KV head ``Hq/Hkv`` times. Returns (out [B,Hq,D], lse [B,Hq]).
    """
    q = from_bits(q_bits)
    k = from_bits(k_bits)
    v = from_bits(v_bits)
    b_count, hq, _ = q.shape
    r = hq // k.shape[2]
    k = np.repeat(k, r, axis=2)
    v = np.repeat(v, r, axis=2)
    out = np.zeros_like(q)
    lse = np.zeros((b_count, hq))
    sc = float(np.float32(scale))
    for b in range(b_count):
        l = int(lens[b])
        s = np.einsum("hd,thd->ht", q[b], k[b, :l]) * sc
        out[b] = np.einsum("ht,thd->hd", scipy.special.softmax(s, axis=1), v[b, :l])
        lse[b] = scipy.special.logsumexp(s, axis=1)
    return out, lse


def _rel(a, b):
    return float(np.max(np.abs(a - b)) / max(1e-300, np.max(np.abs(b))))


def _random_problem(rng, b_count=3, hq=8, hkv=2, lens=(5, 17, 40)):
    lmax = max(lens)
    q = to_bf16_bits(rng.standard_normal((b_count, hq, D)))
    k = to_bf16_bits(rng.standard_normal((b_count, lmax, hkv, D)))
    v = to_bf16_bits(rng.standard_normal((b_count, lmax, hkv, D)))
    return q, k, v, np.array(lens, dtype=np.int32)


def pin_brute_force(orc, seed=0):
    rng = np.random.default_rng(seed)
    for hq, hkv, lens, ps in [(8, 2, (5, 17, 40), 16), (6, 3, (1, 2, 33), 4), (4, 4, (64, 7, 9), 8)]:
        q, k, v, lens = _random_problem(rng, len(lens), hq, hkv, lens)
        scale = 1.0 / math.sqrt(D)
        kp, bt = pack_pages(k, lens, ps, rng)
        vp = np.empty_like(kp)
        # V shares the block table: pack V into the same physical slots
        for b in range(len(lens)):
            for j in range(-(-int(lens[b]) // ps)):
                take = min(ps, int(lens[b]) - j * ps)
                vp[bt[b, j], :take] = v[b, j * ps:j * ps + take]
        vp[np.isin(np.arange(kp.shape[0]), bt, invert=True)] = 0x7FC0
        out, lse = orc.decode(q, kp, vp, bt, lens, scale)
        ref_o, ref_l = dense_reference(q, k, v, lens, scale)
        assert _rel(out, ref_o) < 1e-12, "decode != dense scipy attention"
        assert np.max(np.abs(lse - ref_l)) < 1e-12 * max(1.0, np.max(np.abs(ref_l))), "lse != scipy logsumexp"


def pin_single_key(orc, seed=1):
    rng = np.random.default_rng(seed)
    q = to_bf16_bits(rng.standard_normal((2, 4, D)))
    k = to_bf16_bits(rng.standard_normal((2, 1, 1, D)))
    v = to_bf16_bits(rng.standard_normal((2, 1, 1, D)))
    lens = np.array([1, 1], np.int32)
    kp, bt = pack_pages(k, lens, 16, rng)
    vp = kp.copy()
    for b in range(2):
        vp[bt[b, 0], 0] = v[b, 0]
    scale = 0.37
    out, lse = orc.decode(q, kp, vp, bt, lens, scale)
    for b in range(2):
        for h in range(4):
            assert np.array_equal(out[b, h], from_bits(v[b, 0, 0])), "single key: out != v exactly"
            s0 = float(np.float32(scale)) * math.fsum(from_bits(q[b, h]) * from_bits(k[b, 0, 0]))
            assert abs(lse[b, h] - s0) <= 1e-13 * max(1.0, abs(s0)), "single key: lse != score"


def pin_uniform_keys(orc, seed=2):
    rng = np.random.default_rng(seed)
    lens = np.array([7, 50], np.int32)
    q = to_bf16_bits(rng.standard_normal((2, 4, D)))
    krow = to_bf16_bits(rng.standard_normal((2, 1, 2, D)))
    k = np.repeat(krow, 50, axis=1)
    v = to_bf16_bits(rng.standard_normal((2, 50, 2, D)))
    kp, bt = pack_pages(k, lens, 8, rng)
    vp = kp.copy()
    for b in range(2):
        for j in range(-(-int(lens[b]) // 8)):
            take = min(8, int(lens[b]) - j * 8)
            vp[bt[b, j], :take] = v[b, j * 8:j * 8 + take]
    scale = 0.11
    out, lse = orc.decode(q, kp, vp, bt, lens, scale)
    for b in range(2):
        l = int(lens[b])
        for h in range(4):
            g = h // 2
            mean = np.mean(from_bits(v[b, :l, g]), axis=0)
            assert _rel(out[b, h], mean) < 1e-13, "uniform keys: out != mean(v)"
            s = float(np.float32(scale)) * math.fsum(from_bits(q[b, h]) * from_bits(krow[b, 0, g]))
            assert abs(lse[b, h] - (s + math.log(l))) < 1e-12, "uniform keys: lse != s + ln L"


def pin_page_invariance(orc, seed=3):
    rng = np.random.default_rng(seed)
    q, k, v, lens = _random_problem(rng, 3, 8, 2, (33, 64, 100))
    results = []
    for ps in (1, 8, 16, 64):
        for rep in range(2):
            kp, bt = pack_pages(k, lens, ps, rng, extra_pages=rep + 1)
            vp = np.full_like(kp, 0x7FC0)
            for b in range(3):
                for j in range(-(-int(lens[b]) // ps)):
                    take = min(ps, int(lens[b]) - j * ps)
                    vp[bt[b, j], :take] = v[b, j * ps:j * ps + take]
            results.append(orc.decode(q, kp, vp, bt, lens, 0.0883883))
    for o, l in results[1:]:
        assert np.array_equal(o, results[0][0]) and np.array_equal(l, results[0][1]), \
            "result depends on page size or physical page order"


def pin_split_merge(orc, seed=4):
    rng = np.random.default_rng(seed)
    qf = from_bits(to_bf16_bits(rng.standard_normal((3, D))))
    k = from_bits(to_bf16_bits(rng.standard_normal((200, D))))
    v = from_bits(to_bf16_bits(rng.standard_normal((200, D))))
    full_o, full_l = orc.attend(qf, k, v, 0.2)
    for _ in range(5):
        cuts = np.sort(rng.choice(np.arange(1, 200), size=rng.integers(1, 6), replace=False))
        bounds = [0, *cuts.tolist(), 200]
        parts = [orc.attend_range(qf, k, v, 0.2, a, b) for a, b in zip(bounds[:-1], bounds[1:])]
        # add an empty part too: it must carry no weight
        parts.append(orc.attend_range(qf, k, v, 0.2, 10, 10))
        o_parts = np.stack([p[0] for p in parts])[None]          # [1, S, 3, D]
        l_parts = np.stack([p[1] for p in parts])[None]          # [1, S, 3]
        mo, ml = orc.merge(o_parts, l_parts, np.array([len(parts)]))
        assert _rel(mo[0], full_o) < 1e-12, "merge of split partials != unsplit output"
        assert np.max(np.abs(ml[0] - full_l)) < 1e-12 * max(1, np.max(np.abs(full_l))), "merged lse"
    eo, el = orc.merge(np.zeros((1, 2, 1, D)), np.full((1, 2, 1), -np.inf), np.array([2]))
    assert np.all(eo == 0) and np.all(el == -np.inf), "all-empty merge must give 0 / -inf"


def pin_extend(orc, seed=5):
    rng = np.random.default_rng(seed)
    hq, hkv, ps = 8, 2, 8
    kv = np.array([23, 9, 40], np.int32)
    n = np.array([5, 9, 1], np.int32)              # second sequence: empty prefix
    indptr = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    q = to_bf16_bits(rng.standard_normal((int(n.sum()), hq, D)))
    k = to_bf16_bits(rng.standard_normal((3, 40, hkv, D)))
    v = to_bf16_bits(rng.standard_normal((3, 40, hkv, D)))
    kp, bt = pack_pages(k, kv, ps, rng)
    vp = np.full_like(kp, 0x7FC0)
    for b in range(3):
        for j in range(-(-int(kv[b]) // ps)):
            take = min(ps, int(kv[b]) - j * ps)
            vp[bt[b, j], :take] = v[b, j * ps:j * ps + take]
    scale = 0.09
    out, lse = orc.extend(q, indptr, kp, vp, bt, kv, scale, row_block=2)
    for b in range(3):
        p = int(kv[b] - n[b])
        for i in range(int(n[b])):
            row = indptr[b] + i
            do, dl = orc.decode(q[row:row + 1], kp, vp, bt[b:b + 1], np.array([p + i + 1]), scale)
            assert _rel(out[row], do[0]) < 1e-13 and np.max(np.abs(lse[row] - dl[0])) < 1e-12, \
                "extend row i != decode over p+i+1 keys"
    # empty prefix: textbook causal self-attention on the chunk (scipy, dense mask)
    b = 1
    qs = from_bits(q[indptr[b]:indptr[b + 1]])          # [n, Hq, D]
    ks = np.repeat(from_bits(k[b, :9]), hq // hkv, axis=1)
    vs = np.repeat(from_bits(v[b, :9]), hq // hkv, axis=1)
    s = np.einsum("ihd,jhd->hij", qs, ks) * float(np.float32(scale))
    s = s + np.triu(np.full((9, 9), -np.inf), k=1)[None]
    ref = np.einsum("hij,jhd->ihd", scipy.special.softmax(s, axis=2), vs)
    assert _rel(out[indptr[b]:indptr[b + 1]], ref) < 1e-12, "extend with empty prefix != causal attention"


def pin_gqa_expansion(orc, seed=6):
    rng = np.random.default_rng(seed)
    q, k, v, lens = _random_problem(rng, 2, 12, 3, (30, 45))
    kp, bt = pack_pages(k, lens, 16, rng)
    vp = np.full_like(kp, 0x7FC0)
    for b in range(2):
        for j in range(-(-int(lens[b]) // 16)):
            take = min(16, int(lens[b]) - j * 16)
            vp[bt[b, j], :take] = v[b, j * 16:j * 16 + take]
    out, lse = orc.decode(q, kp, vp, bt, lens, 0.1)
    kp_mha = np.repeat(kp, 4, axis=2)                  # KV head g -> query heads 4g..4g+3
    vp_mha = np.repeat(vp, 4, axis=2)
    out2, lse2 = orc.decode(q, kp_mha, vp_mha, bt, lens, 0.1)
    assert _rel(out, out2) < 1e-13 and np.max(np.abs(lse - lse2)) < 1e-12, "GQA != expanded MHA"


def pin_scale_homogeneity(orc, seed=7):
    rng = np.random.default_rng(seed)
    q, k, v, lens = _random_problem(rng, 2, 4, 2, (20, 31))
    kp, bt = pack_pages(k, lens, 8, rng)
    vp = np.full_like(kp, 0x7FC0)
    for b in range(2):
        for j in range(-(-int(lens[b]) // 8)):
            take = min(8, int(lens[b]) - j * 8)
            vp[bt[b, j], :take] = v[b, j * 8:j * 8 + take]
    scale = np.float32(0.0883883)
    o1, l1 = orc.decode(q, kp, vp, bt, lens, float(scale))
    q2 = to_bf16_bits(2.0 * from_bits(q))              # exact: exponent + 1
    o2, l2 = orc.decode(q2, kp, vp, bt, lens, float(scale / np.float32(2)))
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2), "(2q, scale/2) must be the same problem"


def pin_batch_and_sharing(orc, seed=8):
    rng = np.random.default_rng(seed)
    q, k, v, lens = _random_problem(rng, 4, 8, 2, (40, 48, 33, 64))
    # sequences 0..3 share their first 32 tokens (4 pages of 8) physically
    k[:, :32] = k[0:1, :32]
    v[:, :32] = v[0:1, :32]
    ps = 8
    kp, bt = pack_pages(k, lens, ps, rng)
    vp = np.full_like(kp, 0x7FC0)
    for b in range(4):
        for j in range(-(-int(lens[b]) // ps)):
            take = min(ps, int(lens[b]) - j * ps)
            vp[bt[b, j], :take] = v[b, j * ps:j * ps + take]
    o_priv, l_priv = orc.decode(q, kp, vp, bt, lens, 0.1)
    bt_shared = bt.copy()
    bt_shared[1:, :4] = bt[0, :4]                      # point members at the leader's prefix pages
    o_sh, l_sh = orc.decode(q, kp, vp, bt_shared, lens, 0.1)
    assert np.array_equal(o_priv, o_sh) and np.array_equal(l_priv, l_sh), "shared prefix pages changed result"
    perm = np.array([2, 0, 3, 1])
    o_p, l_p = orc.decode(q[perm], kp, vp, bt[perm], lens[perm], 0.1)
    assert np.array_equal(o_p, o_priv[perm]) and np.array_equal(l_p, l_priv[perm]), "batch order changed result"


def pin_golden(orc):
    with open(os.path.join(GOLDEN, "closed_form_cases.json")) as f:
        cases = json.load(f)["cases"]
    env = {"e": math.e, "log": math.log, "exp": math.exp, "sqrt": math.sqrt}
    for case in cases:
        lens = np.array(case["lens"], np.int32)
        hq, hkv, ps = case["hq"], case["hkv"], case["page_size"]
        q = np.zeros((len(lens), hq, D), np.float32)
        kd = np.zeros((len(lens), max(lens), hkv, D), np.float32)
        vd = np.zeros_like(kd)
        for b, h, d, x in case["q"]:
            q[b, h, d] = x
        for b, t, g, d, x in case["k"]:
            kd[b, t, g, d] = x
        for b, t, g, d, x in case["v"]:
            vd[b, t, g, d] = x
        rng = np.random.default_rng(0)
        kp, bt = pack_pages(to_bf16_bits(kd), lens, ps, rng)
        vp = np.full_like(kp, 0x7FC0)
        for b in range(len(lens)):
            for j in range(-(-int(lens[b]) // ps)):
                take = min(ps, int(lens[b]) - j * ps)
                vp[bt[b, j], :take] = to_bf16_bits(vd[b, j * ps:j * ps + take])
        out, lse = orc.decode(to_bf16_bits(q), kp, vp, bt, lens, case["scale"])
        for b, h, d, expr in case["expect_out"]:
            want = eval(expr, {"__builtins__": {}}, env)   # closed forms from the fixture
            assert abs(out[b, h, d] - want) < 1e-14 * max(1.0, abs(want)), f"{case['name']}: out[{b},{h},{d}]"
        for b, h, expr in case["expect_lse"]:
            want = eval(expr, {"__builtins__": {}}, env)
            assert abs(lse[b, h] - want) < 1e-14 * max(1.0, abs(want)), f"{case['name']}: lse[{b},{h}]"


def _fp8_values_torch(codes: np.ndarray) -> np.ndarray:
    """FP8 E4M3 codes -> float64 through torch's float8_e4m3fn (an implementation independent of the oracle)."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(codes, dtype=np.uint8)).view(torch.float8_e4m3fn)
    return t.to(torch.float64).numpy()


def _fp8_problem(rng, lens=(21, 40, 9), hq=8, hkv=2, ps=8):
    """Random FP8 codes (finite only) for K and V, paged; and the same values as bf16 bits."""
    import torch

    lens = np.array(lens, dtype=np.int32)
    b_count, lmax = len(lens), int(max(lens))
    q = to_bf16_bits(rng.standard_normal((b_count, hq, D)))
    pages = []
    for _ in range(2):
        x = torch.from_numpy(rng.standard_normal((b_count, lmax, hkv, D)).astype(np.float32) * 3.0)
        codes = x.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        pages.append(codes)
    rng_pages = np.random.default_rng(int(rng.integers(1 << 30)))
    kp, bt = pack_pages(pages[0].astype(np.uint16), lens, ps, rng_pages)      # pack as uint16, keep uint8 values
    vp = np.full_like(kp, 0x7F)
    for b in range(b_count):
        for j in range(-(-int(lens[b]) // ps)):
            take = min(ps, int(lens[b]) - j * ps)
            vp[bt[b, j], :take] = pages[1][b, j * ps:j * ps + take]
    kp = np.where(kp == 0x7FC0, 0x7F, kp).astype(np.uint8)                  # NaN filler -> FP8 NaN code
    vp = vp.astype(np.uint8)
    return q, kp, vp, bt, lens


def _fp8_as_bf16_bits(codes: np.ndarray, factor=None) -> np.ndarray:
    """The FP8 values (times an optional per-KV-head power of two) as bf16 bits, via torch (exact)."""
    vals = _fp8_values_torch(codes)
    if factor is not None:
        vals = vals * np.asarray(factor, dtype=np.float64)[None, None, :, None]
    return to_bf16_bits(vals.astype(np.float32))


def pin_fp8_codes(orc):
    codes = np.arange(256, dtype=np.uint8)
    mine = orc.fp8_e4m3_to_f64(codes)
    ref = _fp8_values_torch(codes)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(mine), nan) and nan.sum() == 2, "NaN codes"
    assert np.array_equal(mine[~nan], ref[~nan]), "FP8 E4M3 decoding differs from torch's float8_e4m3fn"
    closed = {0x00: 0.0, 0x01: 2.0 ** -9, 0x07: 7 * 2.0 ** -9, 0x08: 2.0 ** -6, 0x38: 1.0, 0x3C: 1.5,
              0x7E: 448.0, 0x80: -0.0, 0xB8: -1.0, 0xFE: -448.0}
    for c, want in closed.items():
        assert mine[c] == want and np.signbit(mine[c]) == np.signbit(want), f"code {c:#04x}"


def pin_fp8_equals_bf16(orc, seed=9):
    rng = np.random.default_rng(seed)
    q, kp, vp, bt, lens = _fp8_problem(rng)
    ones = np.ones(2, np.float32)
    o8, l8 = orc.decode(q, kp, vp, bt, lens, 0.0883883, k_scale=ones, v_scale=ones)
    ob, lb = orc.decode(q, _fp8_as_bf16_bits(kp), _fp8_as_bf16_bits(vp), bt, lens, 0.0883883)
    assert np.array_equal(o8, ob) and np.array_equal(l8, lb), "FP8 pages differ from the same values in bf16"
    qo = np.array([0, 5, 45, 54], np.int32)[: len(lens) + 1]
    qe = to_bf16_bits(rng.standard_normal((int(qo[-1]), 8, D)))
    kvl = np.maximum(lens, np.diff(qo))
    e8, m8 = orc.extend(qe, qo, kp, vp, bt, kvl, 0.1, k_scale=ones, v_scale=ones)
    eb, mb = orc.extend(qe, qo, _fp8_as_bf16_bits(kp), _fp8_as_bf16_bits(vp), bt, kvl, 0.1)
    assert np.array_equal(e8, eb) and np.array_equal(m8, mb), "FP8 extend differs from bf16"


def pin_fp8_scales(orc, seed=10):
    rng = np.random.default_rng(seed)
    q, kp, vp, bt, lens = _fp8_problem(rng, lens=(33, 7), hq=4, hkv=2)
    ks = np.array([0.25, 4.0], np.float32)
    vs = np.array([2.0, 0.5], np.float32)
    o8, l8 = orc.decode(q, kp, vp, bt, lens, 0.07, k_scale=ks, v_scale=vs)
    ob, lb = orc.decode(q, _fp8_as_bf16_bits(kp, ks), _fp8_as_bf16_bits(vp, vs), bt, lens, 0.07)
    assert np.array_equal(o8, ob) and np.array_equal(l8, lb), "per-KV-head scales are not applied per head"
    # arbitrary scales against dense brute force (scipy) on the dequantised values
    ks = np.array([0.013, 0.71], np.float32)
    vs = np.array([1.7, 0.0042], np.float32)
    o8, l8 = orc.decode(q, kp, vp, bt, lens, 0.07, k_scale=ks, v_scale=vs)
    lmax = int(lens.max())
    kd = np.zeros((len(lens), lmax, 2, D))
    vd = np.zeros_like(kd)
    for b in range(len(lens)):
        for t in range(int(lens[b])):
            kd[b, t] = _fp8_values_torch(kp[bt[b, t // 8], t % 8]) * ks[:, None].astype(np.float64)
            vd[b, t] = _fp8_values_torch(vp[bt[b, t // 8], t % 8]) * vs[:, None].astype(np.float64)
    qf = from_bits(q)
    for b in range(len(lens)):
        for h in range(4):
            g, l = h // 2, int(lens[b])
            s = float(np.float32(0.07)) * (kd[b, :l, g] @ qf[b, h])
            want_o = scipy.special.softmax(s) @ vd[b, :l, g]
            assert _rel(o8[b, h], want_o) < 1e-12, "FP8 decode vs brute force"
            assert abs(l8[b, h] - scipy.special.logsumexp(s)) < 1e-12 * max(1.0, abs(l8[b, h]))


def _fp8_encode_torch(x: np.ndarray) -> np.ndarray:
    """torch's float8_e4m3fn cast (round to nearest even) as uint8 codes; an independent encoder."""
    import torch

    return torch.from_numpy(np.asarray(x, np.float32).copy()).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def pin_fp8_encode(orc, seed=11):
    rng = np.random.default_rng(seed)
    # every finite value and every midpoint between neighbours (exact in float32), both signs
    finite = _fp8_values_torch(np.arange(0x7F, dtype=np.uint8))
    mids = (finite[:-1] + finite[1:]) / 2
    mag = np.exp2(rng.uniform(-12, np.log2(448.0), 4000))
    x = np.concatenate([finite, mids, mag, [0.0, 440.0, 447.9, 448.0]]).astype(np.float32)
    x = np.concatenate([x, -x])
    got = orc.fp8_e4m3_encode(x)
    assert np.array_equal(got, _fp8_encode_torch(x)), "E4M3 encoding differs from torch's float8_e4m3fn cast"
    # round trip of every finite code, and brute-force nearest with ties to the even code
    codes = np.array([c for c in range(256) if c & 0x7F != 0x7F], dtype=np.uint8)
    assert np.array_equal(orc.fp8_e4m3_encode(_fp8_values_torch(codes).astype(np.float32)), codes)
    y = (rng.standard_normal(2000) * np.exp2(rng.uniform(-10, 8, 2000))).astype(np.float32)
    y = y[np.abs(y) <= 448]
    dec = _fp8_values_torch(orc.fp8_e4m3_encode(y))
    dist = np.abs(y.astype(np.float64)[:, None] - np.concatenate([finite, -finite])[None, :])
    assert np.all(np.abs(dec - y) <= dist.min(axis=1)), "not the nearest E4M3 value"
    # saturation and NaN
    sat = orc.fp8_e4m3_encode(np.array([449.0, 480.0, 1e6, np.inf, -500.0, -np.inf], np.float32))
    assert list(sat) == [0x7E] * 4 + [0xFE] * 2, "magnitudes above 448 must saturate"
    assert orc.fp8_e4m3_encode(np.array([np.nan], np.float32))[0] & 0x7F == 0x7F


def _append_problem(rng, lens=(40, 9, 71, 16), chunk=(7, 9, 1, 16), hkv=2, page_size=8):
    lens = np.array(lens, np.int32)
    rows = to_bf16_bits(rng.standard_normal((len(lens), int(lens.max()), hkv, D)))
    vrows = to_bf16_bits(rng.standard_normal((len(lens), int(lens.max()), hkv, D)))
    kp, bt = pack_pages(rows, lens, page_size, np.random.default_rng(99))
    vp, _ = pack_pages(vrows, lens, page_size, np.random.default_rng(99))
    n = np.array(chunk, np.int32)
    qo = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    k_new = np.concatenate([rows[b, lens[b] - n[b]:lens[b]] for b in range(len(lens))])
    v_new = np.concatenate([vrows[b, lens[b] - n[b]:lens[b]] for b in range(len(lens))])
    return rows, vrows, kp, vp, bt, lens, qo, k_new, v_new


def pin_append_roundtrip(orc, seed=12):
    """Clearing the last n_b rows of each sequence and appending them again restores the pages bitwise."""
    rng = np.random.default_rng(seed)
    _, _, kp, vp, bt, lens, qo, k_new, v_new = _append_problem(rng)
    kc, vc = kp.copy(), vp.copy()
    for b in range(len(lens)):
        n = int(qo[b + 1] - qo[b])
        for t in range(int(lens[b]) - n, int(lens[b])):
            kc[bt[b, t // 8], t % 8] = 0x1234
            vc[bt[b, t // 8], t % 8] = 0x4321
    ka, va = orc.append_kv(kc, vc, bt, lens, qo, k_new, v_new)
    assert np.array_equal(ka, kp) and np.array_equal(va, vp), "append does not restore the removed rows"
    assert not np.array_equal(kc, kp), "the problem must clear something"


def pin_append_fp8(orc, seed=13):
    """FP8 pages receive torch's E4M3 cast of the float32 quotient by the head's scale, and only
    at the appended positions; dequantised values are within half an E4M3 step of the input."""
    rng = np.random.default_rng(seed)
    rows, vrows, _, _, bt, lens, qo, k_new, v_new = _append_problem(rng)
    pool = np.full((bt.max() + 3, 8, 2, D), 0x5A, np.uint8)
    # |x| / scale stays below 448 (torch's cast does not saturate; saturation is pinned above)
    ks = np.array([0.013, 0.021], np.float32)
    vs = np.array([0.017, 0.0125], np.float32)
    ka, va = orc.append_kv(pool, pool, bt, lens, qo, k_new, v_new, k_scale=ks, v_scale=vs)
    for pages, new, sc in ((ka, k_new, ks), (va, v_new, vs)):
        quot = (from_bits(new).astype(np.float32) / sc[None, :, None]).astype(np.float32)
        assert np.abs(quot).max() < 448
        want = _fp8_encode_torch(quot)
        touched = np.zeros(pool.shape[:2], bool)
        r = 0
        for b in range(len(lens)):
            n = int(qo[b + 1] - qo[b])
            for i in range(n):
                t = int(lens[b]) - n + i
                p, s = bt[b, t // 8], t % 8
                assert np.array_equal(pages[p, s], want[r]), "appended codes"
                touched[p, s] = True
                r += 1
        assert np.all(pages[~touched] == 0x5A), "append wrote outside the new positions"
        x = from_bits(new)
        deq = _fp8_values_torch(want) * sc[None, :, None].astype(np.float64)
        assert np.all(np.abs(deq - x) <= np.abs(x) / 16 + 2.0 ** -10 * sc.max()), "dequantisation error"
    # near-ties found by search, where the rounding of the quotient decides the code: the
    # float32 quotient x / s, not x times the reciprocal of s, and not the exact quotient
    tie = np.zeros((1, 2, D), np.uint16)
    tie[0, 0, :2] = [0x3B90, 0x3B60]
    tie[0, 1, :3] = [0x3A80, 0x3BA0, 0x3C10]
    sc = np.array([0.3, 1 / 3], np.float32)
    quot = (from_bits(tie).astype(np.float32) / sc[None, :, None]).astype(np.float32)
    assert np.array_equal(orc.quantize_rows(tie, sc), _fp8_encode_torch(quot)), "quotient rounding"


ALL_PINS = [pin_brute_force, pin_single_key, pin_uniform_keys, pin_page_invariance, pin_split_merge,
            pin_extend, pin_gqa_expansion, pin_scale_homogeneity, pin_batch_and_sharing, pin_golden,
            pin_fp8_codes, pin_fp8_equals_bf16, pin_fp8_scales, pin_fp8_encode, pin_append_roundtrip,
            pin_append_fp8]
