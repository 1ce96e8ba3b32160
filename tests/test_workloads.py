"""Seeded input generator: determinism and structure (CPU only)."""

import numpy as np
import torch

from paper_2609_08368_amd import workloads as wl


def test_metadata_deterministic():
    for name, fn in wl.WORKLOADS.items():
        a, b = fn(), fn()
        assert np.array_equal(a.block_table, b.block_table), name
        assert np.array_equal(a.kv_lens, b.kv_lens), name
        assert np.array_equal(a.q_lens, b.q_lens), name


def test_config_shapes():
    c1 = wl.decode_tiny()
    assert c1.num_pages == 256 and list(c1.kv_lens) == [128, 256, 384, 512] and c1.page_size == 16
    assert c1.kv_bytes() == 1_310_720
    c2 = wl.decode_uniform()
    assert c2.kv_bytes() == 2_147_483_648 and c2.num_pages == 64 * 128 + 1
    c3 = wl.decode_ragged()
    assert c3.kv_lens.min() >= 1024 and c3.kv_lens.max() <= 65536 and c3.batch == 128 and c3.hq == 96
    assert c3.kv_head_scale.shape == (8,) and np.all((c3.kv_head_scale >= 0.5) & (c3.kv_head_scale <= 2.0))
    c4 = wl.decode_group_prefix()
    assert c4.batch == 128
    for g in range(16):
        rows = c4.block_table[8 * g:8 * g + 8, :64]
        assert np.all(rows == rows[0]), "group members must share their 64 prefix page ids"
        if g:
            assert not np.intersect1d(rows[0], c4.block_table[0, :64]).size
    priv = c4.kv_lens - 4096
    assert priv.min() >= 512 and priv.max() <= 16384
    # unique bytes: 16 shared prefixes + private continuations
    assert c4.kv_bytes(unique=True) == (16 * 4096 + int(priv.sum())) * 4096
    c5 = wl.extend_multiturn()
    p = c5.kv_lens - c5.q_lens
    assert p.min() >= 8192 and p.max() <= 65536 and c5.q_lens.min() >= 64 and c5.q_lens.max() <= 2048
    assert c5.qo_indptr[-1] == c5.total_q


def test_physical_pages_distinct_and_in_pool():
    for fn in (wl.decode_tiny, wl.decode_uniform, wl.extend_multiturn):
        w = fn()
        ids = []
        for b in range(w.batch):
            used = -(-int(w.kv_lens[b]) // w.page_size)
            ids.extend(w.block_table[b, :used].tolist())
        assert len(ids) == len(set(ids))
        assert min(ids) >= 0 and max(ids) < w.num_pages
        assert w.poison_page not in ids


def test_materialize_cpu_deterministic_and_poisoned():
    w = wl.decode_tiny()
    a = wl.materialize(w, "cpu")
    b = wl.materialize(w, "cpu")
    for key in ("q", "k_pages", "v_pages"):
        assert torch.equal(a[key].view(torch.int16), b[key].view(torch.int16))
    used = wl.referenced_pages(w)
    unused = np.setdiff1d(np.arange(w.num_pages), used)
    assert torch.isnan(a["k_pages"][torch.from_numpy(unused)].float()).all()
    assert not torch.isnan(a["k_pages"][torch.from_numpy(used)].float()).any()   # lengths are page multiples


def test_tail_poison_and_head_scale():
    w = wl.custom(3, "decode", [5, 16, 17], hq=4, hkv=2, page_size=8, kv_head_scale=[0.5, 2.0])
    t = wl.materialize(w, "cpu")
    k = t["k_pages"].float()
    for b, l in enumerate(w.kv_lens):
        last = (int(l) - 1) // 8
        pid = int(w.block_table[b, last])
        n = int(l) - last * 8
        assert not torch.isnan(k[pid, :n]).any()
        assert torch.isnan(k[pid, n:]).all()
    # the second KV head was drawn with a 4x larger multiplier
    good = torch.from_numpy(wl.referenced_pages(w))
    s0 = k[good][:, :, 0][~torch.isnan(k[good][:, :, 0])].std()
    s1 = k[good][:, :, 1][~torch.isnan(k[good][:, :, 1])].std()
    assert 2.5 < float(s1 / s0) < 6.0
