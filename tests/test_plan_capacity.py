"""The host's workspace sizing against the device planners' needs (host only).

The decode and extend planners run on the device and write work lists and
partial-result slots into a workspace whose capacities the host fixes before
the launch, from sizes alone. A planner that needs more reports
kErrCapacity instead of racing or dropping work, but that must never happen for
a valid call. This test models the planners' counts in plain Python (split
size, trajectory groups and sub-groups, shared items, equal-work worker shares
and the pieces they cut, partial slots, extend work units), evaluates them on
drawn batches (ragged and uniform lengths, empty sequences, trajectory groups
with shared prefixes, forced splits, 1-64 query tokens, batches up to 3,000),
and checks each count against the capacities the library's host code computes
(rl_attn_diag_decode_capacity / rl_attn_diag_extend_capacity).
"""

import math

import numpy as np
import pytest

from paper_2609_08368_amd import rl_attn as ra

TILE = 32            # keys per private-pass tile
MIN_SPLIT = 256      # smallest automatic split of shared keys
MIN_WORKER_KEYS = 256
GROUP_MAX = 1024     # batches up to this size get trajectory-group detection


def ceil_div(a, b):
    return -(-a // b)


def plan_decode(lens, table, P, caps, forced_split):
    """Counts the decode planner produces: (shared items, partial slots)."""
    B = len(lens)
    total = int(sum(lens))
    if forced_split > 0:
        C = forced_split
    else:
        per = ceil_div(total, caps["target_items"])
        per = ceil_div(per, 64) * 64
        C = max(per, MIN_SPLIT)
    cap = caps["group_cap"]
    grouping = cap >= 2 and B <= GROUP_MAX
    shared = [0] * B
    subgroups = []       # (leader, members in the sub-group, shared keys)
    if grouping:
        lead = list(range(B))
        first = {}
        for b in range(B):
            if lens[b] // P > 0:
                key = int(table[b][0])
                first.setdefault(key, b)
                lead[b] = first[key]
        kmin = {b: None for b in range(B)}
        cnt = [0] * B
        for m in range(B):
            l = lead[m]
            if l == m:
                continue
            lim = min(lens[m], lens[l]) // P
            k = lim
            for j in range(lim):
                if table[m][j] != table[l][j]:
                    k = j
                    break
            kmin[l] = k if kmin[l] is None else min(kmin[l], k)
            cnt[l] += 1
        for b in range(B):
            l = lead[b]
            if cnt[l] >= 1 and kmin[l] is not None and kmin[l] >= 1:
                shared[b] = kmin[l] * P
        tot_sh = 0
        for l in range(B):
            if lead[l] == l and shared[l] > 0:
                members = cnt[l] + 1
                for s0 in range(0, members, cap):
                    subgroups.append((l, min(cap, members - s0), shared[l]))
                tot_sh += ceil_div(members, cap) * shared[l]
        if forced_split <= 0 and tot_sh > 0:
            per = ceil_div(tot_sh * caps["hkv"], caps["prefix_grid"])
            per = ceil_div(per, 64) * 64
            C = max(C, per)
    priv = [ceil_div(lens[b] - shared[b], TILE) for b in range(B)]
    pref = np.concatenate([[0], np.cumsum(priv)]).astype(np.int64)
    W = int(pref[-1])
    nwork = 1
    if W > 0:
        per_w = (forced_split if forced_split > 0 else MIN_WORKER_KEYS) // TILE
        nwork = min(ceil_div(W, per_w), caps["max_workers"])

    def starts_before(y):
        return (y * nwork + W - 1) // W

    slots = 0
    for b in range(B):
        S = shared[b]
        nsh = ceil_div(S, C) if S > 0 else 0
        p0, p1 = int(pref[b]), int(pref[b + 1])
        npriv = 1 + starts_before(p1) - starts_before(p0 + 1) if p1 > p0 else 0
        direct = S == 0 and npriv == 1
        if not (direct or lens[b] == 0):
            slots += nsh + npriv
    items = sum(ceil_div(S, C) for (_, _, S) in subgroups)
    return items, slots, nwork


def group_batch(rng, groups, gsize, shared_pages, P, priv_hi):
    """Lengths and block table of trajectory groups sharing their first pages."""
    lens, rows, nxt = [], [], 0
    for _ in range(groups):
        base = list(range(nxt, nxt + shared_pages))
        nxt += shared_pages
        for _ in range(gsize):
            priv = int(rng.integers(0, priv_hi + 1))
            L = shared_pages * P + priv
            own = ceil_div(L, P) - shared_pages
            rows.append(base + list(range(nxt, nxt + own)))
            nxt += own
            lens.append(L)
    width = max(1, max(len(r) for r in rows))
    table = np.zeros((len(rows), width), np.int32)
    for i, r in enumerate(rows):
        table[i, :len(r)] = r
    order = rng.permutation(len(lens))
    return [lens[i] for i in order], table[order]


def plain_batch(rng, B, P, kind):
    if kind == "ragged":
        lens = np.clip(np.rint(rng.lognormal(math.log(16384), 1.0, size=B)), 0, 65536).astype(int)
    elif kind == "short":
        lens = rng.integers(0, 300, size=B)
    else:
        lens = np.full(B, int(rng.integers(1, 9000)))
    lens[rng.random(B) < 0.05] = 0
    width = max(1, ceil_div(int(lens.max()), P))
    table = np.arange(B * width, dtype=np.int64).reshape(B, width).astype(np.int32)
    return [int(x) for x in lens], table


CONFIGS = []
_rng = np.random.default_rng(2024)
for i in range(160):
    kind = ["ragged", "short", "uniform", "groups"][i % 4]
    P = int(_rng.choice([8, 16, 32, 64, 128]))
    hkv = int(_rng.choice([1, 2, 4, 8]))
    R = int(_rng.choice([1, 4, 8, 12, 16, 20]))
    n_tok = int(_rng.choice([1, 1, 2, 4, 8, 16, 64]))
    split = int(_rng.choice([0, 0, 0, 64, 256, 1024, 8192]))
    B = int(_rng.choice([1, 7, 64, 128, 500, 1024, 1500, 3000])) if kind != "groups" else None
    CONFIGS.append((i, kind, P, hkv, R, n_tok, split, B))


@pytest.mark.parametrize("cfg", CONFIGS, ids=[f"{c[0]}_{c[1]}" for c in CONFIGS])
def test_decode_capacity_covers_planner(cfg):
    i, kind, P, hkv, R, n_tok, split, B = cfg
    rng = np.random.default_rng(1000 + i)
    if kind == "groups":
        gsize = int(rng.choice([2, 3, 8, 20, 33]))
        groups = int(rng.integers(1, 1024 // gsize + 1))
        lens, table = group_batch(rng, groups, gsize, int(rng.integers(1, 40)), P, int(rng.integers(0, 5000)))
    else:
        lens, table = plain_batch(rng, B, P, kind)
    if kind != "groups" and B > 500 and kind == "ragged":
        lens = [min(x, 4096) for x in lens]        # keep the model fast on large batches
    B = len(lens)
    max_pages = table.shape[1]
    lens = [min(x, max_pages * P) for x in lens]
    hq = hkv * R
    if B * n_tok * hq >= 2 ** 31:
        pytest.skip("beyond the accepted sizes")
    for cus, wpc in ((256, 1), (256, 2), (80, 3)):
        caps = ra.diag_decode_capacity(B, hq, hkv, max_pages, P, n_tok, split, True, cus, wpc)
        caps["hkv"] = hkv
        items, slots, nwork = plan_decode(lens, table, P, caps, split)
        assert nwork <= caps["max_workers"]
        assert items <= caps["max_items"], f"shared items {items} > capacity {caps['max_items']} ({caps})"
        assert slots <= caps["max_slots"], f"partial slots {slots} > capacity {caps['max_slots']} ({caps})"
        # the sized workspace covers every carved array
        assert caps["bytes"] >= caps["max_slots"] * hq * n_tok * 129 * 4


@pytest.mark.parametrize("seed", range(40))
def test_extend_capacity_covers_planner(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.choice([1, 3, 32, 1000, 2500]))
    hkv = int(rng.choice([1, 2, 8]))
    R = int(rng.choice([1, 3, 8, 12, 64, 256]))
    n = rng.integers(0, int(rng.choice([2, 70, 2100])), size=B)
    total_q = int(n.sum())
    caps = ra.diag_extend_capacity(B, total_q, hkv * R, hkv)
    units = sum(ceil_div(int(x), caps["tile_tokens"]) for x in n) * hkv * caps["head_blocks"]
    assert units <= caps["max_items"]
    # decode through the extend kernel: B sequences of n_tok rows
    for n_tok in (1, 4, 64):
        caps = ra.diag_extend_capacity(B, B * n_tok, hkv * R, hkv)
        units = B * ceil_div(n_tok, caps["tile_tokens"]) * hkv * caps["head_blocks"]
        assert units <= caps["max_items"]


def test_capacity_model_reaches_its_bounds():
    """The model is not vacuous: a forced small split on a long batch uses most of the
    slot capacity, and trajectory groups produce shared items."""
    lens, table = plain_batch(np.random.default_rng(5), 64, 64, "uniform")
    lens = [8192] * 64
    table = np.arange(64 * 128, dtype=np.int32).reshape(64, 128)
    caps = ra.diag_decode_capacity(64, 64, 8, 128, 64, 1, 64, True, 256, 1)
    caps["hkv"] = 8
    items, slots, nwork = plan_decode(lens, table, 64, caps, 64)
    assert slots >= 0.4 * caps["max_slots"]
    lens, table = group_batch(np.random.default_rng(6), 16, 8, 64, 64, 16384)
    caps = ra.diag_decode_capacity(128, 64, 8, table.shape[1], 64, 1, 0, True, 256, 1)
    caps["hkv"] = 8
    items, slots, nwork = plan_decode(lens, table, 64, caps, 0)
    assert items > 0 and slots > 128
