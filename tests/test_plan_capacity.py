"""The host's workspace sizing against the device planners' needs (host only).

The decode and extend planners run on the device and write work lists and
partial-result slots into a workspace whose capacities the host fixes before
the launch, from sizes alone. A planner that needs more reports
kErrCapacity instead of racing or dropping work, but that must never happen for
a valid call. This test models the planners' counts in plain Python (split
size, the nodes of nested shared prefix ranges and their sub-groups, shared
items, equal-work worker shares and the pieces they cut, partial slots, extend
work units), evaluates them on drawn batches (ragged and uniform lengths, empty
sequences, trajectory groups with shared prefixes, branching sessions with up
to three nested shared ranges, forced splits, 1-64 query tokens, batches up to
3,000),
and checks each count against the capacities the library's host code computes
(rl_attn_diag_decode_capacity / rl_attn_diag_extend_capacity).
"""

import math

import numpy as np
import pytest

from paper_2609_08368_amd import rl_attn as ra
from paper_2609_08368_amd import workloads as wl

TILE = 32            # keys per private-pass tile
MIN_SPLIT = 256      # smallest automatic split of shared keys
MIN_WORKER_KEYS = 64
GROUP_MAX = 1024     # batches up to this size get trajectory-group detection


def ceil_div(a, b):
    return -(-a // b)


LEVELS = 3          # nested levels of shared prefix pages the planner detects


def plan_decode(lens, table, P, caps, forced_split):
    """Counts the decode planner produces: (shared items, partial slots, workers)."""
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
    lead = [[-1] * B for _ in range(LEVELS)]
    end = [[0] * B for _ in range(LEVELS)]
    num = [[0] * B for _ in range(LEVELS)]
    if grouping:
        for v in range(LEVELS):
            leads, first = [-1] * B, {}
            for b in range(B):
                parent = lead[v - 1][b] if v else -1
                start = end[v - 1][b] if v else 0
                if (v == 0 or parent >= 0) and lens[b] // P > start // P:
                    key = (parent, int(table[b][start // P]))
                    first.setdefault(key, b)
                    leads[b] = first[key]
            kmin, cnt = {}, [0] * B
            for m in range(B):
                l = leads[m]
                if l < 0 or l == m:
                    continue
                p0 = (end[v - 1][m] if v else 0) // P
                lim = min(lens[m], lens[l]) // P
                k = lim
                for j in range(p0, lim):
                    if table[m][j] != table[l][j]:
                        k = j
                        break
                kmin[l] = min(kmin.get(l, k), k)
                cnt[l] += 1
            for b in range(B):
                l = leads[b]
                start = end[v - 1][b] if v else 0
                kept = l >= 0 and cnt[l] >= 1 and kmin[l] > start // P
                lead[v][b] = l if kept else -1
                end[v][b] = kmin[l] * P if kept else start
                num[v][b] = cnt[b] + 1 if kept and l == b else 0
        tot_sh = 0
        for v in range(LEVELS):
            for l in range(B):
                if lead[v][l] == l:
                    start = end[v - 1][l] if v else 0
                    tot_sh += ceil_div(num[v][l], cap) * (end[v][l] - start)
        if forced_split <= 0 and tot_sh > 0:
            per = ceil_div(tot_sh * caps["hkv"], caps["prefix_grid"])
            per = ceil_div(per, 64) * 64
            C = max(C, per)
    shared = [end[LEVELS - 1][b] if grouping else 0 for b in range(B)]
    nsh = [0] * B
    items = 0
    if grouping:
        for v in range(LEVELS):
            for b in range(B):
                if lead[v][b] >= 0:
                    start = end[v - 1][b] if v else 0
                    nsh[b] += ceil_div(end[v][b] - start, C)
                    if lead[v][b] == b:
                        items += ceil_div(num[v][b], cap) * ceil_div(end[v][b] - start, C)
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
        p0, p1 = int(pref[b]), int(pref[b + 1])
        npriv = 1 + starts_before(p1) - starts_before(p0 + 1) if p1 > p0 else 0
        direct = shared[b] == 0 and npriv == 1
        if not (direct or lens[b] == 0):
            slots += nsh[b] + npriv
    return items, slots, nwork


def tree_batch(rng, P):
    """Branching sessions: groups whose members share a prompt, with subsets sharing more."""
    fan = [int(x) for x in rng.choice([2, 3, 4], size=int(rng.integers(1, 4)))]
    sizes = []
    size = int(np.prod(fan))
    for f in fan:
        sizes.append(size)
        size //= f
    levels = [(s, P * int(rng.integers(1, 20))) for s in sizes]
    groups = int(rng.integers(1, max(2, 600 // sizes[0])))
    base = sum(t for _, t in levels)
    lens = [base + int(rng.integers(0, 3000)) for _ in range(groups * sizes[0])]
    table, _, _ = wl._assign_tree_pages(rng, np.array(lens), P, levels)
    order = rng.permutation(len(lens))
    return [lens[i] for i in order], table[order]


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
    kind = ["ragged", "short", "uniform", "groups", "tree"][i % 5]
    P = int(_rng.choice([8, 16, 32, 64, 128]))
    hkv = int(_rng.choice([1, 2, 4, 8]))
    R = int(_rng.choice([1, 4, 8, 12, 16, 20]))
    n_tok = int(_rng.choice([1, 1, 2, 4, 8, 16, 64]))
    split = int(_rng.choice([0, 0, 0, 64, 256, 1024, 8192]))
    B = int(_rng.choice([1, 7, 64, 128, 500, 1024, 1500, 3000])) if kind not in ("groups", "tree") else None
    CONFIGS.append((i, kind, P, hkv, R, n_tok, split, B))


@pytest.mark.parametrize("cfg", CONFIGS, ids=[f"{c[0]}_{c[1]}" for c in CONFIGS])
def test_decode_capacity_covers_planner(cfg):
    i, kind, P, hkv, R, n_tok, split, B = cfg
    rng = np.random.default_rng(1000 + i)
    if kind == "groups":
        gsize = int(rng.choice([2, 3, 8, 20, 33]))
        groups = int(rng.integers(1, 1024 // gsize + 1))
        lens, table = group_batch(rng, groups, gsize, int(rng.integers(1, 40)), P, int(rng.integers(0, 5000)))
    elif kind == "tree":
        lens, table = tree_batch(rng, P)
    else:
        lens, table = plain_batch(rng, B, P, kind)
    if kind == "ragged" and B > 500:
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
    # a three-level tree: 16 groups of 8, halves and pairs sharing further pages
    w = wl.decode_branching()
    caps = ra.diag_decode_capacity(w.batch, 64, 8, w.block_table.shape[1], 64, 1, 0, True, 256, 1)
    caps["hkv"] = 8
    items_t, _, _ = plan_decode([int(x) for x in w.kv_lens], w.block_table, 64, caps, 0)
    assert items_t >= 16 + 32 + 64       # at least one split per node of each level


def align256(x):
    return (x + 255) // 256 * 256


@pytest.mark.parametrize("n_tok", [2, 4, 8, 64])
def test_multi_token_workspace_covers_both_passes(n_tok):
    """With prefix sharing on, a multi-token decode call queues the split passes and an
    extend pass, and carves the extend work list after the decode workspace: the size
    query (what a caller reserves before capturing a graph) covers both."""
    for B, hq, hkv, max_pages, P in ((128, 96, 8, 1024, 64), (3, 8, 2, 40, 16), (1000, 64, 8, 64, 64)):
        dec = ra.diag_decode_capacity(B, hq, hkv, max_pages, P, n_tok, 0, True, 256, 1)["bytes"]
        ext = ra.diag_extend_capacity(B, B * n_tok, hq, hkv)
        need = align256(dec) + 256 + align256(ext["max_items"] * 16)
        assert ra.decode_workspace_size(B, hq, hkv, max_pages, P, query_tokens=n_tok) >= need
