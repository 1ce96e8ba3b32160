"""Shapes at the limits the library accepts, through the C-ABI, against the oracle:
a very long single sequence (hundreds of thousands of keys, a block-table row of
thousands of pages), a 128-wide GQA group (128 query heads on one KV head),
the most query tokens per sequence a multi-token decode takes (64), a whole
prompt prefilled as one chunk, and batches of thousands of sequences.
"""

import numpy as np
import pytest

from paper_2609_08368_amd import workloads as wl
from tests import gpu_helpers as H
from tests.test_gpu_mtp import check as mtp_check
from tests.test_gpu_mtp import mtp_problem, run_mtp

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.mark.parametrize("split", [0, 8192])
@pytest.mark.parametrize("fp8", [False, True])
def test_decode_long_single_sequence(split, fp8):
    """200,003 keys in 1,563 pages of 128 next to two short sequences: the equal-work
    split spreads the long one over many workers (or 25 forced pieces)."""
    lens = [200_003, 1, 777]
    w = wl.custom(301, "decode", lens, hq=8, hkv=1, page_size=128)
    H.say(f"long decode split={split} fp8={fp8}")
    t = (wl.materialize_fp8 if fp8 else wl.materialize)(w, DEV)
    out, lse = H.run_decode(w, t, split_tokens=split)
    ref_o, ref_l = H.oracle_full(w, t)
    H.say("  ", H.compare(out, ref_o, lse, ref_l, what=f"long decode split={split} fp8={fp8}"))


@pytest.mark.parametrize("split", [0, 128])
def test_decode_gqa_128(split):
    """128 query heads on one KV head: eight 16-head blocks per KV head."""
    w = wl.custom(302, "decode", [1, 63, 64, 65, 3000], hq=128, hkv=1, page_size=64)
    H.say(f"decode R=128 split={split}")
    t = wl.materialize(w, DEV)
    out, lse = H.run_decode(w, t, split_tokens=split)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what=f"decode R=128 split={split}")


def test_extend_gqa_128():
    """128 query heads per KV head: a unit holds two chunk tokens of all 128 heads."""
    w = wl.custom(303, "extend", [300, 64, 1000], q_lens=[300, 1, 37], hq=128, hkv=1, page_size=64)
    H.say("extend R=128")
    t = wl.materialize(w, DEV)
    out, lse = H.run_extend(w, t)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what="extend R=128")


def test_extend_whole_prompt_prefill():
    """A 5,000-token prompt prefilled as one chunk (no cached prefix), next to a chunk
    that appends to a long cache."""
    w = wl.custom(304, "extend", [5000, 9000], q_lens=[5000, 700], hq=8, hkv=1, page_size=64)
    H.say("extend whole-prompt prefill")
    t = wl.materialize(w, DEV)
    out, lse = H.run_extend(w, t)
    ref_o, ref_l = H.oracle_full(w, t)
    H.say("  ", H.compare(out, ref_o, lse, ref_l, what="prefill 5000"))


@pytest.mark.parametrize("case", [(16, 8, 2, [64, 100, 700], 0), (32, 2, 2, [64, 65, 500], 64)],
                         ids=["rows256", "rows64"])
def test_mtp_64_tokens(case):
    """64 query tokens per sequence, the most the multi-token decode takes: 256 rows
    per KV head (two row blocks) and 64 rows."""
    ps, hq, hkv, lens, split = case
    n = 64
    w, t = mtp_problem(305 + hq, lens, n, hq, hkv, ps)
    H.say(f"mtp n=64 case {case}")
    out, lse = run_mtp(w, t, n, split_tokens=split)
    mtp_check(w, t, n, out, lse, what=f"mtp n=64 {case}")


def test_extend_large_batch_unsorted_plan():
    """2,500 sequences (more than the planner sorts by key count, so units keep batch
    order), chunks of 0-3 tokens over caches of 1-300 keys."""
    rng = np.random.default_rng(307)
    kv = rng.integers(1, 301, size=2500)
    ql = np.minimum(rng.integers(0, 4, size=2500), kv)
    w = wl.custom(307, "extend", kv.tolist(), q_lens=ql.tolist(), hq=8, hkv=2, page_size=16)
    H.say(f"extend B=2500 total_q={w.total_q}")
    t = wl.materialize(w, DEV)
    out, lse = H.run_extend(w, t)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what="extend B=2500")


@pytest.mark.parametrize("deterministic", [False, True])
def test_decode_large_batch(deterministic):
    """3,000 sequences of 0-400 keys; the deterministic mode runs them as 3,000
    one-row extend units through the unsorted planner path."""
    rng = np.random.default_rng(308)
    lens = rng.integers(0, 401, size=3000)
    w = wl.custom(308, "decode", lens.tolist(), hq=12, hkv=1, page_size=32)
    H.say(f"decode B=3000 deterministic={deterministic}")
    t = wl.materialize(w, DEV)
    out, lse = H.run_decode(w, t, deterministic=deterministic)
    ref_o, ref_l = H.oracle_full(w, t)
    H.compare(out, ref_o, lse, ref_l, what=f"decode B=3000 det={deterministic}")
