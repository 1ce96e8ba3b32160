"""The log-sum-exp merge kernel fed oracle partials (rounded to fp32)."""

import numpy as np
import pytest
import torch

import oracle
from paper_2609_08368_amd import rl_attn as ra
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def test_merge_oracle_partials():
    rng = np.random.default_rng(3)
    N, S, Hh, D = 6, 5, 4, 128
    o_parts = np.zeros((N, S, Hh, D))
    l_parts = np.full((N, S, Hh), -np.inf)
    num = np.array([5, 1, 3, 0, 5, 2], np.int32)
    for n in range(N):
        for h in range(Hh):
            q = rng.standard_normal((1, D))
            L = int(rng.integers(40, 400))
            k = rng.standard_normal((L, D))
            v = rng.standard_normal((L, D)) * (1 + h)
            cuts = np.sort(rng.choice(np.arange(1, L), size=S - 1, replace=False))
            bounds = [0, *cuts.tolist(), L]
            for s in range(num[n]):
                if n == 4 and s == 2:
                    continue                          # an empty part: lse = -inf
                o, l = oracle.attend_range(q, k, v, 0.09, bounds[s], bounds[s + 1])
                o_parts[n, s, h], l_parts[n, s, h] = o[0], l[0]
    o32 = o_parts.astype(np.float32)
    l32 = l_parts.astype(np.float32)
    ref_o, ref_l = oracle.merge(o32.astype(np.float64), l32.astype(np.float64), num)
    H.say("merge")
    out = torch.full((N, Hh, D), float("nan"), device=DEV)
    lse = torch.full((N, Hh), float("nan"), device=DEV)
    ra.merge(torch.from_numpy(o32).to(DEV), torch.from_numpy(l32).to(DEV), torch.from_numpy(num).to(DEV),
             out=out, lse=lse)
    torch.cuda.synchronize()
    g = out.cpu().numpy().astype(np.float64)
    assert np.all(g[3] == 0) and np.all(np.isneginf(lse[3].cpu().numpy()))
    err = g - ref_o
    assert np.sqrt((err ** 2).sum() / (ref_o ** 2).sum()) <= 1e-4
    assert np.abs(err).max() <= 1e-4 * np.abs(ref_o).max()
    H.compare(out, ref_o, lse, ref_l, max_abs=1e-4 * np.abs(ref_o).max(), rel_rms=1e-4, what="merge")
