"""Measurement aids on the GPU: plausible ceilings."""

import pytest
import torch

from paper_2609_08368_amd import rl_attn as ra

pytestmark = pytest.mark.gpu


def test_read_bandwidth_and_mfma_loop():
    buf = torch.zeros(1 << 28, dtype=torch.uint8, device="cuda:0")
    gbps = ra.diag_read_bandwidth(buf, reps=5)
    assert 500.0 < gbps < 10000.0, gbps
    tflops = ra.diag_mfma_bf16(2000)
    assert 200.0 < tflops < 2600.0, tflops
