"""Float64 CPU oracle for paged-KV grouped-query attention.

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import, call or
execute this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it. It shares no code, constants or
helpers with the HIP library; the only thing both sides share is the seeded
input generator, which holds none of the attention arithmetic.

What it computes (the plain definition, evaluated directly in float64):

* decode  -- one query token per sequence attending to its whole cached
  context (the batched generation of the rollout engines, paper section
  "Fast Agentic Rollout with SGLang" and the rollout stage of the RL loop);
* extend  -- a chunk of appended tokens attending to the cached prefix plus,
  causally, to the chunk itself ("each turn prefills only the newly generated
  suffix", same section, and the session server of section "Token-In-Token-Out");
* merge   -- the log-sum-exp combination of attention results over disjoint
  key ranges (split-KV partials);
* append  -- writing new tokens' K/V rows into their pages (``kv_append``),
  with the FP8 E4M3 encoding of the quotient by the KV head's scale.

Pages hold bf16 values, or OCP FP8 E4M3 codes with one dequantisation scale
per KV head (the FP8 key-value cache of the paper's case-study rollout,
section "Case Study", subsection "Configuration").

The paper names the attention kernels its engines run (section "True-On-Policy
Alignment") but never writes the operation down; the definition used here is
textbook scaled dot-product attention (Vaswani et al., 2017) with grouped-query
head sharing (query head h reads KV head h // (Hq // Hkv)).

Pins: see tests/test_oracle_pins.py (brute-force dense attention via scipy,
single-key exactness, uniform-key closed form, page-size/page-order
invariance, split/merge identity, extend<->decode and causal brute force,
GQA expansion, scale homogeneity, batch permutation, closed-form golden file,
FP8 E4M3 decoding against torch's float8_e4m3fn and the format's closed forms,
FP8 pages against the same values in bf16, per-KV-head scales; KV append
positions against a removal/append round trip, and the E4M3 encoder against
torch's float8_e4m3fn cast, its own decoder and brute-force nearest values);
tests/test_oracle_properties.py draws shapes, page layouts and lengths and
compares decode and extend with dense attention computed by scipy.
Parity with values printed in the paper is unpinned: the paper prints none.
"""

from .attention import (  # noqa: F401
    bf16_bits_to_f64,
    gather_head,
    attend,
    attend_range,
    decode,
    extend,
    fp8_e4m3_to_f64,
    merge,
)
from .kv_append import append_kv, fp8_e4m3_encode, quantize_rows  # noqa: F401
