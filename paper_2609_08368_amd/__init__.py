"""Paged-KV grouped-query attention for rollout engines, hand-written HIP for gfx950.

The compute lives in ``librlattn.so`` (C-ABI declared in ``include/rl_attn.h``);
this package only marshals torch tensors into the ABI's tensor views.
"""
