"""Shared helpers for the GPU parity tests (HIP path vs float64 oracle)."""

from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
from paper_2609_08368_amd import rl_attn as ra
from paper_2609_08368_amd import workloads as wl

# Tolerances of the path (bf16 inputs, fp32 accumulation, bf16 output).
MAX_ABS = 2e-2
REL_RMS = 5e-3
LSE_REL = 1e-4


def say(*args):
    print(*args, flush=True)
    sys.stdout.flush()


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def compare(gpu_out, ref_out, gpu_lse=None, ref_lse=None, max_abs=MAX_ABS, rel_rms=REL_RMS, lse_rel=LSE_REL,
            what=""):
    g = f64(gpu_out) if isinstance(gpu_out, torch.Tensor) else gpu_out
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    err = g - ref_out
    ma = float(np.max(np.abs(err))) if err.size else 0.0
    denom = float(np.sqrt(np.sum(ref_out ** 2)))
    rr = float(np.sqrt(np.sum(err ** 2)) / denom) if denom > 0 else float(np.sqrt(np.sum(err ** 2)))
    res = {"max_abs": ma, "rel_rms": rr}
    assert ma <= max_abs, f"{what}: max-abs {ma:.3e} > {max_abs}"
    assert rr <= rel_rms, f"{what}: rel-RMS {rr:.3e} > {rel_rms}"
    if gpu_lse is not None:
        gl = f64(gpu_lse) if isinstance(gpu_lse, torch.Tensor) else gpu_lse
        both_inf = np.isneginf(gl) & np.isneginf(ref_lse)
        assert np.array_equal(np.isneginf(gl), np.isneginf(ref_lse)), f"{what}: -inf lse mismatch"
        d = np.where(both_inf, 0.0, np.abs(gl - ref_lse) / np.maximum(1.0, np.abs(np.where(both_inf, 0, ref_lse))))
        res["lse_rel"] = float(d.max()) if d.size else 0.0
        assert res["lse_rel"] <= lse_rel, f"{what}: lse rel {res['lse_rel']:.3e} > {lse_rel}"
    return res


def poison_like(t: torch.Tensor) -> torch.Tensor:
    """Fill an output buffer with NaN so an unwritten element cannot pass."""
    return t.fill_(float("nan"))


def is_fp8(tensors: dict) -> bool:
    return "k_scale" in tensors


def run_decode(w: wl.Paged, tensors: dict, out_dtype=torch.bfloat16, **opts):
    """The bf16 entry point, or the FP8 one for tensors from ``materialize_fp8``."""
    q = tensors["q"]
    out = poison_like(torch.empty(q.shape, dtype=out_dtype, device=q.device))
    lse = poison_like(torch.empty(q.shape[:2], dtype=torch.float32, device=q.device))
    if is_fp8(tensors):
        ra.decode_fp8(q, tensors["k_pages"], tensors["v_pages"], tensors["k_scale"], tensors["v_scale"],
                      tensors["block_table"], tensors["kv_lens"], tensors["scale"], out=out, lse=lse, **opts)
    else:
        ra.decode(q, tensors["k_pages"], tensors["v_pages"], tensors["block_table"], tensors["kv_lens"],
                  tensors["scale"], out=out, lse=lse, **opts)
    torch.cuda.synchronize()
    return out, lse


def run_extend(w: wl.Paged, tensors: dict, out_dtype=torch.bfloat16, **opts):
    q = tensors["q"]
    out = poison_like(torch.empty(q.shape, dtype=out_dtype, device=q.device))
    lse = poison_like(torch.empty(q.shape[:2], dtype=torch.float32, device=q.device))
    if is_fp8(tensors):
        ra.extend_fp8(q, tensors["qo_indptr"], tensors["k_pages"], tensors["v_pages"], tensors["k_scale"],
                      tensors["v_scale"], tensors["block_table"], tensors["kv_lens"], tensors["scale"], out=out,
                      lse=lse, **opts)
    else:
        ra.extend(q, tensors["qo_indptr"], tensors["k_pages"], tensors["v_pages"], tensors["block_table"],
                  tensors["kv_lens"], tensors["scale"], out=out, lse=lse, **opts)
    torch.cuda.synchronize()
    return out, lse


def host_scales(tensors: dict) -> dict:
    """Per-KV-head dequantisation scales as float64 host arrays (FP8 workloads), else {}."""
    if not is_fp8(tensors):
        return {}
    return {k: tensors[k].cpu().numpy().astype(np.float64) for k in ("k_scale", "v_scale")}


def oracle_decode_rows(w: wl.Paged, tensors: dict, rows):
    """Oracle decode of the sequences ``rows`` (compacted host copy of their pages)."""
    sub = wl.compact_subset(w, tensors, rows)
    return oracle.decode(sub["q"], sub["k_pages"], sub["v_pages"], sub["block_table"], sub["kv_lens"],
                         tensors["scale"], **host_scales(tensors))


def oracle_extend_rows(w: wl.Paged, tensors: dict, seq: int, chunk_rows):
    """Oracle of chunk rows ``chunk_rows`` of sequence ``seq``: row i is decode over p + i + 1 keys."""
    sub = wl.compact_subset(w, tensors, [seq])
    n = int(w.q_lens[seq])
    p = int(w.kv_lens[seq]) - n
    outs, lses = [], []
    for i in chunk_rows:
        o, l = oracle.decode(sub["q"][i:i + 1], sub["k_pages"], sub["v_pages"], sub["block_table"],
                             np.array([p + i + 1]), tensors["scale"], **host_scales(tensors))
        outs.append(o[0])
        lses.append(l[0])
    return np.stack(outs), np.stack(lses)


def to_host(v: torch.Tensor) -> np.ndarray:
    """bf16 -> uint16 bits, FP8 E4M3 -> uint8 codes, anything else as is."""
    if v.dtype == torch.bfloat16:
        return wl.to_numpy_bits(v)
    if v.dtype == torch.float8_e4m3fn:
        return v.view(torch.uint8).cpu().numpy()
    return v.cpu().numpy()


def oracle_full(w: wl.Paged, tensors: dict):
    host = {k: to_host(v) for k, v in tensors.items() if isinstance(v, torch.Tensor) and not k.endswith("_scale")}
    sc = host_scales(tensors)
    if w.kind == "decode":
        return oracle.decode(host["q"], host["k_pages"], host["v_pages"], host["block_table"], host["kv_lens"],
                             tensors["scale"], **sc)
    return oracle.extend(host["q"], host["qo_indptr"], host["k_pages"], host["v_pages"], host["block_table"],
                         host["kv_lens"], tensors["scale"], **sc)
