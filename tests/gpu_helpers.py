"""Shared helpers for the GPU parity tests (HIP path vs float64 oracle)."""

from __future__ import annotations

import math
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


def pages_below(tensors: dict, size: int) -> dict:
    """The same keys in pages of fewer than `size` keys: each halving turns page i
    into pages 2i and 2i + 1 (K, V and the block table; nothing else changes). bf16
    pages of fewer than 64 keys take the 64-key steps, so this gives the reference
    for paths that advance 64 keys per step whatever the page size."""
    t = dict(tensors)
    while t["k_pages"].shape[1] >= size:
        for name in ("k_pages", "v_pages"):
            n, p = t[name].shape[:2]
            t[name] = t[name].reshape(2 * n, p // 2, *t[name].shape[2:])
        bt = t["block_table"]
        two = torch.stack((2 * bt, 2 * bt + 1), dim=-1).reshape(bt.shape[0], -1)
        t["block_table"] = torch.where(two >= 0, two, torch.full_like(two, -1)).contiguous()
    return t


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


# ---------------------------------------------------------------- full-row parity
# Every output row of a full-size call against the float64 oracle. The oracle is
# called once per task (decode: one sequence with all its query heads; extend and
# multi-token decode: one (sequence, KV head) pair, i.e. the pair's query heads
# and that KV head of the pools) from a thread pool on the host cores: numpy
# releases the GIL inside BLAS and large ufuncs, and BLAS runs one thread per
# task so the pool does not oversubscribe the cores. Error sums are accumulated
# per task, so host memory stays bounded by the tasks in flight.

def host_workers(cap: int = 16) -> int:
    """Worker threads for host-side oracle work: the affinity set, at most ``cap``."""
    import os

    return max(1, min(cap, len(os.sched_getaffinity(0))))


class ParityAcc:
    """Running error statistics of one comparison (max-abs, rel-RMS, lse)."""

    def __init__(self):
        self.sq_err = 0.0
        self.sq_ref = 0.0
        self.max_abs = 0.0
        self.lse_rel = 0.0      # |d| / max(1, |ref|)  (the stated criterion)
        self.lse_pure = 0.0     # |d| / |ref| over rows with |ref| >= 1e-3 (diagnostic)
        self.lse_small_abs = 0.0  # |d| over rows with |ref| < 1 (diagnostic)
        self.rows = 0
        self.bad = []

    def add(self, g, ref, gl, rl, what):
        g = np.asarray(g, dtype=np.float64)
        if not np.all(np.isfinite(g)):
            self.bad.append(f"{what}: non-finite output")
            return
        err = g - ref
        self.sq_err += float(np.sum(err * err))
        self.sq_ref += float(np.sum(ref * ref))
        if err.size:
            self.max_abs = max(self.max_abs, float(np.max(np.abs(err))))
        self.rows += int(np.prod(ref.shape[:-1]))
        gl = np.asarray(gl, dtype=np.float64)
        if not np.array_equal(np.isneginf(gl), np.isneginf(rl)):
            self.bad.append(f"{what}: -inf lse mismatch")
            return
        fin = ~np.isneginf(rl)
        if np.any(fin):
            d = np.abs(gl[fin] - rl[fin])
            a = np.abs(rl[fin])
            self.lse_rel = max(self.lse_rel, float(np.max(d / np.maximum(1.0, a))))
            big = a >= 1e-3
            if np.any(big):
                self.lse_pure = max(self.lse_pure, float(np.max(d[big] / a[big])))
            small = a < 1.0
            if np.any(small):
                self.lse_small_abs = max(self.lse_small_abs, float(np.max(d[small])))

    def merge(self, o):
        self.sq_err += o.sq_err
        self.sq_ref += o.sq_ref
        self.max_abs = max(self.max_abs, o.max_abs)
        self.lse_rel = max(self.lse_rel, o.lse_rel)
        self.lse_pure = max(self.lse_pure, o.lse_pure)
        self.lse_small_abs = max(self.lse_small_abs, o.lse_small_abs)
        self.rows += o.rows
        self.bad += o.bad

    def result(self):
        rr = math.sqrt(self.sq_err / self.sq_ref) if self.sq_ref > 0 else math.sqrt(self.sq_err)
        return {"rows": self.rows, "max_abs": self.max_abs, "rel_rms": rr, "lse_rel": self.lse_rel,
                "lse_rel_pure": self.lse_pure, "lse_abs_small": self.lse_small_abs}

    def check(self, what, max_abs=MAX_ABS, rel_rms=REL_RMS, lse_rel=LSE_REL):
        assert not self.bad, f"{what}: {self.bad[:5]}"
        r = self.result()
        assert r["max_abs"] <= max_abs, f"{what}: max-abs {r['max_abs']:.3e} > {max_abs}"
        assert r["rel_rms"] <= rel_rms, f"{what}: rel-RMS {r['rel_rms']:.3e} > {rel_rms}"
        assert r["lse_rel"] <= lse_rel, f"{what}: lse rel {r['lse_rel']:.3e} > {lse_rel}"
        return r


class HostCall:
    """Host copies of one call's inputs and outputs (numpy; bf16 as uint16 bits,
    FP8 E4M3 as uint8 codes): what the full-row comparison reads."""

    def __init__(self, kind, q, k_pages, v_pages, block_table, kv_lens, scale, out, lse, qo_indptr=None,
                 k_scale=None, v_scale=None):
        self.kind = kind                 # "decode": q [B, Hq, 128]; "extend": q [total_q, Hq, 128]
        self.q = q
        self.k_pages, self.v_pages = k_pages, v_pages
        self.block_table = block_table
        self.kv_lens = np.asarray(kv_lens)
        self.qo_indptr = None if qo_indptr is None else np.asarray(qo_indptr)
        self.scale = scale
        self.out = out                   # float32 / float64 host array, q's shape
        self.lse = lse                   # float32 host array [rows, Hq]
        self.k_scale, self.v_scale = k_scale, v_scale

    @staticmethod
    def from_gpu(kind, tensors: dict, out: torch.Tensor, lse: torch.Tensor, q: torch.Tensor = None,
                 qo_indptr=None):
        q = tensors["q"] if q is None else q
        sc = host_scales(tensors)
        if kind == "extend" and qo_indptr is None:
            qo_indptr = tensors["qo_indptr"].cpu().numpy()
        return HostCall(kind, to_host(q.contiguous()), to_host(tensors["k_pages"]), to_host(tensors["v_pages"]),
                        tensors["block_table"].cpu().numpy(), tensors["kv_lens"].cpu().numpy(), tensors["scale"],
                        out.float().cpu().numpy(), lse.float().cpu().numpy(), qo_indptr=qo_indptr,
                        k_scale=sc.get("k_scale"), v_scale=sc.get("v_scale"))

    def tasks(self):
        """(cost, task) pairs: decode -> sequence b; extend -> (b, KV head g)."""
        hkv = self.k_pages.shape[2]
        if self.kind == "decode":
            return [(int(self.kv_lens[b]) + 1, (b,)) for b in range(len(self.kv_lens))]
        res = []
        for b in range(len(self.kv_lens)):
            n = int(self.qo_indptr[b + 1] - self.qo_indptr[b])
            p = int(self.kv_lens[b]) - n
            for g in range(hkv):
                res.append((n * p + n * (n + 1) // 2 + 1, (b, g)))
        return res

    def run_task(self, task, what):
        acc = ParityAcc()
        if self.kind == "decode":
            (b,) = task
            ref_o, ref_l = oracle.decode(self.q[b:b + 1], self.k_pages, self.v_pages, self.block_table[b:b + 1],
                                         self.kv_lens[b:b + 1], self.scale, k_scale=self.k_scale,
                                         v_scale=self.v_scale)
            acc.add(self.out[b:b + 1], ref_o, self.lse[b:b + 1], ref_l, f"{what} seq {b}")
            return acc
        b, g = task
        q0, q1 = int(self.qo_indptr[b]), int(self.qo_indptr[b + 1])
        if q1 == q0:
            return acc
        hkv = self.k_pages.shape[2]
        r = self.q.shape[1] // hkv
        hs = slice(g * r, (g + 1) * r)
        ks = None if self.k_scale is None else self.k_scale[g:g + 1]
        vs = None if self.v_scale is None else self.v_scale[g:g + 1]
        ref_o, ref_l = oracle.extend(self.q[q0:q1, hs], np.array([0, q1 - q0], np.int32),
                                     self.k_pages[:, :, g:g + 1], self.v_pages[:, :, g:g + 1],
                                     self.block_table[b:b + 1], self.kv_lens[b:b + 1], self.scale,
                                     k_scale=ks, v_scale=vs)
        acc.add(self.out[q0:q1, hs], ref_o, self.lse[q0:q1, hs], ref_l, f"{what} seq {b} kv head {g}")
        return acc


def full_parity(call: HostCall, what: str, part: int = 0, parts: int = 1, workers: int = None,
                progress_s: float = 20.0) -> ParityAcc:
    """Compare every row of ``call`` (or of its ``part``-th of ``parts`` shares of
    tasks, dealt longest first) with the oracle; returns the accumulated errors."""
    import concurrent.futures
    import time

    from threadpoolctl import threadpool_limits

    tasks = sorted(call.tasks(), key=lambda x: -x[0])
    mine = [t for i, (_, t) in enumerate(tasks) if i % parts == part]
    workers = workers or host_workers()
    acc = ParityAcc()
    t0 = time.perf_counter()
    last = t0
    with threadpool_limits(1, "blas"), concurrent.futures.ThreadPoolExecutor(workers) as ex:
        futs = [ex.submit(call.run_task, t, what) for t in mine]
        for i, f in enumerate(concurrent.futures.as_completed(futs)):
            acc.merge(f.result())
            now = time.perf_counter()
            if now - last >= progress_s:
                say(f"  {what}: {i + 1}/{len(mine)} tasks, {now - t0:.0f} s")
                last = now
    say(f"  {what}: {len(mine)} tasks on {workers} threads in {time.perf_counter() - t0:.1f} s: {acc.result()}")
    return acc
