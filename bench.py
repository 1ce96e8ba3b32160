"""Benchmark of the rollout-attention hot path on one MI355X.

One step = one pass of the whole path over resident synthetic batches:
  * decode, agentic ragged batch (B=128, 96 query / 8 KV heads, lognormal
    contexts, median 16K, clipped to [1K, 64K], page 64)  -> the headline;
  * decode with trajectory-group prefix sharing (16 prompts x G=8, shared
    4096-token prefix, private continuations U{512..16384});
  * extend (B=32, cached prefix U{8K..64K}, appended chunk U{64..2048}).
The tiny (B=4) and uniform (B=64 x 8192 keys) decode batches are timed beside
the step. Prints one JSON line. ``value`` is the decode KV-bytes rate of the
ragged 64K batch; every other workload's figures (mean, median, min and p90
call times, rates, roofline fractions) and the float64 oracle's rate on the
host cores for each workload are reported beside it.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)


def _host_threads() -> int:
    """Host threads of the oracle baseline: the affinity set, capped by an
    OMP_NUM_THREADS the environment already sets."""
    n = len(os.sched_getaffinity(0))
    try:
        n = min(n, int(os.environ.get("OMP_NUM_THREADS", n)))
    except ValueError:
        pass
    return max(1, n)


# BLAS thread counts are pinned before numpy is first imported
HOST_THREADS = _host_threads()
for _v in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
    os.environ[_v] = str(HOST_THREADS)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2516.6  # MI355X dense bf16 MFMA (256 CU x 4096 flop/clk x 2.4 GHz)
METRIC = "decode-attention KV GB/s (% of HBM peak) + extend TFLOP/s at 64k ctx"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_oracle(w, tensors, budget_s: float, threads: int = HOST_THREADS) -> dict:
    """The float64 oracle, as it stands, on a bounded sample of one workload, on the host cores.

    Decode: one sequence (all its heads) at a time in batch order, BLAS on
    ``threads`` threads (the oracle's page gather is a Python loop, so a thread
    pool would only contend for the interpreter). Extend: independent (sequence,
    KV head) pairs in a seeded random order on a pool of ``threads`` threads with
    one BLAS thread each (large matrix products and ufuncs, which release the
    interpreter), in rounds of ``threads`` pairs. Either runs until ``budget_s``
    of wall time has passed (or all are done). Returns the rate over the tasks
    done, scaled to the metric's units."""
    import concurrent.futures

    import numpy as np
    import torch
    from threadpoolctl import threadpool_limits

    import oracle
    from paper_2609_08368_amd import workloads as wl

    def bits(t):
        return wl.to_numpy_bits(t) if t.dtype == torch.bfloat16 else t.cpu().numpy()

    q, kp, vp = bits(tensors["q"]), bits(tensors["k_pages"]), bits(tensors["v_pages"])
    bt, lens, scale = w.block_table, w.kv_lens, tensors["scale"]
    hkv, hq = w.hkv, w.hq
    r = hq // hkv
    if w.kind == "decode":
        tasks = [(b,) for b in range(w.batch)]
    else:
        indptr = w.qo_indptr
        tasks = [(b, g) for b in range(w.batch) for g in range(hkv) if w.q_lens[b] > 0]
        tasks = [tasks[i] for i in np.random.default_rng(w.seed).permutation(len(tasks))]

    def run(task):
        if w.kind == "decode":
            (b,) = task
            oracle.decode(q[b:b + 1], kp, vp, bt[b:b + 1], lens[b:b + 1], scale)
            return int(lens[b]) * hkv * 512, 1.0, 4.0 * hq * 128 * int(lens[b])
        b, g = task
        q0, q1 = int(indptr[b]), int(indptr[b + 1])
        n, p = q1 - q0, int(lens[b]) - (q1 - q0)
        oracle.extend(q[q0:q1, g * r:(g + 1) * r], np.array([0, n], np.int32), kp[:, :, g:g + 1], vp[:, :, g:g + 1],
                      bt[b:b + 1], lens[b:b + 1], scale)
        return (n + p) * 512, n / hkv, 4.0 * r * 128 * (n * p + n * (n + 1) / 2)

    done = 0
    kv_bytes = tokens = flops = 0.0
    t0 = time.perf_counter()
    if w.kind == "decode":
        with threadpool_limits(threads, "blas"):
            while done < len(tasks) and time.perf_counter() - t0 < budget_s:
                kb, tk, fl = run(tasks[done])
                kv_bytes, tokens, flops, done = kv_bytes + kb, tokens + tk, flops + fl, done + 1
        how = f"one sequence at a time, BLAS on {threads} threads"
    else:
        with threadpool_limits(1, "blas"), concurrent.futures.ThreadPoolExecutor(threads) as ex:
            while done < len(tasks) and time.perf_counter() - t0 < budget_s:
                for kb, tk, fl in ex.map(run, tasks[done:done + threads]):
                    kv_bytes += kb
                    tokens += tk
                    flops += fl
                done = min(len(tasks), done + threads)
        how = f"{threads} threads, one BLAS thread each"
    wall = time.perf_counter() - t0
    unit_what = "sequences" if w.kind == "decode" else "(sequence, KV head) pairs"
    res = {"cores": int(threads), "kind": "oracle", "wall_s": round(wall, 3), "tasks": done, "of": len(tasks),
           "tokens_per_s": round(tokens / wall, 2),
           "sample": f"float64 oracle over {done} of {len(tasks)} {unit_what} of {w.name} "
                     f"({kv_bytes / 1e9:.3f} GB of KV, {flops / 1e12:.3f} TFLOP) in {wall:.2f} s ({how})"}
    if w.kind == "decode":
        res.update({"value": round(kv_bytes / wall / 1e9, 4), "unit": "GB/s"})
    else:
        res.update({"value": round(flops / wall / 1e12, 6), "unit": "TFLOP/s"})
    return res


def calls_then_kernel(fn, kind: str, steps: int):
    """Mean call time (ms) from HIP events around `steps` calls, then, in a second
    pass with the library's kernel timer on, the number of timed launches and the
    mean duration (ms) of the call's main kernel. The timer's events sit between
    the kernels of a call, so they are kept out of the call timing."""
    import torch

    from paper_2609_08368_amd import rl_attn as ra

    stream = torch.cuda.current_stream()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(steps):
        fn()
    b.record(stream)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    ra.profile_read(kind)
    ra.profile_enable(True)
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    ra.profile_enable(False)
    n_k, kern_ms = ra.profile_read(kind)
    return ms, n_k, kern_ms


def timing_stats(v) -> dict:
    """Mean, median, min and 90th percentile of per-call times (ms)."""
    v = sorted(v)
    n = len(v)
    p90 = v[min(n - 1, int(math.ceil(0.9 * n)) - 1)]
    return {"ms_mean": round(sum(v) / n, 4), "ms_median": round(v[n // 2] if n % 2 else 0.5 * (v[n // 2 - 1] + v[n // 2]), 4),
            "ms_min": round(v[0], 4), "ms_p90": round(p90, 4), "calls": n}


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "decode_ragged64k_hbm_traffic.json")
TRAFFIC_FILE_FP8 = os.path.join(ROOT, "profiles", "decode_ragged64k_fp8_hbm_traffic.json")
CALIB_BYTES = 2 << 30   # bytes read and bytes written by the calibration copy


def kernel_source_hash() -> str:
    """Hash of the HIP sources and build flags the decode kernel is built from."""
    import hashlib

    h = hashlib.sha256()
    pkg = os.path.join(ROOT, "paper_2609_08368_amd")
    csrc = os.path.join(pkg, "csrc")
    files = [os.path.join(csrc, n) for n in sorted(os.listdir(csrc)) if n.endswith((".hip", ".hpp", ".cpp"))]
    for path in files + [os.path.join(pkg, "build.py")]:
        with open(path, "rb") as f:
            h.update(os.path.basename(path).encode() + f.read())
    return h.hexdigest()[:16]


def pmc_workload(kind: str = "ragged"):
    """What the counter runs profile.

    ragged: three ragged-64K decode calls, then three copies of CALIB_BYTES (the
    calibration kernel for FETCH_SIZE / WRITE_SIZE); ragged-fp8: the same with FP8
    E4M3 pages; ragged-mtp2 / -mtp4 / -mtp8: the same pages with 2, 4 or 8 query tokens
    per sequence;
    extend: two multi-turn extend calls; group / group-noshare: three decode calls
    of the 16x8 trajectory-group batch with prefix sharing on / off, then the same
    calibration copies; branch / branch-noshare: the same for the 16x8 branching
    batch (prompt, half-group and pair prefixes shared)."""
    import torch

    from paper_2609_08368_amd import rl_attn as ra
    from paper_2609_08368_amd import workloads as wl

    dev = torch.device("cuda:0")
    mtp = int(kind[len("ragged-mtp"):]) if kind.startswith("ragged-mtp") else 0
    w = {"ragged": wl.decode_ragged, "ragged-fp8": wl.decode_ragged, "extend": wl.extend_multiturn,
         "branch": wl.decode_branching, "branch-noshare": wl.decode_branching}.get(
             "ragged" if mtp else kind, wl.decode_group_prefix)()
    fp8 = kind == "ragged-fp8"
    t = (wl.materialize_fp8 if fp8 else wl.materialize)(w, dev, poison=False)
    out = torch.empty_like(t["q"])
    def calibrate():
        src = torch.empty(CALIB_BYTES // 2, dtype=torch.bfloat16, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()

    if kind == "extend":
        for _ in range(2):
            ra.extend_plain(t["q"], t["qo_indptr"], t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"],
                            t["scale"], out=out)
        torch.cuda.synchronize()
        del t, out
        torch.cuda.empty_cache()
        calibrate()
        print(json.dumps({"pmc_workload": kind, "flops": w.flops(), "kv_bytes": w.kv_bytes(),
                          "calib_bytes": CALIB_BYTES}), flush=True)
        return
    share = {"prefix_share": not kind.endswith("-noshare")}
    if mtp:
        g = torch.Generator(device=dev)
        g.manual_seed(900 + mtp)
        t["q"] = torch.randn((w.batch, mtp, w.hq, 128), generator=g, device=dev).to(torch.bfloat16)
        out = torch.empty_like(t["q"])
    for _ in range(3):
        if fp8:
            ra.decode_fp8(t["q"], t["k_pages"], t["v_pages"], t["k_scale"], t["v_scale"], t["block_table"],
                          t["kv_lens"], t["scale"], out=out)
        else:
            ra.decode(t["q"], t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], out=out,
                      **share)
    calibrate()
    per_elem = 0.5 if fp8 else 1.0     # kv_bytes() counts bf16 elements
    print(json.dumps({"pmc_workload": kind, "kv_bytes": int(w.kv_bytes(unique=True) * per_elem),
                      "logical_kv_bytes": int(w.kv_bytes() * per_elem), "calib_bytes": CALIB_BYTES}), flush=True)


def prefix_study(steps: int = 20):
    """Group-prefix decode with prefix sharing on and off: the 16x8 group batch
    (4096 shared tokens), its long-prompt variant (32768 shared tokens) and the
    16x8 branching batch (4096 tokens per group, 2048 per half, 1024 per pair)."""
    import torch

    from paper_2609_08368_amd import rl_attn as ra
    from paper_2609_08368_amd import workloads as wl

    dev = torch.device("cuda:0")
    res = {}
    for w in (wl.decode_group_prefix(), wl.decode_group_long_prefix(), wl.decode_branching()):
        t = wl.materialize(w, dev, poison=False)
        out = torch.empty_like(t["q"])
        row = {"unique_kv_bytes": w.kv_bytes(unique=True), "logical_kv_bytes": w.kv_bytes()}
        for share in (True, False):
            call = lambda: ra.decode(t["q"], t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"],
                                     out=out, prefix_share=share)
            for _ in range(3):
                call()
            torch.cuda.synchronize()
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            ev[0].record()
            for _ in range(steps):
                call()
            ev[1].record()
            torch.cuda.synchronize()
            row["ms_share" if share else "ms_no_share"] = round(ev[0].elapsed_time(ev[1]) / steps, 4)
        row["speedup"] = round(row["ms_no_share"] / row["ms_share"], 3)
        res[w.name] = row
        del t, out
        torch.cuda.empty_cache()
    print(json.dumps(res), flush=True)


def summarize_counters(d: str):
    """Per kernel and counter: dispatches and the mean value per dispatch (summed over
    the counter's dimensions) of a rocprofv3 --pmc output directory."""
    import csv
    import glob

    per = {}
    for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(path)):
            name = r["Kernel_Name"].replace("(anonymous namespace)::", "").split("(")[0]
            key = (name, r["Counter_Name"], int(r["Dispatch_Id"]))
            per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
    agg = {}
    for (kern, ctr, _), v in per.items():
        agg.setdefault((kern, ctr), []).append(v)
    for (kern, ctr), vals in sorted(agg.items()):
        print(f"{kern[-40:]:40s} {ctr:32s} dispatches {len(vals):3d}  mean {sum(vals) / len(vals):.6g}")


def summarize_pmc(fetch_dir: str, write_dir: str, fp8: bool = False, extend: bool = False):
    """Turn the FETCH_SIZE and WRITE_SIZE runs into the committed traffic summary
    (``fp8``: runs of the ``ragged-fp8`` workload; ``extend``: of the ``extend``
    workload)."""
    import csv
    import glob

    from paper_2609_08368_amd import workloads as wl

    kname = "extend_mfma_kernel" if extend else "decode_mfma_kernel"

    def per_kernel(d, counter):
        # KiB per dispatch of the attention kernel, and of the calibration copies
        # (the copy dispatches issued after the last attention dispatch)
        rows = []
        for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            rows += [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        per = {}
        for r in rows:
            key = (int(r["Dispatch_Id"]), r["Kernel_Name"])
            per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
        dec = {k: v for k, v in per.items() if kname in k[1]}
        last_dec = max(k[0] for k in dec)
        cal = {k: v for k, v in per.items() if "copy" in k[1].lower() and k[0] > last_dec}
        return {"decode": sum(dec.values()) / len(dec), "copy": sum(cal.values()) / len(cal)}

    if extend:
        return summarize_extend_pmc(per_kernel(fetch_dir, "FETCH_SIZE"), per_kernel(write_dir, "WRITE_SIZE"),
                                    fetch_dir.rstrip("/"), write_dir.rstrip("/"))

    fetch = per_kernel(fetch_dir, "FETCH_SIZE")
    write = per_kernel(write_dir, "WRITE_SIZE")
    f_scale = CALIB_BYTES / (fetch["copy"] * 1024.0)
    w_scale = CALIB_BYTES / (write["copy"] * 1024.0)
    dec_fetch = fetch["decode"] * 1024.0 * f_scale
    dec_write = write["decode"] * 1024.0 * w_scale
    w = wl.decode_ragged()
    algo = w.kv_bytes() // 2 if fp8 else w.kv_bytes()
    res = {
        "kernel": "decode_mfma_kernel<true>" if fp8 else "decode_mfma_kernel<false>",
        "workload": "ragged 64K decode batch (B128, Hq96/Hkv8, page 64)" + (", FP8 E4M3 pages" if fp8 else ", bf16 pages"),
        "source_hash": kernel_source_hash(),
        "fetch_kib_per_dispatch": fetch["decode"], "write_kib_per_dispatch": write["decode"],
        "copy_fetch_kib": fetch["copy"], "copy_write_kib": write["copy"], "calib_bytes": CALIB_BYTES,
        "fetch_scale": f_scale, "write_scale": w_scale,
        "hbm_read_bytes": dec_fetch, "hbm_write_bytes": dec_write, "traffic_bytes": dec_fetch + dec_write,
        "algorithmic_bytes": algo,
        "traffic_over_algorithmic": (dec_fetch + dec_write) / algo,
    }
    path = TRAFFIC_FILE_FP8 if fp8 else TRAFFIC_FILE
    with open(path, "w") as f:
        json.dump(res, f, indent=1)
    with open(path[:-5] + ".md", "w") as f:
        f.write(traffic_markdown(res, fp8, os.path.basename(path), fetch_dir.rstrip("/"), write_dir.rstrip("/")))
    print(json.dumps(res, indent=1))


def traffic_markdown(d: dict, fp8: bool, json_name: str, fetch_dir: str, write_dir: str) -> str:
    """The committed summary of one traffic measurement (written by --summarize-pmc from the two
    counter runs' output directories)."""
    kind = "ragged-fp8" if fp8 else "ragged"
    pages = "FP8 E4M3 pages" if fp8 else "bf16 pages"
    flag = " --fp8" if fp8 else ""
    return f"""# HBM traffic of {d['kernel']} on the ragged 64K decode batch with {pages}

Workload: B 128, Hq 96 / Hkv 8, lognormal contexts (median 16K, clipped 1K-64K), page 64;
sum of L = 2,544,208 keys, algorithmic KV bytes {d['algorithmic_bytes']:,} per launch.

Commands (repo root, one MI355X), one counter per pass:

    rocprofv3 --pmc FETCH_SIZE --output-format csv -d {fetch_dir} -o run -- python bench.py --pmc-workload {kind}
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d {write_dir} -o run -- python bench.py --pmc-workload {kind}
    python bench.py --summarize-pmc {fetch_dir} {write_dir}{flag}

`--pmc-workload {kind}` runs three decode launches and then three device copies of 2 GiB
(torch `copy_`, dispatched as `__amd_rocclr_copyBuffer`), which calibrate the counters:

| counter | calibration copy (KiB / dispatch) | known bytes | scale |
|---|---|---|---|
| FETCH_SIZE | {d['copy_fetch_kib']:,.0f} | 2 GiB read | {d['fetch_scale']:.3f} |
| WRITE_SIZE | {d['copy_write_kib']:,.0f} | 2 GiB written | {d['write_scale']:.3f} |

| {d['kernel']} | raw KiB / dispatch | scaled bytes |
|---|---|---|
| FETCH_SIZE | {d['fetch_kib_per_dispatch']:,.0f} | {d['hbm_read_bytes']:,.0f} ({d['hbm_read_bytes'] / d['algorithmic_bytes']:.4f} x algorithmic) |
| WRITE_SIZE | {d['write_kib_per_dispatch']:,.0f} | {d['hbm_write_bytes']:,.0f} (split partials) |
| traffic | | {d['traffic_bytes']:,.0f} ({d['traffic_over_algorithmic']:.4f} x algorithmic) |

Reads equal the algorithmic KV bytes: every K and V byte is fetched from HBM once, with no
re-reads. Writes are the fp32 partials of the pieces that split a sequence (at most one per
worker plus one per sequence). `bench.py` reports this traffic figure only while the kernel
sources hash to the value recorded in `{json_name}` (sources under csrc/ plus build.py;
hash {d['source_hash']}).
"""


EXTEND_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "extend_multiturn_hbm_traffic.json")


def summarize_extend_pmc(fetch: dict, write: dict, fetch_dir: str, write_dir: str):
    """The extend kernel's HBM traffic summary from the calibrated counter means."""
    from paper_2609_08368_amd import workloads as wl

    w = wl.extend_multiturn()
    f_scale = CALIB_BYTES / (fetch["copy"] * 1024.0)
    w_scale = CALIB_BYTES / (write["copy"] * 1024.0)
    rd = fetch["decode"] * 1024.0 * f_scale
    wr = write["decode"] * 1024.0 * w_scale
    q_bytes = w.total_q * w.hq * 128 * 2
    res = {"kernel": "extend_mfma_kernel<false, 0>", "workload": "multi-turn extend batch (B32, Hq64/Hkv8, page 64)",
           "source_hash": kernel_source_hash(), "fetch_kib_per_dispatch": fetch["decode"],
           "write_kib_per_dispatch": write["decode"], "copy_fetch_kib": fetch["copy"], "copy_write_kib": write["copy"],
           "fetch_scale": f_scale, "write_scale": w_scale, "hbm_read_bytes": rd, "hbm_write_bytes": wr,
           "kv_bytes": w.kv_bytes(), "q_bytes": q_bytes, "out_bytes": q_bytes,
           "read_over_kv_plus_q": rd / (w.kv_bytes() + q_bytes), "write_over_out": wr / q_bytes}
    with open(EXTEND_TRAFFIC_FILE, "w") as f:
        json.dump(res, f, indent=1)
    with open(EXTEND_TRAFFIC_FILE[:-5] + ".md", "w") as f:
        f.write(f"""# HBM traffic of {res['kernel']} on the multi-turn extend batch

Workload: B 32, cached prefix U{{8192..65536}}, chunk U{{64..2048}}, Hq 64 / Hkv 8, page 64;
36,098 chunk rows. Every K and V byte a sequence needs, read once: {res['kv_bytes']:,} B; q
{q_bytes:,} B read and out {q_bytes:,} B written.

Commands (repo root, one MI355X), one counter per pass:

    rocprofv3 --pmc FETCH_SIZE --output-format csv -d {fetch_dir} -o run -- python bench.py --pmc-workload extend
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d {write_dir} -o run -- python bench.py --pmc-workload extend
    python bench.py --summarize-pmc {fetch_dir} {write_dir} --extend

`--pmc-workload extend` runs two extend launches, then three 2 GiB device copies that
calibrate the counters (FETCH_SIZE scale {f_scale:.3f}, WRITE_SIZE scale {w_scale:.3f}).

| counter | raw KiB / dispatch | scaled bytes | reading |
|---|---|---|---|
| FETCH_SIZE | {fetch['decode']:,.0f} | {rd:,.0f} | {res['read_over_kv_plus_q']:.3f} x (KV + q) |
| WRITE_SIZE | {write['decode']:,.0f} | {wr:,.0f} | {res['write_over_out']:.3f} x out |

The kernel is bound by the matrix cores, not by HBM: at about 42 ms per launch these bytes move
at about {(rd + wr) / 42e-3 / 1e9:,.0f} GB/s. The work units of one (sequence, KV head) run
on one XCD and share their keys through its L2, so the keys beyond the first unit's reads
mostly come from L2. Sources hash {res['source_hash']}.
""")
    print(json.dumps(res, indent=1))


def traffic_bytes(fp8: bool = False):
    """HBM bytes per decode launch from the committed counter summary, or None
    when the summary is missing or the kernel sources changed since it was taken."""
    try:
        with open(TRAFFIC_FILE_FP8 if fp8 else TRAFFIC_FILE) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return None
    return d["traffic_bytes"] if d.get("source_hash") == kernel_source_hash() else None


def fp8_study(steps: int, warmup: int, w_dec, w_ext, bf16_dec_ms: float, bf16_ext_ms: float) -> dict:
    """Time decode and extend of the same batches with FP8 E4M3 KV pages."""
    import torch

    from paper_2609_08368_amd import rl_attn as ra
    from paper_2609_08368_amd import workloads as wl

    dev = torch.device("cuda:0")
    log("FP8 KV pages: materialising ...")
    res = {"format": "OCP E4M3 codes, one fp32 dequantisation scale per KV head (amax / 448)"}
    for name, w in (("decode_ragged", w_dec), ("extend_multiturn", w_ext)):
        t = wl.materialize_fp8(w, dev, poison=False)
        out = torch.empty_like(t["q"])
        if w.kind == "decode":
            def fn():
                ra.decode_fp8(t["q"], t["k_pages"], t["v_pages"], t["k_scale"], t["v_scale"], t["block_table"],
                              t["kv_lens"], t["scale"], out=out)
        else:
            def fn():
                ra.extend_fp8(t["q"], t["qo_indptr"], t["k_pages"], t["v_pages"], t["k_scale"], t["v_scale"],
                              t["block_table"], t["kv_lens"], t["scale"], out=out)
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        kind = "decode" if w.kind == "decode" else "extend"
        ms, n_k, kern_ms = calls_then_kernel(fn, kind, steps)
        fp8_bytes = w.kv_bytes() // 2          # one byte per element
        row = {"ms_mean": round(ms, 4), "kernel_ms": round(kern_ms, 4) if n_k else None,
               "speedup_vs_bf16": round((bf16_dec_ms if kind == "decode" else bf16_ext_ms) / ms, 3)}
        if kind == "decode":
            row.update({"kv_bytes": fp8_bytes, "traffic": traffic_bytes(fp8=True),
                        "kv_GBps": round(fp8_bytes / (ms * 1e-3) / 1e9, 2),
                        "hbm_frac": round(fp8_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                        "kernel_GBps": round(fp8_bytes / (kern_ms * 1e-3) / 1e9, 2) if n_k else None,
                        "tokens_per_s": round(w.batch / (ms * 1e-3), 1)})
        else:
            row.update({"tflops": round(w.flops() / (ms * 1e-3) / 1e12, 2),
                        "mfma_frac": round(w.flops() / (ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)})
        res[name] = row
        log(f"FP8 {name}: {row}")
        del t, out
        torch.cuda.empty_cache()
    return res


def deterministic_study(steps: int, warmup: int, w, t, split_ms: float) -> dict:
    """Time the batch-invariant decode (one extend row per sequence, no key split)."""
    import torch

    from paper_2609_08368_amd import rl_attn as ra

    out = torch.empty_like(t["q"])

    def fn():
        ra.decode(t["q"], t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], out=out,
                  deterministic=True)

    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(steps):
        fn()
    b.record(stream)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    gbps = w.kv_bytes() / (ms * 1e-3) / 1e9
    res = {"workload": "ragged 64K decode batch, bf16 pages", "ms_mean": round(ms, 4), "kv_GBps": round(gbps, 2),
           "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4), "slowdown_vs_split_kv": round(ms / split_ms, 3)}
    log(f"deterministic decode: {res}")
    return res


def append_study(steps: int, warmup: int, w_ext, w_dec) -> dict:
    """Time KV append: the multi-turn batch's chunk tokens, and one decode step's tokens of
    the ragged batch, into bf16 and FP8 pages (new rows resident in HBM)."""
    import torch

    from paper_2609_08368_amd import rl_attn as ra
    from paper_2609_08368_amd import workloads as wl

    dev = torch.device("cuda:0")
    res = {}
    for wname, w in (("extend_chunks", w_ext), ("decode_step", w_dec)):
        total = w.total_q if w.kind == "extend" else w.batch
        g = torch.Generator(device=dev)
        g.manual_seed(77)
        k = torch.randn((total, w.hkv, 128), generator=g, device=dev).to(torch.bfloat16)
        v = torch.randn((total, w.hkv, 128), generator=g, device=dev).to(torch.bfloat16)
        for fp8 in (False, True):
            t = (wl.materialize_fp8 if fp8 else wl.materialize)(w, dev, poison=False)
            if w.kind == "extend":
                indptr = t["qo_indptr"]
            else:
                indptr = torch.arange(w.batch + 1, dtype=torch.int32, device=dev)

            def fn():
                if fp8:
                    ra.append_kv_fp8(k, v, indptr, t["block_table"], t["kv_lens"], t["k_pages"], t["v_pages"],
                                     t["k_scale"], t["v_scale"])
                else:
                    ra.append_kv(k, v, indptr, t["block_table"], t["kv_lens"], t["k_pages"], t["v_pages"])

            for _ in range(warmup):
                fn()
            torch.cuda.synchronize()
            ms, _, kern_ms = calls_then_kernel(fn, "append", steps)
            elems = 2 * total * w.hkv * 128
            moved = elems * 2 + elems * (1 if fp8 else 2)        # read bf16 rows, write pages
            res[f"{wname}_{'fp8' if fp8 else 'bf16'}"] = {
                "rows": total, "ms_per_call": round(ms, 5), "kernel_ms": round(kern_ms, 5), "bytes": moved,
                "kernel_GBps": round(moved / (kern_ms * 1e-3) / 1e9, 1),
                "hbm_frac": round(moved / (kern_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)}
            del t
            torch.cuda.empty_cache()
    log(f"append: {res}")
    return res


def mtp_study(steps: int, warmup: int, w, t, single_ms: float) -> dict:
    """Multi-token decode (n query tokens per sequence, as when verifying multi-token-prediction
    drafts) on the ragged batch's pages: the KV bytes are read once for all n tokens."""
    import torch

    from paper_2609_08368_amd import rl_attn as ra

    dev = torch.device("cuda:0")
    res = {"workload": "ragged 64K decode batch, bf16 pages, n query tokens per sequence (the last n keys)",
           "route": "prefix sharing on: the decode planner finds no shared page in this batch, so the queued "
                    "extend pass computes the rows (one unit per sequence and KV head) and the split passes "
                    "return at once; kernel_ms spans every kernel of the call, planners included",
           "prefix_share_off": {"note": "the same calls with prefix sharing off, which run through the extend "
                                        "kernel directly (no split of the keys, no decode planner)"}}
    for n in (2, 4, 8):
        g = torch.Generator(device=dev)
        g.manual_seed(900 + n)
        q = torch.randn((w.batch, n, w.hq, 128), generator=g, device=dev).to(torch.bfloat16)
        out = torch.empty_like(q)
        for share in (True, False):
            def fn():
                ra.decode(q, t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"], out=out,
                          prefix_share=share)

            for _ in range(warmup):
                fn()
            torch.cuda.synchronize()
            ms, _, kern_ms = calls_then_kernel(fn, "decode", steps)
            gbps = w.kv_bytes() / (ms * 1e-3) / 1e9
            row = {"ms_mean": round(ms, 4), "kernel_ms": round(kern_ms, 4), "kv_GBps": round(gbps, 2),
                   "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4),
                   "query_tokens_per_s": round(w.batch * n / (ms * 1e-3), 1),
                   "time_vs_single_token": round(ms / single_ms, 3)}
            (res if share else res["prefix_share_off"])[f"n{n}"] = row
    log(f"multi-token decode: {res}")
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="scales the oracle baseline's wall-time budgets (15: 33 s over the five workloads)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--pmc-workload", nargs="?", const="ragged",
                    choices=["ragged", "ragged-fp8", "ragged-mtp2", "ragged-mtp4", "ragged-mtp8", "extend", "group",
                             "group-noshare", "branch", "branch-noshare"],
                    help="run only what a counter run profiles")
    ap.add_argument("--summarize-counters", metavar="PMC_DIR", help="per-kernel means of a rocprofv3 --pmc run")
    ap.add_argument("--prefix-study", action="store_true", help="time group-prefix decode with sharing on and off")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write the HBM traffic summary from two rocprofv3 --pmc output directories")
    ap.add_argument("--fp8", action="store_true", help="with --summarize-pmc: runs of --pmc-workload ragged-fp8")
    ap.add_argument("--extend", action="store_true", help="with --summarize-pmc: runs of --pmc-workload extend")
    args = ap.parse_args()
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, fp8=args.fp8, extend=args.extend)
        return
    if args.pmc_workload:
        pmc_workload(args.pmc_workload)
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters)
        return
    if args.prefix_study:
        prefix_study()
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (each GPU would serve its own "
              "sequences or KV heads, with no exchange inside attention). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_08368_amd import rl_attn as ra
    from paper_2609_08368_amd import workloads as wl

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    ra.lib()
    log("materialising inputs on the GPU ...")
    w_tiny = wl.decode_tiny()
    w_uni = wl.decode_uniform()
    w_dec = wl.decode_ragged()
    w_grp = wl.decode_group_prefix()
    w_ext = wl.extend_multiturn()
    t_tiny = wl.materialize(w_tiny, dev, poison=False)
    t_uni = wl.materialize(w_uni, dev, poison=False)
    t_dec = wl.materialize(w_dec, dev, poison=False)
    t_grp = wl.materialize(w_grp, dev, poison=False)
    t_ext = wl.materialize(w_ext, dev, poison=False)
    outs = {id(t): torch.empty_like(t["q"]) for t in (t_tiny, t_uni, t_dec, t_grp, t_ext)}
    torch.cuda.synchronize()
    log(f"ragged decode: sum(L)={int(w_dec.kv_lens.sum())}  group decode: sum(L)={int(w_grp.kv_lens.sum())}  "
        f"extend: total_q={w_ext.total_q}")

    def decode(t):
        ra.decode_plain(t["q"], t["k_pages"], t["v_pages"], t["block_table"], t["kv_lens"], t["scale"],
                        out=outs[id(t)])

    def extend():
        ra.extend_plain(t_ext["q"], t_ext["qo_indptr"], t_ext["k_pages"], t_ext["v_pages"], t_ext["block_table"],
                        t_ext["kv_lens"], t_ext["scale"], out=outs[id(t_ext)])

    # one step: the headline decode, the trajectory-group decode and the extend
    parts = [("decode_ragged", lambda: decode(t_dec)),
             ("decode_group_prefix", lambda: decode(t_grp)),
             ("extend_multiturn", extend)]
    for _ in range(args.warmup):
        for _, fn in parts:
            fn()
    torch.cuda.synchronize()
    log(f"warmup done; timing {args.steps} steps")

    stream = torch.cuda.current_stream()
    ev = {name: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                 for _ in range(args.steps)] for name, _ in parts}
    torch.cuda.synchronize()
    step_start = torch.cuda.Event(enable_timing=True)
    step_stop = torch.cuda.Event(enable_timing=True)
    step_start.record(stream)
    for i in range(args.steps):
        for name, fn in parts:
            ev[name][i][0].record(stream)
            fn()
            ev[name][i][1].record(stream)
    step_stop.record(stream)
    torch.cuda.synchronize()
    total_ms = step_start.elapsed_time(step_stop)
    ms = {name: [a.elapsed_time(b) for a, b in ev[name]] for name in ev}

    # kernel-level timing in passes of their own, with the library's kernel
    # timer on (its events would otherwise sit inside the timed calls): the
    # ragged decode kernel (the roofline) and the extend kernel
    ra.profile_read("decode")
    ra.profile_enable(True)
    for _ in range(args.steps):
        parts[0][1]()
    torch.cuda.synchronize()
    ra.profile_enable(False)
    n_k, dec_kernel_ms = ra.profile_read("decode")
    ra.profile_read("extend")
    ra.profile_enable(True)
    for _ in range(args.steps):
        extend()
    torch.cuda.synchronize()
    ra.profile_enable(False)
    n_ext, ext_kernel_ms = ra.profile_read("extend")

    # the tiny and the uniform decode batches, timed call by call outside the step
    for name, t in (("decode_tiny", t_tiny), ("decode_uniform", t_uni)):
        for _ in range(args.warmup):
            decode(t)
        torch.cuda.synchronize()
        pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                 for _ in range(max(args.steps, 20))]
        for a, b in pairs:
            a.record(stream)
            decode(t)
            b.record(stream)
        torch.cuda.synchronize()
        ms[name] = [a.elapsed_time(b) for a, b in pairs]
    st = {name: timing_stats(v) for name, v in ms.items()}
    mean = {name: v["ms_mean"] for name, v in st.items()}

    kv_dec = w_dec.kv_bytes()
    kv_uni = w_uni.kv_bytes()
    kv_grp_unique = w_grp.kv_bytes(unique=True)
    kv_grp_logical = w_grp.kv_bytes()
    kv_ext = w_ext.kv_bytes()
    flops_ext = w_ext.flops()
    dec_gbps = kv_dec / (mean["decode_ragged"] * 1e-3) / 1e9
    kern_gbps = kv_dec / (dec_kernel_ms * 1e-3) / 1e9
    uni_gbps = kv_uni / (mean["decode_uniform"] * 1e-3) / 1e9
    ext_tflops = flops_ext / (mean["extend_multiturn"] * 1e-3) / 1e12
    ext_kern_tflops = flops_ext / (ext_kernel_ms * 1e-3) / 1e12 if n_ext else None
    grp_s = mean["decode_group_prefix"] * 1e-3

    result = {
        "metric": METRIC,
        "value": round(dec_gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(total_ms / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "step = decode of the agentic ragged batch (B128, Hq96/Hkv8, lognormal median 16K clipped "
                        "1K-64K, page 64; value) + decode with trajectory-group prefix sharing (16x8, shared 4096, "
                        "private 512-16384, Hq64/Hkv8) + extend (B32, prefix 8K-64K, chunk 64-2048, Hq64/Hkv8); "
                        "the tiny (B4, Hq8/Hkv2, 128-512 keys, page 16) and uniform (B64, Hq64/Hkv8, 8192 keys, "
                        "page 64) decode batches are timed beside the step",
            "decode_batch": w_dec.batch, "decode_sum_kv_tokens": int(w_dec.kv_lens.sum()),
            "decode_kv_bytes": kv_dec, "head_dim": 128, "page_size": 64, "seed": w_dec.seed,
        },
        "decode_ragged": dict(st["decode_ragged"], **{
            "kv_GBps": round(dec_gbps, 2), "hbm_frac": round(dec_gbps / HBM_PEAK_GBPS, 4),
            "kv_GBps_at_median": round(kv_dec / (st["decode_ragged"]["ms_median"] * 1e-3) / 1e9, 2),
            "tokens_per_s": round(w_dec.batch / (mean["decode_ragged"] * 1e-3), 1),
        }),
        "decode_group_prefix": dict(st["decode_group_prefix"], **{
            "unique_kv_GBps": round(kv_grp_unique / grp_s / 1e9, 2),
            "logical_kv_GBps": round(kv_grp_logical / grp_s / 1e9, 2),
            "hbm_frac_unique": round(kv_grp_unique / grp_s / 1e9 / HBM_PEAK_GBPS, 4),
            "tokens_per_s": round(w_grp.batch / grp_s, 1),
        }),
        "extend_multiturn": dict(st["extend_multiturn"], **{
            "tflops": round(ext_tflops, 2),
            "mfma_frac": round(ext_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
            "kernel_ms": round(ext_kernel_ms, 4) if n_ext else None,
            "kernel_tflops": round(ext_kern_tflops, 2) if ext_kern_tflops else None,
            "tokens_per_s": round(w_ext.total_q / (mean["extend_multiturn"] * 1e-3), 1),
            "flops": flops_ext, "kv_bytes": kv_ext,
        }),
        "decode_uniform": dict(st["decode_uniform"], **{
            "kv_bytes": kv_uni, "kv_GBps": round(uni_gbps, 2), "hbm_frac": round(uni_gbps / HBM_PEAK_GBPS, 4),
            "tokens_per_s": round(w_uni.batch / (mean["decode_uniform"] * 1e-3), 1),
        }),
        "decode_tiny": dict(st["decode_tiny"], **{
            "kv_bytes": w_tiny.kv_bytes(), "bound": "launch latency (time only)",
            "tokens_per_s": round(w_tiny.batch / (mean["decode_tiny"] * 1e-3), 1),
        }),
        "roofline": {
            "kernel": "decode_mfma_kernel (ragged 64K decode batch)",
            "bound": "hbm", "achieved": round(kern_gbps, 2), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(kern_gbps / HBM_PEAK_GBPS, 4), "traffic": traffic_bytes(),
            "kernel_ms": round(dec_kernel_ms, 4), "launches": n_k,
            "algorithmic_bytes": kv_dec,
        },
    }
    # the same ragged decode and extend batches with FP8 E4M3 KV pages (per-KV-head scales):
    # reported beside the bf16 step, not part of it
    host_inputs = {"decode_tiny": (w_tiny, t_tiny), "decode_uniform": (w_uni, t_uni),
                   "decode_ragged": (w_dec, t_dec), "decode_group_prefix": (w_grp, t_grp),
                   "extend_multiturn": (w_ext, t_ext)}
    result["deterministic_decode"] = deterministic_study(args.steps, args.warmup, w_dec, t_dec,
                                                         mean["decode_ragged"])
    result["multi_token_decode"] = mtp_study(args.steps, args.warmup, w_dec, t_dec, mean["decode_ragged"])
    result["kv_append"] = append_study(args.steps, args.warmup, w_ext, w_dec)
    result["fp8_kv"] = fp8_study(args.steps, args.warmup, w_dec, w_ext, mean["decode_ragged"],
                                 mean["extend_multiturn"])
    # measured ceilings on this device, beside the specification peaks
    torch.cuda.empty_cache()
    buf = torch.ones(4 << 30, dtype=torch.uint8, device=dev)
    read_gbps = ra.diag_read_bandwidth(buf, reps=10)
    del buf
    loop_tflops = ra.diag_mfma_bf16(20000)
    result["ceilings"] = {
        "read_loop_GBps": round(read_gbps, 1), "read_loop_frac_of_spec": round(read_gbps / HBM_PEAK_GBPS, 4),
        "decode_over_read_loop": round(dec_gbps / read_gbps, 4),
        "decode_kernel_over_read_loop": round(kern_gbps / read_gbps, 4),
        "mfma_bf16_loop_TFLOPs": round(loop_tflops, 1),
        "mfma_loop_frac_of_spec": round(loop_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
        "extend_frac_of_mfma_loop": round(ext_tflops / loop_tflops, 4),
    }
    if not args.no_cpu_baseline:
        log(f"timing the oracle on {HOST_THREADS} host threads ...")
        per = {}
        budgets = {"decode_tiny": 1.0, "decode_uniform": 6.0, "decode_ragged": 10.0, "decode_group_prefix": 6.0,
                   "extend_multiturn": 10.0}
        for name, (w, t) in host_inputs.items():
            per[name] = cpu_oracle(w, t, budgets[name] * args.cpu_budget / 15.0)
            log(f"oracle {name}: {per[name]}")
        result["cpu_baseline"] = dict(per["decode_ragged"])
        result["cpu_baseline_per_config"] = per
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
