"""Host-side pieces of bench.py (no GPU): the one-GPU guard, timing statistics and the
traffic profiles' source hash."""

import importlib
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
_THREAD_VARS = ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")


def _bench(monkeypatch):
    """bench.py pins the BLAS thread variables when it is imported: record them so the
    test restores them afterwards."""
    for v in _THREAD_VARS:
        if v in os.environ:
            monkeypatch.setenv(v, os.environ[v])
        else:
            monkeypatch.delenv(v, raising=False)
    return importlib.import_module("bench")


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0
    assert "--gpus 1" in r.stderr
    assert not r.stdout.strip()            # no JSON line for an unsupported run


def test_timing_stats(monkeypatch):
    bench = _bench(monkeypatch)
    st = bench.timing_stats([5.0, 1.0, 3.0, 2.0, 4.0])
    assert st == {"ms_mean": 3.0, "ms_median": 3.0, "ms_min": 1.0, "ms_p90": 5.0, "calls": 5}
    st = bench.timing_stats([2.0, 4.0])
    assert st["ms_median"] == 3.0 and st["ms_p90"] == 4.0 and st["calls"] == 2
    st = bench.timing_stats([1.0] * 9 + [10.0])
    assert st["ms_p90"] == 1.0 and st["ms_mean"] == 1.9


def test_traffic_profiles_name_the_current_sources(monkeypatch):
    """The committed HBM-traffic summaries carry the hash of the kernel sources they were
    measured on; bench.py reports their traffic only while the sources still hash to it."""
    h = _bench(monkeypatch).kernel_source_hash()
    assert len(h) == 16
    for name in ("decode_ragged64k_hbm_traffic.json", "decode_ragged64k_fp8_hbm_traffic.json"):
        with open(os.path.join(ROOT, "profiles", name)) as f:
            prof = json.load(f)
        assert set(prof) >= {"source_hash", "algorithmic_bytes", "traffic_bytes", "traffic_over_algorithmic"}
        assert 0.99 < prof["traffic_over_algorithmic"] < 1.02
