"""bench.py's JSON line on the GPU: one short run of the small signature
workload and one of the timing workload, each checked for the fields of the
line's contract (metric, value, roofline with frac = achieved / peak, the
oracle's cpu_baseline) and for the parity the run reports against the
oracle."""
import json
import math
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args):
    print("CASE bench", *args, flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + list(args), cwd=ROOT,
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1, r.stdout[-2000:]
    return json.loads(lines[0])


def _contract(d, steps, warmup):
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
              "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
              "roofline", "cpu_baseline"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == steps and d["warmup"] == warmup
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["higher_is_better"] is True
    assert d["data"] == "synthetic" and "workload" in d["config"]
    rf = d["roofline"]
    assert rf["bound"] == "hbm" and rf["unit"] == "GB/s" and rf["peak"] == 8000.0
    assert math.isclose(rf["frac"], rf["achieved"] / rf["peak"], rel_tol=1e-3)
    alg = rf["algorithmic_bytes_per_launch"]
    # counter-based traffic is reported only while the kernel's sources are
    # those the counters were taken on
    assert rf["traffic"] is None or 0.99 * alg <= rf["traffic"] <= 1.05 * alg
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] == 1 and cb["value"] > 0 and cb["sample"]


def test_signature_bench_line_small_workload():
    d = _bench("--config", "1", "--steps", "3", "--warmup", "2")
    _contract(d, 3, 2)
    assert d["metric"] == "replica GB/s fingerprinted+localized; % of MI355X HBM peak"
    assert d["config"]["workload"] == "r3_f32_1m_chunk4096el"
    assert d["parity"]["ok"] is True and d["parity"]["records_differing"] == 0
    # the planted flip: replica 2, one chunk
    assert d["config"]["outliers"] == 1


def test_timing_bench_line():
    d = _bench("--config", "5", "--steps", "3", "--warmup", "2")
    _contract(d, 3, 2)
    assert d["config"]["workload"] == "ranks32768_g8_iters1024_fp64_time_f32"
    p = d["parity"]
    assert p["ok"] is True and p["per_unit_results_equal"] is True
    assert p["units_compared"] == 1024 * 4096 and p["verdict_fields_differing"] == 0
    assert d["config"]["stragglers_found"] == 5 and d["config"]["protocol_outliers_found"] == 3
