"""Host-side pieces of the benchmark (CPU only): the refusal of more than
one GPU, the algorithmic flop and byte counts the roofline entry divides by,
the regret and bootstrap helpers of the sweep, and the traffic entry's
kernel-source check."""
import json
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from workloads import config  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_algorithmic_counts_of_the_headline_workload():
    """2 Mtot I H flops; x, W2, Y written and read back, ids and gates, out."""
    w = config("dsv2lite")
    flops, gemm_bytes, combine_bytes, min_bytes = bench.algorithmic(w)
    assert (w.T, w.H, w.I, w.E, w.topk, w.Mtot) == (16384, 2048, 704, 32, 6, 98304)
    assert flops == 2 * 98304 * 704 * 2048 == 283467841536
    x, w2, y = 98304 * 704 * 2, 32 * 704 * 2048 * 2, 98304 * 2048 * 2
    assert gemm_bytes == x + w2 + y
    assert combine_bytes == y + 98304 * 8 + 16384 * 2048 * 4
    assert min_bytes == x + w2 + 98304 * 8 + 16384 * 2048 * 4 == 365690880
    assert gemm_bytes + combine_bytes == 1170997248


def test_sweep_helpers():
    st = {0: (100.0, 99.0, 101.0), 1: (110.0, 108.0, 112.0), 2: (95.0, 94.0, 96.0)}
    assert bench._pick(st, [0, 1, 2]) == 2
    assert bench._pick(st, [0, 1]) == 0
    assert bench._regret(st, 0, 2) == (100.0 - 95.0) / 95.0
    assert bench._regret(st, 2, 2) == 0.0
    rng = np.random.default_rng(3)
    v = rng.normal(400.0, 10.0, size=30)
    med, lo, hi = bench.median_ci(v)
    assert med == float(np.median(v)) and lo <= med <= hi
    assert bench._agg([0.01, 0.03]) == {"mean": 0.02, "max": 0.03}


def test_traffic_entry_follows_the_kernel_source(tmp_path, monkeypatch):
    f = tmp_path / "traffic.json"
    f.write_text(json.dumps({"kernel_sha": bench.kernel_sha(), "workload": "dsv2lite",
                             "hbm_bytes_per_launch": 123}))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    assert bench.traffic_entry("dsv2lite") == 123
    assert bench.traffic_entry("qwen") is None
    f.write_text(json.dumps({"kernel_sha": "0" * 16, "workload": "dsv2lite",
                             "hbm_bytes_per_launch": 123}))
    assert bench.traffic_entry("dsv2lite") is None
