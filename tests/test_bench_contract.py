"""Host-side parts of bench.py's output contract (no GPU): the one-GPU
guard, the traffic lookup that the kernels' hash gates, and the shape of
the CPU baseline record."""
import json
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_is_reported_only_for_the_kernels_it_was_measured_on(tmp_path, monkeypatch):
    path = tmp_path / "traffic.json"
    entry = {"fetch_bytes": 1000, "write_bytes": 234}
    monkeypatch.setattr(bench, "TRAFFIC", str(path))
    path.write_text(json.dumps({"kernels_sha256": bench.kernels_sha256(),
                                "kernels": {"k_encode": entry}}))
    assert bench.measured_traffic("k_encode") == 1234
    assert bench.measured_traffic("k_decode") is None
    path.write_text(json.dumps({"kernels_sha256": "0" * 64, "kernels": {"k_encode": entry}}))
    assert bench.measured_traffic("k_encode") is None
    path.write_text("not json")
    assert bench.measured_traffic("k_encode") is None
    monkeypatch.setattr(bench, "TRAFFIC", str(tmp_path / "missing.json"))
    assert bench.measured_traffic("k_encode") is None


def test_cpu_baseline_record():
    g = np.random.default_rng(7)
    host = g.integers(0, 256, 96 * 65536, dtype=np.uint8)
    out = bench.cpu_baseline(host, target_s=0.05)
    assert out["kind"] == "oracle" and out["unit"] == "GB/s"
    assert out["value"] > 0 and out["cores"] >= 1
    assert "64 KiB chunks" in out["sample"]
