"""bench.py's contract on a host without a GPU: the single-GPU guard and the traffic record."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_record_is_its_counters_scaled():
    for wl, t in bench.TRAFFIC.items():
        kib = t["fetch_kib_per_launch"] * t["fetch_scale"] + t["write_kib_per_launch"] * t["write_scale"]
        assert abs(kib * 1024 - t["bytes_per_launch"]) <= 1e-4 * t["bytes_per_launch"], wl
        assert len(t["source_sha256"]) == 64


def test_traffic_is_reported_only_for_the_measured_source(monkeypatch):
    monkeypatch.setitem(bench.TRAFFIC, "sweep", dict(bench.TRAFFIC["sweep"], source_sha256="0" * 64))
    assert bench.measured_traffic("sweep") is None
    assert bench.measured_traffic("no-such-workload") is None
