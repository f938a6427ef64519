"""Host-side parts of bench.py (CPU): the one-GPU rule, the traffic record's
guard on the kernel sources, and the products it times."""

import os
import subprocess
import sys

from conftest import ROOT

sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""  # no JSON line


def test_traffic_is_reported_only_for_the_measured_sources(monkeypatch):
    stored = dict(bench.TRAFFIC)
    monkeypatch.setattr(bench, "TRAFFIC", dict(stored, sources_sha256=bench.sources_sha256()))
    for product in bench.PRODUCTS:
        assert bench.traffic_bytes(product) == stored["bytes"][product]
    monkeypatch.setattr(bench, "TRAFFIC", dict(stored, sources_sha256="0" * 64))
    assert all(bench.traffic_bytes(p) is None for p in bench.PRODUCTS)
    monkeypatch.setattr(bench, "TRAFFIC", None)
    assert bench.traffic_bytes("dW") is None


def test_timed_products_are_phases_of_the_call():
    assert set(bench.PRODUCTS) <= set(bench.PHASES)
    assert set(bench.PRODUCTS) == {"logits", "dW", "dhidden"}
    assert bench.PEAK_BF16 == 2.5e15 and bench.PEAK_HBM == 8.0e12
    assert bench.spread([3.0, 1.0, 2.0]) == {"min": 1.0, "median": 2.0, "max": 3.0}
