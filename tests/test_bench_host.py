"""Host-side parts of bench.py that need no GPU: the one-GPU guard, the
measured-traffic table and its tie to the kernel sources."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_table_entries_are_complete():
    with open(bench.TRAFFIC_FILE) as f:
        t = json.load(f)
    assert 1.9 < t["read_factor"] < 2.1 and 0.9 < t["write_factor"] < 1.1
    assert t["workloads"], "no measured workloads"
    for key, e in t["workloads"].items():
        assert e["fetch_kib"] > 0 and e["write_kib"] > 0 and e["dispatches"] > 0, key
        assert len(e["kernel_source_sha"]) == 16, key
        assert os.path.exists(os.path.join(ROOT, e["profile"])), (key, e["profile"])


def test_traffic_is_reported_only_for_the_measured_sources(monkeypatch):
    with open(bench.TRAFFIC_FILE) as f:
        t = json.load(f)
    key, e = next((k, v) for k, v in t["workloads"].items() if k.startswith("f16_full:"))
    expected = e["fetch_kib"] * 1024.0 * t["read_factor"] + e["write_kib"] * 1024.0 * t["write_factor"]
    monkeypatch.setattr(bench, "kernel_source_hash", lambda inst: e["kernel_source_sha"])
    assert bench.measured_traffic(key, "op") == pytest.approx(expected)
    monkeypatch.setattr(bench, "kernel_source_hash", lambda inst: "0" * 16)
    assert bench.measured_traffic(key, "op") is None
    assert bench.measured_traffic("no-such-workload", "op") is None


def test_source_hash_covers_each_kernel_family():
    hashes = {inst: bench.kernel_source_hash(inst) for inst in bench.KERNEL_SOURCES}
    assert all(len(h) == 16 for h in hashes.values())
    # each family hashes a different kernel source
    assert len(set(hashes.values())) == len(hashes)
