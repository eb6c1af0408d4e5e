"""Host logic of bench.py (no GPU): the one-GPU refusal and the traffic records."""
import hashlib
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout.strip() == ""


def test_recorded_traffic_scaling_and_source_check(monkeypatch):
    """Bytes = FETCH_SIZE x (1 GiB / copy fetch KiB) + WRITE_SIZE x (1 GiB / copy write
    KiB); a record whose sources no longer hash to its sha256 gives None."""
    src = "paper_2608_02947_amd/csrc/atf_internal.hpp"
    h = hashlib.sha256(open(os.path.join(ROOT, src), "rb").read()).hexdigest()
    fake = {"k": {"sources": [src], "sha256": h, "fetch_kib": 524299.5 * 3, "write_kib": 1048576.0}}
    monkeypatch.setattr(bench, "TRAFFIC_RECORDS", fake)
    t = bench.recorded_traffic("k")
    assert t["fetch_bytes"] == 3 << 30 and t["write_bytes"] == 1 << 30
    assert t["bytes"] == 4 << 30
    fake["k"]["sha256"] = "0" * 64
    assert bench.recorded_traffic("k") is None
