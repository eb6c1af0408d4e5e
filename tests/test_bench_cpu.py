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
    cal = bench.COPY_CALIBRATION_KIB
    fake = {"k": {"sources": [src], "sha256": h, "fetch_kib": cal["fetch"] * 3,
                  "write_kib": cal["write"]}}
    monkeypatch.setattr(bench, "TRAFFIC_RECORDS", fake)
    t = bench.recorded_traffic("k")
    assert t["fetch_bytes"] == 3 << 30 and t["write_bytes"] == 1 << 30
    assert t["bytes"] == 4 << 30
    fake["k"]["sha256"] = "0" * 64
    assert bench.recorded_traffic("k") is None


def test_every_timed_table_has_a_full_size_parity_test():
    """Each (workload, window table) bench.py times is checked by a GPU parity test at
    the same size, and the named test exists."""
    import re
    from parity import BENCH_TABLE_TESTS
    missing = [(n, t) for n, tags in bench.timed_tables().items() for t in tags
               if (n, t) not in BENCH_TABLE_TESTS]
    assert not missing, missing
    for where in set(BENCH_TABLE_TESTS.values()):
        path, name = where.split("::")
        src = open(os.path.join(ROOT, "tests", path)).read()
        assert re.search(rf"^def {name}\(", src, re.M), where


def test_cpu_baseline_rows_are_the_parity_sample():
    """bench.py's oracle sample of each full-size prefill is the GPU parity test's
    sample: >= 256 (row, head) pairs over every head."""
    import numpy as np
    import oracle
    import workloads as W
    from parity import bench_rows, table_windows
    for name in ("qwen7b1m_prefill_chunk", "qwen05b_prefill_32k", "llama3b_prefill_32k",
                 "llama3b_prefill_128k"):
        wl = W.WORKLOADS[name]
        _, widths, _ = table_windows(wl, "default")
        th = W.workload_theta(wl)
        w_bench = oracle.window_widths(wl.head_dim, wl.rope_base, wl.k,
                                       None if th is None else th.numpy(),
                                       n_ctx=wl.q_pos0 + wl.n_q)
        a, b = bench.sample_rows(wl, w_bench), bench_rows(wl, widths)
        assert np.array_equal(a, b), name
        assert len(a) >= 256 and set(a[:, 1].tolist()) == set(range(wl.h_q))
