"""Benchmark of the windowed-attention hot path on one MI355X.

Workload: the Qwen2.5-7B-1M-shaped case -- a prefill of one 131072-row chunk
(positions 917504 .. 1048575) against a 1,048,576-key causal context, plus a
single-token decode at position 1,048,576 over the same cache; 28 query heads,
4 KV heads, head_dim 128, RoPE base 1e7, k = 2, seeded N(0,1) bf16 inputs.

One step = one windowed prefill call + one windowed decode call (all of the
hot path: window table, tile classification, K/V staging, QK and PV MFMAs,
boundary and causal masking, online softmax, epilogue, decode split + merge).
The same kernels at an infinite window (k = +inf) are timed too, for the
speedup the window buys, and the same prefill and decode from unrotated caches
(RoPE applied as the kernels read, App. B).  Inputs are resident in HBM before
timing starts.

Prints ONE JSON line.  Effective TFLOP/s counts only the work the method must
do: per query head 4*T + 2*d*C flops, T = retained (cell, pair) terms, C =
causal cells (softmax not counted).  Decode GB/s counts 4 bytes per retained
(token, pair) of K, all V rows (2*d bytes each), q and o.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import platform
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

METRIC = ("prefill ms + effective TFLOP/s vs full-window at 32K-128K; decode GB/s at 1M")
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
# dense v_mfma_f32_32x32x16_bf16 throughput measured on the device by `bench.py --peaks`
# (back-to-back MFMAs on one wave per SIMD; the clock drops below its 2.4 GHz peak under
# this load); a reference figure beside the published peak, which the roofline uses
MEASURED_MFMA_BF16_TFLOPS = 1965.9
# v_exp_f32 throughput measured the same way (16 independent chains per thread, every SIMD)
MEASURED_V_EXP_PER_S = 1.321e13


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--decode-iters", type=int, default=50)
    ap.add_argument("--no-full-window", action="store_true",
                    help="skip the k=inf reference timing")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-configuration table (the other workloads)")
    ap.add_argument("--no-family", action="store_true",
                    help="skip the other windows (variable-k profile, uniform k=64, rounded slice)")
    ap.add_argument("--peaks", action="store_true",
                    help="only time the device-limit microbenchmarks (libatf_peaks.so): dense "
                         "bf16 MFMA, v_exp_f32 and HBM read rates")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy (for scaling rocprof byte counters)")
    ap.add_argument("--profile-workload", default=None,
                    help="profiling driver: run only this workload's kernel (a name from "
                         "workloads.WORKLOADS) --profile-iters times and print its timings")
    ap.add_argument("--profile-iters", type=int, default=3)
    ap.add_argument("--profile-kinf", action="store_true", help="profiling driver at k = +inf")
    ap.add_argument("--profile-raw-base", action="store_true",
                    help="profiling driver: window table from the raw RoPE base (Llama shapes)")
    ap.add_argument("--profile-unrotated", action="store_true",
                    help="profiling driver: atf_prefill_unrotated / atf_decode_unrotated (RoPE "
                         "at read time) on the same buffers")
    return ap.parse_args()


def profile_driver(name, iters, kinf, raw_base=False, unrotated=False):
    """Run one workload's prefill or decode `iters` times (for rocprofv3 runs)."""
    import paper_2608_02947_amd as atf
    import workloads as W
    wl = W.WORKLOADS[name]
    dev = torch.device("cuda:0")
    inp = W.make_inputs(wl, device=dev)
    th = W.workload_theta(wl)
    win = atf.Window(wl.head_dim, wl.rope_base, math.inf if kinf else wl.k,
                     None if th is None or raw_base else th.numpy())
    stream = torch.cuda.current_stream()
    d = wl.head_dim
    if wl.kind == "prefill":
        o = torch.empty_like(inp["q"])
        lse = torch.empty((wl.batch, wl.h_q, wl.n_q), dtype=torch.float32, device=dev)
        kp = torch.empty(atf.kcache_shape(wl.batch, wl.n_k, wl.h_kv, d), dtype=torch.bfloat16,
                         device=dev)
        atf.atf_pack_kcache(inp["k"], kp)
        vp = torch.empty(atf.vcache_shape(wl.batch, wl.n_k, wl.h_kv, d), dtype=torch.bfloat16,
                         device=dev)
        atf.atf_pack_vcache(inp["v"], vp)
        pre = atf.atf_prefill_unrotated if unrotated else atf.atf_prefill
        run = lambda: pre(inp["q"], kp, vp, o, lse, wl.q_pos0, win, stream=stream)
    else:
        kp = torch.empty((wl.batch, wl.h_kv, d // 16, wl.n_k, 16), dtype=torch.bfloat16,
                         device=dev)
        atf.atf_pack_kcache(inp["k"], kp)
        vp = torch.empty(atf.vcache_shape(wl.batch, wl.n_k, wl.h_kv, d), dtype=torch.bfloat16,
                         device=dev)
        atf.atf_pack_vcache(inp["v"], vp)
        qd = inp["q"][:, 0].contiguous()
        od = torch.empty_like(qd)
        lsed = torch.empty((wl.batch, wl.h_q), dtype=torch.float32, device=dev)
        ws = torch.empty(atf.atf_decode_workspace_bytes(wl.batch, wl.h_q, wl.h_kv, wl.n_k, d),
                         dtype=torch.uint8, device=dev)
        dec = atf.atf_decode_unrotated if unrotated else atf.atf_decode
        run = lambda: dec(qd, kp, vp, od, lsed, wl.q_pos0, win, ws, stream=stream)
    ms = []
    for _ in range(iters):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        run()
        b.record(stream)
        ms.append((a, b))
    torch.cuda.synchronize()
    print(json.dumps({"profile_workload": name, "k": "inf" if kinf else wl.k,
                      "ms": [round(a.elapsed_time(b), 4) for a, b in ms]}))


def measure_peaks():
    """Dense bf16 MFMA rate (back-to-back v_mfma_f32_32x32x16_bf16 on 1, 2 and 4 waves per SIMD),
    v_exp_f32 rate (16 independent chains per thread) and HBM read rate (16-byte loads
    streaming an 8 GiB buffer, and a torch device copy), timed with HIP events on the
    current stream; the median of 5 launches after one warm-up."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2608_02947_amd", "libatf_peaks.so"))
    P, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
    lib.atf_probe_mfma_bf16.argtypes = [P, i32, i32, P]
    lib.atf_probe_exp2.argtypes = [P, i32, i32, P]
    lib.atf_probe_mfma_bf16_k8.argtypes = [P, i32, i32, P]
    lib.atf_probe_read.argtypes = [P, i64, P, i32, P]
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    blocks = 1024  # 4096 waves: four per SIMD on 256 CUs
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")

    def timed(fn):
        fn()
        evs = []
        for _ in range(5):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            rc = fn()
            b.record(stream)
            assert rc in (0, None), rc
            evs.append((a, b))
        torch.cuda.synchronize()
        return statistics.median(a.elapsed_time(b) for a, b in evs) * 1e-3

    it_m = 2000
    mfma = {}
    for waves_per_simd in (1, 2, 4):
        nb = 256 * waves_per_simd
        t = timed(lambda: lib.atf_probe_mfma_bf16(ctypes.c_void_p(out.data_ptr()), nb, it_m, sp))
        mfma[waves_per_simd] = nb * 4 * 4 * it_m * 32768 / t / 1e12
    mfma_tflops = max(mfma.values())
    # the 16-deep MFMA (4 rotary pairs per K-step) on one wave per SIMD: time per
    # instruction relative to the 32-deep one
    t8 = timed(lambda: lib.atf_probe_mfma_bf16_k8(ctypes.c_void_p(out.data_ptr()), 256, it_m, sp))
    t16 = timed(lambda: lib.atf_probe_mfma_bf16(ctypes.c_void_p(out.data_ptr()), 256, it_m, sp))
    it_e = 20000
    t = timed(lambda: lib.atf_probe_exp2(ctypes.c_void_p(out.data_ptr()), blocks, it_e, sp))
    exps = blocks * 256 * 16 * it_e / t
    nbytes = 8 << 30
    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    words = torch.empty(2048 * 256, dtype=torch.int32, device="cuda")
    t = timed(lambda: lib.atf_probe_read(ctypes.c_void_p(src.data_ptr()), nbytes,
                                         ctypes.c_void_p(words.data_ptr()), 2048, sp))
    read_gbs = nbytes / t / 1e9
    dst = torch.empty_like(src)

    def copy_once():
        dst.copy_(src)
    t = timed(copy_once)
    copy_gbs = 2 * nbytes / t / 1e9
    print(json.dumps({"peaks": {
        "mfma_bf16_dense_tflops": round(mfma_tflops, 1),
        "mfma_bf16_dense_tflops_by_waves_per_simd": {str(k): round(v, 1) for k, v in mfma.items()},
        "mfma_32x32x8_time_per_instr_vs_32x32x16": round(t8 / t16, 3),
        "frac_of_2500": round(mfma_tflops / PEAK_BF16_TFLOPS, 4),
        "v_exp_f32_per_s": float(f"{exps:.4g}"),
        "v_exp_f32_lanes_per_clk_per_simd_at_2.4GHz": round(exps / (1024 * 2.4e9), 2),
        "hbm_read_GBps": round(read_gbs, 1), "hbm_copy_read_plus_write_GBps": round(copy_gbs, 1),
        "frac_read_of_8000": round(read_gbs / PEAK_HBM_GBS, 4)}}))


def copy_calibration():
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n, "launches": 3}))


PREFILL_CONFIGS = ["qwen05b_prefill_1k", "qwen05b_prefill_8k", "qwen05b_prefill_32k",
                   "llama3b_prefill_32k", "llama3b_prefill_128k"]
DECODE_CONFIGS = ["llama3b_decode_32k", "llama3b_decode_128k"]
# configurations also timed under the variable-k profile 16 -> 2, uniform k = 64 and
# the rounded slice
FAMILY_CONFIGS = ("qwen05b_prefill_32k", "llama3b_prefill_128k", "llama3b_decode_128k")


FAMILY_TAGS = ("var16to2", "k64", "rounded8")


def timed_tables():
    """{workload: [window tags]} of every call this benchmark times; the GPU parity tests
    check each entry at the same size (tests/parity.py BENCH_TABLE_TESTS)."""
    import workloads as W
    t = {"qwen7b1m_prefill_chunk": ["default", "kinf", *FAMILY_TAGS],
         "qwen7b1m_decode": ["default", "kinf", *FAMILY_TAGS, "unrotated", "unrotated_kinf"]}
    for name in PREFILL_CONFIGS + DECODE_CONFIGS:
        tags = ["default", "kinf"]
        if W.WORKLOADS[name].llama3:
            tags.append("raw_base")
        if name in FAMILY_CONFIGS:
            tags += list(FAMILY_TAGS)
        t[name] = tags
    t["llama3b_decode_128k"] += ["ragged", "ragged_kinf", "paged", "paged_kinf"]
    return t


def sample_rows(wl, widths):
    """The stratified (b, hq, i) sample of a full-size prefill that the oracle times here
    and the GPU parity tests check: >= 256 rows over all heads (workloads.stratified_rows),
    with the prefill workgroup's position tiles floor(rows / G) (rows = 256 at d = 128;
    128 for the windowed and 256 for the window-off kernel at d = 64)."""
    import workloads as W
    G = wl.group
    tiles = (256 // G,) if wl.head_dim == 128 else (128 // G, 256 // G)
    return W.stratified_rows(wl.batch, wl.n_q, wl.h_q, wl.q_pos0, G, tiles, widths, seed=wl.seed)


def family_windows(atf, d, base, theta, k=2.0):
    """Windows timed beside the default one: two members of the window family of
    App. A, and the default window with the rounded slice of Sec. 3.3 (8-pair steps)."""
    return {"var16to2": atf.Window(d, base, 16.0, theta,
                                   k_profile=atf.atf_retention_profile(d, "arithmetic", 16.0, 2.0)),
            "k64": atf.Window(d, base, 64.0, theta),
            "rounded8": atf.Window(d, base, k, theta, slice_pairs=8)}


def _median_ms(fn, stream, warm, iters):
    for _ in range(warm):
        fn()
    evs = []
    for _ in range(iters):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        fn()
        b.record(stream)
        evs.append((a, b))
    torch.cuda.synchronize()
    return statistics.median(a.elapsed_time(b) for a, b in evs)


# configurations the fp64 oracle runs in full (every row) on the host cores, timed beside
# the GPU; the others it runs on the stratified row sample and the time is extrapolated
ORACLE_FULL = ("qwen05b_prefill_1k", "qwen05b_prefill_8k", "llama3b_decode_32k",
               "llama3b_decode_128k")
ORACLE_SAMPLED = ("qwen05b_prefill_32k", "llama3b_prefill_32k", "llama3b_prefill_128k")


def host_cores():
    avail = len(os.sched_getaffinity(0))
    return min(avail, int(os.environ.get("OMP_NUM_THREADS") or avail))


def oracle_full(wl, q, k, v, theta):
    """Wall time of the oracle over every row of workload wl (host tensors), on the host
    cores; the CPU leg of a configuration's line."""
    import oracle
    cores = host_cores()
    widths = oracle.window_widths(wl.head_dim, wl.rope_base, wl.k, theta,
                                  n_ctx=wl.q_pos0 + wl.n_q)
    t = time.perf_counter()
    oracle.attend(q, k, v, wl.q_pos0, widths, threads=cores)
    return {"seconds": round(time.perf_counter() - t, 3), "cores": cores, "kind": "oracle",
            "sample": "every (row, head), fp64, OpenMP over rows"}


def oracle_sampled(wl, q, k, v, theta):
    """The oracle on the stratified row sample of workload wl (the GPU parity sample),
    timed on the host cores; the whole workload's time extrapolated by causal cells
    (the oracle's work per row is proportional to the keys it visits)."""
    import oracle
    cores = host_cores()
    widths = oracle.window_widths(wl.head_dim, wl.rope_base, wl.k, theta,
                                  n_ctx=wl.q_pos0 + wl.n_q)
    rows = sample_rows(wl, widths)
    t = time.perf_counter()
    oracle.attend(q, k, v, wl.q_pos0, widths, rows=rows, threads=cores)
    dt = time.perf_counter() - t
    pos = wl.q_pos0 + np.arange(wl.n_q, dtype=np.float64)
    cells_all = wl.batch * wl.h_q * float(np.sum(np.minimum(pos, wl.n_k - 1) + 1))
    cells_sample = float(np.sum(np.minimum(wl.q_pos0 + rows[:, 2], wl.n_k - 1) + 1))
    return {"seconds_extrapolated": round(dt * cells_all / cells_sample, 1),
            "label": "extrapolated", "sample_seconds": round(dt, 3),
            "sample_rows": int(len(rows)), "cores": cores, "kind": "oracle",
            "sample": f"{len(rows)} stratified (row, head) pairs over all heads, fp64, OpenMP "
                      "over rows; extrapolated to every row by causal-cell count"}


def config_table(atf, W, dev, stream, with_oracle=True):
    """ms, effective TFLOP/s (prefill) or GB/s (decode), fraction of the roofline and
    speedup over the same kernel at k = +inf for each of the other configurations.
    Llama tables: the effective-frequency window (default) and, as a second row,
    the raw-base window, both on inputs rotated with the effective frequencies.
    FAMILY_CONFIGS add the variable-k profile 16 -> 2 and uniform k = 64."""
    out = {}
    for name in PREFILL_CONFIGS:
        wl = W.WORKLOADS[name]
        d = wl.head_dim
        inp = W.make_inputs(wl, device=dev)
        kp = torch.empty(atf.kcache_shape(wl.batch, wl.n_k, wl.h_kv, d), dtype=torch.bfloat16,
                         device=dev)
        atf.atf_pack_kcache(inp["k"], kp)
        vp = torch.empty(atf.vcache_shape(wl.batch, wl.n_k, wl.h_kv, d), dtype=torch.bfloat16,
                         device=dev)
        atf.atf_pack_vcache(inp["v"], vp)
        host = None
        if with_oracle and (name in ORACLE_FULL or name in ORACLE_SAMPLED):
            host = (inp["q"].cpu(), inp["k"].cpu(), inp["v"].cpu())
        del inp["k"], inp["v"]
        o = torch.empty_like(inp["q"])
        lse = torch.empty((wl.batch, wl.h_q, wl.n_q), dtype=torch.float32, device=dev)
        th = W.workload_theta(wl)
        tables = {"": None if th is None else th.numpy()}
        if th is not None:
            tables["raw_base"] = None
        iters = 5 if wl.n_q * wl.h_q >= 1 << 21 else 20
        off = atf.Window(d, wl.rope_base, math.inf)
        run = lambda w: atf.atf_prefill(inp["q"], kp, vp, o, lse, wl.q_pos0, w, stream=stream)
        t_off = _median_ms(lambda: run(off), stream, 2, iters)
        wins = {tag: atf.Window(d, wl.rope_base, wl.k, table) for tag, table in tables.items()}
        if name in FAMILY_CONFIGS:
            wins.update(family_windows(atf, d, wl.rope_base, tables[""], wl.k))
        for tag, win in wins.items():
            T, C = atf.atf_count_terms(win, wl.n_q, wl.q_pos0, wl.n_k)
            flops = wl.batch * wl.h_q * (4 * T + 2 * d * C)
            t = _median_ms(lambda: run(win), stream, 2, iters)
            tf = flops / (t * 1e-3) / 1e12
            out[name + ("_" + tag if tag else "")] = {
                "ms": round(t, 4), "effective_tflops": round(tf, 1),
                "frac_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4),
                "full_window_ms": round(t_off, 4), "speedup_vs_full_window": round(t_off / t, 4),
                "qk_pruned": round(1 - T / (C * d / 2), 4)}
        if host is not None:
            if name in ORACLE_FULL:
                cpu = oracle_full(wl, *host, tables[""])
                cpu["gpu_speedup"] = round(cpu["seconds"] * 1e3 / out[name]["ms"], 1)
            else:
                cpu = oracle_sampled(wl, *host, tables[""])
                cpu["gpu_speedup_extrapolated"] = round(
                    cpu["seconds_extrapolated"] * 1e3 / out[name]["ms"], 1)
            out[name]["oracle"] = cpu
        del inp, kp, vp, o, lse, host
        torch.cuda.empty_cache()
    for name in DECODE_CONFIGS:
        wl = W.WORKLOADS[name]
        d = wl.head_dim
        inp = W.make_inputs(wl, device=dev)
        per_set = 2 * wl.batch * wl.n_k * wl.h_kv * d * 2
        nset = max(1, -(-(1 << 30) // per_set))  # cache sets rotated: >= 1 GiB in all
        sets = []
        for i in range(nset):
            kp = torch.empty(atf.kcache_shape(wl.batch, wl.n_k, wl.h_kv, d), dtype=torch.bfloat16,
                             device=dev)
            vp = torch.empty(atf.vcache_shape(wl.batch, wl.n_k, wl.h_kv, d), dtype=torch.bfloat16,
                             device=dev)
            atf.atf_pack_kcache(inp["k"], kp)
            atf.atf_pack_vcache(inp["v"], vp)
            sets.append((kp, vp))
        host = None
        if with_oracle and name in ORACLE_FULL:
            host = (inp["q"].cpu(), inp["k"].cpu(), inp["v"].cpu())
        del inp["k"], inp["v"]
        qd = inp["q"][:, 0].contiguous()
        od = torch.empty_like(qd)
        lsed = torch.empty((wl.batch, wl.h_q), dtype=torch.float32, device=dev)
        ws = torch.empty(atf.atf_decode_workspace_bytes(wl.batch, wl.h_q, wl.h_kv, wl.n_k, d),
                         dtype=torch.uint8, device=dev)
        th = W.workload_theta(wl)
        tables = {"": None if th is None else th.numpy()}
        if th is not None:
            tables["raw_base"] = None
        off = atf.Window(d, wl.rope_base, math.inf)
        state = {"i": 0}

        def run(w):
            kp, vp = sets[state["i"] % nset]
            state["i"] += 1
            atf.atf_decode(qd, kp, vp, od, lsed, wl.q_pos0, w, ws, stream=stream)
        t_off = _median_ms(lambda: run(off), stream, 3, 30)
        R_off, Cd = atf.atf_count_terms(off, 1, wl.q_pos0, wl.n_k)
        wins = {tag: atf.Window(d, wl.rope_base, wl.k, table) for tag, table in tables.items()}
        if name in FAMILY_CONFIGS:
            wins.update(family_windows(atf, d, wl.rope_base, tables[""], wl.k))
        for tag, win in wins.items():
            R, Cd = atf.atf_count_terms(win, 1, wl.q_pos0, wl.n_k)
            nbytes = wl.batch * wl.h_kv * (4 * R + 2 * d * Cd) + wl.batch * wl.h_q * d * 4
            t = _median_ms(lambda: run(win), stream, 3, 30)
            gbs = nbytes / (t * 1e-3) / 1e9
            out[name + ("_" + tag if tag else "")] = {
                "ms": round(t, 4), "GBps": round(gbs, 1), "frac_hbm_peak": round(gbs / PEAK_HBM_GBS, 4),
                "algorithmic_bytes": nbytes, "full_window_ms": round(t_off, 4),
                "speedup_vs_full_window": round(t_off / t, 4), "cache_sets": nset}
        if host is not None:
            cpu = oracle_full(wl, *host, tables[""])
            cpu["gpu_speedup"] = round(cpu["seconds"] * 1e3 / out[name]["ms"], 1)
            out[name]["oracle"] = cpu
        del sets, qd, od, lsed, ws
        torch.cuda.empty_cache()
    out.update(ragged_decode_config(atf, W, dev, stream))
    return out


RAGGED_ROWS = [131072, 98304, 65536, 32768, 16384, 8192, 120000, 4096]


def ragged_decode_config(atf, W, dev, stream):
    """A ragged decode batch on the Llama-3.2-3B-shaped 128K caches: row b holds
    RAGGED_ROWS[b] keys and its query at that position (atf_decode_ragged, row
    arrays on the device).  Bytes are summed per row like the uniform decode."""
    wl = W.WORKLOADS["llama3b_decode_128k"]
    d, B = wl.head_dim, wl.batch
    assert len(RAGGED_ROWS) == B and max(RAGGED_ROWS) <= wl.n_k
    inp = W.make_inputs(wl, device=dev)
    kp = torch.empty(atf.kcache_shape(B, wl.n_k, wl.h_kv, d), dtype=torch.bfloat16, device=dev)
    vp = torch.empty(atf.vcache_shape(B, wl.n_k, wl.h_kv, d), dtype=torch.bfloat16, device=dev)
    atf.atf_pack_kcache(inp["k"], kp)
    atf.atf_pack_vcache(inp["v"], vp)
    qd = inp["q"][:, 0].contiguous()  # timing only: the query values do not change the work
    del inp
    od = torch.empty_like(qd)
    lsed = torch.empty((B, wl.h_q), dtype=torch.float32, device=dev)
    ws = torch.empty(atf.atf_decode_workspace_bytes(B, wl.h_q, wl.h_kv, wl.n_k, d),
                     dtype=torch.uint8, device=dev)
    rows = torch.tensor(RAGGED_ROWS, dtype=torch.int32, device=dev)
    th = W.workload_theta(wl)
    win = atf.Window(d, wl.rope_base, wl.k, None if th is None else th.numpy())
    off = atf.Window(d, wl.rope_base, math.inf)

    def nbytes(w):
        tot = 0
        for nk in RAGGED_ROWS:
            R, Cd = atf.atf_count_terms(w, 1, nk, nk)
            tot += wl.h_kv * (4 * R + 2 * d * Cd) + wl.h_q * d * 4
        return tot
    run = lambda w: atf.atf_decode_ragged(qd, kp, vp, od, lsed, rows, rows, wl.n_k, w, ws,
                                          stream=stream)
    t_off = _median_ms(lambda: run(off), stream, 3, 30)
    t = _median_ms(lambda: run(win), stream, 3, 30)
    nb = nbytes(win)
    gbs = nb / (t * 1e-3) / 1e9
    out = {"llama3b_decode_ragged_b8": {
        "ms": round(t, 4), "GBps": round(gbs, 1), "frac_hbm_peak": round(gbs / PEAK_HBM_GBS, 4),
        "algorithmic_bytes": nb, "rows": RAGGED_ROWS, "full_window_ms": round(t_off, 4),
        "speedup_vs_full_window": round(t_off / t, 4)}}
    del kp, vp
    torch.cuda.empty_cache()
    # the same rows over paged caches: 128-token pages, each row's pages in shuffled
    # order in one pool (atf_cache_append_paged fills them from the same inputs)
    pt = 128
    maxp = wl.n_k // pt
    counts = [-(-n // pt) for n in RAGGED_ROWS]
    perm = np.random.default_rng(20260099).permutation(sum(counts))
    bt = np.full((B, maxp), -1, dtype=np.int32)
    at = 0
    for b, c in enumerate(counts):
        bt[b, :c] = perm[at:at + c]
        at += c
    btd = torch.from_numpy(bt).to(dev)
    kpool = torch.empty(atf.kpages_shape(sum(counts), pt, wl.h_kv, d), dtype=torch.bfloat16, device=dev)
    vpool = torch.empty(atf.vpages_shape(sum(counts), pt, wl.h_kv, d), dtype=torch.bfloat16, device=dev)
    inp = W.make_inputs(wl, device=dev)
    for b, c in enumerate(counts):  # each row writes only its own pages
        atf.atf_cache_append_paged(inp["k"][b:b + 1, :c * pt].contiguous(),
                                   inp["v"][b:b + 1, :c * pt].contiguous(), kpool, vpool,
                                   btd[b:b + 1], 0, stream=stream)
    del inp
    runp = lambda w: atf.atf_decode_paged(qd, kpool, vpool, od, lsed, btd, rows, rows, wl.n_k, w, ws,
                                          stream=stream)
    tp_off = _median_ms(lambda: runp(off), stream, 3, 30)
    tp = _median_ms(lambda: runp(win), stream, 3, 30)
    gbsp = nb / (tp * 1e-3) / 1e9
    out["llama3b_decode_paged_b8"] = {
        "ms": round(tp, 4), "GBps": round(gbsp, 1), "frac_hbm_peak": round(gbsp / PEAK_HBM_GBS, 4),
        "algorithmic_bytes": nb, "rows": RAGGED_ROWS, "page_tokens": pt,
        "full_window_ms": round(tp_off, 4), "speedup_vs_full_window": round(tp_off / tp, 4)}
    del kpool, vpool, qd, od, lsed, ws, btd
    torch.cuda.empty_cache()
    return out


# HBM bytes moved by one launch of a kernel at the benchmark workload, from two
# rocprofv3 --pmc runs over the profiling driver (FETCH_SIZE, then WRITE_SIZE, KiB
# summed per dispatch), each scaled by what the same counter reads for a 1 GiB
# device-to-device copy.  A record holds only for the kernel sources it was
# taken on (sha256 of the files below); otherwise traffic is reported as null.
TRAFFIC_RECORDS = {
    "prefill_kernel<128, true, false>": {
        "sources": ["paper_2608_02947_amd/csrc/prefill.hip",
                    "paper_2608_02947_amd/csrc/atf_internal.hpp",
                    "paper_2608_02947_amd/csrc/rope.hpp"],
        "sha256": "d9c9dcc43bb67ee7c2dd97170a5956149d9e7ae00eb24c84b92ab89fad06588d",
        "fetch_kib": 80922943.38, "write_kib": 933525.17,
    },
    "decode_split_kernel<128, false>": {
        "sources": ["paper_2608_02947_amd/csrc/decode.hip",
                    "paper_2608_02947_amd/csrc/atf_internal.hpp",
                    "paper_2608_02947_amd/csrc/rope.hpp"],
        "sha256": "a45523c72cc5dbb7bffda3e4d025f689c4ccb579daa1f199c7bde058204a3889",
        "fetch_kib": 737788.15, "write_kib": 4071.24,
    },
}
COPY_CALIBRATION_KIB = {"fetch": 524302.02, "write": 1048576.0}  # counters for a 1 GiB copy


def recorded_traffic(kernel):
    """Bytes per launch from the record of `kernel`, or None if its sources changed."""
    import hashlib
    rec = TRAFFIC_RECORDS[kernel]
    h = hashlib.sha256()
    for f in rec["sources"]:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    if h.hexdigest() != rec["sha256"]:
        return None
    gib_kib = 1024 * 1024
    fetch = rec["fetch_kib"] * 1024 * gib_kib / COPY_CALIBRATION_KIB["fetch"]
    write = rec["write_kib"] * 1024 * gib_kib / COPY_CALIBRATION_KIB["write"]
    return {"bytes": int(round(fetch + write)), "fetch_bytes": int(round(fetch)),
            "write_bytes": int(round(write))}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path, so --gpus must "
              "be 1 (and WORLD_SIZE unset or 1).", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.peaks:
        measure_peaks()
        return
    if args.profile_workload:
        profile_driver(args.profile_workload, args.profile_iters, args.profile_kinf,
                       args.profile_raw_base, args.profile_unrotated)
        return

    import paper_2608_02947_amd as atf
    import workloads as W

    dev = torch.device("cuda:0")
    pf = W.WORKLOADS["qwen7b1m_prefill_chunk"]
    dc = W.WORKLOADS["qwen7b1m_decode"]
    d, B = pf.head_dim, pf.batch

    # ---- inputs, resident in HBM
    inp = W.make_inputs(pf, device=dev)
    q, k, v = inp["q"], inp["k"], inp["v"]
    gq = torch.Generator(device=dev)
    gq.manual_seed(dc.seed + 17)
    qd = torch.randn((dc.batch, 1, dc.h_q, d), generator=gq, device=dev).to(torch.bfloat16)
    qd = W.rotate_half(qd, torch.tensor([dc.q_pos0]), W.rotation_theta(dc))[:, 0].contiguous()
    kp = torch.empty((B, pf.h_kv, d // 16, pf.n_k, 16), dtype=torch.bfloat16, device=dev)
    atf.atf_pack_kcache(k, kp)
    vp = torch.empty(atf.vcache_shape(B, pf.n_k, pf.h_kv, d), dtype=torch.bfloat16, device=dev)
    atf.atf_pack_vcache(v, vp)
    o = torch.empty_like(q)
    lse = torch.empty((B, pf.h_q, pf.n_q), dtype=torch.float32, device=dev)
    od = torch.empty_like(qd)
    lsed = torch.empty((dc.batch, dc.h_q), dtype=torch.float32, device=dev)
    ws = torch.empty(atf.atf_decode_workspace_bytes(dc.batch, dc.h_q, dc.h_kv, dc.n_k, d),
                     dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()

    win = atf.Window(d, pf.rope_base, pf.k)
    win_off = atf.Window(d, pf.rope_base, math.inf)

    # ---- algorithmic work
    T, C = atf.atf_count_terms(win, pf.n_q, pf.q_pos0, pf.n_k)
    T_full, _ = atf.atf_count_terms(win_off, pf.n_q, pf.q_pos0, pf.n_k)
    flops_prefill = B * pf.h_q * (4 * T + 2 * d * C)
    flops_prefill_full = B * pf.h_q * (4 * T_full + 2 * d * C)
    Td, Cd = atf.atf_count_terms(win, 1, dc.q_pos0, dc.n_k)
    Td_full, _ = atf.atf_count_terms(win_off, 1, dc.q_pos0, dc.n_k)
    flops_decode = dc.batch * dc.h_q * (4 * Td + 2 * d * Cd)
    bytes_decode = dc.batch * dc.h_kv * (4 * Td + 2 * d * Cd) + dc.batch * dc.h_q * d * 4
    bytes_decode_full = dc.batch * dc.h_kv * (4 * Td_full + 2 * d * Cd) + dc.batch * dc.h_q * d * 4

    stream = torch.cuda.current_stream()

    def prefill(w):
        atf.atf_prefill(q, kp, vp, o, lse, pf.q_pos0, w, stream=stream)

    def decode(w):
        atf.atf_decode(qd, kp, vp, od, lsed, dc.q_pos0, w, ws, stream=stream)

    def ev():
        return torch.cuda.Event(enable_timing=True)

    # ---- warmup
    for _ in range(args.warmup):
        prefill(win)
        decode(win)
    torch.cuda.synchronize()

    # ---- timed steps (events on the stream the kernels run on)
    t0, t1 = ev(), ev()
    pre_ev, dec_ev = [], []
    torch.cuda.synchronize()
    t0.record(stream)
    for _ in range(args.steps):
        a, b = ev(), ev()
        a.record(stream)
        prefill(win)
        b.record(stream)
        c, e = ev(), ev()
        c.record(stream)
        decode(win)
        e.record(stream)
        pre_ev.append((a, b))
        dec_ev.append((c, e))
    t1.record(stream)
    torch.cuda.synchronize()
    ms_step = t0.elapsed_time(t1) / args.steps
    pre_ms = [a.elapsed_time(b) for a, b in pre_ev]
    # decode alone: many back-to-back calls (its 1.45 GB of reads exceed the 256 MB MALL)
    dec_ms = []
    for _ in range(args.decode_iters):
        a, b = ev(), ev()
        a.record(stream)
        decode(win)
        b.record(stream)
        dec_ms.append((a, b))
    torch.cuda.synchronize()
    dec_ms = [a.elapsed_time(b) for a, b in dec_ms]

    full = None
    if not args.no_full_window:
        prefill(win_off)
        torch.cuda.synchronize()
        pf_full = []
        for _ in range(args.steps):
            a, b = ev(), ev()
            a.record(stream)
            prefill(win_off)
            b.record(stream)
            pf_full.append((a, b))
        dfull = []
        for _ in range(args.decode_iters):
            a, b = ev(), ev()
            a.record(stream)
            decode(win_off)
            b.record(stream)
            dfull.append((a, b))
        torch.cuda.synchronize()
        full = {"prefill_ms": statistics.median(a.elapsed_time(b) for a, b in pf_full),
                "decode_ms": statistics.median(a.elapsed_time(b) for a, b in dfull)}

    pre_med = statistics.median(pre_ms)
    pre_mean = statistics.fmean(pre_ms)
    dec_med = statistics.median(dec_ms)
    step_flops = flops_prefill + flops_decode
    value = step_flops / (ms_step * 1e-3) / 1e12
    achieved = flops_prefill / (pre_mean * 1e-3) / 1e12

    prefill_info = {
        "ms_median": round(pre_med, 3), "ms_min": round(min(pre_ms), 3),
        "ms_max": round(max(pre_ms), 3),
        "effective_tflops": round(flops_prefill / (pre_med * 1e-3) / 1e12, 1),
        "frac_bf16_peak": round(flops_prefill / (pre_med * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "frac_measured_mfma_peak": round(
            flops_prefill / (pre_med * 1e-3) / 1e12 / MEASURED_MFMA_BF16_TFLOPS, 4),
        "retained_terms_per_head": T, "causal_cells_per_head": C,
        "qk_pruned": round(1 - T / (C * d / 2), 4),
        "ceiling_2_over_1_plus_s": round(flops_prefill_full / flops_prefill, 4),
        # the transcendental lower bound beside the MFMA roofline: one v_exp_f32 per causal
        # (row, key) cell of every query head, at the measured v_exp_f32 rate
        "exp_floor_ms": round(B * pf.h_q * C / MEASURED_V_EXP_PER_S * 1e3, 2),
    }
    decode_info = {
        "ms_median": round(dec_med, 4), "ms_min": round(min(dec_ms), 4),
        "GBps": round(bytes_decode / (dec_med * 1e-3) / 1e9, 1),
        "frac_hbm_peak": round(bytes_decode / (dec_med * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "algorithmic_bytes": bytes_decode, "retained_token_pairs_per_kv_head": Td,
        "byte_ceiling_full_over_window": round(bytes_decode_full / bytes_decode, 4),
    }
    if full is not None:
        prefill_info["full_window_ms"] = round(full["prefill_ms"], 3)
        prefill_info["speedup_vs_full_window"] = round(full["prefill_ms"] / pre_med, 4)
        prefill_info["full_window_dense_tflops"] = round(
            flops_prefill_full / (full["prefill_ms"] * 1e-3) / 1e12, 1)
        decode_info["full_window_ms"] = round(full["decode_ms"], 4)
        decode_info["speedup_vs_full_window"] = round(full["decode_ms"] / dec_med, 4)
        decode_info["full_window_GBps"] = round(
            bytes_decode_full / (full["decode_ms"] * 1e-3) / 1e9, 1)

    # ---- the same decode from unrotated caches (RoPE applied at read time, App. B): the
    # same bytes, plus one rotation per kept (token, pair) in the kernel; timed on the
    # same buffers (the work does not depend on the values)
    def decode_unrot(w):
        atf.atf_decode_unrotated(qd, kp, vp, od, lsed, dc.q_pos0, w, ws, stream=stream)

    tu = _median_ms(lambda: decode_unrot(win), stream, 3, args.decode_iters)
    decode_info["unrotated_cache"] = {
        "ms": round(tu, 4), "GBps": round(bytes_decode / (tu * 1e-3) / 1e9, 1),
        "frac_hbm_peak": round(bytes_decode / (tu * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "time_vs_rotated_cache": round(tu / dec_med, 4),
        "rotated_token_pairs_per_kv_head": Td, "full_window_rotations_per_kv_head": Td_full}
    if full is not None:
        tu_off = _median_ms(lambda: decode_unrot(win_off), stream, 3, args.decode_iters)
        decode_info["unrotated_cache"]["full_window_ms"] = round(tu_off, 4)
        decode_info["unrotated_cache"]["speedup_vs_full_window"] = round(tu_off / tu, 4)

    # ---- the same prefill from unrotated caches: the same matrix work, plus the rotation
    # of each query row once and of each kept (key, pair-chunk) once per workgroup that
    # loads it; timed on the same buffers (the work does not depend on the values)
    def prefill_unrot(w):
        atf.atf_prefill_unrotated(q, kp, vp, o, lse, pf.q_pos0, w, stream=stream)

    tpu = _median_ms(lambda: prefill_unrot(win), stream, 1, args.steps)
    prefill_info["unrotated_cache"] = {
        "ms": round(tpu, 3), "effective_tflops": round(flops_prefill / (tpu * 1e-3) / 1e12, 1),
        "frac_bf16_peak": round(flops_prefill / (tpu * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "time_vs_rotated_cache": round(tpu / pre_med, 4)}
    if full is not None:
        tpu_off = _median_ms(lambda: prefill_unrot(win_off), stream, 1, args.steps)
        prefill_info["unrotated_cache"]["full_window_ms"] = round(tpu_off, 3)
        prefill_info["unrotated_cache"]["speedup_vs_full_window"] = round(tpu_off / tpu, 4)
    # the write-time alternative: the whole K cache rotated once into a copy
    # (atf_rotate_kcache), which the pre-rotated prefill then reads
    k_rot = torch.empty_like(kp)
    trk = _median_ms(lambda: atf.atf_rotate_kcache(kp, k_rot, win, stream=stream), stream, 1,
                     args.steps)
    rot_bytes = 2 * kp.numel() * 2
    prefill_info["unrotated_cache"]["rotate_kcache_ms"] = round(trk, 4)
    prefill_info["unrotated_cache"]["rotate_kcache_GBps"] = round(rot_bytes / (trk * 1e-3) / 1e9, 1)
    prefill_info["unrotated_cache"]["rotate_then_prefill_ms"] = round(trk + pre_med, 3)
    del k_rot

    # ---- other windows on the same inputs: the variable-k profile 16 -> 2 and uniform
    # k = 64 (App. A, tab:absbench), and the rounded slice (Sec. 3.3, tab:c2e2e)
    family = None
    if not args.no_family:
        family = {}
        for tag, fw in family_windows(atf, d, pf.rope_base, None, pf.k).items():
            Tf, Cf = atf.atf_count_terms(fw, pf.n_q, pf.q_pos0, pf.n_k)
            fl = B * pf.h_q * (4 * Tf + 2 * d * Cf)
            tp = _median_ms(lambda: prefill(fw), stream, 1, args.steps)
            Rf, Cdf = atf.atf_count_terms(fw, 1, dc.q_pos0, dc.n_k)
            nb = dc.batch * dc.h_kv * (4 * Rf + 2 * d * Cdf) + dc.batch * dc.h_q * d * 4
            td = _median_ms(lambda: decode(fw), stream, 3, args.decode_iters)
            family[tag] = {
                "prefill_ms": round(tp, 3), "prefill_qk_pruned": round(1 - Tf / (Cf * d / 2), 4),
                "prefill_effective_tflops": round(fl / (tp * 1e-3) / 1e12, 1),
                "prefill_speedup_vs_full_window":
                    None if full is None else round(full["prefill_ms"] / tp, 4),
                "decode_ms": round(td, 4), "decode_GBps": round(nb / (td * 1e-3) / 1e9, 1),
                "decode_speedup_vs_full_window":
                    None if full is None else round(full["decode_ms"] / td, 4)}

    tr = recorded_traffic("prefill_kernel<128, true, false>")
    roofline = {"kernel": "prefill_kernel<128, true, false>", "bound": "mfma",
                "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": None if tr is None else tr["bytes"],
                "flops_per_launch": flops_prefill, "avg_launch_ms": round(pre_mean, 3)}
    if tr is not None:
        roofline["traffic_fetch_bytes"] = tr["fetch_bytes"]
        roofline["traffic_write_bytes"] = tr["write_bytes"]
    trd = recorded_traffic("decode_split_kernel<128, false>")
    decode_info["hbm_traffic_bytes"] = None if trd is None else trd["bytes"]

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(inp, pf, qd, dc, dec_med)
    del inp, q, k, v, kp, vp, o, lse
    torch.cuda.empty_cache()
    configs = None if args.no_configs else config_table(atf, W, dev, stream,
                                                        not args.no_cpu_baseline)

    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1), RoPE-rotated; stands in for LongBench-v2 documents)",
        "config": {"workload": "Qwen2.5-7B-1M-shaped: prefill of a 131072-row chunk at "
                               "positions 917504..1048575 over 1048576 keys + decode at 1048576",
                   "batch": B, "n_q": pf.n_q, "q_pos0": pf.q_pos0, "n_k": pf.n_k,
                   "h_q": pf.h_q, "h_kv": pf.h_kv, "head_dim": d, "rope_base": pf.rope_base,
                   "k": pf.k, "parallelism": "single GPU"},
        "prefill": prefill_info, "decode": decode_info, "window_variants": family,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "configs": configs,
    }
    print(json.dumps(out))


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.machine()


def cpu_baseline(inp, pf, qd, dc, decode_ms):
    """The fp64 oracle on the host cores: the stratified row sample of the same prefill
    chunk (the rows the GPU parity test checks; the headline leg, in the metric's unit),
    and the whole decode at 1M (every head)."""
    import oracle
    cores = host_cores()
    qc, kc, vc = inp["q"].cpu(), inp["k"].cpu(), inp["v"].cpu()
    widths = oracle.window_widths(pf.head_dim, pf.rope_base, pf.k, n_ctx=pf.n_k)
    rows = sample_rows(pf, widths)
    t = time.perf_counter()
    _, _, terms = oracle.attend(qc, kc, vc, pf.q_pos0, widths, rows=rows, threads=cores)
    dt = time.perf_counter() - t
    causal = np.minimum(pf.q_pos0 + rows[:, 2], pf.n_k - 1) + 1
    flops = float(np.sum(4.0 * terms.astype(np.float64) + 2.0 * pf.head_dim * causal))
    widths_d = oracle.window_widths(dc.head_dim, dc.rope_base, dc.k, n_ctx=dc.q_pos0 + 1)
    td = time.perf_counter()
    oracle.attend(qd.cpu()[:, None], kc, vc, dc.q_pos0, widths_d, threads=cores)
    td = time.perf_counter() - td
    return {"value": float(f"{flops / dt / 1e12:.6g}"), "unit": "TFLOP/s", "cores": cores,
            "kind": "oracle", "seconds": round(dt, 2), "cpu": cpu_model(),
            "sample": f"{len(rows)} stratified (query row, head) pairs of the 131072-row chunk "
                      "over all heads (the GPU parity sample), each over its ~1M causal keys, "
                      "fp64, OpenMP over rows",
            "decode_1m_full": {"seconds": round(td, 3), "cores": cores,
                               "sample": "every head of the decode at 1,048,576, fp64",
                               "gpu_speedup": round(td * 1e3 / decode_ms, 1)}}


if __name__ == "__main__":
    main()
