"""Helpers of the GPU parity tests: run the HIP path through the C ABI, run the
oracle on the same seeded inputs, and compare to the stated tolerances.

Tolerances (bf16 inputs, fp32 accumulation, bf16 output): O max-abs <= 1e-2 and
mean-abs <= 1e-3, LSE max-abs <= 1e-3.  Term counts are compared bit-exactly.
"""
from __future__ import annotations

import math
import sys
import zlib

import numpy as np
import torch

import oracle
import workloads as W

O_MAX_ABS = 1e-2
O_MEAN_ABS = 1e-3
LSE_MAX_ABS = 1e-3


def case_seed(case) -> int:
    """A seed for a parametrised test case that is the same in every process (Python
    salts the hash of a str per process, so hash() of a case holding a name is not)."""
    return zlib.crc32(repr(case).encode()) % 10000


def note(msg: str):
    """Name the GPU step about to run (visible even if the process dies)."""
    print(f"[gpu-step] {msg}", flush=True)
    sys.stdout.flush()


def windows_for(head_dim, rope_base, k, theta, n_ctx, slice_pairs=0):
    """(GPU window, oracle widths) built independently on each side.  slice_pairs > 1
    selects the rounded slice on the GPU side; the oracle applies its own rounding
    rule when called with atom=slice_pairs."""
    import paper_2608_02947_amd as atf
    th = None if theta is None else np.asarray(theta, dtype=np.float64)
    return (atf.Window(head_dim, rope_base, k, th, slice_pairs=slice_pairs),
            oracle.window_widths(head_dim, rope_base, k, th, n_ctx=n_ctx))


# members of the window family of App. A (eq:family) used by the GPU tests:
# name -> (profile (kind, k_hi, k_lo), gamma, a, beta, cap)
FAMILIES = {
    "var16to2": (("arithmetic", 16.0, 2.0), 1.0, 0.0, 0.0, math.inf),
    "geo16to2": (("geometric", 16.0, 2.0), 1.0, 0.0, 0.0, math.inf),
    "k64": (("constant", 64.0, 0.0), 1.0, 0.0, 0.0, math.inf),
    "k2_floor40_cap180": (("constant", 2.0, 0.0), 1.0, 0.0, 40.0, 180.0),
    "gamma0.8": (("constant", 2.0, 0.0), 0.8, 0.0, 0.0, math.inf),
    "gamma1.25": (("constant", 2.0, 0.0), 1.25, 0.0, 0.0, math.inf),
    "sliding100": (("constant", 0.0, 0.0), 1.0, 0.0, 100.0, 100.0),
    "linear256": (("constant", 0.0, 0.0), 1.0, 256.0, 0.0, math.inf),
}


def family_windows_for(head_dim, rope_base, theta, family):
    """(GPU window, oracle widths) of a window-family member, built independently
    on each side (the library's profile and table, the oracle's profile and widths)."""
    import paper_2608_02947_amd as atf
    (kind, hi, lo), gamma, a, beta, cap = FAMILIES[family]
    th = None if theta is None else np.asarray(theta, dtype=np.float64)
    win = atf.Window(head_dim, rope_base, hi, th,
                     k_profile=atf.atf_retention_profile(head_dim, kind, hi, lo),
                     gamma=gamma, a=a, beta=beta, cap=cap)
    widths = oracle.family_widths(head_dim, rope_base, oracle.retention_profile(head_dim, kind, hi, lo),
                                  gamma=gamma, a=a, beta=beta, cap=cap, theta=th)
    return win, widths


def gpu_prefill(q, k, v, q_pos0, win, scale=0.0, kp=None, n_k=None, vp=None):
    """q [B, n_q, h_q, d]; k, v [B, C, h_kv, d], packed into the caches by the library
    first unless kp / vp are given; keys 0 .. n_k - 1 (default C) are used."""
    import paper_2608_02947_amd as atf
    B, n_q, h_q, d = q.shape
    if kp is None:
        kp = pack_kcache(k)
    if vp is None:
        vp = pack_vcache(v)
    o = torch.empty_like(q)
    lse = torch.empty((B, h_q, n_q), dtype=torch.float32, device=q.device)
    atf.atf_prefill(q, kp, vp, o, lse, q_pos0, win, scale, n_k=n_k)
    torch.cuda.synchronize()
    return o, lse


def pack_kcache(k_bshd):
    import paper_2608_02947_amd as atf
    B, n_k, h_kv, d = k_bshd.shape
    kp = torch.empty((B, h_kv, d // 16, n_k, 16), dtype=torch.bfloat16, device=k_bshd.device)
    atf.atf_pack_kcache(k_bshd, kp)
    return kp


def pack_vcache(v_bshd):
    import paper_2608_02947_amd as atf
    B, n_k, h_kv, d = v_bshd.shape
    vp = torch.empty(atf.vcache_shape(B, n_k, h_kv, d), dtype=torch.bfloat16, device=v_bshd.device)
    atf.atf_pack_vcache(v_bshd, vp)
    return vp


def gpu_decode(q, k_bshd, v_bshd, q_pos, win, scale=0.0, kp=None, vp=None, n_k=None):
    """q [B, h_q, d]; caches given in BSHD [B, C, h_kv, d] are packed by the library
    first; keys 0 .. n_k - 1 (default C) are used."""
    import paper_2608_02947_amd as atf
    B, h_q, d = q.shape
    if kp is None:
        kp = pack_kcache(k_bshd)
    _, h_kv, _, cap, _ = kp.shape
    if vp is None:
        vp = pack_vcache(v_bshd)
    if n_k is None:
        n_k = cap
    ws = torch.empty(atf.atf_decode_workspace_bytes(B, h_q, h_kv, n_k, d), dtype=torch.uint8,
                     device=q.device)
    o = torch.empty_like(q)
    lse = torch.empty((B, h_q), dtype=torch.float32, device=q.device)
    atf.atf_decode(q, kp, vp, o, lse, q_pos, win, ws, scale, n_k=n_k)
    torch.cuda.synchronize()
    return o, lse


def compare(o_gpu, lse_gpu, o_ref, lse_ref, label=""):
    """Element-wise comparison; returns (max_abs_o, mean_abs_o, max_abs_lse)."""
    og = np.asarray(o_gpu, dtype=np.float64)
    lg = np.asarray(lse_gpu, dtype=np.float64)
    assert og.shape == o_ref.shape and lg.shape == lse_ref.shape, label
    assert np.all(np.isfinite(og)) and np.all(np.isfinite(lg)), f"{label}: non-finite output"
    eo = np.abs(og - o_ref)
    el = np.abs(lg - lse_ref)
    mx, mean, ml = float(eo.max()), float(eo.mean()), float(el.max())
    assert mx <= O_MAX_ABS, f"{label}: O max-abs {mx}"
    assert mean <= O_MEAN_ABS, f"{label}: O mean-abs {mean}"
    assert ml <= LSE_MAX_ABS, f"{label}: LSE max-abs {ml}"
    return mx, mean, ml


# Unit roundoffs and instruction accuracies of the error budget below.
U32 = 2.0 ** -24      # fp32, round to nearest even (24 significant bits)
U16 = 2.0 ** -8       # bf16, round to nearest even (8 significant bits)
EXP_ULP = 2.0 ** -23  # v_exp_f32 (the hardware 2^x): accurate to 1 ulp of fp32
LN2 = math.log(2.0)
LOG2E = 1.0 / LN2


def error_budget(s, sabs, v, o_ref, scale, head_dim, tile_keys, extra_states=0):
    """Worst-case bound on |O_kernel - O| per output element of one (batch, head),
    derived from the arithmetic the kernels perform (no fitted factor).

    s [n, n_k]: exact scaled scores (oracle, fp64; -inf where a key is not valid);
    sabs [n, n_k]: the same sum over kept pairs of |q_r k_r| + |q_{r+h} k_{r+h}|,
    unscaled; v [n_k, d]; o_ref [n, d] the oracle's output.  tile_keys: keys per
    running-max update (64 prefill, 32 decode); extra_states: partial states merged
    after the key loop (decode: 4 waves + the splits + 32 merge lanes; prefill 0).

    Error sources, per valid key j of row i (w_ij the exact softmax weights):
      score:  fp32 MFMA accumulation of the bf16 x bf16 products (exact in fp32);
              each kept product passes through at most d additions in the d/16
              K-steps plus d/2 masked partial-pair additions, so
              |dx| <= (3d/2) u32 sabs_ij; the weight exp(scale x) moves by
              scale (3d/2) u32 sabs_ij relative.  The scale itself is an fp32
              constant: u32 |s_ij| more.
      exp:    every exp2 that multiplies the weight (its own, plus one per rescale
              of the running max or merge of partial states: R_i = 1 +
              ceil(n_i / tile_keys) + 2 [decode merges]) is accurate to 1 ulp and
              takes an argument rounded once in fp32, |arg| <= T_i = (max_j s_ij -
              min_j s_ij) log2 e + 8 (the lazy rescale admits probabilities up to
              2^8), plus one fp32 multiply: R_i (2^-23 + ln2 u32 T_i + u32).
      These multiply the weight by (1 + e'_ij), |e'_ij| <= eps_ij, in the output's
      numerator and in the normaliser alike, so with ebar = sum_j w eps:
        d_w  = (sum_j w eps |v_j| + ebar A + 2 ebar |O|) / (1 - ebar),  A = sum_j w |v_j|
      bf16 P (numerator only):            d_p = U16 (A + E1) / (1 - ebar)
      fp32 accumulation of the numerator, depth n_i + R_i + 3 + extra_states:
                                          d_n = g_n (1 + U16) (A + E1) / (1 - ebar)
      fp32 normaliser sum, rescale and reciprocal (depth n_i + R_i + 4 +
      extra_states):                      d_l = g_l / (1 - g_l) * (|O| + d_w + d_p + d_n)
      bf16 rounding of the output:        U16 (|O| + d_w + d_p + d_n + d_l)
      probabilities below 2^-126 flushed to zero: n_i 2^-126 max|v| (the normaliser
      is at least 1: the row's largest probability is at least 2^0).
    The bound is the sum of these terms."""
    s = np.asarray(s, dtype=np.float64)
    valid = np.isfinite(s)
    n_i = valid.sum(axis=1).astype(np.float64)
    M = np.max(np.where(valid, s, -np.inf), axis=1)
    mn = np.min(np.where(valid, s, np.inf), axis=1)
    w = np.where(valid, np.exp(np.where(valid, s, 0.0) - M[:, None]), 0.0)
    w /= w.sum(axis=1, keepdims=True)
    R = 1.0 + np.ceil(n_i / tile_keys) + (2.0 if extra_states else 0.0)
    T = (M - mn) * LOG2E + 8.0
    g_s = 1.5 * head_dim * U32
    eps = (scale * g_s * np.where(valid, sabs, 0.0) + U32 * np.abs(np.where(valid, s, 0.0))
           + (R * (EXP_ULP + LN2 * U32 * T + U32))[:, None])
    eps = np.where(valid, eps, 0.0)
    av = np.abs(np.asarray(v, dtype=np.float64))
    ao = np.abs(np.asarray(o_ref, dtype=np.float64))
    A = w @ av
    E1 = (w * eps) @ av
    ebar = (w * eps).sum(axis=1)[:, None]
    d_w = (E1 + ebar * A + 2.0 * ebar * ao) / (1.0 - ebar)
    d_p = U16 * (A + E1) / (1.0 - ebar)
    g_n = ((n_i + R + 3 + extra_states) * U32)[:, None]
    d_n = g_n * (1.0 + U16) * (A + E1) / (1.0 - ebar)
    g_l = ((n_i + R + 4 + extra_states) * U32)[:, None]
    pre = ao + d_w + d_p + d_n
    d_l = g_l / (1.0 - g_l) * pre
    flush = (n_i * 2.0 ** -126)[:, None] * av.max()
    return d_w + d_p + d_n + d_l + U16 * (pre + d_l) + flush


def prefill_budget(q, k, v, q_pos0, widths, scale, o_ref):
    """error_budget for every row of a prefill (oracle scores per (batch, head));
    returns [B, n_q, h_q, d] like o_ref."""
    B, n_q, h_q, d = q.shape
    h_kv = k.shape[2]
    G = h_q // h_kv
    qa, ka = q.abs(), k.abs()
    vv = v.double().numpy()
    out = np.empty(o_ref.shape, dtype=np.float64)
    for b in range(B):
        for h in range(h_q):
            s = oracle.scores(q, k, q_pos0, widths, b=b, hq=h, scale=scale)
            sabs = oracle.scores(qa, ka, q_pos0, widths, b=b, hq=h, scale=1.0)
            out[b, :, h] = error_budget(s, sabs, vv[b, :, h // G], o_ref[b, :, h], scale, d,
                                        tile_keys=64)
    return out


def decode_budget(q, k, v, q_pos, widths, scale, o_ref):
    """error_budget for every (batch, head) row of a decode (q [B, 1, h_q, d]);
    partial states merged after the key loop: 4 waves, at most ceil(n_k / 128)
    splits (the split plan's cap), 32 merge lanes.  Returns [B, h_q, d]."""
    B, _, h_q, d = q.shape
    n_k, h_kv = k.shape[1], k.shape[2]
    G = h_q // h_kv
    qa, ka = q.abs(), k.abs()
    vv = v.double().numpy()
    extra = 4 + (n_k + 127) // 128 + 32
    out = np.empty(o_ref.shape, dtype=np.float64)
    for b in range(B):
        for h in range(h_q):
            s = oracle.scores(q, k, q_pos, widths, b=b, hq=h, scale=scale)
            sabs = oracle.scores(qa, ka, q_pos, widths, b=b, hq=h, scale=1.0)
            out[b, h] = error_budget(s, sabs, vv[b, :, h // G], o_ref[b, h][None], scale, d,
                                     tile_keys=32, extra_states=extra)[0]
    return out


def compare_rounding_bound(o_gpu, lse_gpu, o_ref, lse_ref, bound, label=""):
    """Element-wise |O_kernel - O| <= bound (the derived error budget) and the LSE
    within the fixed 1e-3.  Returns (largest error / bound ratio, LSE max-abs)."""
    og = np.asarray(o_gpu, dtype=np.float64)
    lg = np.asarray(lse_gpu, dtype=np.float64)
    assert og.shape == o_ref.shape == bound.shape and lg.shape == lse_ref.shape, label
    assert np.all(np.isfinite(og)) and np.all(np.isfinite(lg)), f"{label}: non-finite output"
    ratio = float(np.max(np.abs(og - o_ref) / bound))
    ml = float(np.max(np.abs(lg - lse_ref)))
    print(f"[bound] {label}: largest error / derived bound = {ratio:.3f}, LSE max-abs {ml:.2e}",
          flush=True)
    assert ratio <= 1.0, f"{label}: O error {ratio:.3f} x its derived bound"
    assert ml <= LSE_MAX_ABS, f"{label}: LSE max-abs {ml}"
    return ratio, ml


def to_f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def workload_window(wl: W.Workload, k=None, family=None, slice_pairs=0):
    th = W.workload_theta(wl)
    if family is not None:
        return family_windows_for(wl.head_dim, wl.rope_base, None if th is None else th.numpy(),
                                  family)
    return windows_for(wl.head_dim, wl.rope_base, wl.k if k is None else k,
                       None if th is None else th.numpy(),
                       n_ctx=max(wl.n_k, wl.q_pos0 + wl.n_q), slice_pairs=slice_pairs)


def table_windows(wl: W.Workload, tag: str):
    """(GPU window, oracle widths, oracle atom) of a window table the benchmark times on
    workload wl: "default" (k of the workload; the llama3-effective table for Llama
    shapes), "kinf" (window off), "raw_base" (the table of the raw RoPE base, Llama
    shapes), "rounded8" (the rounded slice of Sec. 3.3), or a window-family member."""
    if tag == "default":
        return (*workload_window(wl), 0)
    if tag == "kinf":
        return (*workload_window(wl, k=math.inf), 0)
    if tag == "raw_base":
        return (*windows_for(wl.head_dim, wl.rope_base, wl.k, None,
                             n_ctx=max(wl.n_k, wl.q_pos0 + wl.n_q)), 0)
    if tag == "rounded8":
        return (*workload_window(wl, slice_pairs=8), 8)
    return (*workload_window(wl, family=tag), 0)


def kernel_position_tiles(head_dim: int, group: int):
    """Positions per prefill workgroup, floor(rows / G): rows = 256 at d = 128; at
    d = 64 the windowed kernel packs 128 rows and the window-off kernel 256."""
    return (256 // group,) if head_dim == 128 else (128 // group, 256 // group)


def bench_rows(wl: W.Workload, widths):
    """The stratified (b, hq, i) sample of a full-size prefill checked against the
    oracle (and timed as the benchmark's CPU baseline on the headline workload)."""
    return W.stratified_rows(wl.batch, wl.n_q, wl.h_q, wl.q_pos0, wl.group,
                             kernel_position_tiles(wl.head_dim, wl.group), widths, seed=wl.seed)


# Every (workload, window table) bench.py times, and the GPU test that checks it at the
# size and in the launch configuration it is timed in.
_T = "test_gpu_bench_tables.py::"
BENCH_TABLE_TESTS = {
    **{("qwen05b_prefill_1k", t): "test_gpu_prefill.py::test_prefill_qwen_1k_workload_all_rows"
       for t in ("default", "kinf")},
    **{(n, t): _T + "test_prefill_bench_tables_sampled_rows"
       for n, ts in {"qwen05b_prefill_8k": ("default", "kinf"),
                     "qwen05b_prefill_32k": ("default", "kinf", "var16to2", "k64", "rounded8"),
                     "llama3b_prefill_32k": ("default", "raw_base", "kinf"),
                     "llama3b_prefill_128k": ("default", "raw_base", "kinf", "var16to2", "k64",
                                              "rounded8"),
                     "qwen7b1m_prefill_chunk": ("default", "kinf", "var16to2", "k64", "rounded8"),
                     }.items() for t in ts},
    **{(n, t): _T + "test_decode_bench_tables_all_rows"
       for n, ts in {"llama3b_decode_32k": ("default", "raw_base", "kinf"),
                     "llama3b_decode_128k": ("default", "raw_base", "kinf", "var16to2", "k64",
                                             "rounded8"),
                     "qwen7b1m_decode": ("default", "kinf", "var16to2", "k64", "rounded8"),
                     }.items() for t in ts},
    **{("qwen7b1m_decode", t): "test_gpu_rope.py::test_decode_unrotated_qwen7b1m_every_head"
       for t in ("unrotated", "unrotated_kinf")},
    **{("llama3b_decode_128k", t): "test_gpu_decode.py::test_decode_ragged_paged_llama_128k_bench_layout"
       for t in ("ragged", "ragged_kinf", "paged", "paged_kinf")},
}


def bench_tables_of(kind: str):
    """{workload: [tags]} of the entries checked by test_gpu_bench_tables.py."""
    out = {}
    for (n, t), where in BENCH_TABLE_TESTS.items():
        if where.startswith(_T) and W.WORKLOADS[n].kind == kind:
            out.setdefault(n, []).append(t)
    return out
