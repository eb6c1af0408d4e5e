"""Helpers of the GPU parity tests: run the HIP path through the C ABI, run the
oracle on the same seeded inputs, and compare to the stated tolerances.

Tolerances (bf16 inputs, fp32 accumulation, bf16 output): O max-abs <= 1e-2 and
mean-abs <= 1e-3, LSE max-abs <= 1e-3.  Term counts are compared bit-exactly.
"""
from __future__ import annotations

import math
import sys

import numpy as np
import torch

import oracle
import workloads as W

O_MAX_ABS = 1e-2
O_MEAN_ABS = 1e-3
LSE_MAX_ABS = 1e-3


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


def compare_rounding_bound(o_gpu, lse_gpu, o_ref, lse_ref, o_absv_ref, label=""):
    """Element-wise check against the error the arithmetic implies when scores are
    large and the softmax is peaked (where a fixed 1e-2 on O does not hold).  Each
    weight p_ij carries the bf16 rounding of P in the PV product (relative 2^-9) and
    the error of its score, accumulated in fp32 at magnitudes up to ~10^3 (up to
    ~2e-3 relative: the order the LSE check below bounds); O is rounded to bf16
    (relative 2^-9).  o_absv_ref is the oracle's output for |V|, i.e.
    sum_j p_ij |v_j| / l_i, and with a factor 2 over 2^-9 + 2e-3 the bound is
        |dO| <= 2^-7 * o_absv_ref + 2^-9 * |O| + 1e-4,   |dLSE| <= 1e-3.
    A missing or wrong rescale of O or of the normaliser gives errors of the order
    of |O| itself."""
    og = np.asarray(o_gpu, dtype=np.float64)
    lg = np.asarray(lse_gpu, dtype=np.float64)
    assert og.shape == o_ref.shape and lg.shape == lse_ref.shape, label
    assert np.all(np.isfinite(og)) and np.all(np.isfinite(lg)), f"{label}: non-finite output"
    bound = 2.0 ** -7 * o_absv_ref + 2.0 ** -9 * np.abs(o_ref) + 1e-4
    ratio = float(np.max(np.abs(og - o_ref) / bound))
    ml = float(np.max(np.abs(lg - lse_ref)))
    assert ratio <= 1.0, f"{label}: O error {ratio:.3f} x its rounding bound"
    assert ml <= LSE_MAX_ABS, f"{label}: LSE max-abs {ml}"
    return ratio, ml


def to_f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def sample_rows(batch, n_q, h_q, n_rows, seed, tile=128):
    """Stratified (b, hq, i) sample: first and last rows, rows at tile edges, random."""
    rng = np.random.default_rng(seed)
    picks = set()
    for i in list(range(min(8, n_q))) + list(range(max(0, n_q - 8), n_q)):
        picks.add(i)
    for t in rng.integers(0, max(1, n_q // tile), size=8):
        for off in (-1, 0, 31, 32, tile - 1):
            i = int(t) * tile + off
            if 0 <= i < n_q:
                picks.add(i)
    while len(picks) < n_rows:
        picks.add(int(rng.integers(0, n_q)))
    rows = []
    for i in sorted(picks)[:max(n_rows, len(picks))]:
        rows.append((int(rng.integers(0, batch)), int(rng.integers(0, h_q)), i))
    return np.array(rows, dtype=np.int64)


def workload_window(wl: W.Workload, k=None, family=None, slice_pairs=0):
    th = W.workload_theta(wl)
    if family is not None:
        return family_windows_for(wl.head_dim, wl.rope_base, None if th is None else th.numpy(),
                                  family)
    return windows_for(wl.head_dim, wl.rope_base, wl.k if k is None else k,
                       None if th is None else th.numpy(),
                       n_ctx=max(wl.n_k, wl.q_pos0 + wl.n_q), slice_pairs=slice_pairs)
