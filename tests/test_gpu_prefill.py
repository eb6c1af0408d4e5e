"""GPU parity of atf_prefill against the fp64 oracle on the same seeded inputs.

Small shapes: every output element; properties that hold at any size (chunked
prefill equal to single-shot, caches longer than the keys used).  The full-size
workloads, in the launch configuration bench.py times, are checked in
test_gpu_bench_tables.py.
"""
import math

import numpy as np
import pytest
import torch

from conftest import gpu_available
import oracle
import workloads as W
from parity import (case_seed, compare_rounding_bound, compare, prefill_budget, family_windows_for, gpu_decode, gpu_prefill, note, pack_kcache,
                    pack_vcache, to_f64, windows_for, workload_window)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]

DEV = "cuda"


def _small_inputs(B, n_q, n_k, q0, h_q, h_kv, d, base, seed, theta=None, scale_k=1.0):
    g = torch.Generator(device="cpu").manual_seed(seed)
    q = torch.randn((B, n_q, h_q, d), generator=g).to(torch.bfloat16)
    k = (torch.randn((B, n_k, h_kv, d), generator=g) * scale_k).to(torch.bfloat16)
    v = torch.randn((B, n_k, h_kv, d), generator=g).to(torch.bfloat16)
    th = torch.as_tensor(theta, dtype=torch.float64) if theta is not None else W.rope_theta(d, base)
    q = W.rotate_half(q, torch.arange(q0, q0 + n_q), th)
    k = W.rotate_half(k, torch.arange(0, n_k), th)
    return q, k, v


def _full_parity(q, k, v, q0, win, widths, label, scale=None, atom=0):
    note(f"prefill {label} shape q={tuple(q.shape)} k={tuple(k.shape)} q0={q0}")
    o, lse = gpu_prefill(q.to(DEV), k.to(DEV), v.to(DEV), q0, win,
                         0.0 if scale is None else scale)
    o_ref, lse_ref, _ = oracle.attend(q, k, v, q0, widths, scale=scale, atom=atom)
    return compare(to_f64(o), to_f64(lse), o_ref, lse_ref, label)


CASES = [
    # B, n_q, n_k, q0, h_q, h_kv, d, base, k
    (1, 128, 128, 0, 1, 1, 64, 1e4, 2.0),
    (1, 300, 300, 0, 6, 2, 128, 5e5, 2.0),
    (2, 45, 45, 0, 4, 4, 64, 1e6, 2.0),           # partial wave, MHA
    (1, 77, 267, 190, 7, 1, 64, 1e6, 2.0),        # chunk at the end of a longer context
    (1, 200, 150, 0, 8, 1, 128, 1e4, 2.0),        # keys end before the last query
    (1, 1, 1, 0, 2, 1, 128, 1e4, 2.0),            # one row, one key
    (1, 257, 257, 0, 3, 3, 128, 100.0, 2.0),      # saturated: every window ends early
    (1, 190, 190, 0, 2, 1, 64, 1e4, 0.05),        # tiny k: empty score sums
    (1, 256, 256, 0, 2, 1, 128, 1e4, math.inf),   # window off
    (1, 333, 500, 167, 16, 2, 64, 1e4, 1.0),      # G = 8, ragged tail
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(str(x) for x in c))
def test_prefill_small_all_rows(case):
    B, n_q, n_k, q0, h_q, h_kv, d, base, kwin = case
    q, k, v = _small_inputs(B, n_q, n_k, q0, h_q, h_kv, d, base, seed=hash(case) % 10000)
    win, widths = windows_for(d, base, kwin, None, n_ctx=max(n_k, q0 + n_q))
    _full_parity(q, k, v, q0, win, widths, f"small{case}")


def test_prefill_llama3_effective_table_all_rows():
    wl = W.WORKLOADS["llama3b_prefill_32k"]
    inp = W.make_inputs(wl, n_k=700, n_q=700, q_pos0=0)
    win, widths = workload_window(wl)
    _full_parity(inp["q"], inp["k"], inp["v"], 0, win, widths, "llama3 700")


def test_prefill_nonmonotone_table_and_position_free_pairs():
    """Per-chunk min/max classification does not assume a monotone table."""
    d = 128
    rng = np.random.default_rng(5)
    theta = rng.uniform(0.005, 3.0, d // 2)
    theta[[3, 17, 40]] = 0.0  # position-free pairs: never pruned
    q, k, v = _small_inputs(1, 260, 260, 0, 4, 2, d, 0.0, seed=9, theta=theta)
    win, widths = windows_for(d, 1e4, 3.0, theta, n_ctx=260)
    _full_parity(q, k, v, 0, win, widths, "nonmonotone")


def test_prefill_custom_scale():
    q, k, v = _small_inputs(1, 160, 160, 0, 2, 1, 64, 1e4, seed=3)
    win, widths = windows_for(64, 1e4, 2.0, None, n_ctx=160)
    _full_parity(q, k, v, 0, win, widths, "scale0.3", scale=0.3)


def test_prefill_qwen_1k_workload_all_rows():
    """The 1K Qwen2.5-0.5B-shaped workload, every row of every head."""
    wl = W.WORKLOADS["qwen05b_prefill_1k"]
    inp = W.make_inputs(wl)
    win, widths = workload_window(wl)
    _full_parity(inp["q"], inp["k"], inp["v"], 0, win, widths, wl.name)
    # k = inf equals the oracle of ordinary causal attention
    win_inf, widths_inf = workload_window(wl, k=math.inf)
    _full_parity(inp["q"], inp["k"], inp["v"], 0, win_inf, widths_inf, wl.name + " k=inf")


FAMILY_CASES = [
    # family, B, n_q, n_k, q0, h_q, h_kv, d, base
    ("var16to2", 2, 260, 260, 0, 4, 4, 64, 1e6),
    ("geo16to2", 1, 300, 300, 0, 6, 2, 128, 5e5),
    ("k64", 1, 333, 500, 167, 16, 2, 64, 1e4),
    ("k2_floor40_cap180", 1, 333, 500, 167, 16, 2, 64, 1e4),   # floor and ceiling bind
    ("gamma0.8", 1, 300, 300, 0, 6, 2, 128, 5e5),
    ("gamma1.25", 1, 200, 450, 250, 8, 1, 128, 1e4),
    ("sliding100", 1, 300, 300, 0, 4, 2, 128, 1e4),            # empty sums past 100
    ("sliding100", 2, 190, 190, 0, 2, 1, 64, 1e4),
    ("linear256", 1, 400, 400, 0, 2, 1, 128, 1e4),
]


@pytest.mark.parametrize("case", FAMILY_CASES, ids=lambda c: "x".join(str(x) for x in c))
def test_prefill_window_family_all_rows(case):
    """Members of the window family of App. A (eq:family): every output element."""
    fam, B, n_q, n_k, q0, h_q, h_kv, d, base = case
    q, k, v = _small_inputs(B, n_q, n_k, q0, h_q, h_kv, d, base, seed=case_seed(case))
    win, widths = family_windows_for(d, base, None, fam)
    _full_parity(q, k, v, q0, win, widths, f"family{case}")


def test_prefill_variable_k_workloads_all_rows():
    """The variable-k profile 16 -> 2 on the 1K Qwen2.5-0.5B-shaped workload and on
    700 rows of the Llama-3.2-3B shape (llama3-effective frequencies)."""
    wl = W.WORKLOADS["qwen05b_prefill_1k"]
    inp = W.make_inputs(wl)
    win, widths = workload_window(wl, family="var16to2")
    _full_parity(inp["q"], inp["k"], inp["v"], 0, win, widths, wl.name + " var16to2")
    wl = W.WORKLOADS["llama3b_prefill_32k"]
    inp = W.make_inputs(wl, n_k=700, n_q=700, q_pos0=0)
    win, widths = workload_window(wl, family="var16to2")
    _full_parity(inp["q"], inp["k"], inp["v"], 0, win, widths, "llama3 700 var16to2")


ROUNDED_CASES = [
    # B, n_q, n_k, q0, h_q, h_kv, d, base, k
    (1, 300, 300, 0, 6, 2, 128, 5e5, 2.0),
    (2, 260, 260, 0, 4, 4, 64, 1e6, 2.0),
    (1, 333, 500, 167, 16, 2, 64, 1e4, 1.0),      # G = 8, ragged tail
    (1, 257, 257, 0, 3, 3, 128, 100.0, 2.0),      # saturated: empty sums
]


@pytest.mark.parametrize("case", ROUNDED_CASES, ids=lambda c: "x".join(str(x) for x in c))
def test_prefill_rounded_slice_all_rows(case):
    """The rounded slice of Sec. 3.3 (8-pair K-steps) against the oracle's rounding rule."""
    B, n_q, n_k, q0, h_q, h_kv, d, base, kwin = case
    q, k, v = _small_inputs(B, n_q, n_k, q0, h_q, h_kv, d, base, seed=hash(case) % 10000 + 1)
    win, widths = windows_for(d, base, kwin, None, n_ctx=max(n_k, q0 + n_q), slice_pairs=8)
    _full_parity(q, k, v, q0, win, widths, f"rounded{case}", atom=8)


def test_prefill_rounded_slice_workloads():
    """Rounded slice: all rows of the 1K Qwen2.5-0.5B shape and of 700 Llama-3.2-3B rows
    (effective table); the full-size workloads are in test_gpu_bench_tables.py."""
    wl = W.WORKLOADS["qwen05b_prefill_1k"]
    inp = W.make_inputs(wl)
    win, widths = workload_window(wl, slice_pairs=8)
    _full_parity(inp["q"], inp["k"], inp["v"], 0, win, widths, wl.name + " rounded", atom=8)
    wl = W.WORKLOADS["llama3b_prefill_32k"]
    inp = W.make_inputs(wl, n_k=700, n_q=700, q_pos0=0)
    win, widths = workload_window(wl, slice_pairs=8)
    _full_parity(inp["q"], inp["k"], inp["v"], 0, win, widths, "llama3 700 rounded", atom=8)


def test_prefill_chunked_equals_single_shot():
    """Prefill in chunks against one pair of caches allocated for the whole sequence
    (q_pos0 offsets, n_k = keys written so far) is bit-identical to one call over
    all rows when every chunk boundary is a multiple of the workgroup's position
    tile, floor(rows / G) positions (rows = 128 at d = 64, 256 at d = 128: 18 for
    the d = 64, G = 7 workload used here)."""
    wl = W.WORKLOADS["qwen05b_prefill_8k"]
    tile = (128 if wl.head_dim == 64 else 256) // wl.group
    chunk = tile * 28
    n = 4 * chunk
    inp = W.make_inputs(wl, device=DEV, n_q=n, n_k=n, q_pos0=0)
    win, _ = workload_window(wl)
    note("prefill chunked vs single")
    kp = pack_kcache(inp["k"])
    vp = pack_vcache(inp["v"])
    o, lse = gpu_prefill(inp["q"], inp["k"], inp["v"], 0, win, kp=kp, vp=vp)
    for s in range(0, n, chunk):
        qc = inp["q"][:, s:s + chunk].contiguous()
        oc, lc = gpu_prefill(qc, inp["k"], inp["v"], s, win, kp=kp, vp=vp, n_k=s + chunk)
        assert torch.equal(oc, o[:, s:s + chunk])
        assert torch.equal(lc, lse[:, :, s:s + chunk])


def test_prefill_chunks_appended_to_shared_caches_then_decode():
    """The pipeline of one request: caches allocated for the whole context; each
    chunk's keys and values are appended (atf_cache_append) and its rows attend the
    keys written so far; the result is bit-identical to one call over the packed
    context; then decode steps append their token and read the same caches.
    Chunk boundaries are multiples of the position tile (floor(256 / G) at d = 128)."""
    import paper_2608_02947_amd as atf
    wl = W.WORKLOADS["llama3b_prefill_32k"]
    tile = 256 // wl.group
    chunk = tile * 9
    n = 3 * chunk + tile   # a shorter last chunk
    cap = n + 40           # room for decode steps, not a multiple of 16
    inp = W.make_inputs(wl, device=DEV, n_q=n + 2, n_k=n + 2, q_pos0=0)
    win, widths = workload_window(wl)
    d, h_kv = wl.head_dim, wl.h_kv
    note("prefill appended chunks")
    o_ref, lse_ref = gpu_prefill(inp["q"][:, :n].contiguous(), inp["k"][:, :n].contiguous(),
                                 inp["v"][:, :n].contiguous(), 0, win)
    kc = torch.full(atf.kcache_shape(wl.batch, cap, h_kv, d), float("nan"), dtype=torch.bfloat16,
                    device=DEV)
    vc = torch.full(atf.vcache_shape(wl.batch, cap, h_kv, d), float("nan"), dtype=torch.bfloat16,
                    device=DEV)
    for s in range(0, n, chunk):
        e = min(s + chunk, n)
        atf.atf_cache_append(inp["k"][:, s:e].contiguous(), inp["v"][:, s:e].contiguous(), kc, vc, s)
        oc, lc = gpu_prefill(inp["q"][:, s:e].contiguous(), None, None, s, win, kp=kc, vp=vc, n_k=e)
        assert torch.equal(oc, o_ref[:, s:e])
        assert torch.equal(lc, lse_ref[:, :, s:e])
    # two decode steps at positions n and n + 1 over the same caches
    for pos in (n, n + 1):
        atf.atf_cache_append(inp["k"][:, pos:pos + 1].contiguous(),
                             inp["v"][:, pos:pos + 1].contiguous(), kc, vc, pos)
        qd = inp["q"][:, pos].contiguous()
        od, ld = gpu_decode(qd, None, None, pos, win, kp=kc, vp=vc, n_k=pos + 1)
        o1, l1, _ = oracle.attend(inp["q"][:, pos:pos + 1].cpu(), inp["k"][:, :pos + 1].cpu(),
                                  inp["v"][:, :pos + 1].cpu(), pos, widths)
        compare(to_f64(od), to_f64(ld), o1[:, 0], l1[:, :, 0], f"decode at {pos}")


def test_prefill_cache_capacity_and_uninitialised_tail():
    """Caches allocated for more tokens than written: keys past n_k (filled with NaN
    here) are never used."""
    B, n_q, n_k, cap, h_q, h_kv, d = 2, 150, 333, 400, 6, 2, 128
    q, k, v = _small_inputs(B, n_q, n_k, n_k - n_q, h_q, h_kv, d, 1e4, seed=21)
    win, widths = windows_for(d, 1e4, 2.0, None, n_ctx=n_k)
    kc = torch.full((B, cap, h_kv, d), float("nan"), dtype=torch.bfloat16)
    vc = torch.full((B, cap, h_kv, d), float("nan"), dtype=torch.bfloat16)
    kc[:, :n_k] = k
    vc[:, :n_k] = v
    note("prefill cache capacity")
    o, lse = gpu_prefill(q.to(DEV), kc.to(DEV), vc.to(DEV), n_k - n_q, win, n_k=n_k)
    o_ref, lse_ref, _ = oracle.attend(q, k, v, n_k - n_q, widths)
    compare(to_f64(o), to_f64(lse), o_ref, lse_ref, "capacity")


def _large_score_inputs(n_q, n_k, q0, h_q, h_kv, d, base, pattern, seed):
    """Scores of order 100s (scaled queries, keys whose magnitude grows along the
    sequence or is log-normal), so the running max of the online softmax is raised
    many times along each row and O and the normaliser are rescaled."""
    g = torch.Generator(device="cpu").manual_seed(seed)
    q = torch.randn((1, n_q, h_q, d), generator=g) * 3.0
    k = torch.randn((1, n_k, h_kv, d), generator=g)
    if pattern == "rising":
        k = k * torch.linspace(0.5, 6.0, n_k)[None, :, None, None]
    else:
        k = k * torch.exp(torch.randn((n_k,), generator=g))[None, :, None, None]
    v = torch.randn((1, n_k, h_kv, d), generator=g)
    th = W.rope_theta(d, base)
    q = W.rotate_half(q.to(torch.bfloat16), torch.arange(q0, q0 + n_q), th)
    k = W.rotate_half(k.to(torch.bfloat16), torch.arange(0, n_k), th)
    return q, k, v.to(torch.bfloat16)


@pytest.mark.parametrize("pattern", ["rising", "lognormal"])
@pytest.mark.parametrize("d,h_q,h_kv", [(128, 6, 2), (64, 7, 1)])
def test_prefill_large_scores_rescale(pattern, d, h_q, h_kv):
    """Every row against the oracle within the error budget derived from the kernel's
    arithmetic (parity.error_budget), windowed and with the window off."""
    q, k, v = _large_score_inputs(700, 700, 0, h_q, h_kv, d, 1e4, pattern, seed=77 + d)
    for kwin in (2.0, math.inf):
        win, widths = windows_for(d, 1e4, kwin, None, n_ctx=700)
        note(f"prefill large scores {pattern} d={d} k={kwin}")
        o, lse = gpu_prefill(q.to(DEV), k.to(DEV), v.to(DEV), 0, win, 1.0)
        o_ref, lse_ref, _ = oracle.attend(q, k, v, 0, widths, scale=1.0)
        bound = prefill_budget(q, k, v, 0, widths, 1.0, o_ref)
        compare_rounding_bound(to_f64(o), to_f64(lse), o_ref, lse_ref, bound,
                               f"large scores {pattern} d={d} k={kwin}")
