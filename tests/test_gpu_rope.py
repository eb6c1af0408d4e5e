"""GPU parity of prefill and decode from UNROTATED caches (RoPE applied at read time,
App. B) through the C ABI: atf_prefill_unrotated, atf_decode_unrotated and its ragged
and paged forms against the oracle, which rotates the same bf16 queries and keys in fp64
(oracle.rope_rotate, pinned in test_oracle_rope.py), stores them in bf16 as a
pre-rotated cache would, and attends them in fp64."""
import math

import numpy as np
import pytest
import torch

from conftest import gpu_available
import oracle
import workloads as W
from parity import (LSE_MAX_ABS, O_MAX_ABS, O_MEAN_ABS, bench_rows, compare, family_windows_for,
                    gpu_prefill, note, pack_kcache, pack_vcache, table_windows, to_f64,
                    windows_for)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X (gfx950) GPU")]

DEV = "cuda"


def _inputs(B, n_k, h_q, h_kv, d, seed):
    """Unrotated bf16 query, keys and values."""
    g = torch.Generator(device="cpu").manual_seed(seed)
    q = torch.randn((B, 1, h_q, d), generator=g).to(torch.bfloat16)
    k = torch.randn((B, n_k, h_kv, d), generator=g).to(torch.bfloat16)
    v = torch.randn((B, n_k, h_kv, d), generator=g).to(torch.bfloat16)
    return q, k, v


def _oracle(q, k, v, q_pos, theta, widths):
    """Rotate in fp64 (query at q_pos, key j at j), store the rotated vectors in bf16
    (round to nearest even) as a pre-rotated cache would hold them, then windowed
    attention: the result an unrotated cache read with RoPE at read time must give."""
    qr = torch.from_numpy(oracle.rope_rotate(q, [q_pos], theta)).to(torch.bfloat16)
    kr = torch.from_numpy(oracle.rope_rotate(k, np.arange(k.shape[1]), theta)).to(torch.bfloat16)
    o, lse, _ = oracle.attend(qr, kr, v, q_pos, widths)
    return o[:, 0], lse[:, :, 0]


def _gpu(q, k, v, q_pos, win, rope_inv_freq=None):
    import paper_2608_02947_amd as atf
    qd = q[:, 0].contiguous().to(DEV)
    kp, vp = pack_kcache(k.to(DEV)), pack_vcache(v.to(DEV))
    B, h_q, d = qd.shape
    h_kv, cap = kp.shape[1], kp.shape[3]
    ws = torch.empty(atf.atf_decode_workspace_bytes(B, h_q, h_kv, cap, d), dtype=torch.uint8,
                     device=DEV)
    o = torch.empty_like(qd)
    lse = torch.empty((B, h_q), dtype=torch.float32, device=DEV)
    atf.atf_decode_unrotated(qd, kp, vp, o, lse, q_pos, win, ws, rope_inv_freq=rope_inv_freq)
    torch.cuda.synchronize()
    return o, lse


CASES = [
    # B, n_k, q_pos, h_q, h_kv, d, base, k
    (2, 300, 300, 6, 2, 128, 5e5, 2.0),
    (3, 1000, 1000, 7, 1, 64, 1e6, 2.0),
    (1, 2049, 5000, 8, 1, 128, 1e4, 2.0),            # query beyond the cache end
    (2, 777, 777, 12, 1, 128, 1e4, 2.0),             # G = 12
    (1, 999, 999, 3, 1, 128, 1e4, math.inf),         # window off: every pair rotated
    (1, 700, (1 << 30) + 5, 4, 1, 128, 1e4, math.inf),  # query at position 2^30 + 5
    (1, 262144, 262144, 4, 1, 64, 1e6, 2.0),         # keys at positions up to 262143
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(str(x) for x in c))
def test_decode_unrotated(case):
    B, n_k, q_pos, h_q, h_kv, d, base, kwin = case
    note(f"decode unrotated {case}")
    q, k, v = _inputs(B, n_k, h_q, h_kv, d, seed=hash(case) % 10000)
    win, widths = windows_for(d, base, kwin, None, n_ctx=q_pos + 1)
    o, lse = _gpu(q, k, v, q_pos, win)
    o_ref, lse_ref = _oracle(q, k, v, q_pos, W.rope_theta(d, base).numpy(), widths)
    compare(to_f64(o), to_f64(lse), o_ref, lse_ref, f"unrotated {case}")


def test_decode_unrotated_llama_frequencies():
    """Llama-3.2-3B shape with the llama3-effective frequencies: rotation from the
    window's own table, and from an explicit table under a raw-base window."""
    wl = W.WORKLOADS["llama3b_decode_32k"]
    d, n_k = wl.head_dim, 4096
    th = W.workload_theta(wl).numpy()
    q, k, v = _inputs(2, n_k, wl.h_q, wl.h_kv, d, seed=wl.seed)
    note("decode unrotated llama effective table")
    win, widths = windows_for(d, wl.rope_base, wl.k, th, n_ctx=n_k + 1)
    o, lse = _gpu(q, k, v, n_k, win)
    o_ref, lse_ref = _oracle(q, k, v, n_k, th, widths)
    compare(to_f64(o), to_f64(lse), o_ref, lse_ref, "llama effective")
    note("decode unrotated llama raw-base window, effective rotation")
    win, widths = windows_for(d, wl.rope_base, wl.k, None, n_ctx=n_k + 1)
    o, lse = _gpu(q, k, v, n_k, win, rope_inv_freq=th)
    o_ref, lse_ref = _oracle(q, k, v, n_k, th, widths)
    compare(to_f64(o), to_f64(lse), o_ref, lse_ref, "llama raw window")


def test_decode_unrotated_deterministic():
    q, k, v = _inputs(1, 3000, 8, 2, 128, seed=41)
    win, _ = windows_for(128, 1e4, 2.0, None, n_ctx=3001)
    note("decode unrotated determinism")
    o1, l1 = _gpu(q, k, v, 3000, win)
    o2, l2 = _gpu(q, k, v, 3000, win)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_decode_paged_unrotated():
    """Pages written with atf_cache_append_paged from unrotated keys, shared pages
    included; row b's token t is rotated to position t."""
    import paper_2608_02947_amd as atf
    n_ks, q_poss = [1500, 1, 700, 0], [1500, 1, 900, 0]
    B, h_q, h_kv, d, pt, base = 4, 6, 2, 128, 64, 1e4
    pages = -(-max(n_ks) // pt)
    cap = pages * pt
    q, k, v = _inputs(B, cap, h_q, h_kv, d, seed=77)
    k[1:, :2 * pt] = k[:1, :2 * pt]   # rows share the first two pages of row 0
    v[1:, :2 * pt] = v[:1, :2 * pt]
    num_pages = B * pages + 1
    rng = np.random.default_rng(5)
    perm = rng.permutation(num_pages)
    bt = np.zeros((B, pages), dtype=np.int32)
    nxt = 0
    for b in range(B):
        for j in range(pages):
            if b > 0 and j < 2:
                bt[b, j] = bt[0, j]
            else:
                bt[b, j] = perm[nxt]
                nxt += 1
    kpool = torch.full(atf.kpages_shape(num_pages, pt, h_kv, d), float("nan"), dtype=torch.bfloat16,
                       device=DEV)
    vpool = torch.full(atf.vpages_shape(num_pages, pt, h_kv, d), float("nan"), dtype=torch.bfloat16,
                       device=DEV)
    btd = torch.from_numpy(bt).to(DEV)
    note("decode paged unrotated")
    atf.atf_cache_append_paged(k.to(DEV), v.to(DEV), kpool, vpool, btd, 0)
    win, _ = windows_for(d, base, 2.0, None, n_ctx=max(q_poss) + 1)
    qd = q[:, 0].contiguous().to(DEV)
    ws = torch.empty(atf.atf_decode_workspace_bytes(B, h_q, h_kv, max(n_ks), d), dtype=torch.uint8,
                     device=DEV)
    o = torch.empty_like(qd)
    lse = torch.empty((B, h_q), dtype=torch.float32, device=DEV)
    atf.atf_decode_paged_unrotated(qd, kpool, vpool, o, lse, btd,
                                   torch.tensor(n_ks, dtype=torch.int32, device=DEV),
                                   torch.tensor(q_poss, dtype=torch.int32, device=DEV), max(n_ks),
                                   win, ws)
    torch.cuda.synchronize()
    o, lse = to_f64(o), to_f64(lse)
    th = W.rope_theta(d, base).numpy()
    for b, (nk, qp) in enumerate(zip(n_ks, q_poss)):
        if nk == 0:
            assert np.all(o[b] == 0.0) and np.all(lse[b] == -np.inf)
            continue
        _, widths = windows_for(d, base, 2.0, None, n_ctx=qp + 1)
        o_ref, lse_ref = _oracle(q[b:b + 1], k[b:b + 1, :nk], v[b:b + 1, :nk], qp, th, widths)
        compare(o[b:b + 1], lse[b:b + 1], o_ref, lse_ref, f"paged unrotated row {b}")


@pytest.mark.parametrize("kwin", [2.0, math.inf], ids=["default", "kinf"])
def test_decode_unrotated_qwen7b1m_every_head(kwin):
    """The benchmark's 1M decode shape (28 query heads / 4 KV heads, d = 128, base 1e7,
    query at 1,048,576 over keys 0 .. 1,048,575) from unrotated caches, at k = 2 and with
    the window off (both timed): every head against the oracle's fp64 rotation and
    attention."""
    wl = W.WORKLOADS["qwen7b1m_decode"]
    d = wl.head_dim
    note(f"decode unrotated qwen7b1m, every head, k={kwin}")
    q, k, v = _inputs(wl.batch, wl.n_k, wl.h_q, wl.h_kv, d, seed=wl.seed + 101)
    win, widths = windows_for(d, wl.rope_base, kwin, None, n_ctx=wl.q_pos0 + 1)
    o, lse = _gpu(q, k, v, wl.q_pos0, win)
    o_ref, lse_ref = _oracle(q, k, v, wl.q_pos0, W.rope_theta(d, wl.rope_base).numpy(), widths)
    compare(to_f64(o), to_f64(lse), o_ref, lse_ref, "unrotated qwen7b1m")


def test_decode_ragged_unrotated():
    """Ragged batch from unrotated contiguous caches: row b's key t at position t, its
    query at q_pos_rows[b] (inside, at and past its cache end; an empty row)."""
    import paper_2608_02947_amd as atf
    n_ks, q_poss = [3000, 1, 1200, 0, 2500], [3000, 1, 1900, 0, 2000]
    B, h_q, h_kv, d, base, cap = 5, 8, 2, 128, 1e4, 3000
    q, k, v = _inputs(B, cap, h_q, h_kv, d, seed=91)
    note("decode ragged unrotated")
    win, _ = windows_for(d, base, 2.0, None, n_ctx=max(q_poss) + 1)
    qd = q[:, 0].contiguous().to(DEV)
    kp, vp = pack_kcache(k.to(DEV)), pack_vcache(v.to(DEV))
    ws = torch.empty(atf.atf_decode_workspace_bytes(B, h_q, h_kv, cap, d), dtype=torch.uint8,
                     device=DEV)
    o = torch.empty_like(qd)
    lse = torch.empty((B, h_q), dtype=torch.float32, device=DEV)
    atf.atf_decode_ragged_unrotated(qd, kp, vp, o, lse,
                                    torch.tensor(n_ks, dtype=torch.int32, device=DEV),
                                    torch.tensor(q_poss, dtype=torch.int32, device=DEV), cap, win, ws)
    torch.cuda.synchronize()
    o, lse = to_f64(o), to_f64(lse)
    th = W.rope_theta(d, base).numpy()
    for b, (nk, qp) in enumerate(zip(n_ks, q_poss)):
        if nk == 0:
            assert np.all(o[b] == 0.0) and np.all(lse[b] == -np.inf)
            continue
        n_used = min(nk, qp + 1)
        _, widths = windows_for(d, base, 2.0, None, n_ctx=qp + 1)
        o_ref, lse_ref = _oracle(q[b:b + 1], k[b:b + 1, :n_used], v[b:b + 1, :n_used], qp, th, widths)
        compare(o[b:b + 1], lse[b:b + 1], o_ref, lse_ref, f"ragged unrotated row {b}")


EXACT_CASES = [
    # B, n_k, q_pos, h_q, h_kv, d, base, k: rows of thousands of keys
    (2, 4096, 4096, 8, 2, 128, 1e4, 2.0),
    (1, 20000, 20000, 7, 1, 128, 1e7, 2.0),
    (1, 4096, 4096, 4, 1, 128, 1e4, math.inf),
    (1, 8192, 8192, 14, 2, 64, 1e6, 2.0),
]


@pytest.mark.parametrize("case", EXACT_CASES, ids=lambda c: "x".join(str(x) for x in c))
def test_decode_unrotated_against_exact_rotation(case):
    """Against attention over the EXACTLY rotated vectors (fp64 rotation, not rounded to
    bf16): the read-time rotation rounds each rotated element to bf16, as a pre-rotated
    cache would, and on rows of thousands of keys those roundings average out below the
    fixed tolerances (O max-abs 1e-2, mean-abs 1e-3, LSE 1e-3)."""
    B, n_k, q_pos, h_q, h_kv, d, base, kwin = case
    note(f"decode unrotated vs exact rotation {case}")
    q, k, v = _inputs(B, n_k, h_q, h_kv, d, seed=(hash(case) + 7) % 10000)
    win, widths = windows_for(d, base, kwin, None, n_ctx=q_pos + 1)
    o, lse = _gpu(q, k, v, q_pos, win)
    theta = W.rope_theta(d, base).numpy()
    qr = torch.from_numpy(oracle.rope_rotate(q, [q_pos], theta))
    kr = torch.from_numpy(oracle.rope_rotate(k, np.arange(n_k), theta))
    o_ref, lse_ref, _ = oracle.attend(qr, kr, v.to(torch.float64), q_pos, widths)
    compare(to_f64(o), to_f64(lse), o_ref[:, 0], lse_ref[:, :, 0], f"exact rotation {case}")


# ---- prefill from unrotated caches ----

def _prefill_inputs(B, n_q, n_k, h_q, h_kv, d, seed):
    """Unrotated bf16 queries, keys and values of a prefill."""
    g = torch.Generator(device="cpu").manual_seed(seed)
    q = torch.randn((B, n_q, h_q, d), generator=g).to(torch.bfloat16)
    k = torch.randn((B, n_k, h_kv, d), generator=g).to(torch.bfloat16)
    v = torch.randn((B, n_k, h_kv, d), generator=g).to(torch.bfloat16)
    return q, k, v


def _rotated_bf16(q, k, q0, theta):
    """The oracle's fp64 rotation (query row i at q0 + i, key j at j), rounded to bf16
    as a pre-rotated cache holds it."""
    n_q, n_k = q.shape[1], k.shape[1]
    qr = torch.from_numpy(oracle.rope_rotate(q, np.arange(q0, q0 + n_q), theta)).to(torch.bfloat16)
    kr = torch.from_numpy(oracle.rope_rotate(k, np.arange(n_k), theta)).to(torch.bfloat16)
    return qr, kr


def _gpu_prefill_unrotated(q, k, v, q0, win, rope_inv_freq=None, kp=None, vp=None, n_k=None):
    import paper_2608_02947_amd as atf
    qd = q.contiguous().to(DEV)
    if kp is None:
        kp, vp = pack_kcache(k.to(DEV)), pack_vcache(v.to(DEV))
    B, n_q, h_q, d = qd.shape
    o = torch.empty_like(qd)
    lse = torch.empty((B, h_q, n_q), dtype=torch.float32, device=DEV)
    atf.atf_prefill_unrotated(qd, kp, vp, o, lse, q0, win, rope_inv_freq=rope_inv_freq, n_k=n_k)
    torch.cuda.synchronize()
    return o, lse


PREFILL_CASES = [
    # B, n_q, n_k, q0, h_q, h_kv, d, base, k
    (1, 300, 300, 0, 6, 2, 128, 5e5, 2.0),
    (2, 45, 45, 0, 4, 4, 64, 1e6, 2.0),                  # partial wave, MHA
    (1, 77, 267, 190, 7, 1, 64, 1e6, 2.0),               # chunk at the end of a longer context
    (1, 200, 150, 0, 8, 1, 128, 1e4, 2.0),               # keys end before the last query
    (1, 1, 1, 0, 2, 1, 128, 1e4, 2.0),                   # one row, one key
    (1, 257, 257, 0, 3, 3, 128, 100.0, 2.0),             # saturated: every window ends early
    (1, 256, 256, 0, 2, 1, 128, 1e4, math.inf),          # window off, d = 128
    (1, 200, 200, 0, 4, 1, 64, 1e4, math.inf),           # window off, d = 64
    (1, 333, 500, 167, 16, 2, 64, 1e4, 1.0),             # G = 8, ragged tail
    (2, 130, 1000, 870, 12, 1, 128, 1e4, 2.0),           # G = 12
    (1, 520, 4100, 3580, 8, 2, 128, 1e7, 2.0),           # many tiles, chunks pruned by tile
    (1, 64, 700, (1 << 30) + 5, 4, 1, 128, 1e4, math.inf),  # queries at 2^30 + 5 ..
    (1, 3, 200, 50, 128, 1, 64, 1e4, 2.0),               # G = 128: one position per workgroup
    (1, 2, 150, 20, 256, 1, 128, 1e4, 2.0),              # G = 256
]


@pytest.mark.parametrize("case", PREFILL_CASES, ids=lambda c: "x".join(str(x) for x in c))
def test_prefill_unrotated(case):
    B, n_q, n_k, q0, h_q, h_kv, d, base, kwin = case
    note(f"prefill unrotated {case}")
    q, k, v = _prefill_inputs(B, n_q, n_k, h_q, h_kv, d, seed=(hash(case) + 3) % 10000)
    win, widths = windows_for(d, base, kwin, None, n_ctx=q0 + n_q)
    o, lse = _gpu_prefill_unrotated(q, k, v, q0, win)
    qr, kr = _rotated_bf16(q, k, q0, W.rope_theta(d, base).numpy())
    o_ref, lse_ref, _ = oracle.attend(qr, kr, v, q0, widths)
    compare(to_f64(o), to_f64(lse), o_ref, lse_ref, f"prefill unrotated {case}")


@pytest.mark.parametrize("case", [PREFILL_CASES[0], PREFILL_CASES[2], PREFILL_CASES[10]],
                         ids=lambda c: "x".join(str(x) for x in c))
def test_prefill_unrotated_matches_prerotated_cache(case):
    """The same attention through atf_prefill over caches the oracle rotated and rounded
    to bf16: the two paths differ only where a rotated element's bf16 rounding falls on
    the other side (fp32 rotation versus fp64), so every output element agrees to within
    one bf16 rounding of itself plus 2e-3, and the LSE to 2e-4."""
    B, n_q, n_k, q0, h_q, h_kv, d, base, kwin = case
    note(f"prefill unrotated vs pre-rotated {case}")
    q, k, v = _prefill_inputs(B, n_q, n_k, h_q, h_kv, d, seed=(hash(case) + 5) % 10000)
    win, _ = windows_for(d, base, kwin, None, n_ctx=q0 + n_q)
    o, lse = _gpu_prefill_unrotated(q, k, v, q0, win)
    qr, kr = _rotated_bf16(q, k, q0, W.rope_theta(d, base).numpy())
    o2, lse2 = gpu_prefill(qr.to(DEV), kr.to(DEV), v.to(DEV), q0, win)
    a, b = o.double(), o2.double()
    # within one bf16 rounding of the output (2^-7 relative at most) plus the scores'
    # perturbation by the rotation's rounding flips
    excess = float(((a - b).abs() - (2.0 ** -7 * torch.maximum(a.abs(), b.abs()) + 2e-3)).max())
    ml = float((lse - lse2).abs().max())
    same = float((o == o2).float().mean())
    print(f"[parity] unrotated vs pre-rotated {case}: bit-identical O {same:.4f}, "
          f"LSE max-abs {ml:.2e}", flush=True)
    assert excess <= 0.0 and ml <= 2e-4, (case, excess, ml)


PREFILL_EXACT_CASES = [
    # B, n_q, n_k, q0, h_q, h_kv, d, base, k: rows of thousands of keys
    (1, 256, 4096, 3840, 8, 2, 128, 1e4, 2.0),
    (1, 128, 8192, 8064, 14, 2, 64, 1e6, 2.0),
    (1, 128, 4096, 3968, 4, 1, 128, 1e4, math.inf),
]


@pytest.mark.parametrize("case", PREFILL_EXACT_CASES, ids=lambda c: "x".join(str(x) for x in c))
def test_prefill_unrotated_against_exact_rotation(case):
    """Against attention over the EXACTLY rotated vectors (fp64, not rounded to bf16):
    the read-time rotation strays from it no further than a pre-rotated bf16 cache does,
    plus the kernel's own arithmetic.  The oracle's attention over its own correctly
    rounded bf16 rotation measures that cache's distance from the exact result (e16);
    by the triangle inequality through that attention, which the parity contract holds
    the kernel to within the fixed tolerances, the kernel's distance is at most e16 plus
    those tolerances.  Over a whole prefill the LSE error of the bf16 rounding alone
    reaches ~1e-3 on some rows (the LSE follows the largest scores, whose rounding shifts
    do not average out), so the fixed LSE tolerance alone is not the yardstick here."""
    B, n_q, n_k, q0, h_q, h_kv, d, base, kwin = case
    note(f"prefill unrotated vs exact rotation {case}")
    q, k, v = _prefill_inputs(B, n_q, n_k, h_q, h_kv, d, seed=(hash(case) + 9) % 10000)
    win, widths = windows_for(d, base, kwin, None, n_ctx=q0 + n_q)
    o, lse = _gpu_prefill_unrotated(q, k, v, q0, win)
    theta = W.rope_theta(d, base).numpy()
    qr = oracle.rope_rotate(q, np.arange(q0, q0 + n_q), theta)
    kr = oracle.rope_rotate(k, np.arange(n_k), theta)
    vv = v.to(torch.float64).numpy()
    o_ex, lse_ex, _ = oracle.attend(qr, kr, vv, q0, widths)
    q16, k16 = (torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy() for x in (qr, kr))
    o_16, lse_16, _ = oracle.attend(q16, k16, vv, q0, widths)
    og, lg = to_f64(o), to_f64(lse)
    e16 = (np.abs(o_16 - o_ex).max(), np.abs(o_16 - o_ex).mean(), np.abs(lse_16 - lse_ex).max())
    eg = (np.abs(og - o_ex).max(), np.abs(og - o_ex).mean(), np.abs(lg - lse_ex).max())
    print(f"[parity] exact rotation {case}: bf16 cache O max {e16[0]:.2e} mean {e16[1]:.2e} "
          f"LSE {e16[2]:.2e}; kernel O max {eg[0]:.2e} mean {eg[1]:.2e} LSE {eg[2]:.2e}",
          flush=True)
    assert np.all(np.isfinite(og)) and np.all(np.isfinite(lg))
    assert eg[0] <= e16[0] + O_MAX_ABS, (case, eg, e16)
    assert eg[1] <= e16[1] + O_MEAN_ABS, (case, eg, e16)
    assert eg[2] <= e16[2] + LSE_MAX_ABS, (case, eg, e16)


@pytest.mark.parametrize("window", ["rounded8", "var16to2", "k2_floor40_cap180", "sliding100"])
@pytest.mark.parametrize("d", [128, 64])
def test_prefill_unrotated_other_windows(window, d):
    """The rounded slice (Sec. 3.3) and members of the window family (App. A) from
    unrotated caches: the rotation follows whatever chunks the window keeps."""
    B, n_q, n_k, q0, h_q, h_kv, base = 1, 300, 900, 600, 6, 2, 1e4
    seed = 211 + d + ["rounded8", "var16to2", "k2_floor40_cap180", "sliding100"].index(window)
    q, k, v = _prefill_inputs(B, n_q, n_k, h_q, h_kv, d, seed=seed)
    if window == "rounded8":
        win, widths = windows_for(d, base, 2.0, None, n_ctx=q0 + n_q, slice_pairs=8)
        atom = 8
    else:
        win, widths = family_windows_for(d, base, None, window)
        atom = 0
    note(f"prefill unrotated {window} d={d}")
    o, lse = _gpu_prefill_unrotated(q, k, v, q0, win)
    qr, kr = _rotated_bf16(q, k, q0, W.rope_theta(d, base).numpy())
    o_ref, lse_ref, _ = oracle.attend(qr, kr, v, q0, widths, atom=atom)
    compare(to_f64(o), to_f64(lse), o_ref, lse_ref, f"unrotated {window} d={d}")


@pytest.mark.parametrize("d", [128, 64])
def test_prefill_unrotated_cache_capacity_and_nan_tail(d):
    """Caches allocated for more tokens than written, the slots past n_k filled with NaN:
    the rotation of a tile that crosses n_k turns only loaded keys (the slots past n_k
    re-read the last key), and the result equals the call over caches of exactly n_k
    tokens bit for bit."""
    import paper_2608_02947_amd as atf
    B, n_q, n_k, cap, h_q, h_kv = 2, 150, 333, 400, 6, 2
    q, k, v = _prefill_inputs(B, n_q, n_k, h_q, h_kv, d, seed=29 + d)
    win, widths = windows_for(d, 1e4, 2.0, None, n_ctx=n_k)
    kc = torch.full((B, cap, h_kv, d), float("nan"), dtype=torch.bfloat16)
    vc = torch.full((B, cap, h_kv, d), float("nan"), dtype=torch.bfloat16)
    kc[:, :n_k] = k
    vc[:, :n_k] = v
    note(f"prefill unrotated cache capacity d={d}")
    kp, vp = pack_kcache(kc.to(DEV)), pack_vcache(vc.to(DEV))
    o, lse = _gpu_prefill_unrotated(q, None, None, n_k - n_q, win, kp=kp, vp=vp, n_k=n_k)
    o2, lse2 = _gpu_prefill_unrotated(q, k, v, n_k - n_q, win)
    assert torch.equal(o, o2) and torch.equal(lse, lse2)
    qr, kr = _rotated_bf16(q, k, n_k - n_q, W.rope_theta(d, 1e4).numpy())
    o_ref, lse_ref, _ = oracle.attend(qr, kr, v, n_k - n_q, widths)
    compare(to_f64(o), to_f64(lse), o_ref, lse_ref, f"unrotated capacity d={d}")


def test_prefill_unrotated_chunked_equals_single_shot():
    """A prefill in three chunks (rows a .. b - 1 against keys 0 .. b - 1 of the same
    caches, capacity larger than the keys used) gives the single-shot result bit for
    bit: a key's angle depends only on its position, not on the chunk that reads it.
    Chunk boundaries are multiples of the position tile (floor(256 / G) = 64)."""
    B, n, h_q, h_kv, d, base = 1, 700, 8, 2, 128, 1e6
    q, k, v = _prefill_inputs(B, n, n + 100, h_q, h_kv, d, seed=123)
    win, _ = windows_for(d, base, 2.0, None, n_ctx=n)
    kp, vp = pack_kcache(k.to(DEV)), pack_vcache(v.to(DEV))
    note("prefill unrotated single shot")
    o1, l1 = _gpu_prefill_unrotated(q, None, None, 0, win, kp=kp, vp=vp, n_k=n)
    for a, b in [(0, 128), (128, 448), (448, 700)]:
        note(f"prefill unrotated chunk {a}..{b}")
        o2, l2 = _gpu_prefill_unrotated(q[:, a:b], None, None, a, win, kp=kp, vp=vp, n_k=b)
        assert torch.equal(o2, o1[:, a:b]) and torch.equal(l2, l1[:, :, a:b]), (a, b)


def test_prefill_unrotated_llama_frequencies():
    """Llama-3.2-3B shape with the llama3-effective frequencies: rotation from the
    window's own table, and from an explicit table under a raw-base window."""
    wl = W.WORKLOADS["llama3b_decode_32k"]
    d, n = wl.head_dim, 1500
    th = W.workload_theta(wl).numpy()
    q, k, v = _prefill_inputs(1, n, n, wl.h_q, wl.h_kv, d, seed=wl.seed + 3)
    qr, kr = _rotated_bf16(q, k, 0, th)
    note("prefill unrotated llama effective table")
    win, widths = windows_for(d, wl.rope_base, wl.k, th, n_ctx=n)
    o, lse = _gpu_prefill_unrotated(q, k, v, 0, win)
    o_ref, lse_ref, _ = oracle.attend(qr, kr, v, 0, widths)
    compare(to_f64(o), to_f64(lse), o_ref, lse_ref, "prefill llama effective")
    note("prefill unrotated llama raw-base window, effective rotation")
    win, widths = windows_for(d, wl.rope_base, wl.k, None, n_ctx=n)
    o, lse = _gpu_prefill_unrotated(q, k, v, 0, win, rope_inv_freq=th)
    o_ref, lse_ref, _ = oracle.attend(qr, kr, v, 0, widths)
    compare(to_f64(o), to_f64(lse), o_ref, lse_ref, "prefill llama raw window")


def test_prefill_unrotated_deterministic():
    q, k, v = _prefill_inputs(1, 600, 2000, 8, 2, 128, seed=43)
    win, _ = windows_for(128, 1e4, 2.0, None, n_ctx=2000)
    note("prefill unrotated determinism")
    o1, l1 = _gpu_prefill_unrotated(q, k, v, 1400, win)
    o2, l2 = _gpu_prefill_unrotated(q, k, v, 1400, win)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


@pytest.mark.parametrize("kwin", [2.0, math.inf], ids=["default", "kinf"])
def test_prefill_unrotated_qwen7b1m_chunk_sampled_rows(kwin):
    """The benchmark's 1M prefill chunk (131,072 query rows at positions 917,504 ..
    1,048,575 over keys 0 .. 1,048,575; 28 query heads / 4 KV heads, d = 128, base 1e7)
    from unrotated caches, in the launch configuration the benchmark times: the
    stratified sample of rows of the pre-rotated test, recomputed by the oracle from its
    own fp64 rotation."""
    wl = W.WORKLOADS["qwen7b1m_prefill_chunk"]
    d = wl.head_dim
    note(f"generate qwen7b1m_prefill_chunk unrotated, k={kwin}")
    inp = W.make_inputs(wl, device=DEV, rotated=False)
    kp, vp = pack_kcache(inp["k"]), pack_vcache(inp["v"])
    win, widths, _ = table_windows(wl, "default" if kwin == 2.0 else "kinf")
    rows = bench_rows(wl, widths)
    assert len(rows) >= 256 and set(rows[:, 1].tolist()) == set(range(wl.h_q))
    note(f"prefill unrotated qwen7b1m chunk k={kwin}: {len(rows)} sampled rows")
    o, lse = _gpu_prefill_unrotated(inp["q"], None, None, wl.q_pos0, win, kp=kp, vp=vp)
    idx = torch.from_numpy(rows).to(DEV)
    og = to_f64(o[idx[:, 0], idx[:, 2], idx[:, 1]])
    lg = to_f64(lse[idx[:, 0], idx[:, 1], idx[:, 2]])
    del o, lse, kp, vp
    # the oracle rotates the sampled query rows and every key
    theta = W.rotation_theta(wl).numpy()
    qs = inp["q"][:, np.unique(rows[:, 2])].cpu()
    uniq = np.unique(rows[:, 2])
    qr = torch.from_numpy(oracle.rope_rotate(qs, wl.q_pos0 + uniq, theta)).to(torch.bfloat16)
    q_full = torch.zeros((wl.batch, wl.n_q, wl.h_q, d), dtype=torch.bfloat16)
    q_full[:, uniq] = qr
    kr = torch.from_numpy(oracle.rope_rotate(inp["k"].cpu(), np.arange(wl.n_k), theta)).to(
        torch.bfloat16)
    o_ref, lse_ref, _ = oracle.attend(q_full, kr, inp["v"].cpu(), wl.q_pos0, widths, rows=rows)
    mx, mean, ml = compare(og, lg, o_ref, lse_ref, f"prefill unrotated qwen7b1m k={kwin}")
    print(f"[parity] prefill unrotated qwen7b1m k={kwin}: O max {mx:.2e} mean {mean:.2e} "
          f"LSE {ml:.2e}", flush=True)


# ---- the whole cache rotated in one pass (write-time alternative) ----

def _unpack_kcache(kp):
    """[B, h_kv, d/16, n, 16] pair-chunk-major -> [B, n, h_kv, d] (pure re-indexing)."""
    B, h_kv, C, n, _ = kp.shape
    g = kp.permute(0, 3, 1, 2, 4)
    lo = g[..., :8].reshape(B, n, h_kv, 8 * C)
    hi = g[..., 8:].reshape(B, n, h_kv, 8 * C)
    return torch.cat([lo, hi], dim=-1)


@pytest.mark.parametrize("shape", [(2, 1000, 1100, 2, 128), (1, 777, 777, 3, 64),
                                   (1, 262144, 262144, 1, 64)],
                         ids=lambda c: "x".join(str(x) for x in c))
def test_rotate_kcache_against_the_oracle(shape):
    """atf_rotate_kcache against the oracle's fp64 rotation rounded to bf16 (key t at
    position t; keys up to position 262143 in the last case), element by element:
    |got - ref| <= one bf16 step of the larger of the two (each is a rounding of its
    own rotation) + 2^-20 (|x_r| + |x_{r+d/2}|) (the fp32 rotation's error: products and
    fma of bf16 inputs with fp32 cosines and sines, and the hardware cosine and sine,
    each within a few fp32 units of the pair's magnitude).  Elements that differ at
    all are rare, and the slots past n_k are untouched."""
    import paper_2608_02947_amd as atf
    B, n_k, cap, h_kv, d = shape
    g = torch.Generator(device="cpu").manual_seed(31 + n_k)
    k = torch.randn((B, cap, h_kv, d), generator=g).to(torch.bfloat16)
    win, _ = windows_for(d, 1e4, 2.0, None, n_ctx=n_k)
    note(f"rotate kcache {shape}")
    kp = pack_kcache(k.to(DEV))
    kr = torch.full_like(kp, float("nan"))
    atf.atf_rotate_kcache(kp, kr, win, n_k=n_k)
    torch.cuda.synchronize()
    theta = W.rope_theta(d, 1e4).numpy()
    ref = torch.from_numpy(oracle.rope_rotate(k[:, :n_k], np.arange(n_k), theta)).to(torch.bfloat16)
    got = _unpack_kcache(kr[:, :, :, :n_k].cpu()).double()
    ref = ref.double()
    x = k[:, :n_k].double().abs()
    mag = torch.cat([x[..., :d // 2] + x[..., d // 2:]] * 2, dim=-1)
    big = torch.maximum(got.abs(), ref.abs())
    step = torch.where(big > 0, torch.exp2(torch.floor(torch.log2(big)) - 7), torch.zeros_like(big))
    excess = float(((got - ref).abs() - (step + 2.0 ** -20 * mag)).max())
    frac = float((got != ref).double().mean())
    print(f"[parity] rotate kcache {shape}: elements that differ {frac:.2e}, "
          f"largest excess over the bound {excess:.2e}", flush=True)
    assert excess <= 0.0 and frac < 1e-3, (shape, excess, frac)
    if cap > n_k:
        assert torch.isnan(kr[:, :, :, n_k:].float()).all()
    # in place: the same bits as into a second buffer
    atf.atf_rotate_kcache(kp, kp, win, n_k=n_k)
    torch.cuda.synchronize()
    assert torch.equal(kp[:, :, :, :n_k], kr[:, :, :, :n_k])


def test_rotate_kcache_then_prefill_and_decode():
    """The rotated copy read as a pre-rotated cache: atf_prefill and atf_decode over it
    against the oracle's attention over its own bf16 rotation."""
    import paper_2608_02947_amd as atf
    B, n_q, n_k, h_q, h_kv, d, base = 1, 300, 2000, 8, 2, 128, 1e6
    q, k, v = _prefill_inputs(B, n_q, n_k, h_q, h_kv, d, seed=57)
    q0 = n_k - n_q
    win, widths = windows_for(d, base, 2.0, None, n_ctx=n_k + 1)
    theta = W.rope_theta(d, base).numpy()
    kp, vp = pack_kcache(k.to(DEV)), pack_vcache(v.to(DEV))
    kr = torch.empty_like(kp)
    note("rotate kcache then prefill and decode")
    atf.atf_rotate_kcache(kp, kr, win, rope_inv_freq=theta)
    qr, kr_ref = _rotated_bf16(q, k, q0, theta)
    o, lse = gpu_prefill(qr.to(DEV), None, None, q0, win, kp=kr, vp=vp)
    o_ref, lse_ref, _ = oracle.attend(qr, kr_ref, v, q0, widths)
    compare(to_f64(o), to_f64(lse), o_ref, lse_ref, "rotated copy, prefill")
    qd = torch.from_numpy(oracle.rope_rotate(q[:, -1:], [n_k], theta)).to(torch.bfloat16)
    ws = torch.empty(atf.atf_decode_workspace_bytes(B, h_q, h_kv, n_k, d), dtype=torch.uint8,
                     device=DEV)
    od = torch.empty((B, h_q, d), dtype=torch.bfloat16, device=DEV)
    lsed = torch.empty((B, h_q), dtype=torch.float32, device=DEV)
    atf.atf_decode(qd[:, 0].contiguous().to(DEV), kr, vp, od, lsed, n_k, win, ws)
    torch.cuda.synchronize()
    o_ref, lse_ref, _ = oracle.attend(qd, kr_ref, v, n_k, widths)
    compare(to_f64(od), to_f64(lsed), o_ref[:, 0], lse_ref[:, :, 0], "rotated copy, decode")


def test_cache_append_rotated():
    """Unrotated keys appended in three chunks with RoPE on the way in: the K cache is
    the one-pass rotation of the whole unrotated cache bit for bit (the same angle and
    rotation per (token, pair)), the V cache is atf_cache_append's, slots past the
    appended tokens keep their contents, and a prefill over the caches matches the
    oracle."""
    import paper_2608_02947_amd as atf
    B, n, cap, h_q, h_kv, d, base = 2, 900, 1000, 8, 2, 128, 1e6
    q, k, v = _prefill_inputs(B, 200, n, h_q, h_kv, d, seed=73)
    win, widths = windows_for(d, base, 2.0, None, n_ctx=n)
    kd, vd = k.to(DEV), v.to(DEV)
    kc = torch.full(atf.kcache_shape(B, cap, h_kv, d), float("nan"), dtype=torch.bfloat16, device=DEV)
    vc = torch.full(atf.vcache_shape(B, cap, h_kv, d), float("nan"), dtype=torch.bfloat16, device=DEV)
    vc2 = vc.clone()
    kc2 = torch.full_like(kc, float("nan"))
    note("cache append rotated")
    for a, b in [(0, 300), (300, 301), (301, 900)]:
        atf.atf_cache_append_rotated(kd[:, a:b].contiguous(), vd[:, a:b].contiguous(), kc, vc, a, win)
        atf.atf_cache_append(kd[:, a:b].contiguous(), vd[:, a:b].contiguous(), kc2, vc2, a)
    kr = torch.full_like(kc, float("nan"))
    atf.atf_rotate_kcache(kc2, kr, win, n_k=n)
    torch.cuda.synchronize()
    assert torch.equal(kc[:, :, :, :n], kr[:, :, :, :n])
    assert torch.isnan(kc[:, :, :, n:].float()).all()
    assert torch.equal(vc.view(torch.int16), vc2.view(torch.int16))
    q0 = n - 200
    theta = W.rope_theta(d, base).numpy()
    qr, kr_ref = _rotated_bf16(q, k, q0, theta)
    o, lse = gpu_prefill(qr.to(DEV), None, None, q0, win, kp=kc, vp=vc, n_k=n)
    o_ref, lse_ref, _ = oracle.attend(qr, kr_ref, v, q0, widths)
    compare(to_f64(o), to_f64(lse), o_ref, lse_ref, "append rotated, prefill")


def test_cache_append_paged_rotated():
    """Unrotated keys appended into shuffled pages in two chunks with RoPE on the way in:
    every written K slot equals the contiguous rotated append's bit for bit, the V pages
    equal atf_cache_append_paged's, pages no row names keep their contents, and the
    paged decode over them matches the oracle."""
    import paper_2608_02947_amd as atf
    B, n, pt, h_q, h_kv, d, base = 3, 700, 64, 6, 2, 128, 1e4
    pages = -(-n // pt)
    num_pages = B * pages + 2
    q, k, v = _prefill_inputs(B, 1, n, h_q, h_kv, d, seed=83)
    win, widths = windows_for(d, base, 2.0, None, n_ctx=n + 1)
    perm = np.random.default_rng(9).permutation(num_pages)[:B * pages].reshape(B, pages)
    btd = torch.from_numpy(perm.astype(np.int32)).to(DEV)
    kd, vd = k.to(DEV), v.to(DEV)
    kpool = torch.full(atf.kpages_shape(num_pages, pt, h_kv, d), float("nan"), dtype=torch.bfloat16,
                       device=DEV)
    vpool = torch.full(atf.vpages_shape(num_pages, pt, h_kv, d), float("nan"), dtype=torch.bfloat16,
                       device=DEV)
    vpool2 = vpool.clone()
    kpool2 = kpool.clone()
    note("cache append paged rotated")
    for a, b in [(0, 250), (250, n)]:
        ka, va = kd[:, a:b].contiguous(), vd[:, a:b].contiguous()
        atf.atf_cache_append_paged_rotated(ka, va, kpool, vpool, btd, a, win)
        atf.atf_cache_append_paged(ka, va, kpool2, vpool2, btd, a)
    kc = torch.empty(atf.kcache_shape(B, n, h_kv, d), dtype=torch.bfloat16, device=DEV)
    vc = torch.empty(atf.vcache_shape(B, n, h_kv, d), dtype=torch.bfloat16, device=DEV)
    atf.atf_cache_append_rotated(kd, vd, kc, vc, 0, win)
    torch.cuda.synchronize()
    # K slot of (row b, token t): page bt[b, t // pt], slot t % pt
    t = torch.arange(n, device=DEV)
    for b in range(B):
        pg = btd[b, t // pt].long()
        got = kpool[pg, :, :, t % pt, :]                   # [n, h_kv, d/16, 16]
        assert torch.equal(got, kc[b].permute(2, 0, 1, 3)), b
    assert torch.equal(vpool.view(torch.int16), vpool2.view(torch.int16))
    unused = sorted(set(range(num_pages)) - set(perm.ravel().tolist()))
    assert torch.isnan(kpool[unused].float()).all()
    qd = torch.from_numpy(oracle.rope_rotate(q, [n], W.rope_theta(d, base).numpy())).to(torch.bfloat16)
    ws = torch.empty(atf.atf_decode_workspace_bytes(B, h_q, h_kv, n, d), dtype=torch.uint8, device=DEV)
    od = torch.empty((B, h_q, d), dtype=torch.bfloat16, device=DEV)
    lsed = torch.empty((B, h_q), dtype=torch.float32, device=DEV)
    rows = torch.full((B,), n, dtype=torch.int32, device=DEV)
    atf.atf_decode_paged(qd[:, 0].contiguous().to(DEV), kpool, vpool, od, lsed, btd, rows, rows, n,
                         win, ws)
    torch.cuda.synchronize()
    _, kr_ref = _rotated_bf16(q, k, n, W.rope_theta(d, base).numpy())
    o_ref, lse_ref, _ = oracle.attend(qd, kr_ref, v, n, widths)
    compare(to_f64(od), to_f64(lsed), o_ref[:, 0], lse_ref[:, :, 0], "paged rotated append, decode")
