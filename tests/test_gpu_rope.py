"""GPU parity of decode from UNROTATED caches (RoPE applied at read time, App. B)
through the C ABI: atf_decode_unrotated and atf_decode_paged_unrotated against the
oracle, which rotates the same bf16 query and keys in fp64 (oracle.rope_rotate, pinned
in test_oracle_rope.py), stores them in bf16 as a pre-rotated cache would, and attends
them in fp64."""
import math

import numpy as np
import pytest
import torch

from conftest import gpu_available
import oracle
import workloads as W
from parity import compare, note, pack_kcache, pack_vcache, to_f64, windows_for

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
