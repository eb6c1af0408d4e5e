"""GPU parity of atf_pack_kcache, atf_pack_vcache and atf_decode against the oracle.

The caches are packed by the library; each pack is checked bit-exactly against
a torch re-indexing of the same tensor.  Decode outputs are compared
for every (batch, query head) row, at small shapes and at the full workload
shapes the benchmark times.
"""
import math

import numpy as np
import pytest
import torch

from conftest import gpu_available
import oracle
import workloads as W
from parity import (case_seed, compare_rounding_bound, compare, decode_budget, family_windows_for, gpu_decode, note, pack_kcache, pack_vcache,
                    to_f64, windows_for, workload_window)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]

DEV = "cuda"


def _ref_pack(k_bshd):
    """[B, n_k, h_kv, d] -> [B, h_kv, d/16, n_k, 16]: chunk c = dims [8c, 8c+8) ++ [d/2+8c, d/2+8c+8)."""
    B, n_k, h_kv, d = k_bshd.shape
    kk = k_bshd.permute(0, 2, 1, 3)
    lo = kk[..., : d // 2].reshape(B, h_kv, n_k, d // 16, 8)
    hi = kk[..., d // 2:].reshape(B, h_kv, n_k, d // 16, 8)
    return torch.cat([lo, hi], dim=-1).permute(0, 1, 3, 2, 4).contiguous()


@pytest.mark.parametrize("shape", [(1, 1, 1, 64), (2, 37, 3, 128), (3, 1000, 2, 64)])
def test_pack_bit_exact(shape):
    note(f"pack {shape}")
    k = W.random_bf16(shape, seed=sum(shape)).to(DEV)
    kp = pack_kcache(k)
    torch.cuda.synchronize()
    ref = _ref_pack(k)
    assert torch.equal(kp.view(torch.int16), ref.view(torch.int16))


def _ref_vpack(v_bshd):
    """[B, n_k, h_kv, d] -> [B, h_kv, ceil(n_k/16), d, 16]; slot 8h + e of a block's
    d-row holds token 8*(e//4) + 4h + e%4 of the block, zero past n_k."""
    B, n_k, h_kv, d = v_bshd.shape
    nb = (n_k + 15) // 16
    vv = torch.zeros((B, nb * 16, h_kv, d), dtype=v_bshd.dtype, device=v_bshd.device)
    vv[:, :n_k] = v_bshd
    blocks = vv.view(B, nb, 16, h_kv, d).permute(0, 3, 1, 4, 2)  # [B, h_kv, nb, d, 16 tokens]
    order = torch.tensor([8 * (e // 4) + 4 * h + e % 4 for h in range(2) for e in range(8)],
                         device=v_bshd.device)
    return blocks[..., order].contiguous()


@pytest.mark.parametrize("shape", [(1, 1, 1, 64), (2, 37, 3, 128), (3, 1000, 2, 64),
                                   (1, 4096, 4, 128)])
def test_vpack_bit_exact(shape):
    note(f"vpack {shape}")
    v = W.random_bf16(shape, seed=sum(shape) + 1).to(DEV)
    vp = pack_vcache(v)
    torch.cuda.synchronize()
    ref = _ref_vpack(v)
    assert vp.shape == ref.shape
    assert torch.equal(vp.view(torch.int16), ref.view(torch.int16))


@pytest.mark.parametrize("shape,cuts", [((2, 100, 3, 128), (0, 7, 40, 41, 100)),
                                        ((1, 333, 2, 64), (0, 16, 17, 300, 333))])
def test_cache_append_bit_exact(shape, cuts):
    """Appending a sequence in pieces at arbitrary offsets writes exactly the packed
    layouts, and slots of tokens not yet appended keep what the cache held."""
    import paper_2608_02947_amd as atf
    B, n, h_kv, d = shape
    cap = n + 21
    note(f"cache append {shape} {cuts}")
    k = W.random_bf16(shape, seed=sum(shape) + 2).to(DEV)
    v = W.random_bf16(shape, seed=sum(shape) + 3).to(DEV)
    sentinel = -7.0
    kc = torch.full(atf.kcache_shape(B, cap, h_kv, d), sentinel, dtype=torch.bfloat16, device=DEV)
    vc = torch.full(atf.vcache_shape(B, cap, h_kv, d), sentinel, dtype=torch.bfloat16, device=DEV)
    for a, b in zip(cuts[:-1], cuts[1:]):
        atf.atf_cache_append(k[:, a:b].contiguous(), v[:, a:b].contiguous(), kc, vc, a)
        torch.cuda.synchronize()
        kfull = torch.full((B, cap, h_kv, d), sentinel, dtype=torch.bfloat16, device=DEV)
        kfull[:, :b] = k[:, :b]
        assert torch.equal(kc.view(torch.int16), _ref_pack(kfull).view(torch.int16))
        vfull = torch.full((B, (cap + 15) // 16 * 16, h_kv, d), sentinel, dtype=torch.bfloat16,
                           device=DEV)
        vfull[:, :b] = v[:, :b]
        ref = _ref_vpack(vfull)
        assert torch.equal(vc.view(torch.int16), ref.view(torch.int16))


def _decode_inputs(B, n_k, q_pos, h_q, h_kv, d, base, seed, theta=None):
    g = torch.Generator(device="cpu").manual_seed(seed)
    q = torch.randn((B, 1, h_q, d), generator=g).to(torch.bfloat16)
    k = torch.randn((B, n_k, h_kv, d), generator=g).to(torch.bfloat16)
    v = torch.randn((B, n_k, h_kv, d), generator=g).to(torch.bfloat16)
    th = torch.as_tensor(theta, dtype=torch.float64) if theta is not None else W.rope_theta(d, base)
    q = W.rotate_half(q, torch.tensor([q_pos]), th)
    k = W.rotate_half(k, torch.arange(0, n_k), th)
    return q, k, v


def _decode_parity(q4, k, v, q_pos, win, widths, label, atom=0):
    """q4 [B, 1, h_q, d] (oracle layout); every (b, head) row compared."""
    note(f"decode {label} q={tuple(q4.shape)} k={tuple(k.shape)} q_pos={q_pos}")
    qd = q4[:, 0].contiguous().to(DEV)
    o, lse = gpu_decode(qd, k.to(DEV), v.to(DEV), q_pos, win)
    o_ref, lse_ref, _ = oracle.attend(q4.cpu(), k.cpu(), v.cpu(), q_pos, widths, atom=atom)
    return compare(to_f64(o), to_f64(lse), o_ref[:, 0], lse_ref[:, :, 0], label)


CASES = [
    # B, n_k, q_pos, h_q, h_kv, d, base, k
    (1, 1, 1, 1, 1, 128, 1e4, 2.0),
    (2, 300, 300, 6, 2, 128, 5e5, 2.0),
    (3, 1000, 1000, 7, 1, 64, 1e6, 2.0),
    (1, 2049, 5000, 8, 1, 128, 1e4, 2.0),       # query beyond the cache end
    (1, 3000, 1500, 4, 2, 64, 1e4, 2.0),        # keys past the query are not causal
    (2, 777, 777, 12, 1, 128, 1e4, 2.0),        # G = 12 in one workgroup
    (1, 1500, 1500, 40, 1, 64, 1e4, 2.0),       # G = 40 in two sub-groups of 20
    (1, 700, 700, 37, 1, 128, 1e4, 2.0),        # G = 37 (prime): one head per workgroup
    (1, 4096, 4096, 16, 2, 128, 100.0, 2.0),    # saturated windows
    (1, 513, 513, 2, 2, 64, 1e4, 0.05),         # tiny k: empty score sums
    (1, 999, 999, 3, 1, 128, 1e4, math.inf),    # window off
    (1, 300000, 300000, 8, 1, 64, 1e6, 2.0),    # 1024 splits: several merge passes per head
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(str(x) for x in c))
def test_decode_small(case):
    B, n_k, q_pos, h_q, h_kv, d, base, kwin = case
    q, k, v = _decode_inputs(B, n_k, q_pos, h_q, h_kv, d, base, seed=hash(case) % 10000)
    win, widths = windows_for(d, base, kwin, None, n_ctx=q_pos + 1)
    _decode_parity(q, k, v, q_pos, win, widths, f"small{case}")


def test_decode_nonmonotone_table():
    d = 128
    rng = np.random.default_rng(8)
    theta = rng.uniform(0.001, 2.0, d // 2)
    theta[[0, 9]] = 0.0
    q, k, v = _decode_inputs(2, 2500, 2500, 6, 3, d, 0.0, seed=4, theta=theta)
    win, widths = windows_for(d, 1e4, 2.0, theta, n_ctx=2501)
    _decode_parity(q, k, v, 2500, win, widths, "nonmonotone")


FAMILY_CASES = [
    # family, B, n_k, q_pos, h_q, h_kv, d, base
    ("var16to2", 2, 777, 777, 12, 1, 128, 1e4),
    ("geo16to2", 1, 1500, 1500, 8, 1, 64, 1e6),
    ("k64", 1, 3000, 3000, 6, 2, 128, 5e5),
    ("k2_floor40_cap180", 1, 3000, 3000, 6, 2, 128, 5e5),
    ("gamma1.25", 3, 1000, 1000, 7, 1, 64, 1e6),
    ("sliding100", 1, 1500, 1500, 8, 1, 128, 1e4),   # every pair pruned past 100
    ("linear256", 1, 2049, 2049, 4, 2, 64, 1e4),
]


@pytest.mark.parametrize("case", FAMILY_CASES, ids=lambda c: "x".join(str(x) for x in c))
def test_decode_window_family(case):
    """Members of the window family of App. A (eq:family)."""
    fam, B, n_k, q_pos, h_q, h_kv, d, base = case
    q, k, v = _decode_inputs(B, n_k, q_pos, h_q, h_kv, d, base, seed=case_seed(case))
    win, widths = family_windows_for(d, base, None, fam)
    _decode_parity(q, k, v, q_pos, win, widths, f"family{case}")


@pytest.mark.parametrize("case", [(2, 777, 777, 12, 1, 128, 1e4, 2.0),
                                  (1, 1500, 1500, 40, 1, 64, 1e4, 2.0),
                                  (1, 4096, 4096, 16, 2, 128, 100.0, 2.0)],
                         ids=lambda c: "x".join(str(x) for x in c))
def test_decode_rounded_slice(case):
    """The rounded slice of Sec. 3.3 (8-pair K-steps) against the oracle's rounding rule."""
    B, n_k, q_pos, h_q, h_kv, d, base, kwin = case
    q, k, v = _decode_inputs(B, n_k, q_pos, h_q, h_kv, d, base, seed=hash(case) % 10000 + 1)
    win, widths = windows_for(d, base, kwin, None, n_ctx=q_pos + 1, slice_pairs=8)
    _decode_parity(q, k, v, q_pos, win, widths, f"rounded{case}", atom=8)


def test_decode_custom_scale_and_determinism():
    q, k, v = _decode_inputs(1, 3001, 3001, 8, 2, 128, 1e4, seed=11)
    win, widths = windows_for(128, 1e4, 2.0, None, n_ctx=3002)
    qd, kd, vd = q[:, 0].contiguous().to(DEV), k.to(DEV), v.to(DEV)
    note("decode scale 0.2")
    o, lse = gpu_decode(qd, kd, vd, 3001, win, scale=0.2)
    o_ref, lse_ref, _ = oracle.attend(q, k, v, 3001, widths, scale=0.2)
    compare(to_f64(o), to_f64(lse), o_ref[:, 0], lse_ref[:, :, 0], "scale0.2")
    o2, lse2 = gpu_decode(qd, kd, vd, 3001, win, scale=0.2)
    assert torch.equal(o, o2) and torch.equal(lse, lse2)


def test_decode_cache_capacity_and_uninitialised_tail():
    """Caches allocated for more tokens than written: tokens past n_k (NaN here,
    including the rest of the 16-token block holding token n_k) are never used."""
    B, n_k, cap, h_q, h_kv, d = 2, 1001, 1200, 8, 2, 128
    q, k, v = _decode_inputs(B, n_k, n_k, h_q, h_kv, d, 1e4, seed=31)
    win, widths = windows_for(d, 1e4, 2.0, None, n_ctx=n_k + 1)
    kc = torch.full((B, cap, h_kv, d), float("nan"), dtype=torch.bfloat16)
    vc = torch.full((B, cap, h_kv, d), float("nan"), dtype=torch.bfloat16)
    kc[:, :n_k] = k
    vc[:, :n_k] = v
    note("decode cache capacity")
    qd = q[:, 0].contiguous().to(DEV)
    o, lse = gpu_decode(qd, kc.to(DEV), vc.to(DEV), n_k, win, n_k=n_k)
    o_ref, lse_ref, _ = oracle.attend(q, k, v, n_k, widths)
    compare(to_f64(o), to_f64(lse), o_ref[:, 0], lse_ref[:, :, 0], "capacity")


# ---------------------------------------------------------------------------
# ragged batch: per-row cache length and query position (device arrays)
# ---------------------------------------------------------------------------
def _ragged_inputs(n_ks, q_poss, cap, h_q, h_kv, d, base, seed, fill=float("nan")):
    """Row b: q at q_poss[b], keys 0 .. n_ks[b] - 1 (rotated at their positions);
    cache slots past n_ks[b] hold `fill` (they must never be used)."""
    B = len(n_ks)
    th = W.rope_theta(d, base)
    g = torch.Generator(device="cpu").manual_seed(seed)
    q = torch.empty((B, 1, h_q, d), dtype=torch.bfloat16)
    kc = torch.full((B, cap, h_kv, d), fill, dtype=torch.bfloat16)
    vc = torch.full((B, cap, h_kv, d), fill, dtype=torch.bfloat16)
    for b, (nk, qp) in enumerate(zip(n_ks, q_poss)):
        qb = torch.randn((1, 1, h_q, d), generator=g).to(torch.bfloat16)
        q[b:b + 1] = W.rotate_half(qb, torch.tensor([qp]), th)
        if nk:
            kb = torch.randn((1, nk, h_kv, d), generator=g).to(torch.bfloat16)
            kc[b:b + 1, :nk] = W.rotate_half(kb, torch.arange(0, nk), th)
            vc[b:b + 1, :nk] = torch.randn((1, nk, h_kv, d), generator=g).to(torch.bfloat16)
    return q, kc, vc


def _gpu_decode_ragged(q, kc, vc, n_ks, q_poss, max_n_k, win):
    import paper_2608_02947_amd as atf
    B, h_q, d = q.shape
    kp, vp = pack_kcache(kc), pack_vcache(vc)
    h_kv = kp.shape[1]
    ws = torch.empty(atf.atf_decode_workspace_bytes(B, h_q, h_kv, max_n_k, d), dtype=torch.uint8,
                     device=DEV)
    o = torch.empty_like(q)
    lse = torch.empty((B, h_q), dtype=torch.float32, device=DEV)
    nk_d = torch.tensor(n_ks, dtype=torch.int32, device=DEV)
    qp_d = torch.tensor(q_poss, dtype=torch.int32, device=DEV)
    atf.atf_decode_ragged(q, kp, vp, o, lse, nk_d, qp_d, max_n_k, win, ws)
    torch.cuda.synchronize()
    return o, lse


def _ragged_parity(n_ks, q_poss, cap, h_q, h_kv, d, base, kwin, seed, max_n_k=None, label=""):
    note(f"decode ragged {label} n_k={n_ks} q_pos={q_poss} cap={cap} h={h_q}/{h_kv} d={d}")
    q, kc, vc = _ragged_inputs(n_ks, q_poss, cap, h_q, h_kv, d, base, seed)
    max_n_k = max(max(n_ks), 1) if max_n_k is None else max_n_k
    win, _ = windows_for(d, base, kwin, None, n_ctx=max(q_poss) + 1)
    o, lse = _gpu_decode_ragged(q[:, 0].contiguous().to(DEV), kc.to(DEV), vc.to(DEV), n_ks,
                                q_poss, max_n_k, win)
    o, lse = to_f64(o), to_f64(lse)
    for b, (nk, qp) in enumerate(zip(n_ks, q_poss)):
        if nk == 0:
            # no key: an empty softmax gives O = 0 and LSE = -inf
            assert np.all(o[b] == 0.0) and np.all(lse[b] == -np.inf), (label, b)
            continue
        _, widths = windows_for(d, base, kwin, None, n_ctx=qp + 1)
        o_ref, lse_ref, _ = oracle.attend(q[b:b + 1], kc[b:b + 1, :nk], vc[b:b + 1, :nk], qp,
                                          widths)
        compare(o[b:b + 1], lse[b:b + 1], o_ref[:, 0], lse_ref[:, :, 0], f"{label} row {b}")


RAGGED_CASES = [
    # n_k per row, q_pos per row, cache capacity, h_q, h_kv, d, base, k
    ([1, 5, 300, 1000, 2049, 777], [1, 5, 300, 1000, 2049, 777], 2100, 7, 1, 128, 1e4, 2.0),
    ([2049, 33, 1500, 1], [5000, 33, 700, 0], 2049, 8, 2, 64, 1e6, 2.0),   # past / inside the cache
    ([0, 400, 0, 129], [0, 400, 10, 129], 512, 6, 2, 128, 5e5, 2.0),       # empty rows
    ([4096, 4000, 17], [4096, 4000, 17], 4096, 16, 2, 128, 100.0, 2.0),   # saturated windows
    ([999, 3, 640], [999, 3, 640], 1024, 3, 1, 128, 1e4, math.inf),       # window off
    ([0, 0, 0], [0, 5, 0], 64, 4, 2, 128, 1e4, 2.0),                       # no key in the batch
]


def _many_rows(n, cap, seed):
    """n row lengths in [0, cap] (some empty, some full) and query positions at,
    past or inside each row's cache."""
    rng = np.random.default_rng(seed)
    n_ks = [int(x) for x in rng.integers(0, cap + 1, size=n)]
    n_ks[3] = n_ks[70] = 0
    n_ks[5] = n_ks[129 % n] = cap
    q_poss = [nk if i % 3 else nk + int(rng.integers(0, 500)) for i, nk in enumerate(n_ks)]
    q_poss[7] = max(0, n_ks[7] // 2)
    return n_ks, q_poss


# more rows than one wave scans at once: the device-side work plan runs over the rows
# in several 64-row steps
RAGGED_CASES.append(_many_rows(130, 2500, 17) + (2500, 4, 2, 64, 1e6, 2.0))
# one KV head: a long row gets over a thousand work items, merged in several passes
RAGGED_CASES.append(([300000, 5, 1000], [300000, 5, 1000], 300000, 8, 1, 64, 1e6, 2.0))


@pytest.mark.parametrize("case", RAGGED_CASES, ids=lambda c: f"B{len(c[0])}_d{c[5]}_k{c[7]}")
def test_decode_ragged_rows(case):
    n_ks, q_poss, cap, h_q, h_kv, d, base, kwin = case
    _ragged_parity(n_ks, q_poss, cap, h_q, h_kv, d, base, kwin, seed=sum(n_ks) % 9973,
                   label=f"ragged d={d}")


def test_decode_ragged_max_bound_above_rows():
    """max_n_k larger than every row (a cache allocated for longer sequences)."""
    _ragged_parity([300, 70, 1], [300, 70, 1], 4096, 14, 2, 64, 1e6, 2.0, seed=5, max_n_k=4000,
                   label="loose bound")


def test_decode_ragged_equals_uniform_bit_exact():
    """Equal rows at a size where both split plans are capped by the 128-token step
    (12 splits) take the same plan and arithmetic as atf_decode: equal bits."""
    B, n_k, h_q, h_kv, d = 4, 1500, 12, 4, 128
    q, kc, vc = _ragged_inputs([n_k] * B, [n_k] * B, n_k, h_q, h_kv, d, 1e4, seed=11)
    win, _ = windows_for(d, 1e4, 2.0, None, n_ctx=n_k + 1)
    qd = q[:, 0].contiguous().to(DEV)
    o_r, lse_r = _gpu_decode_ragged(qd, kc.to(DEV), vc.to(DEV), [n_k] * B, [n_k] * B, n_k, win)
    o_u, lse_u = gpu_decode(qd, kc.to(DEV), vc.to(DEV), n_k, win)
    assert torch.equal(o_r, o_u) and torch.equal(lse_r, lse_u)


def test_decode_ragged_llama_128k_rows():
    """Llama-3.2-3B-shaped ragged batch of 8 up to 128K keys (llama3-effective
    table): every (row, head) against the oracle."""
    wl = W.WORKLOADS["llama3b_decode_128k"]
    d, cap = wl.head_dim, wl.n_k
    n_ks = [cap, 65536, 100000, 3, 1, 77777, cap - 5, 32768]
    note(f"decode ragged llama 128K n_k={n_ks}")
    th = W.workload_theta(wl)
    g = torch.Generator(device="cpu").manual_seed(wl.seed)
    q = torch.empty((8, 1, wl.h_q, d), dtype=torch.bfloat16)
    kc = torch.zeros((8, cap, wl.h_kv, d), dtype=torch.bfloat16)
    vc = torch.zeros((8, cap, wl.h_kv, d), dtype=torch.bfloat16)
    rth = W.rotation_theta(wl)
    for b, nk in enumerate(n_ks):
        q[b:b + 1] = W.rotate_half(torch.randn((1, 1, wl.h_q, d), generator=g).to(torch.bfloat16),
                                   torch.tensor([nk]), rth)
        kc[b:b + 1, :nk] = W.rotate_half(
            torch.randn((1, nk, wl.h_kv, d), generator=g).to(torch.bfloat16), torch.arange(0, nk), rth)
        vc[b:b + 1, :nk] = torch.randn((1, nk, wl.h_kv, d), generator=g).to(torch.bfloat16)
    win, _ = windows_for(d, wl.rope_base, wl.k, th, n_ctx=cap + 1)
    o, lse = _gpu_decode_ragged(q[:, 0].contiguous().to(DEV), kc.to(DEV), vc.to(DEV), n_ks, n_ks,
                                cap, win)
    o, lse = to_f64(o), to_f64(lse)
    for b, nk in enumerate(n_ks):
        _, widths = windows_for(d, wl.rope_base, wl.k, th, n_ctx=nk + 1)
        o_ref, lse_ref, _ = oracle.attend(q[b:b + 1], kc[b:b + 1, :nk], vc[b:b + 1, :nk], nk, widths)
        compare(o[b:b + 1], lse[b:b + 1], o_ref[:, 0], lse_ref[:, :, 0], f"llama128k row {b}")


@pytest.mark.parametrize("pattern", ["rising", "lognormal"])
def test_decode_large_scores_rescale(pattern):
    """Scores of order 100s along the cache: split partials with very different
    maxima and repeated raises of the running max within each split."""
    B, n_k, h_q, h_kv, d = 2, 5000, 8, 2, 128
    g = torch.Generator(device="cpu").manual_seed(123)
    q = torch.randn((B, 1, h_q, d), generator=g) * 3.0
    k = torch.randn((B, n_k, h_kv, d), generator=g)
    if pattern == "rising":
        k = k * torch.linspace(0.5, 6.0, n_k)[None, :, None, None]
    else:
        k = k * torch.exp(torch.randn((n_k,), generator=g))[None, :, None, None]
    v = torch.randn((B, n_k, h_kv, d), generator=g).to(torch.bfloat16)
    th = W.rope_theta(d, 1e4)
    q = W.rotate_half(q.to(torch.bfloat16), torch.tensor([n_k]), th)
    k = W.rotate_half(k.to(torch.bfloat16), torch.arange(0, n_k), th)
    win, widths = windows_for(d, 1e4, 2.0, None, n_ctx=n_k + 1)
    note(f"decode large scores {pattern}")
    o, lse = gpu_decode(q[:, 0].contiguous().to(DEV), k.to(DEV), v.to(DEV), n_k, win, scale=1.0)
    o_ref, lse_ref, _ = oracle.attend(q, k, v, n_k, widths, scale=1.0)
    bound = decode_budget(q, k, v, n_k, widths, 1.0, o_ref[:, 0])
    compare_rounding_bound(to_f64(o), to_f64(lse), o_ref[:, 0], lse_ref[:, :, 0], bound,
                           f"large {pattern}")


# ---------------------------------------------------------------------------
# paged caches: page pools + block tables
# ---------------------------------------------------------------------------
def _block_tables(n_rows, pages_per_row, num_pages, seed, share_prefix=0):
    """Distinct pages per row from a shuffled pool; with share_prefix > 0 every row
    reuses row 0's first share_prefix pages (a shared prompt prefix)."""
    rng = np.random.default_rng(seed)
    perm = rng.permutation(num_pages)
    bt = np.full((n_rows, pages_per_row), -1, dtype=np.int32)
    nxt = 0
    for b in range(n_rows):
        for j in range(pages_per_row):
            if b > 0 and j < share_prefix:
                bt[b, j] = bt[0, j]
            else:
                bt[b, j] = perm[nxt]
                nxt += 1
    assert nxt <= num_pages
    return bt


def _ref_pages(k_bshd, v_bshd, bt, num_pages, pt):
    """Reference page pools from the contiguous reference layouts: page bt[b, j] holds
    row b's tokens j*pt .. j*pt + pt - 1 (rows written in order, later rows win on
    shared pages)."""
    B, n, h_kv, d = k_bshd.shape
    kref = _ref_pack(k_bshd)          # [B, h_kv, d/16, n, 16]
    vref = _ref_vpack(v_bshd)         # [B, h_kv, n/16, d, 16]
    kp = torch.zeros((num_pages, h_kv, d // 16, pt, 16), dtype=torch.bfloat16, device=k_bshd.device)
    vp = torch.zeros((num_pages, h_kv, pt // 16, d, 16), dtype=torch.bfloat16, device=k_bshd.device)
    for b in range(B):
        for j in range(n // pt):
            kp[bt[b, j]] = kref[b, :, :, j * pt:(j + 1) * pt]
            vp[bt[b, j]] = vref[b, :, j * pt // 16:(j + 1) * pt // 16]
    return kp, vp


@pytest.mark.parametrize("pt,d", [(32, 64), (64, 128), (128, 128)])
def test_cache_append_paged_bit_exact(pt, d):
    """Pools written by atf_cache_append_paged in three appends (ragged cuts inside
    pages and 16-token blocks) equal the reference pages bit for bit."""
    import paper_2608_02947_amd as atf
    B, h_kv, pages = 3, 2, 5
    n = pages * pt
    num_pages = B * pages + 3
    bt = _block_tables(B, pages, num_pages, seed=pt + d)
    k = W.random_bf16((B, n, h_kv, d), seed=d).to(DEV)
    v = W.random_bf16((B, n, h_kv, d), seed=d + 1).to(DEV)
    note(f"append paged pt={pt} d={d}")
    kpool = torch.zeros(atf.kpages_shape(num_pages, pt, h_kv, d), dtype=torch.bfloat16, device=DEV)
    vpool = torch.zeros(atf.vpages_shape(num_pages, pt, h_kv, d), dtype=torch.bfloat16, device=DEV)
    btd = torch.from_numpy(bt).to(DEV)
    cuts = [0, 7, pt + 21, n]
    for a, c in zip(cuts[:-1], cuts[1:]):
        atf.atf_cache_append_paged(k[:, a:c].contiguous(), v[:, a:c].contiguous(), kpool, vpool,
                                   btd, a)
    torch.cuda.synchronize()
    kref, vref = _ref_pages(k, v, bt, num_pages, pt)
    assert torch.equal(kpool.view(torch.int16), kref.view(torch.int16))
    assert torch.equal(vpool.view(torch.int16), vref.view(torch.int16))


def _paged_setup(n_ks, q_poss, pt, h_q, h_kv, d, base, seed, share_prefix=0):
    import paper_2608_02947_amd as atf
    B = len(n_ks)
    pages = max(1, -(-max(max(n_ks), 1) // pt))
    cap = pages * pt
    q, kc, vc = _ragged_inputs(n_ks, q_poss, cap, h_q, h_kv, d, base, seed, fill=0.0)
    if share_prefix:
        kc[1:, :share_prefix * pt] = kc[:1, :share_prefix * pt]
        vc[1:, :share_prefix * pt] = vc[:1, :share_prefix * pt]
    num_pages = B * pages + 2
    bt = _block_tables(B, pages, num_pages, seed, share_prefix)
    kpool = torch.full(atf.kpages_shape(num_pages, pt, h_kv, d), float("nan"), dtype=torch.bfloat16,
                       device=DEV)
    vpool = torch.full(atf.vpages_shape(num_pages, pt, h_kv, d), float("nan"), dtype=torch.bfloat16,
                       device=DEV)
    btd = torch.from_numpy(bt).to(DEV)
    atf.atf_cache_append_paged(kc.to(DEV), vc.to(DEV), kpool, vpool, btd, 0)
    return q, kc, vc, kpool, vpool, btd, cap


def _gpu_decode_paged(q, kpool, vpool, btd, n_ks, q_poss, max_n_k, win):
    import paper_2608_02947_amd as atf
    B, h_q, d = q.shape
    h_kv = kpool.shape[1]
    ws = torch.empty(atf.atf_decode_workspace_bytes(B, h_q, h_kv, max_n_k, d), dtype=torch.uint8,
                     device=DEV)
    o = torch.empty_like(q)
    lse = torch.empty((B, h_q), dtype=torch.float32, device=DEV)
    atf.atf_decode_paged(q, kpool, vpool, o, lse, btd, torch.tensor(n_ks, dtype=torch.int32, device=DEV),
                         torch.tensor(q_poss, dtype=torch.int32, device=DEV), max_n_k, win, ws)
    torch.cuda.synchronize()
    return o, lse


PAGED_CASES = [
    # n_k per row, q_pos per row, page tokens, h_q, h_kv, d, base, k, shared prefix pages
    ([1000, 1, 333, 0, 700], [1000, 1, 333, 0, 700], 64, 7, 1, 128, 1e4, 2.0, 0),
    ([2049, 100, 1500], [3000, 100, 900], 128, 8, 2, 64, 1e6, 2.0, 0),
    ([4096, 4000, 2300], [4096, 4000, 2300], 32, 6, 2, 128, 5e5, 2.0, 0),
    ([1500, 1700, 1300], [1500, 1700, 1300], 64, 12, 4, 128, 1e4, 2.0, 16),   # shared prefix
    ([999, 640], [999, 640], 128, 3, 1, 128, 1e4, math.inf, 0),                 # window off
]


@pytest.mark.parametrize("case", PAGED_CASES, ids=lambda c: f"B{len(c[0])}_pt{c[2]}_d{c[5]}_share{c[8]}")
def test_decode_paged_rows(case):
    n_ks, q_poss, pt, h_q, h_kv, d, base, kwin, share = case
    note(f"decode paged n_k={n_ks} q_pos={q_poss} pt={pt} d={d} share={share}")
    q, kc, vc, kpool, vpool, btd, cap = _paged_setup(n_ks, q_poss, pt, h_q, h_kv, d, base,
                                                     seed=sum(n_ks) % 997, share_prefix=share)
    win, _ = windows_for(d, base, kwin, None, n_ctx=max(q_poss) + 1)
    max_n_k = max(max(n_ks), 1)
    qd = q[:, 0].contiguous().to(DEV)
    o, lse = _gpu_decode_paged(qd, kpool, vpool, btd, n_ks, q_poss, max_n_k, win)
    # the same batch over contiguous caches takes the same plan and arithmetic
    o_c, lse_c = _gpu_decode_ragged(qd, kc.to(DEV), vc.to(DEV), n_ks, q_poss, max_n_k, win)
    assert torch.equal(o, o_c) and torch.equal(lse, lse_c)
    o, lse = to_f64(o), to_f64(lse)
    for b, (nk, qp) in enumerate(zip(n_ks, q_poss)):
        if nk == 0:
            assert np.all(o[b] == 0.0) and np.all(lse[b] == -np.inf)
            continue
        _, widths = windows_for(d, base, kwin, None, n_ctx=qp + 1)
        o_ref, lse_ref, _ = oracle.attend(q[b:b + 1], kc[b:b + 1, :nk], vc[b:b + 1, :nk], qp, widths)
        compare(o[b:b + 1], lse[b:b + 1], o_ref[:, 0], lse_ref[:, :, 0], f"paged row {b}")


@pytest.mark.parametrize("tag", ["default", "kinf"])
def test_decode_ragged_paged_llama_128k_bench_layout(tag):
    """The benchmark's ragged and paged batches at full size: Llama-3.2-3B-shaped rows of
    131072 .. 4096 keys, contiguous (atf_decode_ragged) and in 128-token pages, each row's
    pages shuffled in one pool and written row by row with atf_cache_append_paged
    (atf_decode_paged).  The two are bit-equal, and every (row, head) matches the oracle;
    the llama3-effective window and the window off, as timed."""
    import paper_2608_02947_amd as atf
    wl = W.WORKLOADS["llama3b_decode_128k"]
    d, B, pt = wl.head_dim, wl.batch, 128
    rows_l = [131072, 98304, 65536, 32768, 16384, 8192, 120000, 4096]
    note(f"decode ragged and paged llama 128K, benchmark layout, {tag}")
    inp = W.make_inputs(wl, device=DEV)
    counts = [-(-n // pt) for n in rows_l]
    perm = np.random.default_rng(20260099).permutation(sum(counts))
    bt = np.full((B, wl.n_k // pt), -1, dtype=np.int32)
    at = 0
    for b, c in enumerate(counts):
        bt[b, :c] = perm[at:at + c]
        at += c
    btd = torch.from_numpy(bt).to(DEV)
    kpool = torch.empty(atf.kpages_shape(sum(counts), pt, wl.h_kv, d), dtype=torch.bfloat16, device=DEV)
    vpool = torch.empty(atf.vpages_shape(sum(counts), pt, wl.h_kv, d), dtype=torch.bfloat16, device=DEV)
    for b, c in enumerate(counts):
        atf.atf_cache_append_paged(inp["k"][b:b + 1, :c * pt].contiguous(),
                                   inp["v"][b:b + 1, :c * pt].contiguous(), kpool, vpool,
                                   btd[b:b + 1], 0)
    th = W.workload_theta(wl)
    kwin = wl.k if tag == "default" else math.inf
    win, _ = windows_for(d, wl.rope_base, kwin, th, n_ctx=wl.n_k + 1)
    qd = inp["q"][:, 0].contiguous()
    o, lse = _gpu_decode_paged(qd, kpool, vpool, btd, rows_l, rows_l, wl.n_k, win)
    del kpool, vpool
    o_c, lse_c = _gpu_decode_ragged(qd, inp["k"], inp["v"], rows_l, rows_l, wl.n_k, win)
    assert torch.equal(o, o_c) and torch.equal(lse, lse_c)
    o, lse = to_f64(o), to_f64(lse)
    q_h, k_h, v_h = inp["q"].cpu(), inp["k"].cpu(), inp["v"].cpu()
    for b, nk in enumerate(rows_l):
        _, widths = windows_for(d, wl.rope_base, kwin, th, n_ctx=nk + 1)
        o_ref, lse_ref, _ = oracle.attend(q_h[b:b + 1], k_h[b:b + 1, :nk], v_h[b:b + 1, :nk],
                                          nk, widths)
        compare(o[b:b + 1], lse[b:b + 1], o_ref[:, 0], lse_ref[:, :, 0], f"bench row {b} {tag}")
