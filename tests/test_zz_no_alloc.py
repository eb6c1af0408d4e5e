"""GPU check of atf_decode_noalloc (the decode entry point that allocates nothing:
its split partials go to the library's own device scratch array) against
atf_decode with a caller workspace, through the C ABI: equal bits, and within the
oracle tolerances; two calls in a row, the second on a smaller input, so that the
second reads the scratch array the first left behind."""
import math

import numpy as np
import pytest
import torch

from conftest import gpu_available
import oracle
import workloads as W
from parity import compare, gpu_decode, note, pack_kcache, pack_vcache, to_f64, windows_for

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]

DEV = "cuda"


def _inputs(B, n_k, h_q, h_kv, d, base, seed):
    g = torch.Generator(device="cpu").manual_seed(seed)
    q = torch.randn((B, 1, h_q, d), generator=g).to(torch.bfloat16)
    k = torch.randn((B, n_k, h_kv, d), generator=g).to(torch.bfloat16)
    v = torch.randn((B, n_k, h_kv, d), generator=g).to(torch.bfloat16)
    th = W.rope_theta(d, base)
    q = W.rotate_half(q, torch.tensor([n_k]), th)
    k = W.rotate_half(k, torch.arange(0, n_k), th)
    return q, k, v


def _noalloc(qd, kp, vp, q_pos, win, n_k):
    import paper_2608_02947_amd as atf
    o = torch.empty_like(qd)
    lse = torch.empty(qd.shape[:2], dtype=torch.float32, device=DEV)
    atf.atf_decode_noalloc(qd, kp, vp, o, lse, q_pos, win, n_k=n_k)
    torch.cuda.synchronize()
    return o, lse


@pytest.mark.parametrize("kwin", [2.0, math.inf], ids=["k2", "kinf"])
def test_decode_noalloc_equals_decode_two_calls(kwin):
    cases = [  # B, n_k, h_q, h_kv, d, base: the second call is smaller than the first
        (2, 20000, 28, 4, 128, 1e7),
        (1, 3001, 14, 2, 64, 1e6),
    ]
    for B, n_k, h_q, h_kv, d, base in cases:
        note(f"decode_noalloc B={B} n_k={n_k} h_q={h_q} h_kv={h_kv} d={d} k={kwin}")
        q, k, v = _inputs(B, n_k, h_q, h_kv, d, base, seed=n_k + d)
        win, widths = windows_for(d, base, kwin, None, n_ctx=n_k + 1)
        qd, kp, vp = q[:, 0].contiguous().to(DEV), pack_kcache(k.to(DEV)), pack_vcache(v.to(DEV))
        o_na, lse_na = _noalloc(qd, kp, vp, n_k, win, n_k)
        o_ws, lse_ws = gpu_decode(qd, None, None, n_k, win, kp=kp, vp=vp, n_k=n_k)
        assert torch.equal(o_na, o_ws) and torch.equal(lse_na, lse_ws)
        o_ref, lse_ref, _ = oracle.attend(q, k, v, n_k, widths)
        compare(to_f64(o_na), to_f64(lse_na), o_ref[:, 0], lse_ref[:, :, 0],
                f"noalloc B={B} n_k={n_k} k={kwin}")


def test_decode_noalloc_rejects_sizes_beyond_the_scratch_array():
    import paper_2608_02947_amd as atf
    B, h_q, h_kv, d, n_k = 64, 64, 1, 128, 4096
    assert atf.atf_decode_workspace_bytes(B, h_q, h_kv, n_k, d) > atf.DECODE_NOALLOC_SCRATCH_BYTES
    qd = torch.zeros((B, h_q, d), dtype=torch.bfloat16, device=DEV)
    kp = torch.zeros(atf.kcache_shape(B, n_k, h_kv, d), dtype=torch.bfloat16, device=DEV)
    vp = torch.zeros(atf.vcache_shape(B, n_k, h_kv, d), dtype=torch.bfloat16, device=DEV)
    win = atf.Window(d, 1e4, 2.0)
    o = torch.empty_like(qd)
    lse = torch.empty((B, h_q), dtype=torch.float32, device=DEV)
    with pytest.raises(atf.AtfError) as e:
        atf.atf_decode_noalloc(qd, kp, vp, o, lse, n_k, win)
    assert e.value.code == atf.ATF_EWORKSPACE
