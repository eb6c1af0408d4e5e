"""Seeded synthetic workloads shared by the oracle side and the GPU side.

This module holds no arithmetic of the windowed-attention method: it only
defines the workload shapes, draws seeded Gaussian tensors, applies the RoPE
rotation that the method takes as already done (q~, k~ of Sec. 3.1), and
computes the llama3-style effective frequencies that a Llama-3.2-3B config
implies (Sec. 3.2 last paragraph: the window table uses the effective theta').

Input recipe (the same on every path):
  1. draw fp32 N(0, 1) Q, K, V in that order from one seeded generator,
     shaped [B, N, H, d] (BSHD);
  2. optionally scale both dims of K's rotary pair r by sigma_r (the Qwen 8K/32K
     workload ramps sigma from 0.5 at the highest frequency to 2.0 at the
     lowest);
  3. round to bf16;
  4. rotate Q at its positions and K at positions 0..N-1 in fp64 with the
     rotate-half convention (pair r = dims r and r + d/2);
  5. round to bf16.
The seeded tensors stand in for the paper's long documents: the window and the
term counts do not depend on the input values.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    kind: str            # "prefill" or "decode"
    batch: int
    n_q: int             # query rows (1 for decode)
    q_pos0: int          # position of query row 0
    n_k: int             # keys at positions 0 .. n_k - 1
    h_q: int
    h_kv: int
    head_dim: int
    rope_base: float
    k: float = 2.0
    llama3: bool = False          # llama3-style rope_scaling (factor 32, lf 1, hf 4, L 8192)
    k_pair_ramp: bool = False     # K pair std ramp 0.5 -> 2.0
    seed: int = 20260000

    @property
    def group(self) -> int:
        return self.h_q // self.h_kv


def _wl(**kw) -> Workload:
    return Workload(**kw)


# The paper's speed and quality shapes (Sec. 6-7); seeds 20260000 + config index.
WORKLOADS = {
    "qwen05b_prefill_1k": _wl(name="qwen05b_prefill_1k", kind="prefill", batch=1, n_q=1024,
                              q_pos0=0, n_k=1024, h_q=14, h_kv=2, head_dim=64, rope_base=1e6,
                              seed=20260000),
    "qwen05b_prefill_8k": _wl(name="qwen05b_prefill_8k", kind="prefill", batch=1, n_q=8192,
                              q_pos0=0, n_k=8192, h_q=14, h_kv=2, head_dim=64, rope_base=1e6,
                              k_pair_ramp=True, seed=20260001),
    "qwen05b_prefill_32k": _wl(name="qwen05b_prefill_32k", kind="prefill", batch=1, n_q=32768,
                               q_pos0=0, n_k=32768, h_q=14, h_kv=2, head_dim=64, rope_base=1e6,
                               k_pair_ramp=True, seed=20260001),
    "llama3b_prefill_32k": _wl(name="llama3b_prefill_32k", kind="prefill", batch=1, n_q=32768,
                               q_pos0=0, n_k=32768, h_q=24, h_kv=8, head_dim=128,
                               rope_base=5e5, llama3=True, seed=20260002),
    "llama3b_prefill_128k": _wl(name="llama3b_prefill_128k", kind="prefill", batch=1,
                                n_q=131072, q_pos0=0, n_k=131072, h_q=24, h_kv=8, head_dim=128,
                                rope_base=5e5, llama3=True, seed=20260002),
    "llama3b_decode_32k": _wl(name="llama3b_decode_32k", kind="decode", batch=8, n_q=1,
                              q_pos0=32768, n_k=32768, h_q=24, h_kv=8, head_dim=128,
                              rope_base=5e5, llama3=True, seed=20260003),
    "llama3b_decode_128k": _wl(name="llama3b_decode_128k", kind="decode", batch=8, n_q=1,
                               q_pos0=131072, n_k=131072, h_q=24, h_kv=8, head_dim=128,
                               rope_base=5e5, llama3=True, seed=20260003),
    "qwen7b1m_prefill_chunk": _wl(name="qwen7b1m_prefill_chunk", kind="prefill", batch=1,
                                  n_q=131072, q_pos0=1048576 - 131072, n_k=1048576, h_q=28,
                                  h_kv=4, head_dim=128, rope_base=1e7, seed=20260004),
    "qwen7b1m_decode": _wl(name="qwen7b1m_decode", kind="decode", batch=1, n_q=1,
                           q_pos0=1048576, n_k=1048576, h_q=28, h_kv=4, head_dim=128,
                           rope_base=1e7, seed=20260004),
}


def rope_theta(head_dim: int, base: float) -> torch.Tensor:
    """RoPE angular velocities theta_r = base^(-2r/d), r = 0 .. d/2-1, fp64."""
    r = torch.arange(head_dim // 2, dtype=torch.float64)
    return torch.pow(torch.tensor(float(base), dtype=torch.float64), -2.0 * r / head_dim)


def llama3_theta(head_dim: int, base: float, factor: float = 32.0, low_freq_factor: float = 1.0,
                 high_freq_factor: float = 4.0, original_context: int = 8192) -> torch.Tensor:
    """Effective theta'_r of the public Llama-3.1 rope_scaling rule (fp64).

    Wavelengths below original_context / high_freq_factor keep theta; those
    above original_context / low_freq_factor are divided by ``factor``; in
    between, theta' interpolates linearly in original_context / wavelength.
    """
    theta = rope_theta(head_dim, base)
    wavelen = 2.0 * math.pi / theta
    low_wl = original_context / low_freq_factor
    high_wl = original_context / high_freq_factor
    smooth = (original_context / wavelen - low_freq_factor) / (high_freq_factor - low_freq_factor)
    mid = (1.0 - smooth) * theta / factor + smooth * theta
    out = torch.where(wavelen < high_wl, theta, torch.where(wavelen > low_wl, theta / factor, mid))
    return out


def workload_theta(w: Workload) -> Optional[torch.Tensor]:
    """The effective theta' table to hand to both sides, or None for plain base^(-2r/d)."""
    if w.llama3:
        return llama3_theta(w.head_dim, w.rope_base)
    return None


def rotation_theta(w: Workload) -> torch.Tensor:
    t = workload_theta(w)
    return t if t is not None else rope_theta(w.head_dim, w.rope_base)


def rotate_half(x: torch.Tensor, positions: torch.Tensor, theta: torch.Tensor,
                chunk: int = 1 << 16) -> torch.Tensor:
    """RoPE-rotate x [B, N, H, d] (any float dtype) at positions [N]; returns bf16.

    Pair r = dims (r, r + d/2): x~_r = x_r cos(p th) - x_{r+h} sin(p th),
    x~_{r+h} = x_{r+h} cos(p th) + x_r sin(p th).  Done in fp64, chunked along N.
    """
    B, N, H, d = x.shape
    h = d // 2
    out = torch.empty(x.shape, dtype=torch.bfloat16, device=x.device)
    th = theta.to(device=x.device, dtype=torch.float64)
    for s in range(0, N, chunk):
        e = min(N, s + chunk)
        xs = x[:, s:e].to(torch.float64)
        ang = positions[s:e].to(device=x.device, dtype=torch.float64)[:, None] * th[None, :]
        c = torch.cos(ang)[None, :, None, :]
        sn = torch.sin(ang)[None, :, None, :]
        lo, hi = xs[..., :h], xs[..., h:]
        out[:, s:e, :, :h] = (lo * c - hi * sn).to(torch.bfloat16)
        out[:, s:e, :, h:] = (hi * c + lo * sn).to(torch.bfloat16)
    return out


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def make_inputs(w: Workload, device="cpu", seed: Optional[int] = None, n_k: Optional[int] = None,
                n_q: Optional[int] = None, q_pos0: Optional[int] = None, batch: Optional[int] = None):
    """Seeded bf16 inputs of workload ``w`` (sizes may be overridden for small tests).

    Returns dict with q [B, n_q, h_q, d], k [B, n_k, h_kv, d], v [B, n_k, h_kv, d]
    (bf16 on ``device``) plus the sizes used.  For decode workloads n_q = 1 and
    the query sits at position q_pos0 (= n_k by default).  Random draws on a
    CUDA device use that device's generator, so values differ from CPU draws of
    the same seed; both sides always consume the same tensors.
    """
    seed = w.seed if seed is None else seed
    B = w.batch if batch is None else batch
    nk = w.n_k if n_k is None else n_k
    nq = w.n_q if n_q is None else n_q
    if q_pos0 is None:
        q_pos0 = w.q_pos0 if (n_k is None and n_q is None) else (
            nk if w.kind == "decode" else max(0, nk - nq))
    d = w.head_dim
    g = _gen(seed, device)
    q = torch.randn((B, nq, w.h_q, d), generator=g, device=device, dtype=torch.float32)
    k = torch.randn((B, nk, w.h_kv, d), generator=g, device=device, dtype=torch.float32)
    v = torch.randn((B, nk, w.h_kv, d), generator=g, device=device, dtype=torch.float32)
    if w.k_pair_ramp:
        h = d // 2
        sig = 0.5 + 1.5 * torch.arange(h, dtype=torch.float32, device=device) / (h - 1)
        k = k * torch.cat([sig, sig])[None, None, None, :]
    q = q.to(torch.bfloat16)
    k = k.to(torch.bfloat16)
    v = v.to(torch.bfloat16)
    th = rotation_theta(w)
    qpos = torch.arange(q_pos0, q_pos0 + nq, dtype=torch.int64)
    kpos = torch.arange(0, nk, dtype=torch.int64)
    q = rotate_half(q, qpos, th)
    k = rotate_half(k, kpos, th)
    return {"q": q, "k": k, "v": v, "n_q": nq, "n_k": nk, "q_pos0": q_pos0, "batch": B}


def random_bf16(shape, seed: int, device="cpu", scale: float = 1.0) -> torch.Tensor:
    """Seeded N(0, scale^2) bf16 tensor (used by small edge-case tests)."""
    g = _gen(seed, device)
    return (torch.randn(shape, generator=g, device=device, dtype=torch.float32) * scale).to(
        torch.bfloat16)
