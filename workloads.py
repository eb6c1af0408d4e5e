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
                n_q: Optional[int] = None, q_pos0: Optional[int] = None, batch: Optional[int] = None,
                rotated: bool = True):
    """Seeded bf16 inputs of workload ``w`` (sizes may be overridden for small tests).

    Returns dict with q [B, n_q, h_q, d], k [B, n_k, h_kv, d], v [B, n_k, h_kv, d]
    (bf16 on ``device``) plus the sizes used.  For decode workloads n_q = 1 and
    the query sits at position q_pos0 (= n_k by default).  rotated=False returns q and k
    as drawn, before the RoPE rotation (the inputs of the unrotated-cache kernels,
    which rotate them as they read them).  Random draws on a
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
    if not rotated:
        return {"q": q, "k": k, "v": v, "n_q": nq, "n_k": nk, "q_pos0": q_pos0, "batch": B}
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


def stratified_rows(batch: int, n_q: int, h_q: int, q_pos0: int, group: int, pos_tiles,
                    widths, seed: int, n_random: int = 64, wave_rows: int = 32,
                    n_threshold_pairs: int = 24, min_rows: int = 256):
    """A stratified sample of (b, hq, i) query rows of a prefill, over all query heads,
    for checking full-size outputs row by row.  Returns an int64 array [n, 3] of
    (batch, query head, query row), sorted, without repeats.

    Strata (positions are q_pos0 + i; a workgroup of the prefill packs
    P = pos_tiles[k] consecutive positions x the `group` heads of one KV head into
    rows f -> (position f // group, head f % group), in blocks of `wave_rows` rows):
      - the first and the last 64 query rows, the head advancing by one per row, so
        that every head appears at both ends;
      - the first and the last row of 8 randomly chosen position tiles, for every
        tile size in pos_tiles;
      - the rows on either side of each seam between two `wave_rows`-row blocks
        (f = wave_rows*w - 1 and wave_rows*w) of 3 randomly chosen tiles per tile size;
      - for up to n_threshold_pairs pairs r whose width W_r = floor(widths[r]) is below
        the largest distance: positions p at which the first key the pair still
        reaches, p - W_r, is the first or last key of a 32-key block or of a 64-key
        tile (residues 0, 31, 32, 63 mod 64), two residues per pair;
      - n_random seeded random rows, and more until there are at least min_rows.
    This module holds no arithmetic of the method: `widths` and `pos_tiles` are inputs.
    """
    import numpy as np
    rng = np.random.default_rng(seed)
    picks = set()

    def add(i, h=None, b=None):
        if 0 <= i < n_q:
            picks.add((int(rng.integers(0, batch)) if b is None else int(b),
                       int(rng.integers(0, h_q)) if h is None else int(h) % h_q, int(i)))

    for t in range(min(64, n_q)):
        add(t, h=t)
        add(n_q - 1 - t, h=t)
    for P in pos_tiles:
        P = int(P)
        n_tiles = (n_q + P - 1) // P
        for t in rng.integers(0, n_tiles, size=8):
            add(int(t) * P)
            add(min(n_q, int(t) * P + P) - 1)
        rows = P * group
        n_kv = max(1, h_q // group)
        for t in rng.integers(0, n_tiles, size=3):
            g = int(rng.integers(0, n_kv))
            for w in range(1, (rows + wave_rows - 1) // wave_rows):
                for f in (wave_rows * w - 1, wave_rows * w):
                    if f < rows:
                        add(int(t) * P + f // group, h=g * group + f % group)
    w = np.asarray(widths, dtype=np.float64)
    p_lo, p_hi = q_pos0, q_pos0 + n_q - 1
    cand = [r for r in range(w.shape[0]) if np.isfinite(w[r]) and np.floor(w[r]) + 1 <= p_hi]
    if len(cand) > n_threshold_pairs:
        cand = sorted(rng.choice(cand, size=n_threshold_pairs, replace=False).tolist())
    for r in cand:
        W_r = int(np.floor(w[r]))
        lo = max(p_lo, W_r + 1)
        for res in rng.choice([0, 31, 32, 63], size=2, replace=False):
            p0 = int(rng.integers(lo, p_hi + 1))
            p = p0 - ((p0 - W_r - int(res)) % 64)
            if p < lo:
                p += 64
            if p <= p_hi:
                add(p - q_pos0)
    target = max(min_rows, len(picks) + n_random) if n_q * h_q * batch >= min_rows else 0
    while len(picks) < target:
        add(int(rng.integers(0, n_q)))
    return np.array(sorted(picks), dtype=np.int64).reshape(-1, 3)
