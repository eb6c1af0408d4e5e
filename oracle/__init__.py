"""fp64 CPU oracle for per-RoPE-wavelength windowed causal attention.

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  It shares no code
with the GPU library and never imports it.

The arithmetic lives in ``oracle.c`` (plain C, fp64, OpenMP over rows); this
module only marshals numpy arrays into it:

- :func:`window_widths` -- w_r = min(k * lambda_r, N), lambda_r = 2*pi/theta_r
  (Sec. 3.1 eq:lambda, Sec. 3.2 eq:window).
- :func:`retention_profile` -- the per-pair retention k_r of App. A: constant,
  k-arithmetic (the variable-k profile 16 -> 2 is one) or k-geometric.
- :func:`family_widths` -- the window family of App. A eq:family.
- :func:`scores` -- the windowed, scaled score matrix of one (batch, head)
  (Sec. 3.1 eq:pair with the keep rule of Sec. 3.2).
- :func:`attend` -- windowed causal attention, plain two-pass softmax, for all
  or a sample of query rows; O, LSE and the per-row retained-term count.
- :func:`count_terms` -- the retained-term and causal-cell counts of Sec. 4.
- :func:`rope_rotate` -- the RoPE rotation of Sec. 3.1 (pair r rotated by
  position * theta_r, rotate-half pairing), in numpy fp64: the reference for
  decode from unrotated caches (App. B, rotation at read time).

Every function whose result is checked against something other than itself is
listed in ``tests/test_oracle.py``; none is "parity unpinned".
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

_F64 = 0
_BF16 = 1


def build(force: bool = True) -> str:
    """Compile ``oracle.c`` with gcc into ``liboracle.so`` next to it."""
    if force or not os.path.exists(_LIB_PATH):
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
               "-Wall", "-Wextra", "-o", _LIB_PATH, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
    return _LIB_PATH


_lib = None


def _load():
    """Load liboracle.so, or the library named by ORACLE_LIB (the mutation test of the
    pins loads deliberately broken builds of oracle.c this way)."""
    global _lib
    if _lib is None:
        path = os.environ.get("ORACLE_LIB") or _LIB_PATH
        if path == _LIB_PATH and not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(path)
        p = ctypes.c_void_p
        i64 = ctypes.c_int64
        dbl = ctypes.c_double
        lib.oracle_window_widths.argtypes = [i64, dbl, dbl, p, dbl, p]
        lib.oracle_family_widths.argtypes = [i64, dbl, p, p, dbl, dbl, dbl, dbl, p]
        lib.oracle_scores.argtypes = [p, p, ctypes.c_int, i64, i64, i64, i64, i64, i64,
                                      i64, p, i64, dbl, i64, i64, p]
        lib.oracle_attend.argtypes = [p, p, p, ctypes.c_int, i64, i64, i64, i64, i64, i64,
                                      i64, p, i64, dbl, i64, p, p, p, p, ctypes.c_int]
        lib.oracle_count_terms.argtypes = [p, i64, i64, i64, i64, p, p]
        lib.oracle_count_terms_by_distance.argtypes = [p, i64, i64, i64, i64, i64, p, p]
        for f in (lib.oracle_window_widths, lib.oracle_family_widths, lib.oracle_scores,
                  lib.oracle_attend, lib.oracle_count_terms, lib.oracle_count_terms_by_distance):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _as_input(x):
    """Return (contiguous ndarray, dtype code): bf16 bits as uint16, else float64."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            x = x.detach().cpu().contiguous()
            if x.dtype == torch.bfloat16:
                return x.view(torch.int16).numpy().view(np.uint16), _BF16
            return x.to(torch.float64).numpy(), _F64
    except ImportError:  # pragma: no cover
        pass
    x = np.ascontiguousarray(x)
    if x.dtype == np.uint16:
        return x, _BF16
    return np.ascontiguousarray(x, dtype=np.float64), _F64


def window_widths(head_dim: int, rope_base: float, k: float, theta=None,
                  n_ctx: float = math.inf) -> np.ndarray:
    """w_r = min(k * 2*pi/theta_r, n_ctx) for r < head_dim/2 (eq:window)."""
    lib = _load()
    w = np.empty(head_dim // 2, dtype=np.float64)
    th = None
    if theta is not None:
        th = np.ascontiguousarray(theta, dtype=np.float64)
        assert th.shape == (head_dim // 2,)
    rc = lib.oracle_window_widths(head_dim, float(rope_base), float(k),
                                  _ptr(th) if th is not None else None, float(n_ctx), _ptr(w))
    if rc != 0:
        raise ValueError("oracle_window_widths: bad arguments")
    return w


def retention_profile(head_dim: int, kind: str, k_hi: float, k_lo: float = None) -> np.ndarray:
    """Per-pair retention k_r, r = 0 (highest frequency) .. d/2 - 1 (App. A).

    "constant": k_r = k_hi.  "arithmetic": k_r falls by the same amount per
    pair, from k_hi at r = 0 to k_lo at r = d/2 - 1 (the variable-k profile of
    the main text is k_hi = 16, k_lo = 2).  "geometric": k_r falls by the same
    ratio per pair between the same end points.  With one pair, k_r = k_hi.
    """
    n = head_dim // 2
    r = np.arange(n, dtype=np.float64)
    if kind == "constant":
        return np.full(n, float(k_hi))
    span = max(n - 1, 1)
    if kind == "arithmetic":
        return k_hi - (k_hi - k_lo) * r / span
    if kind == "geometric":
        return k_hi * (k_lo / k_hi) ** (r / span)
    raise ValueError(kind)


def family_widths(head_dim: int, rope_base: float, k_profile, gamma: float = 1.0,
                  a: float = 0.0, beta: float = 0.0, cap: float = math.inf,
                  theta=None) -> np.ndarray:
    """w_r = min(max(k_r lambda_r^gamma + a (r+1)/(d/2), beta), cap) (App. A eq:family);
    a position-free pair (theta_r = 0) gets +inf."""
    lib = _load()
    kp = np.ascontiguousarray(np.broadcast_to(np.asarray(k_profile, dtype=np.float64),
                                              (head_dim // 2,)))
    th = None
    if theta is not None:
        th = np.ascontiguousarray(theta, dtype=np.float64)
        assert th.shape == (head_dim // 2,)
    w = np.empty(head_dim // 2, dtype=np.float64)
    rc = lib.oracle_family_widths(head_dim, float(rope_base), _ptr(th) if th is not None else None,
                                  _ptr(kp), float(gamma), float(a), float(beta), float(cap),
                                  _ptr(w))
    if rc != 0:
        raise ValueError("oracle_family_widths: bad arguments")
    return w


def scores(q, k, q_pos0: int, widths, b: int = 0, hq: int = 0, scale=None,
           atom: int = 0) -> np.ndarray:
    """Windowed scaled scores [n_q, n_k] of one (batch, query head); -inf above the diagonal.
    atom > 0: the rounded slice of Sec. 3.3 (kept slice rounded up to atom-pair steps)."""
    lib = _load()
    qa, dt = _as_input(q)
    ka, dt2 = _as_input(k)
    assert dt == dt2
    B, n_q, h_q, d = qa.shape
    _, n_k, h_kv, _ = ka.shape
    w = np.ascontiguousarray(widths, dtype=np.float64)
    sc = 1.0 / math.sqrt(d) if scale is None else float(scale)
    out = np.empty((n_q, n_k), dtype=np.float64)
    rc = lib.oracle_scores(_ptr(qa), _ptr(ka), dt, B, n_q, n_k, q_pos0, h_q, h_kv, d,
                           _ptr(w), int(atom), sc, b, hq, _ptr(out))
    if rc != 0:
        raise ValueError("oracle_scores: bad arguments")
    return out


def all_rows(batch: int, n_q: int, h_q: int) -> np.ndarray:
    """(b, hq, i) triples of every query row, in [B][n_q][h_q] order."""
    b, i, h = np.meshgrid(np.arange(batch), np.arange(n_q), np.arange(h_q), indexing="ij")
    return np.stack([b.ravel(), h.ravel(), i.ravel()], axis=1).astype(np.int64)


def attend(q, k, v, q_pos0: int, widths, scale=None, rows=None, threads: int = 0,
           atom: int = 0):
    """Windowed causal attention in fp64.

    atom > 0 applies the rounded slice of Sec. 3.3: at each distance the kept
    low-frequency slice is rounded up to a whole number of atom-pair K-steps.

    q [B, n_q, h_q, d], k/v [B, n_k, h_kv, d] (bf16 torch tensors, uint16 bf16
    bits, or float arrays).  ``rows`` is an (n, 3) array of (b, hq, i); None
    means all rows, and the outputs are then shaped o [B, n_q, h_q, d],
    lse [B, h_q, n_q], terms [B, h_q, n_q].  Otherwise o [n, d], lse [n],
    terms [n] in the order of ``rows``.
    """
    lib = _load()
    qa, dt = _as_input(q)
    ka, dt2 = _as_input(k)
    va, dt3 = _as_input(v)
    assert dt == dt2 == dt3, "q, k, v must share one element type"
    B, n_q, h_q, d = qa.shape
    _, n_k, h_kv, _ = ka.shape
    w = np.ascontiguousarray(widths, dtype=np.float64)
    assert w.shape == (d // 2,)
    sc = 1.0 / math.sqrt(d) if scale is None else float(scale)
    full = rows is None
    r = all_rows(B, n_q, h_q) if full else np.ascontiguousarray(rows, dtype=np.int64)
    n = r.shape[0]
    o = np.empty((n, d), dtype=np.float64)
    lse = np.empty(n, dtype=np.float64)
    terms = np.empty(n, dtype=np.uint64)
    rc = lib.oracle_attend(_ptr(qa), _ptr(ka), _ptr(va), dt, B, n_q, n_k, q_pos0, h_q, h_kv, d,
                           _ptr(w), int(atom), sc, n, _ptr(r), _ptr(o), _ptr(lse), _ptr(terms),
                           int(threads))
    if rc != 0:
        raise ValueError("oracle_attend: bad arguments")
    if full:
        o = o.reshape(B, n_q, h_q, d)
        lse = lse.reshape(B, n_q, h_q).transpose(0, 2, 1).copy()
        terms = terms.reshape(B, n_q, h_q).transpose(0, 2, 1).copy()
    return o, lse, terms


def count_terms(widths, n_q: int, q_pos0: int, n_k: int, atom: int = 0, by_distance=None):
    """(retained terms, causal cells) of one (batch, query head), Sec. 4.

    atom == 0: per pair and row in closed form.  atom > 0 (the rounded slice of
    Sec. 3.3), or by_distance=True: summed over distances z with the pairs kept at z.
    """
    lib = _load()
    w = np.ascontiguousarray(widths, dtype=np.float64)
    ret = np.zeros(1, dtype=np.uint64)
    cau = np.zeros(1, dtype=np.uint64)
    if atom > 0 or by_distance:
        rc = lib.oracle_count_terms_by_distance(_ptr(w), w.shape[0], int(atom), n_q, q_pos0,
                                                n_k, _ptr(ret), _ptr(cau))
    else:
        rc = lib.oracle_count_terms(_ptr(w), w.shape[0], n_q, q_pos0, n_k, _ptr(ret), _ptr(cau))
    if rc != 0:
        raise ValueError("oracle_count_terms: bad arguments")
    return int(ret[0]), int(cau[0])


def rope_rotate(x, positions, theta):
    """RoPE rotation in fp64 (Sec. 3.1): x [..., n, h, d] at positions [n]; pair r
    is dims (r, r + d/2), rotated by angle positions[i] * theta[r]:
    x'_r = x_r cos - x_{r+d/2} sin, x'_{r+d/2} = x_{r+d/2} cos + x_r sin.
    x may be a bf16 torch tensor, bf16 bits as uint16, or a float array."""
    xa, dt = _as_input(x)
    if dt == _BF16:
        xa = (xa.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    d = xa.shape[-1]
    h = d // 2
    pos = np.asarray(positions, dtype=np.float64)
    th = np.asarray(theta, dtype=np.float64)
    assert th.shape == (h,) and pos.shape == (xa.shape[-3],)
    ang = pos[:, None] * th[None, :]                 # [n, h]
    c = np.cos(ang)[:, None, :]                      # [n, 1, h]: the same for every head
    s_ = np.sin(ang)[:, None, :]
    a, b = xa[..., :h], xa[..., h:]
    out = np.empty_like(xa)
    out[..., :h] = a * c - b * s_
    out[..., h:] = b * c + a * s_
    return out
