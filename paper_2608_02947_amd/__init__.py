"""Python binding of libatf.so: per-RoPE-wavelength windowed causal attention on MI355X.

Argument marshalling only.  Every step of prefill and decode runs in the HIP
kernels of ``libatf.so`` (built from ``csrc/`` by ``python
paper_2608_02947_amd/build.py``); torch supplies device memory and the current HIP
stream.  Importing this package loads the library and raises if it is missing:
there is no fallback path.

The functions carry the C names of ``include/atf.h``:

- :func:`atf_window_table`, :func:`atf_retention_profile`, :func:`atf_count_terms`
  -- host only.
- :func:`atf_prefill` -- windowed prefill (chunked via ``q_pos0``).
- :func:`atf_pack_kcache`, :func:`atf_kcache_chunk_pairs` -- decode K-cache layout.
- :func:`atf_pack_vcache`, :func:`atf_vcache_bytes` -- V-cache layout.
- :func:`atf_cache_append` -- write new tokens into both caches at a position.
- :func:`atf_decode_workspace_bytes`, :func:`atf_decode` -- split-KV decode.
- :func:`atf_decode_noalloc` -- the same without a workspace (library scratch array).
- :func:`atf_decode_ragged` -- the same for a batch of sequences of different lengths.
- :func:`atf_cache_append_paged`, :func:`atf_decode_paged` -- paged caches (block tables).
- :func:`atf_prefill_unrotated`, :func:`atf_decode_unrotated` (and its ragged and paged
  forms) -- the same from unrotated caches, RoPE applied as the kernels read them.
- :func:`atf_rotate_kcache` -- RoPE over a whole unrotated K cache in one pass, into a
  pre-rotated copy; :func:`atf_cache_append_rotated`, :func:`atf_cache_append_paged_rotated`
  -- the appends with RoPE on the way in.
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# ATF_LIB names another build of the same library (the sanitizer test of the host code
# loads one built with AddressSanitizer this way); by default the in-package libatf.so
LIB_PATH = os.environ.get("ATF_LIB") or os.path.join(_HERE, "libatf.so")

ATF_OK = 0
ATF_EINVAL = -1
ATF_EUNSUPPORTED = -2
ATF_EWORKSPACE = -3
ATF_EHIP = -4


class AtfError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"atf error {code}: {message}")
        self.code = code


class _CWindow(ctypes.Structure):
    _fields_ = [("head_dim", ctypes.c_int32), ("rope_base", ctypes.c_double),
                ("k", ctypes.c_double), ("inv_freq", ctypes.c_void_p),
                ("family", ctypes.c_int32), ("k_profile", ctypes.c_void_p),
                ("gamma", ctypes.c_double), ("a", ctypes.c_double),
                ("beta", ctypes.c_double), ("cap", ctypes.c_double),
                ("slice_pairs", ctypes.c_int32)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python paper_2608_02947_amd/build.py`")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    i32, i64, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    W = ctypes.POINTER(_CWindow)
    sig = {
        "atf_window_table": (ctypes.c_int, [W, P]),
        "atf_retention_profile": (ctypes.c_int, [i32, i32, ctypes.c_double, ctypes.c_double, P]),
        "atf_count_terms": (ctypes.c_int, [W, i64, i64, i64, P, P]),
        "atf_prefill": (ctypes.c_int, [P, P, P, P, P, i32, i64, i64, i64, i32, i32, i64, W, f32, P]),
        "atf_kcache_chunk_pairs": (ctypes.c_int32, [i32]),
        "atf_pack_kcache": (ctypes.c_int, [P, P, i32, i64, i32, i32, P]),
        "atf_vcache_bytes": (ctypes.c_size_t, [i32, i64, i32, i32]),
        "atf_pack_vcache": (ctypes.c_int, [P, P, i32, i64, i32, i32, P]),
        "atf_cache_append": (ctypes.c_int, [P, P, P, P, i32, i64, i64, i32, i32, i64, P]),
        "atf_decode_workspace_bytes": (ctypes.c_size_t, [i32, i32, i32, i64, i32]),
        "atf_decode": (ctypes.c_int, [P, P, P, P, P, i32, i64, i64, i32, i32, i64, W, f32, P,
                                      ctypes.c_size_t, P]),
        "atf_decode_noalloc": (ctypes.c_int, [P, P, P, P, P, i32, i64, i64, i32, i32, i64, W, f32,
                                              P]),
        "atf_decode_ragged": (ctypes.c_int, [P, P, P, P, P, i32, P, P, i64, i32, i32, i64, W, f32,
                                             P, ctypes.c_size_t, P]),
        "atf_cache_append_paged": (ctypes.c_int, [P, P, P, P, P, i32, i32, i32, i32, i64, i64,
                                                  i32, i32, P]),
        "atf_decode_paged": (ctypes.c_int, [P, P, P, P, P, i32, P, i32, i32, i32, P, P, i64, i32,
                                            i32, W, f32, P, ctypes.c_size_t, P]),
        "atf_rotate_kcache": (ctypes.c_int, [P, P, i32, i64, i32, i64, W, P, P]),
        "atf_cache_append_rotated": (ctypes.c_int, [P, P, P, P, i32, i64, i64, i32, i64, W, P, P]),
        "atf_cache_append_paged_rotated": (ctypes.c_int, [P, P, P, P, P, i32, i32, i32, i32, i64,
                                                          i64, i32, W, P, P]),
        "atf_prefill_unrotated": (ctypes.c_int, [P, P, P, P, P, i32, i64, i64, i64, i32, i32, i64,
                                                 W, P, f32, P]),
        "atf_decode_unrotated": (ctypes.c_int, [P, P, P, P, P, i32, i64, i64, i32, i32, i64, W, P,
                                                f32, P, ctypes.c_size_t, P]),
        "atf_decode_ragged_unrotated": (ctypes.c_int, [P, P, P, P, P, i32, P, P, i64, i32, i32, i64,
                                                       W, P, f32, P, ctypes.c_size_t, P]),
        "atf_decode_paged_unrotated": (ctypes.c_int, [P, P, P, P, P, i32, P, i32, i32, i32, P, P,
                                                      i64, i32, i32, W, P, f32, P, ctypes.c_size_t,
                                                      P]),
        "atf_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


_lib = _load()
EXPORTED = ("atf_window_table", "atf_retention_profile", "atf_count_terms", "atf_prefill", "atf_kcache_chunk_pairs",
            "atf_pack_kcache", "atf_vcache_bytes", "atf_pack_vcache", "atf_cache_append",
            "atf_decode_workspace_bytes", "atf_decode", "atf_decode_noalloc", "atf_decode_ragged",
            "atf_cache_append_paged",
            "atf_decode_paged", "atf_rotate_kcache", "atf_cache_append_rotated",
            "atf_cache_append_paged_rotated",
            "atf_prefill_unrotated", "atf_decode_unrotated", "atf_decode_ragged_unrotated",
            "atf_decode_paged_unrotated", "atf_last_error")


def library():
    """The loaded ctypes library (for tests of the raw C interface)."""
    return _lib


def atf_last_error() -> str:
    return _lib.atf_last_error().decode()


def _check(rc: int):
    if rc != ATF_OK:
        raise AtfError(rc, atf_last_error())


ATF_PROFILE_CONSTANT = 0
ATF_PROFILE_ARITHMETIC = 1
ATF_PROFILE_GEOMETRIC = 2
_PROFILE_KINDS = {"constant": ATF_PROFILE_CONSTANT, "arithmetic": ATF_PROFILE_ARITHMETIC,
                  "geometric": ATF_PROFILE_GEOMETRIC}


@dataclasses.dataclass
class Window:
    """atf_window: d, RoPE base B, retained periods k (+inf = off), optional theta'_r.

    Any of ``k_profile``, ``gamma``, ``a``, ``beta``, ``cap`` away from the default
    window selects the window family of App. A (eq:family):
    w_r = min(max(k_r lambda_r^gamma + a (r+1)/(d/2), beta), cap).
    ``slice_pairs`` = 8 selects the rounded slice of Sec. 3.3 (the kept low-frequency
    slice rounded up to 16-element MMA K-steps at each distance); 0 is the exact window.
    """
    head_dim: int
    rope_base: float
    k: float
    inv_freq: Optional[Sequence[float]] = None
    k_profile: Optional[Sequence[float]] = None
    gamma: float = 1.0
    a: float = 0.0
    beta: float = 0.0
    cap: float = math.inf
    slice_pairs: int = 0

    @property
    def family(self) -> bool:
        return (self.k_profile is not None or self.gamma != 1.0 or self.a != 0.0
                or self.beta != 0.0 or self.cap != math.inf)

    def as_c(self):
        def arr(x):
            if x is None:
                return None
            return np.ascontiguousarray(np.asarray(x, dtype=np.float64))
        th, kp = arr(self.inv_freq), arr(self.k_profile)
        for x, name in ((th, "inv_freq"), (kp, "k_profile")):
            if x is not None and x.shape != (self.head_dim // 2,):
                raise ValueError(f"{name} must hold head_dim/2 = {self.head_dim // 2} values")
        cw = _CWindow(int(self.head_dim), float(self.rope_base), float(self.k),
                      th.ctypes.data if th is not None else None, int(self.family),
                      kp.ctypes.data if kp is not None else None, float(self.gamma),
                      float(self.a), float(self.beta), float(self.cap),
                      int(self.slice_pairs))
        return cw, (th, kp)  # keep the arrays alive for the duration of the call


def atf_retention_profile(head_dim: int, kind: str, k_hi: float, k_lo: float = 0.0) -> np.ndarray:
    """k_r of App. A: "constant", "arithmetic" (variable-k: 16 -> 2) or "geometric"."""
    if kind not in _PROFILE_KINDS:
        raise ValueError(f"unknown profile kind {kind!r}")
    out = np.zeros(head_dim // 2 if head_dim >= 2 else 1, dtype=np.float64)
    _check(_lib.atf_retention_profile(head_dim, _PROFILE_KINDS[kind], float(k_hi), float(k_lo),
                                      out.ctypes.data))
    return out


def atf_window_table(window: Window) -> np.ndarray:
    cw, keep = window.as_c()
    out = np.zeros(window.head_dim // 2, dtype=np.int32)
    _check(_lib.atf_window_table(ctypes.byref(cw), out.ctypes.data))
    return out


def atf_count_terms(window: Window, n_q: int, q_pos0: int, n_k: int):
    """(retained terms, causal cells) per (batch, query head)."""
    cw, keep = window.as_c()
    r = ctypes.c_uint64()
    c = ctypes.c_uint64()
    _check(_lib.atf_count_terms(ctypes.byref(cw), n_q, q_pos0, n_k, ctypes.byref(r),
                                ctypes.byref(c)))
    return r.value, c.value


def atf_kcache_chunk_pairs(head_dim: int) -> int:
    return int(_lib.atf_kcache_chunk_pairs(head_dim))


def atf_decode_workspace_bytes(batch: int, h_q: int, h_kv: int, n_k: int, head_dim: int) -> int:
    return int(_lib.atf_decode_workspace_bytes(batch, h_q, h_kv, n_k, head_dim))


# ---------------------------------------------------------------------------
# device entry points (torch tensors on the current HIP device)
# ---------------------------------------------------------------------------
def _torch():
    import torch
    return torch


def _dev_ptr(t, dtype, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream_ptr(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def kcache_shape(batch: int, cache_tokens: int, h_kv: int, head_dim: int):
    """Shape of the pair-chunk-major K cache: [B, h_kv, d/16, cache_tokens, 16]."""
    return (batch, h_kv, head_dim // 16, cache_tokens, 16)


def atf_prefill(q, k_cache, v_cache, o, lse, q_pos0: int, window: Window,
                softmax_scale: float = 0.0, stream=None, n_k: Optional[int] = None):
    """q [B, n_q, h_q, d] bf16; k_cache [B, h_kv, d/16, C, 16] pair-chunk-major (see
    atf_pack_kcache); v_cache [B, h_kv, ceil(C/16), d, 16] (see atf_pack_vcache); o like
    q; lse [B, h_q, n_q] fp32.  C is the caches' token capacity; keys 0 .. n_k - 1 are
    used (n_k defaults to C)."""
    torch = _torch()
    B, n_q, h_q, d = q.shape
    if k_cache.dim() != 5:
        raise ValueError("atf_prefill: k_cache must be [B, h_kv, d/16, C, 16]")
    _, h_kv, _, cap, _ = k_cache.shape
    n_k = cap if n_k is None else int(n_k)
    if tuple(k_cache.shape) != kcache_shape(B, cap, h_kv, d) or \
            tuple(v_cache.shape) != vcache_shape(B, cap, h_kv, d) or \
            tuple(o.shape) != tuple(q.shape) or tuple(lse.shape) != (B, h_q, n_q):
        raise ValueError("atf_prefill: inconsistent shapes")
    cw, keep = window.as_c()
    rc = _lib.atf_prefill(_dev_ptr(q, torch.bfloat16, "q"), _dev_ptr(k_cache, torch.bfloat16, "k"),
                          _dev_ptr(v_cache, torch.bfloat16, "v"), _dev_ptr(o, torch.bfloat16, "o"),
                          _dev_ptr(lse, torch.float32, "lse"), B, n_q, n_k, q_pos0, h_q, h_kv,
                          cap, ctypes.byref(cw), float(softmax_scale), _stream_ptr(stream))
    _check(rc)


def atf_pack_kcache(k_bshd, k_pcm, stream=None):
    """k_bshd [B, C, h_kv, d] -> k_pcm [B, h_kv, d/16, C, 16] (bf16)."""
    torch = _torch()
    B, n_k, h_kv, d = k_bshd.shape
    if k_pcm.numel() != k_bshd.numel():
        raise ValueError("atf_pack_kcache: destination size mismatch")
    _check(_lib.atf_pack_kcache(_dev_ptr(k_bshd, torch.bfloat16, "k_bshd"),
                                _dev_ptr(k_pcm, torch.bfloat16, "k_pcm"), B, n_k, h_kv, d,
                                _stream_ptr(stream)))


def atf_vcache_bytes(batch: int, n_k: int, h_kv: int, head_dim: int) -> int:
    return int(_lib.atf_vcache_bytes(batch, n_k, h_kv, head_dim))


def vcache_shape(batch: int, n_k: int, h_kv: int, head_dim: int):
    """Shape of the packed V cache: [B, h_kv, ceil(n_k/16), d, 16]."""
    return (batch, h_kv, (n_k + 15) // 16, head_dim, 16)


def atf_cache_append(k_new, v_new, k_cache, v_cache, pos0: int, stream=None):
    """k_new, v_new [B, n_new, h_kv, d] -> positions pos0 .. pos0 + n_new - 1 of
    k_cache [B, h_kv, d/16, C, 16] and v_cache [B, h_kv, ceil(C/16), d, 16] (bf16)."""
    torch = _torch()
    B, n_new, h_kv, d = k_new.shape
    if k_cache.dim() != 5:
        raise ValueError("atf_cache_append: k_cache must be [B, h_kv, d/16, C, 16]")
    cap = k_cache.shape[3]
    if tuple(v_new.shape) != tuple(k_new.shape) or \
            tuple(k_cache.shape) != kcache_shape(B, cap, h_kv, d) or \
            tuple(v_cache.shape) != vcache_shape(B, cap, h_kv, d):
        raise ValueError("atf_cache_append: inconsistent shapes")
    _check(_lib.atf_cache_append(_dev_ptr(k_new, torch.bfloat16, "k_new"),
                                 _dev_ptr(v_new, torch.bfloat16, "v_new"),
                                 _dev_ptr(k_cache, torch.bfloat16, "k_cache"),
                                 _dev_ptr(v_cache, torch.bfloat16, "v_cache"),
                                 B, n_new, int(pos0), h_kv, d, cap, _stream_ptr(stream)))


def atf_pack_vcache(v_bshd, v_pack, stream=None):
    """v_bshd [B, n_k, h_kv, d] -> v_pack [B, h_kv, ceil(n_k/16), d, 16] (bf16)."""
    torch = _torch()
    B, n_k, h_kv, d = v_bshd.shape
    if tuple(v_pack.shape) != vcache_shape(B, n_k, h_kv, d):
        raise ValueError("atf_pack_vcache: destination shape mismatch")
    _check(_lib.atf_pack_vcache(_dev_ptr(v_bshd, torch.bfloat16, "v_bshd"),
                                _dev_ptr(v_pack, torch.bfloat16, "v_pack"), B, n_k, h_kv, d,
                                _stream_ptr(stream)))


def atf_decode(q, k_pcm, v_pack, o, lse, q_pos: int, window: Window, workspace,
               softmax_scale: float = 0.0, stream=None, n_k: Optional[int] = None):
    """q [B, h_q, d]; k_pcm [B, h_kv, d/16, C, 16]; v_pack [B, h_kv, ceil(C/16), d, 16];
    o [B, h_q, d]; lse [B, h_q]; workspace: uint8 device tensor of
    atf_decode_workspace_bytes().  C is the caches' token capacity; keys
    0 .. n_k - 1 are used (n_k defaults to C)."""
    torch = _torch()
    B, h_q, d = q.shape
    if k_pcm.dim() != 5:
        raise ValueError("atf_decode: k_pcm must be [B, h_kv, d/16, C, 16]")
    _, h_kv, _, cap, _ = k_pcm.shape
    n_k = cap if n_k is None else int(n_k)
    if tuple(o.shape) != tuple(q.shape) or tuple(lse.shape) != (B, h_q) or \
            tuple(k_pcm.shape) != kcache_shape(B, cap, h_kv, d) or \
            tuple(v_pack.shape) != vcache_shape(B, cap, h_kv, d):
        raise ValueError("atf_decode: inconsistent shapes")
    cw, keep = window.as_c()
    rc = _lib.atf_decode(_dev_ptr(q, torch.bfloat16, "q"), _dev_ptr(k_pcm, torch.bfloat16, "k"),
                         _dev_ptr(v_pack, torch.bfloat16, "v"), _dev_ptr(o, torch.bfloat16, "o"),
                         _dev_ptr(lse, torch.float32, "lse"), B, n_k, q_pos, h_q, h_kv, cap,
                         ctypes.byref(cw), float(softmax_scale),
                         _dev_ptr(workspace, torch.uint8, "workspace"), workspace.numel(),
                         _stream_ptr(stream))
    _check(rc)


# Size of the library's decode scratch array (ATF_DECODE_NOALLOC_SCRATCH_BYTES)
DECODE_NOALLOC_SCRATCH_BYTES = 16 << 20


def atf_decode_noalloc(q, k_pcm, v_pack, o, lse, q_pos: int, window: Window,
                       softmax_scale: float = 0.0, stream=None, n_k: Optional[int] = None):
    """atf_decode without a workspace: the split partials go to the library's own
    device scratch array (no allocation; calls on one device must not overlap)."""
    torch = _torch()
    B, h_q, d = q.shape
    if k_pcm.dim() != 5:
        raise ValueError("atf_decode_noalloc: k_pcm must be [B, h_kv, d/16, C, 16]")
    _, h_kv, _, cap, _ = k_pcm.shape
    n_k = cap if n_k is None else int(n_k)
    if tuple(o.shape) != tuple(q.shape) or tuple(lse.shape) != (B, h_q) or \
            tuple(k_pcm.shape) != kcache_shape(B, cap, h_kv, d) or \
            tuple(v_pack.shape) != vcache_shape(B, cap, h_kv, d):
        raise ValueError("atf_decode_noalloc: inconsistent shapes")
    cw, keep = window.as_c()
    rc = _lib.atf_decode_noalloc(_dev_ptr(q, torch.bfloat16, "q"),
                                 _dev_ptr(k_pcm, torch.bfloat16, "k"),
                                 _dev_ptr(v_pack, torch.bfloat16, "v"),
                                 _dev_ptr(o, torch.bfloat16, "o"),
                                 _dev_ptr(lse, torch.float32, "lse"), B, n_k, q_pos, h_q, h_kv,
                                 cap, ctypes.byref(cw), float(softmax_scale), _stream_ptr(stream))
    _check(rc)


def _rope_freq(rope_inv_freq, d):
    """Host double array [d/2] of rotation frequencies (pointer, owner), or (None, None)."""
    if rope_inv_freq is None:
        return None, None
    import numpy as np
    arr = np.ascontiguousarray(np.asarray(rope_inv_freq, dtype=np.float64))
    if arr.shape != (d // 2,):
        raise ValueError(f"rope_inv_freq must have d/2 = {d // 2} entries")
    return arr.ctypes.data_as(ctypes.c_void_p), arr


def atf_rotate_kcache(k_pcm, k_rot, window: Window, n_k: Optional[int] = None,
                      rope_inv_freq=None, stream=None):
    """k_pcm [B, h_kv, d/16, C, 16] unrotated -> k_rot (same shape) with key t turned to
    position t, for t < n_k (default C); later slots of k_rot are not written.  k_rot may
    be k_pcm itself (in place)."""
    torch = _torch()
    if k_pcm.dim() != 5 or tuple(k_rot.shape) != tuple(k_pcm.shape):
        raise ValueError("atf_rotate_kcache: caches must both be [B, h_kv, d/16, C, 16]")
    B, h_kv, nc, cap, _ = k_pcm.shape
    d = 16 * nc
    n_k = cap if n_k is None else int(n_k)
    cw, keep = window.as_c()
    fp, keep2 = _rope_freq(rope_inv_freq, d)
    _check(_lib.atf_rotate_kcache(_dev_ptr(k_pcm, torch.bfloat16, "k_pcm"),
                                  _dev_ptr(k_rot, torch.bfloat16, "k_rot"), B, n_k, h_kv, cap,
                                  ctypes.byref(cw), fp, _stream_ptr(stream)))


def atf_cache_append_rotated(k_new, v_new, k_cache, v_cache, pos0: int, window: Window,
                             rope_inv_freq=None, stream=None):
    """atf_cache_append with the new keys given unrotated: key t is turned to its cache
    position pos0 + t as it is written.  k_new, v_new [B, n_new, h_kv, d] bf16."""
    torch = _torch()
    B, n_new, h_kv, d = k_new.shape
    if k_cache.dim() != 5 or tuple(v_new.shape) != tuple(k_new.shape):
        raise ValueError("atf_cache_append_rotated: inconsistent shapes")
    cap = k_cache.shape[3]
    if tuple(k_cache.shape) != kcache_shape(B, cap, h_kv, d) or \
            tuple(v_cache.shape) != vcache_shape(B, cap, h_kv, d):
        raise ValueError("atf_cache_append_rotated: inconsistent cache shapes")
    cw, keep = window.as_c()
    fp, keep2 = _rope_freq(rope_inv_freq, d)
    _check(_lib.atf_cache_append_rotated(
        _dev_ptr(k_new, torch.bfloat16, "k_new"), _dev_ptr(v_new, torch.bfloat16, "v_new"),
        _dev_ptr(k_cache, torch.bfloat16, "k_cache"), _dev_ptr(v_cache, torch.bfloat16, "v_cache"),
        B, n_new, int(pos0), h_kv, cap, ctypes.byref(cw), fp, _stream_ptr(stream)))


def atf_prefill_unrotated(q, k_cache, v_cache, o, lse, q_pos0: int, window: Window,
                          softmax_scale: float = 0.0, stream=None, n_k: Optional[int] = None,
                          rope_inv_freq=None):
    """atf_prefill with q and the K cache UNROTATED: the kernel applies RoPE (query row i
    at q_pos0 + i, key j at position j) to q and to the key pairs the window keeps.
    rope_inv_freq: the rotation's theta_r (d/2 floats) or None for the window's
    frequencies."""
    torch = _torch()
    B, n_q, h_q, d = q.shape
    if k_cache.dim() != 5:
        raise ValueError("atf_prefill_unrotated: k_cache must be [B, h_kv, d/16, C, 16]")
    _, h_kv, _, cap, _ = k_cache.shape
    n_k = cap if n_k is None else int(n_k)
    if tuple(k_cache.shape) != kcache_shape(B, cap, h_kv, d) or \
            tuple(v_cache.shape) != vcache_shape(B, cap, h_kv, d) or \
            tuple(o.shape) != tuple(q.shape) or tuple(lse.shape) != (B, h_q, n_q):
        raise ValueError("atf_prefill_unrotated: inconsistent shapes")
    cw, keep = window.as_c()
    fp, keep2 = _rope_freq(rope_inv_freq, d)
    rc = _lib.atf_prefill_unrotated(
        _dev_ptr(q, torch.bfloat16, "q"), _dev_ptr(k_cache, torch.bfloat16, "k"),
        _dev_ptr(v_cache, torch.bfloat16, "v"), _dev_ptr(o, torch.bfloat16, "o"),
        _dev_ptr(lse, torch.float32, "lse"), B, n_q, n_k, q_pos0, h_q, h_kv, cap,
        ctypes.byref(cw), fp, float(softmax_scale), _stream_ptr(stream))
    _check(rc)


def atf_decode_unrotated(q, k_pcm, v_pack, o, lse, q_pos: int, window: Window, workspace,
                         softmax_scale: float = 0.0, stream=None, n_k: Optional[int] = None,
                         rope_inv_freq=None):
    """atf_decode with q and the K cache UNROTATED: the kernel applies RoPE (query at
    q_pos, key j at position j) to the pairs the window keeps.  rope_inv_freq: the
    rotation's theta_r (d/2 floats) or None for the window's frequencies."""
    torch = _torch()
    B, h_q, d = q.shape
    if k_pcm.dim() != 5:
        raise ValueError("atf_decode_unrotated: k_pcm must be [B, h_kv, d/16, C, 16]")
    _, h_kv, _, cap, _ = k_pcm.shape
    n_k = cap if n_k is None else int(n_k)
    if tuple(o.shape) != tuple(q.shape) or tuple(lse.shape) != (B, h_q) or \
            tuple(k_pcm.shape) != kcache_shape(B, cap, h_kv, d) or \
            tuple(v_pack.shape) != vcache_shape(B, cap, h_kv, d):
        raise ValueError("atf_decode_unrotated: inconsistent shapes")
    cw, keep = window.as_c()
    fp, keep2 = _rope_freq(rope_inv_freq, d)
    rc = _lib.atf_decode_unrotated(
        _dev_ptr(q, torch.bfloat16, "q"), _dev_ptr(k_pcm, torch.bfloat16, "k"),
        _dev_ptr(v_pack, torch.bfloat16, "v"), _dev_ptr(o, torch.bfloat16, "o"),
        _dev_ptr(lse, torch.float32, "lse"), B, n_k, q_pos, h_q, h_kv, cap, ctypes.byref(cw), fp,
        float(softmax_scale), _dev_ptr(workspace, torch.uint8, "workspace"), workspace.numel(),
        _stream_ptr(stream))
    _check(rc)


def atf_decode_ragged(q, k_pcm, v_pack, o, lse, n_k_rows, q_pos_rows, max_n_k: int,
                      window: Window, workspace, softmax_scale: float = 0.0, stream=None):
    """Ragged batch: q [B, h_q, d]; row b attends keys 0 .. min(q_pos_rows[b],
    n_k_rows[b] - 1) of its cache entry.  n_k_rows and q_pos_rows: int32 device tensors
    [B]; max_n_k bounds n_k_rows and sizes the workspace
    (atf_decode_workspace_bytes(B, h_q, h_kv, max_n_k, d)).  Other arguments as
    atf_decode."""
    torch = _torch()
    B, h_q, d = q.shape
    if k_pcm.dim() != 5:
        raise ValueError("atf_decode_ragged: k_pcm must be [B, h_kv, d/16, C, 16]")
    _, h_kv, _, cap, _ = k_pcm.shape
    if tuple(o.shape) != tuple(q.shape) or tuple(lse.shape) != (B, h_q) or \
            tuple(k_pcm.shape) != kcache_shape(B, cap, h_kv, d) or \
            tuple(v_pack.shape) != vcache_shape(B, cap, h_kv, d) or \
            tuple(n_k_rows.shape) != (B,) or tuple(q_pos_rows.shape) != (B,):
        raise ValueError("atf_decode_ragged: inconsistent shapes")
    cw, keep = window.as_c()
    rc = _lib.atf_decode_ragged(
        _dev_ptr(q, torch.bfloat16, "q"), _dev_ptr(k_pcm, torch.bfloat16, "k"),
        _dev_ptr(v_pack, torch.bfloat16, "v"), _dev_ptr(o, torch.bfloat16, "o"),
        _dev_ptr(lse, torch.float32, "lse"), B, _dev_ptr(n_k_rows, torch.int32, "n_k_rows"),
        _dev_ptr(q_pos_rows, torch.int32, "q_pos_rows"), int(max_n_k), h_q, h_kv, cap,
        ctypes.byref(cw), float(softmax_scale), _dev_ptr(workspace, torch.uint8, "workspace"),
        workspace.numel(), _stream_ptr(stream))
    _check(rc)


def kpages_shape(num_pages: int, page_tokens: int, h_kv: int, head_dim: int):
    """K page pool [num_pages, h_kv, d/16, page_tokens, 16] (pair-chunk-major pages)."""
    return (num_pages, h_kv, head_dim // 16, page_tokens, 16)


def vpages_shape(num_pages: int, page_tokens: int, h_kv: int, head_dim: int):
    """V page pool [num_pages, h_kv, page_tokens/16, d, 16] (16-token blocks)."""
    return (num_pages, h_kv, page_tokens // 16, head_dim, 16)


def _pages(k_pages, v_pages, fn):
    if k_pages.dim() != 5 or v_pages.dim() != 5:
        raise ValueError(f"{fn}: page pools must be 5-d (see kpages_shape, vpages_shape)")
    num_pages, h_kv, c16, pt, _ = k_pages.shape
    d = 16 * c16
    if tuple(k_pages.shape) != kpages_shape(num_pages, pt, h_kv, d) or \
            tuple(v_pages.shape) != vpages_shape(num_pages, pt, h_kv, d):
        raise ValueError(f"{fn}: inconsistent page pool shapes")
    return num_pages, h_kv, pt, d


def atf_cache_append_paged(k_new, v_new, k_pages, v_pages, block_table, pos0: int, stream=None):
    """Write k_new, v_new [B, n_new, h_kv, d] at row positions pos0 .. into the pages
    block_table [B, max_pages] (int32, device) names."""
    torch = _torch()
    num_pages, h_kv, pt, d = _pages(k_pages, v_pages, "atf_cache_append_paged")
    B, n_new, hk, dd = k_new.shape
    if tuple(v_new.shape) != tuple(k_new.shape) or hk != h_kv or dd != d or \
            block_table.dim() != 2 or block_table.shape[0] != B:
        raise ValueError("atf_cache_append_paged: inconsistent shapes")
    rc = _lib.atf_cache_append_paged(
        _dev_ptr(k_new, torch.bfloat16, "k_new"), _dev_ptr(v_new, torch.bfloat16, "v_new"),
        _dev_ptr(k_pages, torch.bfloat16, "k_pages"), _dev_ptr(v_pages, torch.bfloat16, "v_pages"),
        _dev_ptr(block_table, torch.int32, "block_table"), block_table.shape[1], num_pages, pt, B,
        n_new, int(pos0), h_kv, d, _stream_ptr(stream))
    _check(rc)


def atf_cache_append_paged_rotated(k_new, v_new, k_pages, v_pages, block_table, pos0: int,
                                   window: Window, rope_inv_freq=None, stream=None):
    """atf_cache_append_paged with the new keys given unrotated: key t of each row is
    turned to its position pos0 + t as it is written into its page."""
    torch = _torch()
    num_pages, h_kv, pt, d = _pages(k_pages, v_pages, "atf_cache_append_paged_rotated")
    B, n_new, hk, dd = k_new.shape
    if tuple(v_new.shape) != tuple(k_new.shape) or hk != h_kv or dd != d or \
            block_table.dim() != 2 or block_table.shape[0] != B or window.head_dim != d:
        raise ValueError("atf_cache_append_paged_rotated: inconsistent shapes")
    cw, keep = window.as_c()
    fp, keep2 = _rope_freq(rope_inv_freq, d)
    _check(_lib.atf_cache_append_paged_rotated(
        _dev_ptr(k_new, torch.bfloat16, "k_new"), _dev_ptr(v_new, torch.bfloat16, "v_new"),
        _dev_ptr(k_pages, torch.bfloat16, "k_pages"), _dev_ptr(v_pages, torch.bfloat16, "v_pages"),
        _dev_ptr(block_table, torch.int32, "block_table"), block_table.shape[1], num_pages, pt, B,
        n_new, int(pos0), h_kv, ctypes.byref(cw), fp, _stream_ptr(stream)))


def atf_decode_paged(q, k_pages, v_pages, o, lse, block_table, n_k_rows, q_pos_rows,
                     max_n_k: int, window: Window, workspace, softmax_scale: float = 0.0,
                     stream=None):
    """atf_decode_ragged over paged caches: row b's keys are read through
    block_table[b] (int32 [B, max_pages], device)."""
    torch = _torch()
    num_pages, h_kv, pt, d = _pages(k_pages, v_pages, "atf_decode_paged")
    B, h_q, dq = q.shape
    if dq != d or tuple(o.shape) != tuple(q.shape) or tuple(lse.shape) != (B, h_q) or \
            block_table.dim() != 2 or block_table.shape[0] != B or \
            tuple(n_k_rows.shape) != (B,) or tuple(q_pos_rows.shape) != (B,):
        raise ValueError("atf_decode_paged: inconsistent shapes")
    cw, keep = window.as_c()
    rc = _lib.atf_decode_paged(
        _dev_ptr(q, torch.bfloat16, "q"), _dev_ptr(k_pages, torch.bfloat16, "k_pages"),
        _dev_ptr(v_pages, torch.bfloat16, "v_pages"), _dev_ptr(o, torch.bfloat16, "o"),
        _dev_ptr(lse, torch.float32, "lse"), B, _dev_ptr(block_table, torch.int32, "block_table"),
        block_table.shape[1], num_pages, pt, _dev_ptr(n_k_rows, torch.int32, "n_k_rows"),
        _dev_ptr(q_pos_rows, torch.int32, "q_pos_rows"), int(max_n_k), h_q, h_kv,
        ctypes.byref(cw), float(softmax_scale), _dev_ptr(workspace, torch.uint8, "workspace"),
        workspace.numel(), _stream_ptr(stream))
    _check(rc)


def atf_decode_ragged_unrotated(q, k_pcm, v_pack, o, lse, n_k_rows, q_pos_rows, max_n_k: int,
                                window: Window, workspace, softmax_scale: float = 0.0,
                                stream=None, rope_inv_freq=None):
    """atf_decode_ragged with q and the K cache UNROTATED (row b's key t at position t,
    its query at q_pos_rows[b]); rope_inv_freq as atf_decode_unrotated."""
    torch = _torch()
    B, h_q, d = q.shape
    if k_pcm.dim() != 5:
        raise ValueError("atf_decode_ragged_unrotated: k_pcm must be [B, h_kv, d/16, C, 16]")
    _, h_kv, _, cap, _ = k_pcm.shape
    if tuple(o.shape) != tuple(q.shape) or tuple(lse.shape) != (B, h_q) or \
            tuple(k_pcm.shape) != kcache_shape(B, cap, h_kv, d) or \
            tuple(v_pack.shape) != vcache_shape(B, cap, h_kv, d) or \
            tuple(n_k_rows.shape) != (B,) or tuple(q_pos_rows.shape) != (B,):
        raise ValueError("atf_decode_ragged_unrotated: inconsistent shapes")
    cw, keep = window.as_c()
    fp, keep2 = _rope_freq(rope_inv_freq, d)
    rc = _lib.atf_decode_ragged_unrotated(
        _dev_ptr(q, torch.bfloat16, "q"), _dev_ptr(k_pcm, torch.bfloat16, "k"),
        _dev_ptr(v_pack, torch.bfloat16, "v"), _dev_ptr(o, torch.bfloat16, "o"),
        _dev_ptr(lse, torch.float32, "lse"), B, _dev_ptr(n_k_rows, torch.int32, "n_k_rows"),
        _dev_ptr(q_pos_rows, torch.int32, "q_pos_rows"), int(max_n_k), h_q, h_kv, cap,
        ctypes.byref(cw), fp, float(softmax_scale), _dev_ptr(workspace, torch.uint8, "workspace"),
        workspace.numel(), _stream_ptr(stream))
    _check(rc)


def atf_decode_paged_unrotated(q, k_pages, v_pages, o, lse, block_table, n_k_rows, q_pos_rows,
                               max_n_k: int, window: Window, workspace,
                               softmax_scale: float = 0.0, stream=None, rope_inv_freq=None):
    """atf_decode_paged with q and the K pages UNROTATED (RoPE at read time, row b's
    token t at position t); rope_inv_freq as atf_decode_unrotated."""
    torch = _torch()
    num_pages, h_kv, pt, d = _pages(k_pages, v_pages, "atf_decode_paged_unrotated")
    B, h_q, dq = q.shape
    if dq != d or tuple(o.shape) != tuple(q.shape) or tuple(lse.shape) != (B, h_q) or \
            block_table.dim() != 2 or block_table.shape[0] != B or \
            tuple(n_k_rows.shape) != (B,) or tuple(q_pos_rows.shape) != (B,):
        raise ValueError("atf_decode_paged_unrotated: inconsistent shapes")
    cw, keep = window.as_c()
    fp, keep2 = _rope_freq(rope_inv_freq, d)
    rc = _lib.atf_decode_paged_unrotated(
        _dev_ptr(q, torch.bfloat16, "q"), _dev_ptr(k_pages, torch.bfloat16, "k_pages"),
        _dev_ptr(v_pages, torch.bfloat16, "v_pages"), _dev_ptr(o, torch.bfloat16, "o"),
        _dev_ptr(lse, torch.float32, "lse"), B, _dev_ptr(block_table, torch.int32, "block_table"),
        block_table.shape[1], num_pages, pt, _dev_ptr(n_k_rows, torch.int32, "n_k_rows"),
        _dev_ptr(q_pos_rows, torch.int32, "q_pos_rows"), int(max_n_k), h_q, h_kv,
        ctypes.byref(cw), fp, float(softmax_scale), _dev_ptr(workspace, torch.uint8, "workspace"),
        workspace.numel(), _stream_ptr(stream))
    _check(rc)
