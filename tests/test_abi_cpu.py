"""Host-side checks of libatf.so that need no GPU.

- the library loads and exports every function include/atf.h declares;
- atf_window_table equals floor(k * lambda_r) from the oracle, bit-exact;
- atf_count_terms (closed form per pair) equals the oracle's count and brute
  force, bit-exact, for every workload shape and for random small cases;
- every validation error is returned before anything is launched.
No call here reaches a kernel launch.
"""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import workloads as W
from conftest import ROOT

atf = pytest.importorskip("paper_2608_02947_amd")


def header_functions():
    src = open(os.path.join(ROOT, "include", "atf.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(atf_[a-z_0-9]+)\s*\(", src)))


def test_exports_every_declared_symbol():
    names = header_functions()
    assert "atf_prefill" in names and "atf_decode" in names and "atf_count_terms" in names
    lib = ctypes.CDLL(atf.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(atf.EXPORTED)


def _oracle_thresholds(oracle_lib, wl_or_args):
    d, base, k, theta = wl_or_args
    w = oracle_lib.window_widths(d, base, k, theta)
    return np.minimum(np.floor(w), 2 ** 31 - 1).astype(np.int64)


@pytest.mark.parametrize("name", sorted(W.WORKLOADS))
@pytest.mark.parametrize("kwin", [2.0, 0.5, 7.0, math.inf])
def test_window_table_matches_oracle(oracle_lib, name, kwin):
    wl = W.WORKLOADS[name]
    th = W.workload_theta(wl)
    th_np = th.numpy() if th is not None else None
    win = atf.Window(wl.head_dim, wl.rope_base, kwin, th_np)
    got = atf.atf_window_table(win).astype(np.int64)
    exp = _oracle_thresholds(oracle_lib, (wl.head_dim, wl.rope_base, kwin, th_np))
    assert np.array_equal(got, exp)
    if math.isinf(kwin):
        assert np.all(got == 2 ** 31 - 1)


@pytest.mark.parametrize("name", sorted(W.WORKLOADS))
def test_count_matches_oracle_for_workloads(oracle_lib, name):
    wl = W.WORKLOADS[name]
    th = W.workload_theta(wl)
    th_np = th.numpy() if th is not None else None
    win = atf.Window(wl.head_dim, wl.rope_base, wl.k, th_np)
    got = atf.atf_count_terms(win, wl.n_q, wl.q_pos0, wl.n_k)
    w = oracle_lib.window_widths(wl.head_dim, wl.rope_base, wl.k, th_np,
                                 n_ctx=max(wl.n_k, wl.q_pos0 + wl.n_q))
    assert got == oracle_lib.count_terms(w, wl.n_q, wl.q_pos0, wl.n_k)


def test_count_known_values():
    # values of the 1K Qwen workload and of the 1M chunk (per head), exact
    wl = W.WORKLOADS["qwen05b_prefill_1k"]
    assert atf.atf_count_terms(atf.Window(64, 1e6, 2.0), 1024, 0, 1024) == (12986186, 524800)
    assert atf.atf_count_terms(atf.Window(128, 1e7, 2.0), 131072, 917504, 1048576) == \
        (2928556179456, 128849084416)
    assert wl.n_q == 1024


@pytest.mark.parametrize("seed", range(25))
def test_count_random_vs_oracle_and_brute(oracle_lib, seed):
    rng = np.random.default_rng(seed)
    d = int(rng.choice([2, 4, 8, 64, 128]))
    base = float(rng.uniform(1.5, 1e6))
    kwin = float(rng.choice([0.01, 0.2, 1.0, 2.0, 9.0, math.inf]))
    n_q = int(rng.integers(0, 300))
    q0 = int(rng.integers(0, 300))
    n_k = int(rng.integers(0, 400))
    theta = None
    if rng.random() < 0.3:
        theta = np.sort(rng.uniform(0.0, 2.0, d // 2))[::-1].copy()
        theta[-1] = 0.0 if rng.random() < 0.5 else theta[-1]
    win = atf.Window(d, base, kwin, theta)
    got = atf.atf_count_terms(win, n_q, q0, n_k)
    w = oracle_lib.window_widths(d, base, kwin, theta)
    assert got == oracle_lib.count_terms(w, n_q, q0, n_k)
    if d <= 8 and n_q * n_k <= 4000:
        T = C = 0
        for i in range(n_q):
            p = q0 + i
            for j in range(min(p, n_k - 1) + 1):
                C += 1
                T += int(np.sum(p - j <= np.floor(w)))
        assert got == (T, C)


def test_window_validation():
    for bad in (atf.Window(63, 1e4, 2.0), atf.Window(0, 1e4, 2.0), atf.Window(8, 1.0, 2.0),
                atf.Window(8, 1e4, 0.0), atf.Window(8, 1e4, float("nan")),
                atf.Window(8, 1e4, 2.0, [1.0, -1.0, 0.5, 0.1]),
                atf.Window(8, 1e4, 2.0, [1.0, float("nan"), 0.5, 0.1])):
        with pytest.raises(atf.AtfError) as e:
            atf.atf_window_table(bad)
        assert e.value.code == atf.ATF_EINVAL
        assert "window" in atf.atf_last_error()
    # position-free pair and an infinite window clamp to 2^31 - 1
    t = atf.atf_window_table(atf.Window(4, 10.0, 2.0, [1.0, 0.0]))
    assert t[1] == 2 ** 31 - 1 and t[0] == math.floor(4 * math.pi)


# window family of App. A: the library's table and counts against the oracle's
# widths, built independently on each side
FAMILY_CASES = {
    # name: (d, base, theta-kind, profile (kind, hi, lo), gamma, a, beta, cap)
    "var16to2_qwen05b": (64, 1e6, None, ("arithmetic", 16.0, 2.0), 1.0, 0.0, 0.0, math.inf),
    "var16to2_qwen7b": (128, 1e7, None, ("arithmetic", 16.0, 2.0), 1.0, 0.0, 0.0, math.inf),
    "var16to2_llama3": (128, 5e5, "llama3", ("arithmetic", 16.0, 2.0), 1.0, 0.0, 0.0, math.inf),
    "geo16to2_qwen7b": (128, 1e7, None, ("geometric", 16.0, 2.0), 1.0, 0.0, 0.0, math.inf),
    "k64_qwen7b": (128, 1e7, None, ("constant", 64.0, 0.0), 1.0, 0.0, 0.0, math.inf),
    "cap_0.25N_32k": (64, 1e6, None, ("constant", 2.0, 0.0), 1.0, 0.0, 0.0, 8192.0),
    "floor_and_cap": (128, 5e5, None, ("constant", 2.0, 0.0), 1.0, 0.0, 100.0, 50000.0),
    "gamma_0.8": (128, 1e7, None, ("constant", 2.0, 0.0), 0.8, 0.0, 0.0, math.inf),
    "gamma_1.25": (64, 1e6, None, ("constant", 2.0, 0.0), 1.25, 0.0, 0.0, math.inf),
    "sliding_300": (64, 1e6, None, ("constant", 0.0, 0.0), 1.0, 0.0, 300.0, 300.0),
    "linear_4096": (128, 1e7, None, ("constant", 0.0, 0.0), 1.0, 4096.0, 0.0, math.inf),
    "additive_and_var": (64, 1e4, None, ("arithmetic", 8.0, 1.0), 1.0, 77.5, 0.0, math.inf),
}


def _family_pair(oracle_lib, case):
    d, base, tk, (kind, hi, lo), gamma, a, beta, cap = FAMILY_CASES[case]
    th = W.llama3_theta(d, base).numpy() if tk == "llama3" else None
    prof = oracle_lib.retention_profile(d, kind, hi, lo)
    widths = oracle_lib.family_widths(d, base, prof, gamma=gamma, a=a, beta=beta, cap=cap,
                                      theta=th)
    win = atf.Window(d, base, hi, th, k_profile=atf.atf_retention_profile(d, kind, hi, lo),
                     gamma=gamma, a=a, beta=beta, cap=cap)
    return win, widths


@pytest.mark.parametrize("case", sorted(FAMILY_CASES))
def test_family_table_and_counts_match_oracle(oracle_lib, case):
    win, widths = _family_pair(oracle_lib, case)
    got = atf.atf_window_table(win).astype(np.int64)
    exp = np.minimum(np.floor(widths), 2 ** 31 - 1).astype(np.int64)
    assert np.array_equal(got, exp)
    for n_q, q0, n_k in [(16384, 0, 16384), (4096, 126976, 131072), (1, 1 << 20, 1 << 20),
                         (300, 0, 200)]:
        assert atf.atf_count_terms(win, n_q, q0, n_k) == oracle_lib.count_terms(widths, n_q, q0, n_k)


@pytest.mark.parametrize("kind", ["constant", "arithmetic", "geometric"])
@pytest.mark.parametrize("d", [2, 8, 64, 128])
def test_retention_profile_matches_oracle(oracle_lib, kind, d):
    got = atf.atf_retention_profile(d, kind, 16.0, 2.0)
    np.testing.assert_allclose(got, oracle_lib.retention_profile(d, kind, 16.0, 2.0),
                               rtol=1e-14, atol=0)


def test_family_defaults_and_validation():
    # the zero-initialised tail (family == 0) is the default window
    cw, keep = atf.Window(64, 1e6, 2.0).as_c()
    assert cw.family == 0 and not cw.k_profile and cw.gamma == 1.0
    cw.gamma, cw.beta = 7.0, 1e9  # ignored while family == 0
    t = np.zeros(32, dtype=np.int32)
    assert atf.library().atf_window_table(ctypes.byref(cw), t.ctypes.data) == 0
    assert np.array_equal(t, atf.atf_window_table(atf.Window(64, 1e6, 2.0)))
    # the family at its default point equals the default window
    same = atf.Window(64, 1e6, 2.0, k_profile=np.full(32, 2.0))
    assert same.family
    assert np.array_equal(atf.atf_window_table(same), t)
    # k = 0 is allowed only in the family
    assert np.all(atf.atf_window_table(atf.Window(8, 1e4, 0.0, beta=5.0)) == 5)
    bad = [atf.Window(8, 1e4, 2.0, gamma=math.inf), atf.Window(8, 1e4, 2.0, gamma=math.nan),
           atf.Window(8, 1e4, 2.0, a=-1.0), atf.Window(8, 1e4, 2.0, a=math.inf),
           atf.Window(8, 1e4, 2.0, beta=-1.0), atf.Window(8, 1e4, 2.0, beta=math.inf),
           atf.Window(8, 1e4, 2.0, cap=-1.0), atf.Window(8, 1e4, 2.0, cap=math.nan),
           atf.Window(8, 1e4, -1.0, beta=1.0),
           atf.Window(8, 1e4, 2.0, k_profile=[1.0, -1.0, 1.0, 1.0]),
           atf.Window(8, 1e4, 2.0, k_profile=[1.0, math.nan, 1.0, 1.0]),
           atf.Window(8, 1e4, 2.0, k_profile=[0.0, 1.0, 1.0, 1.0], gamma=1e6)]  # 0 * inf
    for w in bad:
        with pytest.raises(atf.AtfError) as e:
            atf.atf_window_table(w)
        assert e.value.code == atf.ATF_EINVAL and "window" in atf.atf_last_error()
    with pytest.raises(ValueError):
        atf.Window(8, 1e4, 2.0, k_profile=[1.0, 2.0]).as_c()
    lib = atf.library()
    out = np.zeros(4)
    assert lib.atf_retention_profile(8, 9, 16.0, 2.0, out.ctypes.data) == atf.ATF_EINVAL
    assert lib.atf_retention_profile(7, 1, 16.0, 2.0, out.ctypes.data) == atf.ATF_EINVAL
    assert lib.atf_retention_profile(8, 2, 16.0, 0.0, out.ctypes.data) == atf.ATF_EINVAL
    assert lib.atf_retention_profile(8, 1, -1.0, 2.0, out.ctypes.data) == atf.ATF_EINVAL
    assert lib.atf_retention_profile(8, 1, 16.0, 2.0, None) == atf.ATF_EINVAL


# the rounded slice of Sec. 3.3: the library's table/counts against the oracle's
# cell-by-cell rounding rule summed by distance
@pytest.mark.parametrize("name", ["qwen05b_prefill_32k", "llama3b_prefill_128k",
                                  "qwen7b1m_prefill_chunk", "qwen7b1m_decode"])
@pytest.mark.parametrize("sp", [2, 3, 8, 16])
def test_rounded_slice_counts_match_oracle(oracle_lib, name, sp):
    wl = W.WORKLOADS[name]
    th = W.workload_theta(wl)
    th_np = th.numpy() if th is not None else None
    win = atf.Window(wl.head_dim, wl.rope_base, wl.k, th_np, slice_pairs=sp)
    widths = oracle_lib.window_widths(wl.head_dim, wl.rope_base, wl.k, th_np)
    n_q = min(wl.n_q, 4096)   # the by-distance sum walks every distance up to the last row
    q0 = wl.q_pos0 + wl.n_q - n_q
    got = atf.atf_count_terms(win, n_q, q0, wl.n_k)
    assert got == oracle_lib.count_terms(widths, n_q, q0, wl.n_k, atom=sp)
    # rounding only adds terms
    assert got[0] >= atf.atf_count_terms(atf.Window(wl.head_dim, wl.rope_base, wl.k, th_np),
                                         n_q, q0, wl.n_k)[0]


def test_rounded_slice_table_and_validation(oracle_lib):
    t = atf.atf_window_table(atf.Window(128, 1e7, 2.0, slice_pairs=8))
    exact = atf.atf_window_table(atf.Window(128, 1e7, 2.0))
    # each 8-pair step takes the threshold of its lowest-frequency pair
    assert np.array_equal(t, np.repeat(exact[7::8], 8))
    assert np.array_equal(atf.atf_window_table(atf.Window(128, 1e7, 2.0, slice_pairs=1)), exact)
    # steps counted from the lowest frequency: with 3-pair steps on 4 pairs, {0} {1,2,3}
    t3 = atf.atf_window_table(atf.Window(8, 100.0, 2.0, slice_pairs=3))
    e3 = atf.atf_window_table(atf.Window(8, 100.0, 2.0))
    assert list(t3) == [e3[0], e3[3], e3[3], e3[3]]
    # the variable-k profile keeps a non-decreasing table: allowed
    var = atf.Window(64, 1e6, 16.0, k_profile=atf.atf_retention_profile(64, "arithmetic", 16, 2),
                     slice_pairs=8)
    atf.atf_window_table(var)
    bad = [atf.Window(8, 1e4, 2.0, slice_pairs=-1), atf.Window(8, 1e4, 2.0, slice_pairs=5),
           atf.Window(8, 1e4, 2.0, [1.0, 0.5, 2.0, 0.1], slice_pairs=2),   # decreasing widths
           atf.Window(64, 1e4, 1e6, gamma=-1.0, slice_pairs=8)]
    for w in bad:
        with pytest.raises(atf.AtfError) as e:
            atf.atf_window_table(w)
        assert e.value.code == atf.ATF_EINVAL and "window" in atf.atf_last_error()


def _raw_prefill(lib, cw, **kw):
    args = dict(q=16, k=16, v=16, o=16, lse=16, batch=1, n_q=4, n_k=4, q_pos0=0, h_q=2, h_kv=1,
                cache_tokens=0)
    args.update(kw)
    return lib.atf_prefill(args["q"], args["k"], args["v"], args["o"], args["lse"], args["batch"],
                           args["n_q"], args["n_k"], args["q_pos0"], args["h_q"], args["h_kv"],
                           args["cache_tokens"], ctypes.byref(cw), 0.0, None)


@pytest.mark.parametrize("name", ["qwen05b_prefill_32k", "llama3b_prefill_128k",
                                  "qwen7b1m_prefill_chunk"])
@pytest.mark.parametrize("kind", ["k2", "k0.5", "k64", "var16to2", "rounded8", "floor64"])
def test_prefill_first_kept_tile_matches_the_chunk_test(name, kind):
    """The prefill stages K chunk c of the 64-key tile at j0 iff some pair of c is kept
    at the tile's smallest distance, max(0, pos_first - j0 - 63), i.e. iff the chunk's
    largest threshold reaches it.  Its load issue replaces that per-tile test by one
    first tile per chunk, ceil((pos_first - 63 - max_c W) / 64) clamped at 0, which
    holds because thresholds are >= 0 and the distance falls as j0 grows.  Both forms
    over the window tables the kernels see, and positions from the first tile to 2^31."""
    wl = W.WORKLOADS[name]
    d = wl.head_dim
    th = W.workload_theta(wl)
    th = None if th is None else th.numpy()
    kw = {"k2": dict(k=2.0), "k0.5": dict(k=0.5), "k64": dict(k=64.0),
          "var16to2": dict(k=16.0, k_profile=atf.atf_retention_profile(d, "arithmetic", 16.0, 2.0)),
          "rounded8": dict(k=2.0, slice_pairs=8), "floor64": dict(k=2.0, beta=64.0)}[kind]
    k = kw.pop("k")
    table = atf.atf_window_table(atf.Window(d, wl.rope_base, k, th, **kw)).astype(np.int64)
    assert table.min() >= 0
    chunk_max = table.reshape(d // 16, 8).max(axis=1)
    rng = np.random.default_rng(7)
    positions = np.concatenate([[0, 1, 62, 63, 64, 65, 127, 128, 4095, 2**31 - 2],
                                rng.integers(0, 2**31 - 1, size=40)])
    for pos_first in positions:
        pos_first = int(pos_first)
        num = pos_first - 63 - chunk_max
        first = np.where(num <= 0, 0, np.minimum(2**31 - 1, -(-num // 64)))
        t_hi = max(0, pos_first + 63) // 64
        tiles = np.unique(np.concatenate([np.arange(0, 64), np.arange(max(0, t_hi - 64), t_hi + 2),
                                          first, np.maximum(first - 1, 0), first + 1]))
        tiles = tiles[(tiles >= 0) & (tiles < 2**25)]
        zlo = np.maximum(0, pos_first - 64 * tiles - 63)
        kept = chunk_max[None, :] >= zlo[:, None]
        by_first = tiles[:, None] >= first[None, :]
        assert np.array_equal(kept, by_first), (pos_first, np.argwhere(kept != by_first)[:4])


def test_prefill_validation_before_launch():
    lib = atf.library()
    good, _ = atf.Window(64, 1e4, 2.0).as_c()
    cases = [
        (atf.Window(96, 1e4, 2.0), {}, atf.ATF_EUNSUPPORTED),
        (atf.Window(64, 1e4, 2.0), {"h_q": 3, "h_kv": 2}, atf.ATF_EINVAL),
        (atf.Window(64, 1e4, 2.0), {"n_k": 0}, atf.ATF_EINVAL),
        (atf.Window(64, 1e4, 2.0), {"batch": 0}, atf.ATF_EINVAL),
        (atf.Window(64, 1e4, 2.0), {"q_pos0": -1}, atf.ATF_EINVAL),
        (atf.Window(64, 1e4, 2.0), {"q_pos0": 2 ** 31 - 2}, atf.ATF_EINVAL),
        (atf.Window(64, 1e4, 2.0), {"q": None}, atf.ATF_EINVAL),
        (atf.Window(64, 1e4, 2.0), {"o": 18}, atf.ATF_EINVAL),        # misaligned
        (atf.Window(64, 1e4, -1.0), {}, atf.ATF_EINVAL),
        (atf.Window(64, 1e4, 2.0), {"cache_tokens": 3}, atf.ATF_EINVAL),   # below n_k
        (atf.Window(64, 1e4, 2.0), {"cache_tokens": 2 ** 31}, atf.ATF_EINVAL),
    ]
    for win, kw, code in cases:
        cw, keep = win.as_c()
        assert _raw_prefill(lib, cw, **kw) == code, (win, kw)
        assert atf.atf_last_error()
    # n_q == 0 is a no-op that touches nothing
    assert _raw_prefill(lib, good, n_q=0, q=None, k=None, v=None, o=None, lse=None) == atf.ATF_OK


def test_decode_validation_before_launch():
    lib = atf.library()
    cw, keep = atf.Window(128, 5e5, 2.0).as_c()
    need = atf.atf_decode_workspace_bytes(8, 24, 8, 131072, 128)
    assert need > 0
    assert atf.atf_decode_workspace_bytes(8, 24, 7, 131072, 128) == 0
    assert atf.atf_decode_workspace_bytes(8, 24, 8, 131072, 96) == 0

    def call(ws=16, ws_bytes=None, d=128, **kw):
        a = dict(batch=8, n_k=131072, q_pos=131072, h_q=24, h_kv=8, cache_tokens=0)
        a.update(kw)
        w, kp = atf.Window(d, 5e5, 2.0).as_c()
        # the default workspace (16 bytes) is too small for any split plan, so a call
        # whose other arguments are valid still fails before launching
        return lib.atf_decode(16, 16, 16, 16, 16, a["batch"], a["n_k"], a["q_pos"], a["h_q"],
                              a["h_kv"], a["cache_tokens"], ctypes.byref(w), 0.0, ws,
                              16 if ws_bytes is None else ws_bytes, None)
    assert call() == atf.ATF_EWORKSPACE
    assert call(ws=None, ws_bytes=need) == atf.ATF_EWORKSPACE
    assert call(d=80) == atf.ATF_EUNSUPPORTED
    assert call(q_pos=-1) == atf.ATF_EINVAL
    assert call(h_kv=5) == atf.ATF_EINVAL
    assert call(n_k=0) == atf.ATF_EINVAL
    assert call(ws_bytes=need, cache_tokens=131071) == atf.ATF_EINVAL   # below n_k


def test_decode_noalloc_validation_before_launch():
    """atf_decode_noalloc: sizes whose partial states exceed the library's scratch array
    fail with ATF_EWORKSPACE, and a NULL window with ATF_EINVAL, before any device call
    (the pointers below are not device memory)."""
    lib = atf.library()
    w, keep = atf.Window(128, 1e4, 2.0).as_c()
    assert atf.atf_decode_workspace_bytes(64, 64, 1, 4096, 128) > atf.DECODE_NOALLOC_SCRATCH_BYTES
    rc = lib.atf_decode_noalloc(16, 16, 16, 16, 16, 64, 4096, 4096, 64, 1, 0, ctypes.byref(w),
                                0.0, None)
    assert rc == atf.ATF_EWORKSPACE and "scratch" in atf.atf_last_error()
    rc = lib.atf_decode_noalloc(16, 16, 16, 16, 16, 1, 4096, 4096, 28, 4, 0, None, 0.0, None)
    assert rc == atf.ATF_EINVAL


def test_decode_ragged_validation_before_launch():
    """Every call below fails validation, so nothing is launched (the pointers are
    placeholders)."""
    lib = atf.library()
    need = atf.atf_decode_workspace_bytes(8, 24, 8, 131072, 128)

    def call(ws=16, ws_bytes=None, d=128, nk_rows=1 << 12, qp_rows=1 << 13, **kw):
        a = dict(batch=8, max_n_k=131072, h_q=24, h_kv=8, cache_tokens=0)
        a.update(kw)
        w, kp = atf.Window(d, 5e5, 2.0).as_c()
        return lib.atf_decode_ragged(16, 16, 16, 16, 16, a["batch"], nk_rows, qp_rows,
                                     a["max_n_k"], a["h_q"], a["h_kv"], a["cache_tokens"],
                                     ctypes.byref(w), 0.0, ws,
                                     16 if ws_bytes is None else ws_bytes, None)
    assert call() == atf.ATF_EWORKSPACE              # everything else valid
    assert call(ws=None, ws_bytes=need) == atf.ATF_EWORKSPACE
    assert call(nk_rows=None) == atf.ATF_EINVAL
    assert call(qp_rows=None) == atf.ATF_EINVAL
    assert call(nk_rows=(1 << 12) + 2) == atf.ATF_EINVAL   # row arrays are int32, 4-byte aligned
    assert call(qp_rows=(1 << 13) + 1) == atf.ATF_EINVAL
    assert call(max_n_k=0) == atf.ATF_EINVAL
    assert call(max_n_k=131072, cache_tokens=1000) == atf.ATF_EINVAL   # bound above the capacity
    assert call(d=80) == atf.ATF_EUNSUPPORTED
    assert call(h_kv=5) == atf.ATF_EINVAL
    assert call(batch=0) == atf.ATF_EINVAL
    assert "decode_ragged" in atf.atf_last_error()


def test_paged_validation_before_launch():
    """Every call below fails validation, so nothing is launched (the pointers are
    placeholders)."""
    lib = atf.library()

    def app(**kw):
        a = dict(k=16, v=16, kp=1 << 20, vp=1 << 21, bt=1 << 12, max_pages=4, num_pages=8, pt=64,
                 batch=2, n_new=10, pos0=0, h_kv=2, d=128)
        a.update(kw)
        return lib.atf_cache_append_paged(a["k"], a["v"], a["kp"], a["vp"], a["bt"], a["max_pages"],
                                          a["num_pages"], a["pt"], a["batch"], a["n_new"],
                                          a["pos0"], a["h_kv"], a["d"], None)
    assert app(pt=48) == atf.ATF_EINVAL
    assert app(pt=0) == atf.ATF_EINVAL
    assert app(num_pages=0) == atf.ATF_EINVAL
    assert app(max_pages=0) == atf.ATF_EINVAL
    assert app(pos0=250) == atf.ATF_EINVAL          # 250 + 10 > 4 pages of 64
    assert app(bt=None) == atf.ATF_EINVAL
    assert app(bt=(1 << 12) + 2) == atf.ATF_EINVAL  # int32 table, 4-byte aligned
    assert app(k=24) == atf.ATF_EINVAL              # 16-byte alignment
    assert app(d=80) == atf.ATF_EUNSUPPORTED
    assert app(n_new=-1) == atf.ATF_EINVAL
    assert app(n_new=0) == atf.ATF_OK               # no-op: nothing launched

    need = atf.atf_decode_workspace_bytes(2, 24, 8, 256, 128)
    assert need > 0

    def dec(ws=16, ws_bytes=16, **kw):
        a = dict(bt=1 << 12, max_pages=4, num_pages=8, pt=64, max_n_k=256, nk=1 << 13, qp=1 << 14)
        a.update(kw)
        w, kp = atf.Window(128, 5e5, 2.0).as_c()
        return lib.atf_decode_paged(16, 16, 16, 16, 16, 2, a["bt"], a["max_pages"], a["num_pages"],
                                    a["pt"], a["nk"], a["qp"], a["max_n_k"], 24, 8, ctypes.byref(w),
                                    0.0, ws, ws_bytes, None)
    assert dec() == atf.ATF_EWORKSPACE              # everything else valid
    assert dec(bt=None) == atf.ATF_EINVAL
    assert dec(bt=(1 << 12) + 1) == atf.ATF_EINVAL
    assert dec(nk=None) == atf.ATF_EINVAL
    assert dec(pt=40) == atf.ATF_EINVAL
    assert dec(num_pages=0) == atf.ATF_EINVAL
    assert dec(max_n_k=257) == atf.ATF_EINVAL       # more than 4 pages of 64 tokens
    assert dec(max_n_k=0) == atf.ATF_EINVAL
    assert "decode_paged" in atf.atf_last_error()


def test_unrotated_validation_before_launch():
    """Rotation frequencies are checked before launch (the window and workspace as for
    atf_decode / atf_decode_paged); every call below fails, so nothing is launched."""
    lib = atf.library()
    w, keep = atf.Window(128, 1e4, 2.0).as_c()
    good = [1e4 ** (-2.0 * r / 128) for r in range(64)]

    def freq(f):
        if f is None:
            return None
        arr = (ctypes.c_double * len(f))(*f)
        freq.keep = arr
        return ctypes.cast(arr, ctypes.c_void_p)

    def dec(f=None):
        return lib.atf_decode_unrotated(16, 16, 16, 16, 16, 1, 1000, 1000, 8, 2, 1000,
                                        ctypes.byref(w), freq(f), 0.0, 16, 16, None)

    def paged(f=None):
        return lib.atf_decode_paged_unrotated(16, 16, 16, 16, 16, 2, 1 << 12, 4, 8, 64, 1 << 13,
                                              1 << 14, 256, 24, 8, ctypes.byref(w), freq(f), 0.0,
                                              16, 16, None)

    def ragged(f=None):
        return lib.atf_decode_ragged_unrotated(16, 16, 16, 16, 16, 2, 1 << 13, 1 << 14, 1000, 8,
                                               2, 1000, ctypes.byref(w), freq(f), 0.0, 16, 16,
                                               None)

    assert ragged(good) == atf.ATF_EWORKSPACE
    bad = list(good)
    bad[0] = -2.0
    assert ragged(bad) == atf.ATF_EINVAL and "decode_ragged_unrotated" in atf.atf_last_error()
    assert dec() == atf.ATF_EWORKSPACE               # the window's frequencies
    assert dec(good) == atf.ATF_EWORKSPACE
    assert paged(good) == atf.ATF_EWORKSPACE
    for bad in (-1.0, float("inf"), float("nan")):
        f = list(good)
        f[5] = bad
        assert dec(f) == atf.ATF_EINVAL
        assert "decode_unrotated" in atf.atf_last_error()
        assert paged(f) == atf.ATF_EINVAL
        assert "decode_paged_unrotated" in atf.atf_last_error()


def test_prefill_unrotated_validation_before_launch():
    """atf_prefill_unrotated checks the rotation frequencies with the window, before the
    n_q == 0 no-op and before any launch; the pre-rotated checks apply unchanged."""
    lib = atf.library()
    w, keep = atf.Window(128, 1e4, 2.0).as_c()
    good = [1e4 ** (-2.0 * r / 128) for r in range(64)]
    keep_f = []

    def pre(f=None, n_q=0, q=16, h_q=8):
        fp = None
        if f is not None:
            arr = (ctypes.c_double * len(f))(*f)
            keep_f.append(arr)
            fp = ctypes.cast(arr, ctypes.c_void_p)
        return lib.atf_prefill_unrotated(q, 16, 16, 16, 16, 1, n_q, 1000, 0, h_q, 2, 1000,
                                         ctypes.byref(w), fp, 0.0, None)

    assert pre(good) == atf.ATF_OK       # n_q = 0: validated, then a no-op
    assert pre() == atf.ATF_OK           # the window's frequencies
    for bad in (-1.0, float("inf"), float("nan")):
        f = list(good)
        f[7] = bad
        assert pre(f) == atf.ATF_EINVAL
        assert "prefill_unrotated" in atf.atf_last_error()
    assert pre(good, n_q=10, q=17) == atf.ATF_EINVAL      # misaligned q
    assert "prefill_unrotated" in atf.atf_last_error()
    assert pre(good, n_q=10, h_q=7) == atf.ATF_EINVAL     # h_q not a multiple of h_kv
    w64, keep64 = atf.Window(96, 1e4, 2.0).as_c()
    assert lib.atf_prefill_unrotated(16, 16, 16, 16, 16, 1, 1, 10, 0, 2, 1, 10,
                                     ctypes.byref(w64), None, 0.0, None) == atf.ATF_EUNSUPPORTED


def test_rotate_kcache_validation_before_launch():
    """Every call below fails host validation, so nothing is launched."""
    lib = atf.library()
    w, keep = atf.Window(128, 1e4, 2.0).as_c()
    w96, keep96 = atf.Window(96, 1e4, 2.0).as_c()
    bad_f = (ctypes.c_double * 64)(*([1.0] * 63 + [float("nan")]))

    def rot(src=16, dst=1 << 30, batch=1, n_k=100, h_kv=2, cap=0, win=w, f=None):
        return lib.atf_rotate_kcache(src, dst, batch, n_k, h_kv, cap, ctypes.byref(win), f, None)

    assert rot(win=w96) == atf.ATF_EUNSUPPORTED
    assert rot(batch=0) == atf.ATF_EINVAL
    assert rot(n_k=0) == atf.ATF_EINVAL
    assert rot(cap=50) == atf.ATF_EINVAL                       # capacity below n_k
    assert rot(batch=4096, h_kv=4) == atf.ATF_EUNSUPPORTED    # 4096 * 4 * 8 streams
    assert rot(f=ctypes.cast(bad_f, ctypes.c_void_p)) == atf.ATF_EINVAL
    assert "rotate_kcache" in atf.atf_last_error()
    assert rot(src=None) == atf.ATF_EINVAL
    assert rot(src=17) == atf.ATF_EINVAL                       # misaligned
    assert rot(src=16, dst=16 + 4096) == atf.ATF_EINVAL        # overlap: 2 * 2 * 128 * 100 bytes


def test_cache_append_rotated_validation_before_launch():
    lib = atf.library()
    w, keep = atf.Window(128, 1e4, 2.0).as_c()
    w96, keep96 = atf.Window(96, 1e4, 2.0).as_c()
    bad_f = (ctypes.c_double * 64)(*([1.0] * 10 + [-1.0] + [1.0] * 53))

    def app(win=w, n_new=10, pos0=0, cap=100, f=None, k_new=16):
        wp = None if win is None else ctypes.byref(win)
        return lib.atf_cache_append_rotated(k_new, 1 << 20, 1 << 24, 1 << 28, 1, n_new, pos0, 2,
                                            cap, wp, f, None)

    assert app(win=None) == atf.ATF_EINVAL
    assert app(win=w96) == atf.ATF_EUNSUPPORTED
    assert app(f=ctypes.cast(bad_f, ctypes.c_void_p)) == atf.ATF_EINVAL
    assert "cache_append_rotated" in atf.atf_last_error()
    assert app(pos0=95) == atf.ATF_EINVAL          # past the capacity
    assert app(k_new=None) == atf.ATF_EINVAL
    assert app(k_new=17) == atf.ATF_EINVAL         # misaligned
    assert app(n_new=0) == atf.ATF_OK              # a no-op after validation


def test_cache_append_paged_rotated_validation_before_launch():
    lib = atf.library()
    w, keep = atf.Window(128, 1e4, 2.0).as_c()
    w96, keep96 = atf.Window(96, 1e4, 2.0).as_c()
    bad_f = (ctypes.c_double * 64)(*([1.0] * 20 + [float("inf")] + [1.0] * 43))

    def app(win=w, pt=64, n_new=10, pos0=0, f=None, bt=16):
        wp = None if win is None else ctypes.byref(win)
        return lib.atf_cache_append_paged_rotated(16, 1 << 20, 1 << 24, 1 << 28, bt, 4, 8, pt, 1,
                                                  n_new, pos0, 2, wp, f, None)

    assert app(win=None) == atf.ATF_EINVAL
    assert app(win=w96) == atf.ATF_EUNSUPPORTED
    assert app(f=ctypes.cast(bad_f, ctypes.c_void_p)) == atf.ATF_EINVAL
    assert "cache_append_paged_rotated" in atf.atf_last_error()
    assert app(pt=48) == atf.ATF_EINVAL            # not a multiple of 32
    assert app(pos0=250) == atf.ATF_EINVAL         # past the row's 4 pages of 64
    assert app(bt=None) == atf.ATF_EINVAL
    assert app(bt=18) == atf.ATF_EINVAL            # misaligned table
    assert app(n_new=0) == atf.ATF_OK              # a no-op after validation


def test_pack_validation_before_launch():
    lib = atf.library()
    assert lib.atf_pack_kcache(16, 16 + 64, 1, 4, 1, 64, None) == atf.ATF_EINVAL   # overlap
    assert lib.atf_pack_kcache(16, 1 << 20, 1, 4, 1, 48, None) == atf.ATF_EUNSUPPORTED
    assert lib.atf_pack_kcache(None, 1 << 20, 1, 4, 1, 64, None) == atf.ATF_EINVAL
    assert lib.atf_pack_kcache(16, 1 << 20, 0, 4, 1, 64, None) == atf.ATF_EINVAL
    assert atf.atf_kcache_chunk_pairs(128) == 8 and atf.atf_kcache_chunk_pairs(64) == 8
    assert atf.atf_kcache_chunk_pairs(32) == 0


def test_vpack_validation_and_size():
    lib = atf.library()
    assert atf.atf_vcache_bytes(1, 17, 2, 64) == 1 * 2 * 2 * 16 * 64 * 2
    assert atf.atf_vcache_bytes(3, 16, 1, 128) == 3 * 1 * 1 * 16 * 128 * 2
    assert atf.atf_vcache_bytes(1, 0, 1, 64) == 0
    assert atf.atf_vcache_bytes(1, 5, 1, 96) == 0
    # destination overlapping the source (the packed size rounds n_k up to 16)
    assert lib.atf_pack_vcache(1 << 20, (1 << 20) + 512, 1, 5, 1, 64, None) == atf.ATF_EINVAL
    assert lib.atf_pack_vcache((1 << 20) + 1024, 1 << 20, 1, 5, 1, 64, None) == atf.ATF_EINVAL
    assert lib.atf_pack_vcache(16, 1 << 20, 1, 4, 1, 48, None) == atf.ATF_EUNSUPPORTED
    assert lib.atf_pack_vcache(None, 1 << 20, 1, 4, 1, 64, None) == atf.ATF_EINVAL
    assert lib.atf_pack_vcache(24, 1 << 20, 1, 4, 1, 64, None) == atf.ATF_EINVAL  # alignment
    assert lib.atf_pack_vcache(16, 1 << 20, 1, 4, 0, 64, None) == atf.ATF_EINVAL
    assert atf.vcache_shape(2, 33, 4, 128) == (2, 4, 3, 128, 16)


def test_cache_append_validation_before_launch():
    lib = atf.library()
    A = 1 << 30  # four far-apart fake device addresses (nothing is launched)
    kn, vn, kc, vc = A, 2 * A, 3 * A, 4 * A
    ok = dict(batch=1, n=4, pos0=8, h_kv=2, d=64, cap=16)

    def call(**kw):
        a = dict(ok, kn=kn, vn=vn, kc=kc, vc=vc)
        a.update(kw)
        return lib.atf_cache_append(a["kn"], a["vn"], a["kc"], a["vc"], a["batch"], a["n"],
                                    a["pos0"], a["h_kv"], a["d"], a["cap"], None)
    assert call(n=0) == atf.ATF_OK                          # nothing to write
    assert call(d=96) == atf.ATF_EUNSUPPORTED
    for bad in (dict(batch=0), dict(h_kv=0), dict(n=-1), dict(pos0=-1), dict(cap=0),
                dict(pos0=13), dict(cap=2 ** 31), dict(kn=None), dict(vc=None),
                dict(kc=kc + 8),                             # misaligned
                dict(kc=vc + 256),                           # K cache inside the V cache
                dict(vn=vc + 512),                           # input inside the V cache
                dict(kn=kc + 64 * 2 * 2 * 4)):               # input inside the K cache
        assert call(**bad) == atf.ATF_EINVAL, bad
        assert "cache_append" in atf.atf_last_error()
