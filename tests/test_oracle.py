"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each oracle function is checked against something other than itself:

- ``window_widths``: the paper's printed term counts (Table 1, Fig. 1 CASE,
  Sec. 4 decode figures, App. C Fig. sndecomp), which fail if lambda, the
  2*pi, the exponent sign or the <= of the keep rule is wrong; saturation.
- ``scores``: eq:pair evaluated in the unrotated frame with an independent
  complex-number rotation (wrong pair index, sign or scale fails it); the
  special cases below.
- ``attend``: (check 1) a textbook dense causal attention in numpy at an
  infinite window, with GQA and query-position offsets; a hand-worked example;
  two special cases that reduce to numpy dense attention (dropped prefix pairs,
  one uniform width); sampled rows equal to the full run.
- ``count_terms``: brute-force triple loop on tiny inputs, the per-row count
  returned by ``attend``, the printed pins, and the paper's closed forms within
  its stated integral-approximation error.
"""
import math

import numpy as np
import pytest

from conftest import kv, read_golden

import workloads as W


# ----------------------------------------------------------------------------
# independent references written in the test
# ----------------------------------------------------------------------------
def dense_attention(q, k, v, q_pos0, scale):
    """Textbook causal attention in fp64 (numpy): softmax(QK^T * scale + mask) V."""
    B, nq, hq, d = q.shape
    nk, hkv = k.shape[1], k.shape[2]
    G = hq // hkv
    kk = np.repeat(k, G, axis=2)
    vv = np.repeat(v, G, axis=2)
    s = np.einsum("bihd,bjhd->bhij", q, kk) * scale
    pos = q_pos0 + np.arange(nq)
    mask = np.arange(nk)[None, :] > pos[:, None]
    s = np.where(mask[None, None], -np.inf, s)
    m = s.max(-1, keepdims=True)
    e = np.exp(s - m)
    l_ = e.sum(-1, keepdims=True)
    o = np.einsum("bhij,bjhd->bihd", e / l_, vv)
    lse = (m + np.log(l_))[..., 0]
    return o, lse


def dense_from_scores(s, v, hq, G):
    """Softmax over a given [nq, nk] score matrix (with -inf) and PV, numpy."""
    m = s.max(-1, keepdims=True)
    e = np.exp(s - m)
    l_ = e.sum(-1, keepdims=True)
    return (e / l_) @ v, (m + np.log(l_))[:, 0]


def bf16_grid(rng, shape, scale=1.0):
    """Random values exactly representable in bf16 (so both sides see the same numbers)."""
    import torch
    x = torch.from_numpy(rng.standard_normal(shape) * scale).to(torch.bfloat16)
    return x.to(torch.float64).numpy()


def rotate_complex(x, positions, theta):
    """RoPE by complex multiplication: u_r = x_r + i x_{r+h}, u~ = u e^{i p theta_r}."""
    assert x.ndim == 4  # [B, N, H, d]
    h = x.shape[-1] // 2
    u = x[..., :h] + 1j * x[..., h:]
    ph = np.exp(1j * positions[:, None] * theta[None, :]).reshape(1, len(positions), 1, h)
    r = u * ph
    return np.concatenate([r.real, r.imag], axis=-1)


# ----------------------------------------------------------------------------
# hand-worked example (tests/golden/hand_example.txt)
# ----------------------------------------------------------------------------
def test_hand_example(oracle_lib):
    recs = read_golden("hand_example.txt")
    q = np.array([[1, 0, 0, 0], [0, 1, 0, 0], [1, 1, 1, 1]], dtype=np.float64)[None, :, None, :]
    k = np.array([[2, 0, 2, 0], [0, 2, 0, 0], [0, 0, 0, 0]], dtype=np.float64)[None, :, None, :]
    v = np.array([[1, 0, 0, 0], [0, 1, 0, 0], [0, 0, 1, 0]], dtype=np.float64)[None, :, None, :]
    w = np.array([1.0, np.inf])
    o, lse, terms = oracle_lib.attend(q, k, v, 0, w, scale=0.5)
    of, lsef, termsf = oracle_lib.attend(q, k, v, 0, np.array([np.inf, np.inf]), scale=0.5)
    for r in recs:
        f = kv(r)
        if r[0] == "row":
            i = int(r[1])
            np.testing.assert_allclose(o[0, i, 0], [float(x) for x in f["o"].split(",")],
                                       atol=1e-15)
            assert abs(lse[0, 0, i] - float(f["lse"])) < 1e-15
        elif r[0] == "full_row":
            i = int(r[1])
            np.testing.assert_allclose(of[0, i, 0], [float(x) for x in f["o"].split(",")],
                                       atol=1e-15)
            assert abs(lsef[0, 0, i] - float(f["lse"])) < 1e-14
        elif r[0] == "terms":
            assert int(terms.sum()) == int(r[1])
            assert oracle_lib.count_terms(w, 3, 0, 3)[0] == int(r[1])
        elif r[0] == "full_terms":
            assert int(termsf.sum()) == int(r[1])
    # rows 0 and 1 are untouched by the window (every distance there is <= 1)
    np.testing.assert_allclose(o[0, :2], of[0, :2], atol=0)


def test_empty_score_sum_is_zero(oracle_lib):
    """d=2 with w_0 = 0: every off-diagonal cell keeps no term, so its score is 0
    and the token stays in the softmax (terms dropped, never tokens: Sec. 3.2)."""
    rng = np.random.default_rng(1)
    q = bf16_grid(rng, (1, 5, 1, 2))
    k = bf16_grid(rng, (1, 5, 1, 2))
    s = oracle_lib.scores(q, k, 0, np.array([0.0]))
    for i in range(5):
        for j in range(5):
            if j > i:
                assert s[i, j] == -np.inf
            elif j < i:
                assert s[i, j] == 0.0
            else:
                assert s[i, j] == pytest.approx(q[0, i, 0] @ k[0, j, 0] / math.sqrt(2), abs=1e-15)


# ----------------------------------------------------------------------------
# check 1: infinite window == ordinary causal RoPE attention (numpy dense)
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("B,nq,nk,q0,hq,hkv,d", [
    (1, 33, 33, 0, 1, 1, 8),
    (2, 37, 37, 0, 4, 2, 8),
    (1, 17, 40, 23, 6, 2, 16),     # chunk at the end of a longer context
    (1, 20, 12, 5, 3, 3, 4),       # keys end before the last query position
    (2, 16, 16, 0, 7, 1, 64),
])
@pytest.mark.parametrize("kwin", [math.inf, 1e9])
def test_check1_matches_dense(oracle_lib, B, nq, nk, q0, hq, hkv, d, kwin):
    rng = np.random.default_rng(B * 1000 + nq * 7 + d)
    q = bf16_grid(rng, (B, nq, hq, d))
    k = bf16_grid(rng, (B, nk, hkv, d))
    v = bf16_grid(rng, (B, nk, hkv, d))
    w = oracle_lib.window_widths(d, 1e4, kwin, n_ctx=max(nk, q0 + nq))
    o, lse, terms = oracle_lib.attend(q, k, v, q0, w)
    od, lsed = dense_attention(q, k, v, q0, 1 / math.sqrt(d))
    np.testing.assert_allclose(o, od, atol=1e-12, rtol=0)
    np.testing.assert_allclose(lse, lsed, atol=1e-12, rtol=0)
    causal = sum(min(q0 + i, nk - 1) + 1 for i in range(nq))
    assert int(terms[0, 0].sum()) == causal * d // 2


def test_sampled_rows_equal_full_run(oracle_lib):
    rng = np.random.default_rng(7)
    q = bf16_grid(rng, (2, 29, 4, 16))
    k = bf16_grid(rng, (2, 29, 2, 16))
    v = bf16_grid(rng, (2, 29, 2, 16))
    w = oracle_lib.window_widths(16, 50.0, 1.0)
    o, lse, t = oracle_lib.attend(q, k, v, 0, w)
    rows = np.array([[1, 3, 28], [0, 0, 0], [1, 1, 13], [0, 2, 7]])
    os_, ls, ts = oracle_lib.attend(q, k, v, 0, w, rows=rows)
    for n, (b, h, i) in enumerate(rows):
        assert np.array_equal(os_[n], o[b, i, h])
        assert ls[n] == lse[b, h, i]
        assert ts[n] == t[b, h, i]


# ----------------------------------------------------------------------------
# check 2: eq:pair -- the rotated score is a sum of per-pair terms
#          a_r cos(z theta_r) + b_r sin(z theta_r) with z = n - m
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("d,base,kwin", [(8, 100.0, math.inf), (8, 100.0, 1.0),
                                          (64, 1e6, 2.0), (128, 5e5, 0.5)])
def test_check2_pair_decomposition(oracle_lib, d, base, kwin):
    rng = np.random.default_rng(d + int(base) % 97)
    h = d // 2
    n_pos = 40
    theta = base ** (-2.0 * np.arange(h) / d)
    qu = rng.standard_normal((1, n_pos, 1, d))
    ku = rng.standard_normal((1, n_pos, 1, d))
    pos = np.arange(n_pos, dtype=np.float64)
    qr = rotate_complex(qu, pos, theta)
    kr = rotate_complex(ku, pos, theta)
    w = oracle_lib.window_widths(d, base, kwin)
    s = oracle_lib.scores(qr, kr, 0, w)
    for i in range(n_pos):
        for j in range(i + 1):
            z = i - j
            a = qu[0, i, 0, :h] * ku[0, j, 0, :h] + qu[0, i, 0, h:] * ku[0, j, 0, h:]
            b = qu[0, i, 0, :h] * ku[0, j, 0, h:] - qu[0, i, 0, h:] * ku[0, j, 0, :h]
            terms = a * np.cos(z * theta) + b * np.sin(z * theta)
            expect = terms[z <= w].sum() / math.sqrt(d)
            assert s[i, j] == pytest.approx(expect, abs=1e-12 * (1 + abs(expect)))
    # (i) with every pair kept the per-pair sum is the plain dot product
    s_full = oracle_lib.scores(qr, kr, 0, np.full(h, np.inf))
    dots = qr[0, :, 0] @ kr[0, :, 0].T / math.sqrt(d)
    tri = np.tril(np.ones((n_pos, n_pos), dtype=bool))
    np.testing.assert_allclose(s_full[tri], dots[tri], atol=1e-12)


def test_scores_depend_only_on_distance(oracle_lib):
    """Shifting query and key positions together leaves every windowed score unchanged."""
    rng = np.random.default_rng(11)
    d, h = 16, 8
    theta = 300.0 ** (-2.0 * np.arange(h) / d)
    qu = rng.standard_normal((1, 1, 1, d))
    ku = rng.standard_normal((1, 1, 1, d))
    w = oracle_lib.window_widths(d, 300.0, 0.7)
    vals = []
    for shift in (0, 5, 123):
        n, m = 9 + shift, 2 + shift
        qr = rotate_complex(qu, np.array([float(n)]), theta)
        kk = np.zeros((1, n + 1, 1, d))
        kk[0, m] = rotate_complex(ku, np.array([float(m)]), theta)[0, 0]
        vals.append(oracle_lib.scores(qr, kk, n, w)[0, m])
    assert vals[0] == pytest.approx(vals[1], abs=1e-12)
    assert vals[0] == pytest.approx(vals[2], abs=1e-12)


# ----------------------------------------------------------------------------
# special cases that reduce to numpy dense attention
# ----------------------------------------------------------------------------
def test_dropped_prefix_pairs_equal_dense_on_sub_dims(oracle_lib):
    """w_r = -1 for r < r0 (never kept), +inf otherwise == dense attention on the
    dims of pairs r >= r0, i.e. dims [r0, h) and [h + r0, d)."""
    rng = np.random.default_rng(3)
    d, h, r0 = 16, 8, 3
    q = bf16_grid(rng, (1, 21, 2, d))
    k = bf16_grid(rng, (1, 21, 1, d))
    v = bf16_grid(rng, (1, 21, 1, d))
    w = np.array([-1.0] * r0 + [np.inf] * (h - r0))
    o, lse, _ = oracle_lib.attend(q, k, v, 0, w)
    keep = np.r_[np.arange(r0, h), np.arange(h + r0, d)]
    od, lsed = dense_attention(q[..., keep], k[..., keep], v, 0, 1 / math.sqrt(d))
    np.testing.assert_allclose(o, od, atol=1e-12)
    np.testing.assert_allclose(lse, lsed, atol=1e-12)


def test_uniform_width_zeroes_far_scores(oracle_lib):
    """One width w0 for every pair: cells at distance z > w0 have score 0, the rest
    the full dot product (dense scores with the far band set to zero)."""
    rng = np.random.default_rng(5)
    d, n, w0 = 8, 19, 4
    q = bf16_grid(rng, (1, n, 1, d))
    k = bf16_grid(rng, (1, n, 1, d))
    v = bf16_grid(rng, (1, n, 1, d))
    o, lse, _ = oracle_lib.attend(q, k, v, 0, np.full(d // 2, float(w0)))
    s = q[0, :, 0] @ k[0, :, 0].T / math.sqrt(d)
    z = np.arange(n)[:, None] - np.arange(n)[None, :]
    s = np.where(z > w0, 0.0, s)
    s = np.where(z < 0, -np.inf, s)
    od, lsed = dense_from_scores(s, v[0, :, 0], 1, 1)
    np.testing.assert_allclose(o[0, :, 0], od, atol=1e-12)
    np.testing.assert_allclose(lse[0, 0], lsed, atol=1e-12)


# ----------------------------------------------------------------------------
# check 3: term counts
# ----------------------------------------------------------------------------
def brute_force_count(w, n_q, q0, n_k):
    T = C = 0
    for i in range(n_q):
        p = q0 + i
        for j in range(n_k):
            if j > p:
                continue
            C += 1
            for wr in w:
                if p - j <= wr:
                    T += 1
    return T, C


@pytest.mark.parametrize("seed", range(12))
def test_count_brute_force(oracle_lib, seed):
    rng = np.random.default_rng(100 + seed)
    d = int(rng.choice([2, 4, 8]))
    base = float(rng.uniform(2.0, 500.0))
    kwin = float(rng.choice([0.05, 0.3, 1.0, 2.0, 7.5]))
    n_q = int(rng.integers(1, 30))
    q0 = int(rng.integers(0, 20))
    n_k = int(rng.integers(1, 50))
    w = oracle_lib.window_widths(d, base, kwin)
    bt, bc = brute_force_count(w, n_q, q0, n_k)
    assert oracle_lib.count_terms(w, n_q, q0, n_k) == (bt, bc)
    if q0 + n_q - 1 >= 0:
        rng2 = np.random.default_rng(seed)
        q = bf16_grid(rng2, (1, n_q, 1, d))
        k = bf16_grid(rng2, (1, n_k, 1, d))
        _, _, terms = oracle_lib.attend(q, k, k, q0, w)
        assert int(terms.sum()) == bt


def _pruned(oracle_lib, rec):
    f = kv(rec)
    d = int(f["d"])
    base = float(f["base"])
    N = int(f["N"])
    theta = W.llama3_theta(d, base).numpy() if rec[1] == "llama3b" else None
    qty = next(x for x in rec[2:] if "=" not in x)  # the quantity's name
    if "to" in f["k"]:  # k-arithmetic retention profile k_hi -> k_lo (App. A)
        hi, lo = (float(x) for x in f["k"].split("to"))
        assert qty == "pruned_prefill"
        prof = oracle_lib.retention_profile(d, "arithmetic", hi, lo)
        w = oracle_lib.family_widths(d, base, prof, cap=N, theta=theta)
        T, C = oracle_lib.count_terms(w, N, 0, N)
        return 100.0 * (1 - T / (C * d / 2))
    kwin = float(f["k"])
    if "atom" in f:  # the rounded slice of Sec. 3.3
        w = oracle_lib.window_widths(d, base, kwin, theta, n_ctx=N)
        T, C = oracle_lib.count_terms(w, N, 0, N, atom=int(f["atom"]))
        s = T / (C * d / 2)
        if qty == "ceiling":
            return 2.0 / (1.0 + s)
        assert qty == "pruned_prefill"
        return 100.0 * (1 - s)
    if qty == "pruned_prefill":
        w = oracle_lib.window_widths(d, base, kwin, theta, n_ctx=N)
        T, C = oracle_lib.count_terms(w, N, 0, N)
        return 100.0 * (1 - T / (C * d / 2))
    if qty == "pruned_decode":   # query at position N over keys 0..N-1
        w = oracle_lib.window_widths(d, base, kwin, theta, n_ctx=N + 1)
        T, C = oracle_lib.count_terms(w, 1, N, N)
        return 100.0 * (1 - T / (C * d / 2))
    if qty == "pruned_row":      # one row with n keys at distances 0..n-1
        w = oracle_lib.window_widths(d, base, kwin, theta, n_ctx=N)
        T, C = oracle_lib.count_terms(w, 1, N - 1, N)
        return 100.0 * (1 - T / (C * d / 2))
    if qty == "terms_last_row_z":
        w = oracle_lib.window_widths(d, base, kwin, theta, n_ctx=N)
        z = int(f["z"])
        return float(np.sum(z <= w))
    raise AssertionError(qty)


@pytest.mark.parametrize("rec", read_golden("paper_pins.txt"), ids=lambda r: r[0])
def test_paper_printed_counts(oracle_lib, rec):
    f = kv(rec)
    got = _pruned(oracle_lib, rec)
    assert abs(got - float(f["value"])) <= float(f["tol"]), (rec[0], got)


def R_interval(n0, n1, d, base, kwin):
    """eq:Rgen with eq:Fdef: reduction of the row interval [n0, n1] (App. C)."""
    wmin = 2 * math.pi * kwin
    F = lambda n: n * n * (math.log(n / wmin) - 1.5) + 2 * wmin * n
    return (F(n1) - F(n0)) / ((n1 * n1 - n0 * n0) * math.log(base))


@pytest.mark.parametrize("rec", read_golden("closed_forms.txt"), ids=lambda r: r[0])
def test_paper_closed_forms(rec):
    """The printed closed-form values follow from the formulas as written."""
    f = kv(rec)
    B = float(f["base"])
    lnB = math.log(B)
    q = rec[1]
    if q == "redprefill":
        kwin, N = float(f["k"]), int(f["N"])
        got = 100 * (math.log(N / (2 * math.pi * kwin)) - 1.5) / lnB
    elif q in ("row_continuous", "rhostar"):
        d, kwin, n = int(f["d"]), float(f["k"]), int(f["n"])
        wmin = 2 * math.pi * kwin
        rho = (d / 2) * math.log(n / wmin) / lnB
        s = d / (2 * lnB) * (n - wmin) + (d / 2 - rho) * n     # eq:Kn
        got = rho if q == "rhostar" else 100 * (1 - s / (d / 2 * n))
    elif q == "gap":
        got = 100 / (2 * lnB)
    elif q == "saturation_decode":
        got = 100 * (1 - 1 / lnB)
    elif q == "half_minus_whole":
        got = 100 * (1.5 - 1.27) / lnB
    else:
        raise AssertionError(q)
    assert abs(got - float(f["value"])) <= float(f["tol"]), (rec[0], got)


@pytest.mark.parametrize("N", [1024, 4096, 32768, 131072, 1048576])
@pytest.mark.parametrize("d,base", [(64, 1e6), (128, 1e7), (128, 5e5)])
def test_count_vs_closed_form_interval(oracle_lib, N, d, base):
    """Exact discrete whole-prefill and decode reductions sit within the paper's
    1-2 point integral-approximation error of eq:Rgen (we allow 2 points)."""
    w = oracle_lib.window_widths(d, base, 2.0, n_ctx=N + 1)
    T, C = oracle_lib.count_terms(w, N, 0, N)
    exact = 1 - T / (C * d / 2)
    assert abs(exact - R_interval(1, N, d, base, 2.0)) < 0.02
    T, C = oracle_lib.count_terms(w, 1, N, N)
    exact_dec = 1 - T / (C * d / 2)
    wmin = 4 * math.pi
    dec = (math.log(N / wmin) - 1 + wmin / N) / math.log(base)   # App. C Step 2, exact last row
    assert abs(exact_dec - dec) < 0.02
    # the appended-context interval [N/2, N] of App. C
    T, C = oracle_lib.count_terms(w, N - N // 2, N // 2, N)
    exact_half = 1 - T / (C * d / 2)
    assert abs(exact_half - R_interval(N // 2, N, d, base, 2.0)) < 0.02


def test_saturation_constant_terms_per_row(oracle_lib):
    """Past N >= k*lambda_max every row keeps the same sum over pairs (Sec. 4 fact
    (iii); App. C Step 3): B=100, d=8, k=2 gives floor widths [12, 39, 125, 397]."""
    w = oracle_lib.window_widths(8, 100.0, 2.0)
    assert list(np.floor(w).astype(int)) == [12, 39, 125, 397]
    per_row = int(np.sum(np.floor(w) + 1))
    assert per_row == 577
    for p in (397, 398, 1000, 5000):
        T, C = oracle_lib.count_terms(w, 1, p, p + 1)
        assert T == per_row
    # O(N) total: the count grows linearly once saturated
    T1, _ = oracle_lib.count_terms(w, 1000, 4000, 10_000)
    T2, _ = oracle_lib.count_terms(w, 2000, 4000, 10_000)
    assert T2 == 2 * T1 == 2 * 1000 * per_row
    # decode reduction tends to 1 beyond saturation
    red = [1 - oracle_lib.count_terms(w, 1, N, N)[0] / (4 * N) for N in (1000, 10_000, 100_000)]
    assert red[0] < red[1] < red[2] < 1


def test_window_widths_basics(oracle_lib):
    # theta' = 0 is a position-free pair: width = N (never pruned within N)
    w = oracle_lib.window_widths(4, 10.0, 2.0, theta=np.array([1.0, 0.0]), n_ctx=1000.0)
    assert w[1] == 1000.0 and w[0] == pytest.approx(4 * math.pi)
    # min(k lambda, N)
    w = oracle_lib.window_widths(8, 100.0, 2.0, n_ctx=50.0)
    assert math.floor(w[0]) == 12 and math.floor(w[1]) == 39
    assert w[2] == 50.0 and w[3] == 50.0
    # non-decreasing in r for every workload table
    for wl in W.WORKLOADS.values():
        th = W.workload_theta(wl)
        ww = oracle_lib.window_widths(wl.head_dim, wl.rope_base, wl.k,
                                      th.numpy() if th is not None else None)
        assert np.all(np.diff(ww) >= 0)
    with pytest.raises(ValueError):
        oracle_lib.window_widths(8, 100.0, 0.0)
    with pytest.raises(ValueError):
        oracle_lib.window_widths(8, 100.0, float("nan"))


# ----------------------------------------------------------------------------
# window family of App. A (eq:family) and the retention profiles
# ----------------------------------------------------------------------------
def test_retention_profiles_follow_app_a(oracle_lib):
    """Variable-k profile: 16 at the highest frequency (r = 0) down to 2 at the
    lowest, falling by 14/(d/2 - 1) per pair; k-geometric: same end points, a
    constant ratio; constant: k everywhere."""
    for d in (64, 128):
        n = d // 2
        ka = oracle_lib.retention_profile(d, "arithmetic", 16.0, 2.0)
        assert ka[0] == 16.0 and ka[-1] == pytest.approx(2.0, abs=1e-12)
        np.testing.assert_allclose(np.diff(ka), -14.0 / (n - 1), rtol=1e-12)
        kg = oracle_lib.retention_profile(d, "geometric", 16.0, 2.0)
        assert kg[0] == 16.0 and kg[-1] == pytest.approx(2.0, rel=1e-12)
        np.testing.assert_allclose(kg[1:] / kg[:-1], (2.0 / 16.0) ** (1.0 / (n - 1)), rtol=1e-12)
        # the geometric profile falls faster at high frequencies
        assert np.all(kg[1:-1] < ka[1:-1])
        assert np.all(oracle_lib.retention_profile(d, "constant", 3.0) == 3.0)


def test_family_default_point_is_the_default_window(oracle_lib):
    """k_r = k, gamma = 1, a = 0, beta = 0, cap = N is eq:window (App. A)."""
    for d, base, kwin, N in [(64, 1e6, 2.0, 32768), (128, 1e7, 2.0, 1 << 20), (8, 100.0, 1.0, 300)]:
        wf = oracle_lib.family_widths(d, base, np.full(d // 2, kwin), cap=N)
        wd = oracle_lib.window_widths(d, base, kwin, n_ctx=N)
        np.testing.assert_array_equal(wf, wd)
    th = W.llama3_theta(128, 5e5).numpy()
    wf = oracle_lib.family_widths(128, 0.0, np.full(64, 2.0), cap=65536, theta=th)
    np.testing.assert_array_equal(wf, oracle_lib.window_widths(128, 0.0, 2.0, th, n_ctx=65536))
    # a position-free pair is never pruned, whatever the knobs (App. A)
    wf = oracle_lib.family_widths(4, 0.0, [2.0, 0.0], gamma=0.5, beta=3.0, cap=10.0,
                                  theta=np.array([1.0, 0.0]))
    assert wf[1] == math.inf and wf[0] == pytest.approx(2.0 * math.sqrt(2 * math.pi))


@pytest.mark.parametrize("gamma", [0.8, 1.3])
@pytest.mark.parametrize("d,base", [(64, 1e6), (128, 5e5)])
def test_family_gamma_acts_as_base_rescaling(oracle_lib, gamma, d, base):
    """eq:gammasub: a gamma-window on base B is the default window on base B^gamma
    with w_min = k (2 pi)^gamma, so eq:redprefill holds with ln B -> gamma ln B
    (within the 1-2 point integral error of Sec. 4; 2 points allowed)."""
    kwin = 2.0
    wg = oracle_lib.family_widths(d, base, np.full(d // 2, kwin), gamma=gamma)
    wd = oracle_lib.window_widths(d, base ** gamma, kwin * (2 * math.pi) ** (gamma - 1))
    np.testing.assert_allclose(wg, wd, rtol=1e-13)
    wmin = kwin * (2 * math.pi) ** gamma
    for N in (32768, 131072):  # below saturation, N < k lambda_max^gamma
        assert N < wg.max()
        T, C = oracle_lib.count_terms(wg, N, 0, N)
        exact = 1 - T / (C * d / 2)
        closed = (math.log(N / wmin) - 1.5) / (gamma * math.log(base))
        assert abs(exact - closed) < 0.02, (N, exact, closed)


def test_family_linear_window_retention(oracle_lib):
    """k_r = 0, a = W degenerates to the linear window w = W (r+1)/(d/2) (App. A,
    App. C Step 4): one row of n keys retains 1 - n/(2W) of its terms for n <= W
    and W/(2n) past it, up to O(1/d) (4/d allowed)."""
    d, Wlin = 2048, 1000.0
    w = oracle_lib.family_widths(d, 1e4, np.zeros(d // 2), a=Wlin)
    np.testing.assert_allclose(w, Wlin * np.arange(1, d // 2 + 1) / (d // 2), rtol=1e-15)
    for n in (100, 500, 1000, 2000, 8000):
        T, C = oracle_lib.count_terms(w, 1, n - 1, n)
        kept = T / (C * d / 2)
        pred = 1 - n / (2 * Wlin) if n <= Wlin else Wlin / (2 * n)
        assert abs(kept - pred) < 4.0 / d, (n, kept, pred)


def test_family_sliding_window_counts_and_scores(oracle_lib):
    """Every pair at one width S (k_r = 0, beta = cap = S): the sliding-window
    special case of App. A.  Count = sum over rows of min(p + 1, S + 1) cells, times
    d/2; scores are the full dot product for z <= S and an empty sum (0) beyond."""
    d, S = 16, 37
    w = oracle_lib.family_widths(d, 1e4, np.zeros(d // 2), beta=S, cap=S)
    assert np.all(w == S)
    for n_q, q0, n_k in [(300, 0, 300), (50, 400, 450), (10, 0, 5)]:
        T, C = oracle_lib.count_terms(w, n_q, q0, n_k)
        cells = sum(min(p + 1, n_k) - max(0, p - S) for p in range(q0, q0 + n_q)
                    if max(0, p - S) <= min(p, n_k - 1))
        assert T == cells * d // 2
    rng = np.random.default_rng(17)
    n = 90
    q = bf16_grid(rng, (1, n, 1, d))
    k = bf16_grid(rng, (1, n, 1, d))
    s = oracle_lib.scores(q, k, 0, w)
    full = q[0, :, 0] @ k[0, :, 0].T / math.sqrt(d)
    z = np.arange(n)[:, None] - np.arange(n)[None, :]
    want = np.where(z < 0, -np.inf, np.where(z > S, 0.0, full))
    np.testing.assert_allclose(s, want, atol=1e-12)


def test_family_floor_and_ceiling(oracle_lib):
    """The floor beta keeps every pair at distances z <= beta (scores equal the full
    dot product there); the ceiling cap prunes every pair past it (scores 0)."""
    d, base, beta, cap = 16, 1e4, 30.0, 200.0
    w = oracle_lib.family_widths(d, base, np.full(d // 2, 2.0), beta=beta, cap=cap)
    wd = oracle_lib.window_widths(d, base, 2.0)
    np.testing.assert_array_equal(w, np.minimum(np.maximum(wd, beta), cap))
    assert w.min() == beta and w.max() == cap  # both clamps bind for this base
    rng = np.random.default_rng(23)
    n = 260
    q = bf16_grid(rng, (1, n, 1, d))
    k = bf16_grid(rng, (1, n, 1, d))
    s = oracle_lib.scores(q, k, 0, w)
    full = q[0, :, 0] @ k[0, :, 0].T / math.sqrt(d)
    z = np.arange(n)[:, None] - np.arange(n)[None, :]
    near = (z >= 0) & (z <= beta)
    np.testing.assert_allclose(s[near], full[near], atol=1e-12)
    assert np.all(s[z > cap] == 0.0)
    with pytest.raises(ValueError):   # 0 * inf: the width is undefined
        oracle_lib.family_widths(4, 10.0, [0.0, 1.0], gamma=1e6)


# ----------------------------------------------------------------------------
# rounded slice of Sec. 3.3 (kept low-frequency slice rounded up to MMA K-steps)
# ----------------------------------------------------------------------------
def test_rounded_slice_exact_window_misses_the_printed_ceilings(oracle_lib):
    """tab:c2e2e and the abstract's 57 % fit the rounded slice, not the exact window."""
    w = oracle_lib.window_widths(128, 1e7, 2.0)
    for N, ceil_printed in [(262144, 1.31), (524288, 1.35), (1048576, 1.40)]:
        T, C = oracle_lib.count_terms(w, N, 0, N)
        s = T / (C * 64)
        assert 2 / (1 + s) - ceil_printed > 0.04


@pytest.mark.parametrize("seed", range(6))
def test_rounded_slice_atom1_is_the_window_and_counts_agree(oracle_lib, seed):
    """atom = 1 rounds nothing; the by-distance count equals the per-pair closed form
    and brute force; rounded counts are at least the exact ones."""
    rng = np.random.default_rng(100 + seed)
    h = int(rng.integers(1, 20))
    w = np.sort(rng.uniform(-1, 60, h))
    n_q, q0, n_k = int(rng.integers(0, 40)), int(rng.integers(0, 50)), int(rng.integers(0, 70))
    exact = oracle_lib.count_terms(w, n_q, q0, n_k)
    assert oracle_lib.count_terms(w, n_q, q0, n_k, by_distance=True) == exact
    assert oracle_lib.count_terms(w, n_q, q0, n_k, atom=1) == exact
    assert exact == brute_force_count(w, n_q, q0, n_k)
    for atom in (2, 3, 8):
        Tr, Cr = oracle_lib.count_terms(w, n_q, q0, n_k, atom=atom)
        assert Cr == exact[1] and Tr >= exact[0]
        # brute force of the rounding rule, cell by cell
        T = 0
        for i in range(n_q):
            p = q0 + i
            for j in range(min(p, n_k - 1) + 1):
                n = int(np.sum(p - j <= w))
                T += min(h, atom * -(-n // atom))
        assert Tr == T


def test_rounded_slice_scores(oracle_lib):
    """Scores under the rounded slice: with one atom spanning every pair, a cell keeps
    all pairs as soon as the window keeps one (full dot product) and none otherwise (0);
    with 8-pair atoms the kept set is the lowest-frequency 8*ceil(n/8) pairs, a superset
    of the window's, and equals it where the widths are constant over each atom."""
    rng = np.random.default_rng(31)
    d, n = 32, 120
    h = d // 2
    q = bf16_grid(rng, (1, n, 1, d))
    k = bf16_grid(rng, (1, n, 1, d))
    w = oracle_lib.window_widths(d, 30.0, 1.0)  # widths 6 .. ~100: every count occurs
    full = q[0, :, 0] @ k[0, :, 0].T / math.sqrt(d)
    z = np.arange(n)[:, None] - np.arange(n)[None, :]
    s_all = oracle_lib.scores(q, k, 0, w, atom=h)
    any_kept = z <= w.max()
    want = np.where(z < 0, -np.inf, np.where(any_kept, full, 0.0))
    np.testing.assert_allclose(s_all, want, atol=1e-12)
    # 8-pair atoms, against the sum over the kept suffix written per cell
    s8 = oracle_lib.scores(q, k, 0, w, atom=8)
    for i in range(0, n, 7):
        for j in range(0, i + 1, 5):
            cnt = int(np.sum(i - j <= w))
            r0 = h - min(h, 8 * -(-cnt // 8))
            x = sum(q[0, i, 0, r] * k[0, j, 0, r] + q[0, i, 0, r + h] * k[0, j, 0, r + h]
                    for r in range(r0, h))
            assert s8[i, j] == pytest.approx(x / math.sqrt(d), abs=1e-12)
    # widths constant over each 8-pair atom: rounding changes nothing
    wc = np.repeat(np.array([5.0, 40.0]), 8)
    np.testing.assert_array_equal(oracle_lib.scores(q, k, 0, wc, atom=8),
                                  oracle_lib.scores(q, k, 0, wc))
    # the rounded slice needs a window whose kept pairs are a low-frequency suffix
    with pytest.raises(ValueError):
        oracle_lib.scores(q, k, 0, w[::-1].copy(), atom=8)
