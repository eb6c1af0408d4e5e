"""Pins of the oracle's RoPE rotation (Sec. 3.1), the reference of decode from
unrotated caches.  Each check compares it with something other than itself: the
complex-exponential form of the rotation, the group law of rotations, the pair
decomposition of the score (eq:pair) and hand-computed values."""
import math

import numpy as np
import pytest
import torch

import oracle


def _theta(d, base):
    return base ** (-2.0 * np.arange(d // 2) / d)


def _x(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def test_rope_matches_complex_exponential():
    """Pair r as the complex number x_r + i x_{r+d/2}, multiplied by e^{i pos theta_r}."""
    d, base = 16, 1e4
    x = _x((2, 7, 3, d), 1)
    pos = np.array([0, 1, 5, 100, 4097, 131071, 1048575])
    th = _theta(d, base)
    y = oracle.rope_rotate(x, pos, th)
    z = (x[..., : d // 2] + 1j * x[..., d // 2:]) * np.exp(1j * pos[:, None] * th)[None, :, None, :]
    assert np.abs(y[..., : d // 2] - z.real).max() < 1e-12
    assert np.abs(y[..., d // 2:] - z.imag).max() < 1e-12


def test_rope_hand_values():
    """d = 2, theta = pi/2: (1, 0) turns a quarter per position."""
    x = np.array([[[1.0, 0.0]]] * 4)[None]            # [1, 4, 1, 2]
    y = oracle.rope_rotate(x, np.arange(4), np.array([math.pi / 2]))
    want = np.array([[1, 0], [0, 1], [-1, 0], [0, -1]], dtype=np.float64)
    assert np.abs(y[0, :, 0, :] - want).max() < 1e-15


def test_rope_identity_at_zero_and_norms():
    d = 64
    x = _x((1, 5, 2, d), 2)
    th = _theta(d, 1e6)
    assert np.array_equal(oracle.rope_rotate(x, np.zeros(5), th), x)
    y = oracle.rope_rotate(x, np.array([3, 77, 1000, 65536, 999999]), th)
    n0 = x[..., : d // 2] ** 2 + x[..., d // 2:] ** 2
    n1 = y[..., : d // 2] ** 2 + y[..., d // 2:] ** 2
    assert np.abs(n1 - n0).max() < 1e-12 * n0.max()


def test_rope_composition():
    """Rotating by m1 and then m2 is rotating by m1 + m2."""
    d = 32
    x = _x((1, 4, 2, d), 3)
    th = _theta(d, 1e4)
    m1, m2 = np.array([1, 10, 300, 7000]), np.array([5, 0, 1234, 90000])
    y = oracle.rope_rotate(oracle.rope_rotate(x, m1, th), m2, th)
    assert np.abs(y - oracle.rope_rotate(x, m1 + m2, th)).max() < 1e-10


@pytest.mark.parametrize("n,m", [(5, 2), (4096, 17), (1048576, 917505)])
def test_rope_score_is_pair_sum_of_relative_position(n, m):
    """eq:pair: q~(n) . k~(m) = sum_r a_r cos(z theta_r) + b_r sin(z theta_r), z = n - m,
    with a_r = q_r k_r + q_{r+h} k_{r+h} and b_r = q_r k_{r+h} - q_{r+h} k_r."""
    d = 128
    h = d // 2
    th = _theta(d, 5e5)
    q = _x((1, 1, 1, d), 4)
    k = _x((1, 1, 1, d), 5)
    s = float((oracle.rope_rotate(q, [n], th) * oracle.rope_rotate(k, [m], th)).sum())
    qv, kv = q.ravel(), k.ravel()
    a = qv[:h] * kv[:h] + qv[h:] * kv[h:]
    b = qv[:h] * kv[h:] - qv[h:] * kv[:h]
    z = n - m
    want = float((a * np.cos(z * th) + b * np.sin(z * th)).sum())
    assert abs(s - want) < 1e-9 * (np.abs(a).sum() + np.abs(b).sum())


def test_rope_bf16_input_is_its_exact_value():
    g = torch.Generator().manual_seed(6)
    x = torch.randn((1, 3, 2, 16), generator=g).to(torch.bfloat16)
    th = _theta(16, 1e4)
    y1 = oracle.rope_rotate(x, [0, 9, 4000], th)
    y2 = oracle.rope_rotate(x.to(torch.float64).numpy(), [0, 9, 4000], th)
    assert np.array_equal(y1, y2)


# ---------------------------------------------------------------------------
# planted mistakes: each plausible slip in a rotation routine fails at least one of
# the checks above (written again here against a rotation passed in)
# ---------------------------------------------------------------------------
def _rot_variant(kind):
    def rot(x, positions, theta):
        x = np.asarray(x, dtype=np.float64)
        d = x.shape[-1]
        h = d // 2
        pos = np.asarray(positions, dtype=np.float64)
        th = np.asarray(theta, dtype=np.float64)
        if kind == "position_off_by_one":
            pos = pos + 1
        if kind == "theta_reversed":
            th = th[::-1]
        ang = pos[:, None] * th[None, :]
        c, s_ = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
        if kind == "interleaved_pairs":
            a, b = x[..., 0::2], x[..., 1::2]
        else:
            a, b = x[..., :h], x[..., h:]
        sgn = -1.0 if kind == "sine_sign" else 1.0
        first = a * c - sgn * b * s_
        second = b * c + sgn * a * s_
        if kind == "cos_sin_swapped":
            first, second = a * s_ - b * c, b * s_ + a * c
        out = np.empty_like(x)
        if kind == "interleaved_pairs":
            out[..., 0::2], out[..., 1::2] = first, second
        else:
            out[..., :h], out[..., h:] = first, second
        return out
    return rot


def _passes_pins(rot):
    d = 16
    th = _theta(d, 1e4)
    x = _x((2, 7, 3, d), 1)
    pos = np.array([0, 1, 5, 100, 4097, 131071, 1048575])
    y = rot(x, pos, th)
    z = (x[..., : d // 2] + 1j * x[..., d // 2:]) * np.exp(1j * pos[:, None] * th)[None, :, None, :]
    if np.abs(y[..., : d // 2] - z.real).max() > 1e-12 or np.abs(y[..., d // 2:] - z.imag).max() > 1e-12:
        return False
    hand = rot(np.array([[[1.0, 0.0]]] * 4)[None], np.arange(4), np.array([math.pi / 2]))
    if np.abs(hand[0, :, 0, :] - np.array([[1, 0], [0, 1], [-1, 0], [0, -1]])).max() > 1e-15:
        return False
    if not np.array_equal(rot(x, np.zeros(7), th), x):
        return False
    return True


def test_pins_accept_the_oracle():
    assert _passes_pins(oracle.rope_rotate)
    assert _passes_pins(_rot_variant("none"))


@pytest.mark.parametrize("kind", ["sine_sign", "interleaved_pairs", "position_off_by_one",
                                  "theta_reversed", "cos_sin_swapped"])
def test_pins_reject_planted_mistake(kind):
    assert not _passes_pins(_rot_variant(kind))
