"""CPU checks of the GPU-parity comparator and its derived error budget (no
device work).

error_budget accepts what the kernels' arithmetic can do to a peaked softmax
(scores accumulated in fp32 from bf16 products, exp2 of an fp32 argument, bf16
probabilities in the PV product, fp32 sums, a bf16 output), and
compare_rounding_bound rejects a missing rescale of O, a wrong normaliser and
probabilities rounded to fewer bits than bf16 keeps."""
import math

import numpy as np
import pytest
import torch

from parity import U16, compare_rounding_bound, error_budget


def _bf16(x):
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16).to(
        torch.float64).numpy()


def _round_bits(x, bits):
    """Round to `bits` significant bits, to nearest (ties away; enough for a mistake)."""
    x = np.asarray(x, dtype=np.float64)
    e = np.floor(np.log2(np.abs(np.where(x == 0, 1.0, x))))
    q = 2.0 ** (e - bits + 1)
    return np.where(x == 0, 0.0, np.round(x / q) * q)


def _case(seed, n_k=600, d=64, scale=0.25, q_amp=1.0):
    """One query row against n_k keys whose magnitude rises along the sequence, so
    the softmax is peaked and its maximum keeps rising; bf16 inputs."""
    rng = np.random.default_rng(seed)
    q = _bf16(rng.normal(size=d) * q_amp)
    k = _bf16(rng.normal(size=(n_k, d)) * np.linspace(0.5, 4.0, n_k)[:, None])
    v = _bf16(rng.normal(size=(n_k, d)))
    s = scale * (k @ q)
    sabs = np.abs(k) @ np.abs(q)
    m = s.max()
    p = np.exp(s - m)
    o = p @ v / p.sum()
    lse = m + np.log(p.sum())
    return q, k, v, s, sabs, o, lse


def _kernel_like(q, k, v, scale, tile=64, p_bits=None):
    """The kernels' arithmetic in numpy: fp32 scores, exp2 in fp32 against a lazily
    raised running max (threshold 2^8), fp32 normaliser, bf16 probabilities (or
    p_bits significant bits) in the PV sum, fp32 accumulation, bf16 output."""
    f32 = np.float32
    sc = f32(scale * math.log2(math.e))
    x = (k.astype(f32) @ q.astype(f32)).astype(f32)
    m_run, l_run = f32(-np.inf), f32(0)
    acc = np.zeros(v.shape[1], dtype=f32)
    for j0 in range(0, len(x), tile):
        xs = x[j0:j0 + tile]
        cand = f32(xs.max() * sc)
        if cand > m_run + f32(8):
            m_new = max(m_run, cand)
            alpha = f32(np.exp2(f32(m_run - m_new))) if np.isfinite(m_run) else f32(0)
            m_run = m_new
            l_run = f32(l_run * alpha)
            acc = (acc * alpha).astype(f32)
        p = np.exp2((xs * sc - m_run).astype(f32)).astype(f32)
        l_run = f32(l_run + p.sum(dtype=f32))
        pb = _bf16(p) if p_bits is None else _round_bits(p, p_bits)
        acc = (acc + (pb.astype(f32) @ v[j0:j0 + tile].astype(f32))).astype(f32)
    o = _bf16(acc / l_run)
    lse = float(m_run) * math.log(2.0) + math.log(float(l_run))
    return o, lse


def _budget(s, sabs, v, o, scale, d):
    return error_budget(s[None], sabs[None], v, o[None], scale, d, tile_keys=64)


def _rows(seed, n_rows=16, scale=0.25, q_amp=1.0, p_bits=None):
    """n_rows independent rows: (kernel-like outputs, exact outputs, budgets)."""
    got, ref, bnd, lg, lr = [], [], [], [], []
    for r in range(n_rows):
        q, k, v, s, sabs, o, lse = _case(100 * seed + r, scale=scale, q_amp=q_amp)
        o_k, lse_k = _kernel_like(q, k, v, scale, p_bits=p_bits)
        got.append(o_k)
        ref.append(o)
        bnd.append(_budget(s, sabs, v, o, scale, q.shape[0])[0])
        lg.append(lse_k)
        lr.append(lse)
    return np.array(got), np.array(lg), np.array(ref), np.array(lr), np.array(bnd)


@pytest.mark.parametrize("seed", [1, 2, 3])
@pytest.mark.parametrize("scale,q_amp", [(1.0, 2.0), (0.25, 1.0), (0.125, 1.0)])
def test_budget_holds_for_the_kernel_arithmetic(seed, scale, q_amp):
    """Scores of order 10^2 (scale 1) down to order 1: the kernels' arithmetic stays
    within the budget; at moderate scores its errors reach a good part of it (the
    budget is not vacuous)."""
    ratio, _ = compare_rounding_bound(*_rows(seed, scale=scale, q_amp=q_amp),
                                      f"seed {seed} scale {scale}")
    if scale < 1.0:
        assert ratio > 0.3


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_budget_rejects_missing_rescale(seed):
    """Keys before the last raise of the running max accumulated without their
    factor exp(m_old - m_new) (as if O were not rescaled when the max rose)."""
    q, k, v, s, sabs, o, lse = _case(seed, q_amp=2.0, scale=1.0)
    n = len(s)
    w = np.exp(s - s.max())
    w[: n // 2] = np.exp(s[: n // 2] - s[: n // 2].max())  # not rescaled
    o_bad = _bf16(w @ v / np.exp(s - s.max()).sum())
    with pytest.raises(AssertionError):
        compare_rounding_bound(o_bad[None], np.array([lse]), o[None], np.array([lse]),
                               _budget(s, sabs, v, o, 1.0, q.shape[0]))


def test_budget_rejects_wrong_normaliser():
    q, k, v, s, sabs, o, lse = _case(5, q_amp=2.0, scale=1.0)
    p = np.exp(s - s.max())
    o_bad = _bf16((_bf16(p) @ v) / (p.sum() * 1.05))
    bound = _budget(s, sabs, v, o, 1.0, q.shape[0])
    with pytest.raises(AssertionError):
        compare_rounding_bound(o_bad[None], np.array([lse]), o[None], np.array([lse]), bound)
    # and the LSE check catches a normaliser off by more than 1e-3
    with pytest.raises(AssertionError):
        compare_rounding_bound(o[None], np.array([lse + np.log(1.01)]), o[None], np.array([lse]),
                               bound)


@pytest.mark.parametrize("seed", [1, 2, 3, 4, 5])
def test_budget_rejects_probabilities_rounded_to_6_bits(seed):
    """Probabilities carried with 6 significant bits instead of bf16's 8 (4x its
    rounding error) exceed the budget on 16 rows of moderate scores."""
    got, lg, ref, lr, bnd = _rows(seed, p_bits=6)
    with pytest.raises(AssertionError):
        compare_rounding_bound(got, lr, ref, lr, bnd)


def test_budget_terms_reduce_to_bf16_rounding_for_exact_scores():
    """With exact scores and exponentials (sabs = 0 and one valid key) the budget is
    the bf16 rounding of P and of O: 2^-8 |v| + 2^-8 |O| plus fp32 terms."""
    v = np.array([[1.0, -2.0, 0.5]])
    o = v.copy()
    b = error_budget(np.array([[0.0]]), np.array([[0.0]]), v, o, 1.0, 64, tile_keys=64)
    expect = U16 * np.abs(v) + U16 * np.abs(o)
    assert np.all(b >= expect) and np.all(b <= expect * 1.01)
