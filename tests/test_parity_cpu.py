"""CPU checks of the GPU-parity comparators themselves (no device work).

compare_rounding_bound accepts what bf16 rounding of the probabilities and of the
output can do to a peaked softmax, and rejects what a missing or wrong rescale of
O or of the normaliser does."""
import numpy as np
import pytest
import torch

from parity import compare_rounding_bound


def _bf16(x):
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16).to(
        torch.float64).numpy()


def _peaked_case(seed, n=600, d=32):
    rng = np.random.default_rng(seed)
    s = rng.normal(size=n) * 40.0 + np.linspace(0, 200, n)  # scores rising along the keys
    v = _bf16(rng.normal(size=(n, d)))
    m = s.max()
    p = np.exp(s - m)
    l = p.sum()
    o = p @ v / l
    oabs = p @ np.abs(v) / l
    lse = m + np.log(l)
    return s, v, p, l, o, oabs, lse


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_bound_accepts_bf16_rounding_of_p_and_o(seed):
    s, v, p, l, o, oabs, lse = _peaked_case(seed)
    o_gpu = _bf16((_bf16(p) @ v) / l)
    compare_rounding_bound(o_gpu[None], np.array([lse]), o[None], np.array([lse]), oabs[None])


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_bound_rejects_missing_rescale(seed):
    """Keys before the last raise of the running max are accumulated without their
    factor exp(m_old - m_new) (as if O were not rescaled when the max rose)."""
    s, v, p, l, o, oabs, lse = _peaked_case(seed)
    n = len(s)
    m_old = s[: n // 2].max()
    w = np.exp(s - s.max())
    w[: n // 2] = np.exp(s[: n // 2] - m_old)  # not rescaled
    o_bad = _bf16((w @ v) / l)
    with pytest.raises(AssertionError):
        compare_rounding_bound(o_bad[None], np.array([lse]), o[None], np.array([lse]), oabs[None])


def test_bound_rejects_wrong_normaliser():
    s, v, p, l, o, oabs, lse = _peaked_case(4)
    o_bad = _bf16((_bf16(p) @ v) / (l * 1.05))
    with pytest.raises(AssertionError):
        compare_rounding_bound(o_bad[None], np.array([lse]), o[None], np.array([lse]), oabs[None])
    # and the LSE check catches a normaliser off by more than 1e-3
    with pytest.raises(AssertionError):
        compare_rounding_bound(o[None], np.array([lse + np.log(1.01)]), o[None], np.array([lse]),
                               oabs[None])
