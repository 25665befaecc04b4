"""CPU checks of the parity bars themselves (tests/parity_util.py).

The LSE bound: the joint and spatial forward sum the probabilities of a row in
the bf16 precision of their P V products. Here that sum is reproduced on the
host (probabilities formed in fp32 against a base, rounded to bf16 to nearest
even, summed in fp32) and its log-sum-exp compared with the exact fp64 value,
on random rows, rows with one dominant key and a constructed near-worst case:
the error must stay within lse_bound, and the worst case must come close to it
(so the bound is not loose by orders of magnitude).
"""
import math

import numpy as np
import pytest

from parity_util import MAX_ABS, assert_close, bf16_spacing, lse_bound

torch = pytest.importorskip("torch")


def _bf16(x: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.bfloat16).to(torch.float32).numpy()


def _lse_bf16_sum(s: np.ndarray, base: float) -> float:
    """log-sum-exp of natural-log scores s, probabilities against `base` (log2 units),
    rounded to bf16, summed in fp32 tile by tile as the forward does."""
    log2e = np.float32(1.4426950408889634)
    p = np.exp2((s.astype(np.float32) * log2e - np.float32(base)).astype(np.float32)).astype(np.float32)
    pb = _bf16(p)
    acc = np.float32(0.0)
    for t in range(0, len(pb), 64):
        acc = np.float32(acc + pb[t:t + 64].sum(dtype=np.float32))
    return float((np.float32(base) + np.log2(acc, dtype=np.float32)) * np.float32(math.log(2.0)))


def _lse_exact(s: np.ndarray) -> float:
    m = s.max()
    return float(m + np.log(np.exp(s - m).sum()))


@pytest.mark.parametrize("n", [1, 144, 4096])
def test_lse_bound_covers_bf16_probability_sums(n):
    rng = np.random.Generator(np.random.PCG64(n))
    worst = 0.0
    for trial in range(200):
        s = rng.standard_normal(n) * rng.choice([0.1, 1.0, 3.0])
        if trial % 4 == 1:
            s[rng.integers(n)] += 12.0  # one dominant key
        s = s.astype(np.float32).astype(np.float64)
        base = float(np.float32(s.max() * 1.4426950408889634 - rng.uniform(0, 13)))
        worst = max(worst, abs(_lse_bf16_sum(s, base) - _lse_exact(s)))
    assert worst <= lse_bound(n), (worst, lse_bound(n))


def test_lse_bound_is_nearly_reached():
    """A single key whose probability against the base sits just below the rounding
    midpoint above 1 (1 + 2^-8 - tiny rounds down to 1): the error approaches 2^-8."""
    x = 1.0 + 2.0 ** -8 - 2.0 ** -20
    s = np.array([math.log(x)])
    err = abs(_lse_bf16_sum(s, 0.0) - _lse_exact(s))
    assert 0.9 * 2.0 ** -8 < err <= lse_bound(1)


def test_bf16_bar_grows_only_past_representability():
    """Below magnitude 4 the bf16 max-abs bar is the stated 2e-2; from 4 on, one bf16
    spacing (0.03125 in [4, 8), 0.0625 in [8, 16)), as 2e-2 is then less than a spacing."""
    ref = np.array([0.5, -3.9] + [1.0] * 98)
    assert bf16_spacing(3.9) < MAX_ABS
    assert_close("o", ref + np.r_[0.0, 0.019, np.zeros(98)], ref)
    with pytest.raises(AssertionError):
        assert_close("o", ref + np.r_[0.0, 0.021, np.zeros(98)], ref)
    for top in (5.0, 9.0):
        ref = np.array([top] + [1.0] * 99)
        assert bf16_spacing(top) > MAX_ABS
        assert_close("dv", ref + np.r_[bf16_spacing(top) * 0.99, np.zeros(99)], ref)
        with pytest.raises(AssertionError):
            assert_close("dv", ref + np.r_[bf16_spacing(top) * 1.01, np.zeros(99)], ref)


def test_lse_bar_is_absolute():
    """LSE keeps an absolute bar (its reference is about ln N, not below 1)."""
    ref = np.full(50, 11.0)
    assert_close("lse", ref + 0.9 * lse_bound(2 ** 17), ref)
    with pytest.raises(AssertionError):
        assert_close("lse", ref + 1.1 * lse_bound(2 ** 17), ref)
