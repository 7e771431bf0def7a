"""The quantisers form a code as rint(x * y) with y = 1 / s (correctly rounded)
and fall back to the correctly rounded divide x / s only when x * y lies within
2^-18 (4-bit) or 2^-14 (8-bit) of a half-integer.  This checks that rule on the
CPU against rint(fl(x / s)) for every finite fp16 x with |x| <= absmax, at
thousands of scales s = fl(absmax / qmax) whose absmax is itself an fp16 value
(so that many x / s fall on or next to half-integers), and that the threshold
is not loose by a large margin: the largest gap between x * y and fl(x / s)
seen is below half of it."""
import numpy as np
import pytest

F32 = np.float32


def rule_codes(x, s, qmax, near):
    with np.errstate(over="ignore", divide="ignore", invalid="ignore"):
        y = F32(1) / s                                   # correctly rounded (numpy float32 divide)
        q0 = x * y                                       # one rounding
    r = np.rint(q0)
    with np.errstate(invalid="ignore"):
        slow = ~((F32(0.5) - np.abs(q0 - r)) > near)      # NaN products take the divide
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(slow, np.rint(x / s), r)
    return np.clip(r, -(qmax + 1), qmax), slow


@pytest.mark.parametrize("qmax,near", [(7, 2.0 ** -18), (127, 2.0 ** -14)])
def test_rule_equals_divide(qmax, near):
    h = np.arange(65536, dtype=np.uint16).view(np.float16)
    h = h[np.isfinite(h)].astype(F32)
    mags = np.unique(np.abs(h[h != 0]))
    rng = np.random.default_rng(qmax)
    picks = np.concatenate([mags[:200], mags[-200:], rng.choice(mags, 2000, replace=False)])
    worst = 0.0
    slow_total = 0
    for a in picks:
        s = F32(a) / F32(qmax)                           # the kernel's scale
        x = h[np.abs(h) <= a]
        want = np.clip(np.rint(x / s), -(qmax + 1), qmax)
        got, slow = rule_codes(x, s, F32(qmax), F32(near))
        assert np.array_equal(got, want), (qmax, a)
        gap = np.abs((x * (F32(1) / s)).astype(np.float64) - (x / s).astype(np.float64))
        worst = max(worst, float(gap.max()))
        slow_total += int(slow.sum())
    assert worst < near / 2, worst                       # the bound the rule relies on, with margin
    assert slow_total > 0                                # the divide path is exercised


def _divide_codes(x, s, qmax):
    with np.errstate(divide="ignore", invalid="ignore"):
        return np.clip(np.rint(x / s), -(qmax + 1), qmax)


@pytest.mark.parametrize("qmax,near", [(7, 2.0 ** -18), (127, 2.0 ** -14)])
def test_rule_fp32_edges(qmax, near):
    """fp32 inputs: subnormal scales (1 / s overflows to inf), zero and
    non-finite values, and x well beyond absmax (the clamp decides)."""
    rng = np.random.default_rng(100 + qmax)
    tiny = np.array([1, 2, 3, 7, 100, 2 ** 20, 2 ** 23 - 1], np.uint32).view(F32)   # subnormals
    scales = np.concatenate([tiny / F32(qmax), tiny,
                             (rng.random(500) * 10.0 ** rng.integers(-30, 30, 500)).astype(F32)])
    scales = scales.astype(F32)
    for s in scales[scales > 0]:                         # s == 0 gives code 0 without the rule
        x = np.concatenate([
            (rng.standard_normal(4000) * s * qmax).astype(F32),
            (rng.integers(-4 * qmax, 4 * qmax, 4000) + F32(0.5)).astype(F32) * s,   # near half-integers
            (rng.standard_normal(200) * s * 1e4).astype(F32),
            np.array([0.0, -0.0, np.inf, -np.inf, np.nan], F32)])
        got, _ = rule_codes(x, s, F32(qmax), F32(near))
        want = _divide_codes(x, s, qmax)
        assert np.array_equal(got, want, equal_nan=True), (qmax, s)
