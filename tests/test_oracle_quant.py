"""Pins of the oracle's per-row symmetric int4 quantiser (Sec. 3.1, Eq. 2-3 and 5, in
the symmetric form z = 0, s = absmax/7, ties to even)."""
import numpy as np
import pytest

from oracle import oracle as O


def test_hand_example():
    # absmax 7 -> s = 1 exactly, so the codes are the half-even roundings of the
    # values themselves: 3.5 -> 4, -3.5 -> -4, 0.5 -> 0, 1.5 -> 2, 2.5 -> 2, -0.5 -> 0.
    x = np.array([[7, -7, 3.5, -3.5, 0.5, 1.5, 2.5, -0.5]], np.float32)
    packed, s, q = O.quant_rows(x)
    assert s[0] == 1.0
    assert q.tolist() == [[7, -7, 4, -4, 0, 2, 2, 0]]
    # byte t = (q[2t] & 15) | (q[2t+1] & 15) << 4:
    # (7, -7) -> 0x97, (4, -4) -> 0xC4, (0, 2) -> 0x20, (2, 0) -> 0x02
    assert packed.tolist() == [[0x97, 0xC4, 0x20, 0x02]]
    assert O.unpack(packed).tolist() == q.tolist()


def test_hand_example_scaled():
    # absmax 14 -> s = 2: x/s = [7, 0.25, 0.75, -1.25, 2.5, -2.5, 3.5, 1] -> [7, 0, 1, -1, 2, -2, 4, 1]
    x = np.array([[14, 0.5, 1.5, -2.5, 5, -5, 7, 2]], np.float32)
    _, s, q = O.quant_rows(x)
    assert s[0] == 2.0
    assert q.tolist() == [[7, 0, 1, -1, 2, -2, 4, 1]]


def test_zero_row():
    packed, s, q = O.quant_rows(np.zeros((2, 64), np.float32))
    assert (s == 0).all() and (q == 0).all() and (packed == 0).all()


@pytest.mark.parametrize("amax", [1.0, 7.0, 0.3, 1234.5, 3.0e-3, 65504.0])
def test_exhaustive_fp16_values_vs_search(amax):
    """Every finite fp16 value with |v| <= amax, quantised in a row whose absmax is amax,
    equals a brute-force search for the code nearest to fl32(v / s), ties to even."""
    h = np.arange(65536, dtype=np.uint16)
    v = h.view(np.float16).astype(np.float32)
    v = v[np.isfinite(v) & (np.abs(v) <= amax)]
    row = np.concatenate([[np.float32(amax)], v]).astype(np.float32)
    pad = (-len(row)) % 2
    row = np.concatenate([row, np.zeros(pad, np.float32)])
    _, s, q = O.quant_rows(row[None, :])
    s32 = np.float32(amax) / np.float32(7.0)
    assert s[0] == s32
    ratio = (row / s32).astype(np.float32)          # IEEE fp32 quotient
    ref = O.nearest_code(ratio)
    assert (q[0] == ref).all()


def test_invariants_random_rows():
    rng = np.random.default_rng(3)
    x = (rng.standard_normal((300, 512)) * rng.uniform(1e-3, 1e3, (300, 1))).astype(np.float32)
    x[::7, rng.integers(0, 512)] *= 40                    # outliers
    _, s, q = O.quant_rows(x)
    amax = np.abs(x).max(axis=1)
    assert (s == (amax / np.float32(7)).astype(np.float32)).all()
    assert q.min() >= -7 and q.max() <= 7
    assert (np.abs(q).max(axis=1) == 7).all()
    # per-element error at most s/2 (up to the fp32 rounding of the quotient)
    err = np.abs(x.astype(np.float64) - s[:, None].astype(np.float64) * q)
    assert (err <= s[:, None] * (0.5 + 2.0 ** -20)).all()
