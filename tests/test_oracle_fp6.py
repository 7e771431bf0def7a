"""Pins of the FP6 reference (int4 codes carried as e3m2 six-bit floats).

The decoder is checked against the landmarks the OCP Microscaling Formats v1.0
specification fixes for FP6 E3M2 (largest normal 28, smallest normal 2^-2,
smallest subnormal 2^-4, no infinities or NaNs, a sign bit), the encoder
against exactness and uniqueness, the layout against hand-placed bits and a
round trip, and the product against brute-force integer dot products."""
import numpy as np
import pytest

from oracle import fp6 as F
from oracle import oracle as O


def test_format_landmarks():
    assert F.e3m2_value(0b011111) == 28.0           # largest normal: 2^(7-3) x 1.75
    assert F.e3m2_value(0b000100) == 0.25           # smallest normal: 2^(1-3)
    assert F.e3m2_value(0b000001) == 0.0625         # smallest subnormal: 2^-2 x 1/4
    assert F.e3m2_value(0b000011) == 0.1875         # largest subnormal
    assert F.e3m2_value(0b001100) == 1.0            # exponent field 3 is 2^0
    vals = [F.e3m2_value(b) for b in range(64)]
    assert all(np.isfinite(vals))                   # no Inf / NaN encodings
    pos = vals[:32]
    assert pos == sorted(pos) and len(set(pos)) == 32          # monotone, no duplicates
    assert [vals[32 + b] for b in range(32)] == [-v for v in pos]   # sign bit


def test_every_int4_code_is_exact_and_unique():
    for q in range(-8, 8):
        b = F.encode(q)
        assert F.e3m2_value(b) == q
        assert sum(1 for x in range(64) if F.e3m2_value(x) == q and not (q == 0 and x >> 5)) == 1
    assert F.encode(0) == 0
    with pytest.raises(ValueError):
        F.encode(9)                                  # 9 = 1.125 x 8 needs a third mantissa bit


def test_products_and_sums_are_exact_in_fp32():
    # every product of two codes is an integer of magnitude <= 64, so a sum of
    # K <= 131072 products stays below 2^24: fp32 accumulation is exact in any order
    prods = {F.e3m2_value(F.encode(a)) * F.e3m2_value(F.encode(b)) for a in range(-8, 8) for b in range(-8, 8)}
    assert max(abs(p) for p in prods) == 64 and all(p == int(p) for p in prods)
    assert 64 * 131072 <= 2 ** 24


def test_hand_placed_bits():
    K = 128
    for k, q in ((0, 1), (1, -8), (21, 7), (22, -3), (31, 5), (32, 2), (127, -1)):
        codes = np.zeros((1, K), np.int64)
        codes[0, k] = q
        data = F.to_fp6(codes)
        c, j = divmod(k, 32)
        bit = 6 * j                                   # within the 192-bit chunk
        frag = bytes(data[0, 16 * c: 16 * c + 16]) + bytes(data[0, 64 + 8 * c: 64 + 8 * c + 8])
        word = int.from_bytes(frag, "little")
        assert word == F.encode(q) << bit
        # everything else in the block is zero
        others = np.delete(data[0], list(range(16 * c, 16 * c + 16)) + list(range(64 + 8 * c, 72 + 8 * c)))
        assert not others.any()
    # code 21 straddles the 16 / 8 byte split: bits 126..131
    codes = np.zeros((1, K), np.int64)
    codes[0, 21] = -8                                 # 0b111000
    d = F.to_fp6(codes)[0]
    assert d[15] == (0b111000 << 6) & 0xFF and d[64] == 0b111000 >> 2


@pytest.mark.parametrize("K", [64, 128, 192, 512])
def test_round_trip_and_padding(K):
    rng = np.random.default_rng(K)
    codes = rng.integers(-8, 8, (5, K))
    data = F.to_fp6(codes)
    assert data.shape == (5, 96 * ((K + 127) // 128))
    assert np.array_equal(F.from_fp6(data, K), codes)
    if K % 128:
        # the padded half block holds zero codes
        assert not data[:, -96 + 32:-32].any() and not data[:, -16:].any()
    # the conversion from the packed int4 layout agrees
    assert np.array_equal(F.codes_to_fp6(F.pack_int4(codes)), data)
    assert np.array_equal(O.unpack(F.pack_int4(codes)), codes)


def test_gemm_is_the_int4_gemm_of_the_codes():
    rng = np.random.default_rng(3)
    M, N, K = 3, 5, 192
    qa = rng.integers(-8, 8, (M, K))
    qw = rng.integers(-8, 8, (N, K))
    s_a = rng.uniform(0.1, 1, M).astype(np.float32)
    s_w = rng.uniform(1e-3, 1e-2, N).astype(np.float32)
    Y, acc = F.gemm(F.to_fp6(qa), s_a, F.to_fp6(qw), s_w, K)
    brute = np.array([[sum(int(qa[i, k]) * int(qw[n, k]) for k in range(K)) for n in range(N)] for i in range(M)])
    assert np.array_equal(acc, brute)
    rY, racc = O.gemm(F.pack_int4(qa), s_a, F.pack_int4(qw), s_w)
    assert np.array_equal(acc, racc) and np.array_equal(Y.view(np.uint16), rY.view(np.uint16))


def test_gemm_rejects_non_codes():
    K = 128
    bad = F.to_fp6(np.zeros((1, K), np.int64))
    bad[0, 0] = 0b000011                               # code 0 becomes 0.1875: a subnormal, not a code
    with pytest.raises(ValueError):
        F.gemm(bad, np.ones(1, np.float32), F.to_fp6(np.zeros((1, K), np.int64)), np.ones(1, np.float32), K)
