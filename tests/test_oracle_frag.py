"""Pins of the fragment-ordered weight reference.

The layout is checked against byte offsets worked out by hand from its
definition, against being a bijection onto the non-padding bytes, against a
round trip with zero padding at a ragged N and a half k step, and the GEMM
against brute-force integer dot products of the codes; the int8 layout at
hand-worked offsets (64 codes a k step) and its GEMM against brute force."""
import numpy as np
import pytest

from oracle import frag as F
from oracle import oracle as O


def test_sizes():
    assert F.frag_bytes(16, 128) == 1024
    assert F.frag_bytes(40, 320) == 3 * 3 * 1024          # 3 groups, K/2 = 160 bytes -> 3 steps
    assert F.frag_bytes(24576, 4096) == 1536 * 32 * 1024
    assert F.frag_bytes(0, 128) == 0


def test_hand_worked_offsets():
    N, K = 40, 320                                         # G = 3, T = 3; last group rows 32..39, last step half
    cases = {(0, 0): 0,                                    # row 0, byte 0: block (0, 0), unit 0
             (1, 0): 16,                                   # row 1: unit 1
             (0, 16): 256,                                 # byte 16: j = 1, unit 16
             (0, 63): 48 * 16 + 15,                        # byte 63: j = 3, unit 48, last byte
             (0, 64): 3 * 1024,                            # byte 64: block (g 0, t 1) = 1 x 3 + 0
             (17, 0): 1024 + 16,                           # row 17: block (g 1, t 0), unit 1
             (17, 64): 4 * 1024 + 16,                      # block (g 1, t 1) = 1 x 3 + 1
             (39, 159): 8 * 1024 + 23 * 16 + 15}           # row 39, byte 159: block (g 2, t 2), unit 16 + 7
    for (row, byte), off in cases.items():
        W = np.zeros((N, K // 2), np.uint8)
        W[row, byte] = 0xA5
        flat = F.to_frag(W, K).reshape(-1)
        assert flat.size == F.frag_bytes(N, K)
        assert flat[off] == 0xA5 and np.count_nonzero(flat) == 1, (row, byte)


@pytest.mark.parametrize("N,K", [(16, 128), (40, 320), (8, 64), (48, 4160)])
def test_bijection(N, K):
    ids = np.arange(1, N * K // 2 + 1, dtype=np.int64).reshape(N, K // 2)
    flat = F.to_frag(ids, K).reshape(-1)
    nz = flat[flat != 0]
    assert np.array_equal(np.sort(nz), ids.reshape(-1))   # every byte exactly once
    assert flat.size - nz.size == F.frag_bytes(N, K) - N * K // 2   # the rest is padding


@pytest.mark.parametrize("N,K", [(16, 128), (24, 192), (40, 320), (8, 64), (136, 4160)])
def test_round_trip_and_padding(N, K):
    W = np.random.default_rng(N + K).integers(0, 256, (N, K // 2)).astype(np.uint8)
    Wf = F.to_frag(W, K)
    assert Wf.dtype == np.uint8 and Wf.shape == ((K + 127) // 128, (N + 15) // 16, 1024)
    assert np.array_equal(F.from_frag(Wf, N, K), W)
    if N % 16 or K % 128:
        bad = Wf.copy().reshape(-1)
        pad = np.flatnonzero(F.to_frag(np.ones_like(W), K).reshape(-1) == 0)
        bad[pad[len(pad) // 2]] = 1
        with pytest.raises(ValueError):
            F.from_frag(bad, N, K)


def test_gemm_is_the_int4_gemm():
    rng = np.random.default_rng(5)
    M, N, K = 3, 24, 192                                  # ragged group and a half k step
    qa, qw = rng.integers(-8, 8, (M, K)), rng.integers(-8, 8, (N, K))
    pack = lambda q: ((q[:, 0::2] & 15) | ((q[:, 1::2] & 15) << 4)).astype(np.uint8)
    s_a = rng.uniform(0.1, 1, M).astype(np.float32)
    s_w = rng.uniform(1e-3, 1e-2, N).astype(np.float32)
    Y, acc = F.gemm(pack(qa), s_a, F.to_frag(pack(qw), K), s_w, N, K)
    brute = np.array([[sum(int(qa[i, k]) * int(qw[n, k]) for k in range(K)) for n in range(N)] for i in range(M)])
    assert np.array_equal(acc, brute)
    rY, _ = O.gemm(pack(qa), s_a, pack(qw), s_w)
    assert np.array_equal(Y.view(np.uint16), rY.view(np.uint16))


def test_q8_hand_worked_offsets():
    N, K = 24, 96                                          # G = 2, T = 2 (64 + 32 bytes a row)
    cases = {(0, 0): 0, (0, 17): 256 + 1,                  # byte 17: j = 1, unit 16
             (0, 64): 2 * 1024,                            # code 64 opens k step 1: block 1 x 2 + 0
             (23, 95): 3 * 1024 + (16 * 1 + 7) * 16 + 15}  # row 23, code 95: block (g 1, t 1), j 1, r 7
    for (row, k), off in cases.items():
        W = np.zeros((N, K), np.int8)
        W[row, k] = -91
        flat = F.to_frag_q8(W, K).reshape(-1)
        assert flat.size == 2 * 2 * 1024
        assert flat[off] == np.uint8(256 - 91) and np.count_nonzero(flat) == 1, (row, k)


def test_gemm_q8_is_the_int8_gemm():
    rng = np.random.default_rng(6)
    M, N, K = 3, 24, 96                                   # ragged group and a half k step
    qa = rng.integers(-128, 128, (M, K)).astype(np.int8)
    qw = rng.integers(-128, 128, (N, K)).astype(np.int8)
    qw[0] = -128
    s_a = rng.uniform(0.1, 1, M).astype(np.float32)
    s_w = rng.uniform(1e-4, 1e-3, N).astype(np.float32)
    Y, acc = F.gemm_q8(qa, s_a, F.to_frag_q8(qw, K), s_w, N, K)
    brute = np.array([[sum(int(qa[i, k]) * int(qw[n, k]) for k in range(K)) for n in range(N)] for i in range(M)])
    assert np.array_equal(acc, brute)
    rY, _ = O.gemm_q8(qa, s_a, qw, s_w)
    assert np.array_equal(Y.view(np.uint16), rY.view(np.uint16))
