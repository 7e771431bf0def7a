"""GPU parity of the FP6 path (int4 codes carried as e3m2 on the FP6 matrix
cores) through the C ABI.

* the conversion of packed int4 codes to the FP6 operand layout equals the
  oracle's bit for bit, half-filled last blocks included;
* the GEMM on operands the oracle encoded (so independent of the GPU converter)
  gives the oracle's int32 accumulators and fp16 outputs bit for bit;
* on GPU-converted operands, at every tile plan and ragged edge, and at the
  largest K with the extreme sum 2^23, acc and Y equal the oracle's and
  w4a4_gemm's."""
import numpy as np
import pytest

import paper_2606_04945_amd as sq
from oracle import fp6 as F
from oracle import oracle as O
from gpu_util import assert_bits, assert_y, dev, host, pack_codes, say

pytestmark = pytest.mark.gpu
THREADS = 16


def codes(R, K, seed, lo=-8, hi=7):
    return np.random.default_rng(seed).integers(lo, hi + 1, (R, K))


@pytest.mark.parametrize("R,K", [(1, 64), (7, 128), (33, 4160), (300, 576)])
def test_conversion_bit_exact(R, K):
    q = codes(R, K, 100 + K)
    got = host(sq.codes_to_fp6(dev(pack_codes(q))))
    assert_bits(got, F.to_fp6(q), "fp6 operand")


def test_gemm_on_oracle_encoded_operands():
    M, N, K = 40, 48, 320                       # two and a half blocks: a half-filled last block
    qa, qw = codes(M, K, 1), codes(N, K, 2)
    rng = np.random.default_rng(3)
    s_a = rng.uniform(0.05, 3, M).astype(np.float32)
    s_w = rng.uniform(1e-4, 5e-3, N).astype(np.float32)
    Y, acc = sq.w4a4_gemm_fp6(dev(F.to_fp6(qa)), dev(s_a), dev(F.to_fp6(qw)), dev(s_w), K, want_acc=True)
    rY, racc = F.gemm(F.to_fp6(qa), s_a, F.to_fp6(qw), s_w, K)
    assert_bits(host(acc), racc, "acc")
    assert_y(host(Y), rY)


# 256 x 256 tiles (>= 512 of them), 128 x 128 (>= 256), 64 x 64; ragged M and N
SHAPES = [(1, 8, 64), (5, 136, 192), (77, 200, 4160), (300, 1032, 576), (1024, 1024, 1024),
          (2100, 4104, 3584), (4096, 8200, 256), (513, 4104, 12288)]


@pytest.mark.parametrize("M,N,K", SHAPES)
def test_gemm_bit_exact(M, N, K):
    qa, qw = codes(M, K, 10 + M), codes(N, K, 20 + N)
    Aq, Wq = pack_codes(qa), pack_codes(qw)
    rng = np.random.default_rng(4)
    s_a = rng.uniform(0.05, 3, M).astype(np.float32)
    s_w = rng.uniform(1e-4, 5e-3, N).astype(np.float32)
    say(f"gemm_fp6 M={M} N={N} K={K}")
    A6, W6 = sq.codes_to_fp6(dev(Aq)), sq.codes_to_fp6(dev(Wq))
    Y, acc = sq.w4a4_gemm_fp6(A6, dev(s_a), W6, dev(s_w), K, want_acc=True)
    Y, acc = host(Y), host(acc)
    rows = np.arange(M) if M * N * K <= 3e9 else np.unique(np.r_[0, M - 1, rng.choice(M, 24)])
    rY, racc = O.gemm(Aq[rows], s_a[rows], Wq, s_w, threads=THREADS)
    assert_bits(acc[rows], racc, "acc")
    assert_y(Y[rows], rY)
    # and the int4 path on the same codes agrees bit for bit
    Y4, acc4 = sq.w4a4_gemm(dev(Aq), dev(s_a), dev(Wq), dev(s_w), want_acc=True)
    assert_bits(acc, host(acc4), "acc vs w4a4_gemm")
    assert_bits(Y, host(Y4), "Y vs w4a4_gemm")


def test_gemm_at_the_largest_K():
    """K = 131072 with every product (-8)(-8) on row 0 / column 0: the sum is 2^23,
    the largest the format has to carry exactly."""
    K, M, N = 131072, 3, 16
    rng = np.random.default_rng(12)
    qa, qw = rng.integers(-8, 8, (M, K)), rng.integers(-8, 8, (N, K))
    qa[0, :] = -8
    qw[0, :] = -8
    Aq, Wq = pack_codes(qa), pack_codes(qw)
    s_a = np.ones(M, np.float32)
    s_w = np.full(N, 1e-7, np.float32)
    Y, acc = sq.w4a4_gemm_fp6(sq.codes_to_fp6(dev(Aq)), dev(s_a), sq.codes_to_fp6(dev(Wq)), dev(s_w), K,
                              want_acc=True)
    ref = qa.astype(np.int64) @ qw.T.astype(np.int64)
    assert ref[0, 0] == 1 << 23
    assert_bits(host(acc), ref.astype(np.int32), "acc")
    rY, _ = O.gemm(Aq, s_a, Wq, s_w, threads=THREADS)
    assert_y(host(Y), rY)


def test_empty_and_acc_only():
    K = 128
    A6 = sq.codes_to_fp6(dev(pack_codes(codes(0, K, 5))))
    assert A6.shape == (0, 96)
    qa, qw = codes(4, K, 6), codes(8, K, 7)
    _, acc = sq.w4a4_gemm_fp6(sq.codes_to_fp6(dev(pack_codes(qa))), dev(np.ones(4, np.float32)),
                              sq.codes_to_fp6(dev(pack_codes(qw))), dev(np.ones(8, np.float32)), K,
                              want_Y=False, want_acc=True)
    assert_bits(host(acc), (qa @ qw.T).astype(np.int32), "acc")
