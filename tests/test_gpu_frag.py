"""GPU parity of the fragment-ordered weight path through the C ABI.

* the conversion of packed int4 weights to fragment order equals the oracle's
  bit for bit (ragged N, half-filled last k step included);
* the GEMM on weights the oracle reordered (so independent of the GPU
  converter) gives the oracle's int32 accumulators and fp16 outputs bit for bit;
* on GPU-converted weights, at every short-M plan (wide, mid-width and narrow
  layers; activations staged in LDS or read from L2; one to four row tiles),
  every tiled plan (with and without K splits; 64 x 64 ... 128 x 256 tiles; k
  groups within a workgroup) and at the largest K with the
  extreme sum 2^23, acc and Y equal the oracle's and w4a4_gemm's;
* the same for int8 codes (W8A8): conversion, GEMM on oracle-ordered weights,
  short-M and tiled plans, and the extreme sum 2^30 at K = 65536."""
import numpy as np
import pytest

import paper_2606_04945_amd as sq
from oracle import frag as F
from oracle import oracle as O
from gpu_util import assert_bits, assert_y, dev, host, pack_codes, say

pytestmark = pytest.mark.gpu
THREADS = 16


def codes(R, K, seed):
    return np.random.default_rng(seed).integers(-8, 8, (R, K))


@pytest.mark.parametrize("N,K", [(8, 64), (40, 320), (4104, 4160), (24576, 4096)])
def test_conversion_bit_exact(N, K):
    Wq = pack_codes(codes(N, K, N + K))
    got = host(sq.weights_to_frag(dev(Wq)))
    assert_bits(got, F.to_frag(Wq, K), "fragment-ordered weights")


def test_gemm_on_oracle_ordered_weights():
    M, N, K = 20, 40, 320                        # two row tiles, a ragged group, a half last k step
    qa, qw = codes(M, K, 1), codes(N, K, 2)
    rng = np.random.default_rng(3)
    s_a = rng.uniform(0.05, 3, M).astype(np.float32)
    s_w = rng.uniform(1e-4, 5e-3, N).astype(np.float32)
    Aq, Wf = pack_codes(qa), F.to_frag(pack_codes(qw), K)
    Y, acc = sq.w4a4_gemm_frag(dev(Aq), dev(s_a), dev(Wf), dev(s_w), want_acc=True)
    rY, racc = F.gemm(Aq, s_a, Wf, s_w, N, K)
    assert_bits(host(acc), racc, "acc")
    assert_y(host(Y), rY)


SHAPES = [
    # short M: wide (>= 1024 column groups), mid-width, narrow; LDS or L2 activations
    (1, 24576, 4096), (16, 24576, 4096), (32, 24576, 4096), (48, 24576, 4096), (33, 37888, 3584),
    (16, 12288, 4096), (17, 12296, 4160), (48, 8200, 12288),
    (1, 4096, 4096), (16, 4096, 12288), (5, 4104, 4160), (48, 3584, 18944), (1, 8, 64), (3, 24, 192),
    (3, 16392, 8192), (40, 16392, 8192),
    # one k step per batch where two would leave zero-weight steps; the two-batch ring of narrow
    # layers at two or three row tiles; activations from L2 where they do not fit in LDS; short K
    (1, 37888, 3584), (32, 37888, 3584), (16, 8192, 2560), (40, 8192, 2560), (32, 12288, 4096),
    (16, 4608, 3584), (48, 4608, 3584), (32, 4096, 4096), (20, 16392, 12288), (32, 8200, 12288),
    (16, 4096, 1024), (32, 4096, 1024),
    # four row tiles at 49 ... 64 tokens for layers up to 12288 wide with K <= 4096
    (64, 12288, 4096), (57, 4608, 3584), (64, 4096, 4096), (50, 3584, 3584), (61, 12288, 2048), (64, 1032, 576),
    # tiled plans: 64 x 64 with K splits, 64 x 128, 128 x 128, 256 x 128, 128 x 256
    (49, 4104, 4160), (64, 24576, 4096), (300, 1032, 576), (1024, 4096, 4096), (2100, 4104, 3584),
    (4096, 8200, 4160), (513, 4104, 12288), (4096, 4096, 192), (4000, 4000, 4160), (3000, 12296, 3584),
    # 128 x 128 in two k groups: ragged M and N, an odd number of k steps with half a last step
    (1000, 3584, 19008), (1024, 3584, 18944), (1024, 4096, 12288),
]


@pytest.mark.parametrize("M,N,K", SHAPES)
def test_gemm_bit_exact(M, N, K):
    qa, qw = codes(M, K, 10 + M), codes(N, K, 20 + N)
    Aq, Wq = pack_codes(qa), pack_codes(qw)
    rng = np.random.default_rng(4)
    s_a = rng.uniform(0.05, 3, M).astype(np.float32)
    s_w = rng.uniform(1e-4, 5e-3, N).astype(np.float32)
    say(f"gemm_frag M={M} N={N} K={K}")
    Wf = sq.weights_to_frag(dev(Wq))
    Y, acc = sq.w4a4_gemm_frag(dev(Aq), dev(s_a), Wf, dev(s_w), want_acc=True)
    Y, acc = host(Y), host(acc)
    rows = np.arange(M) if M * N * K <= 3e9 else np.unique(np.r_[0, M - 1, rng.choice(M, 24)])
    rY, racc = O.gemm(Aq[rows], s_a[rows], Wq, s_w, threads=THREADS)
    assert_bits(acc[rows], racc, "acc")
    assert_y(Y[rows], rY)
    # and the row-major path on the same codes agrees bit for bit
    Y4, acc4 = sq.w4a4_gemm(dev(Aq), dev(s_a), dev(Wq), dev(s_w), want_acc=True)
    assert_bits(acc, host(acc4), "acc vs w4a4_gemm")
    assert_bits(Y, host(Y4), "Y vs w4a4_gemm")


@pytest.mark.parametrize("M", [3, 64])
def test_gemm_at_the_largest_K(M):
    """K = 131072 with every product (-8)(-8) on row 0 / column 0: the sum is 2^23,
    whose scaled int32 value wraps (short-M and tiled kernels)."""
    K, N = 131072, 16
    rng = np.random.default_rng(12)
    qa, qw = rng.integers(-8, 8, (M, K)), rng.integers(-8, 8, (N, K))
    qa[0, :] = -8
    qw[0, :] = -8
    Aq, Wq = pack_codes(qa), pack_codes(qw)
    s_a = np.ones(M, np.float32)
    s_w = np.full(N, 1e-7, np.float32)
    say(f"gemm_frag largest K M={M}")
    Y, acc = sq.w4a4_gemm_frag(dev(Aq), dev(s_a), sq.weights_to_frag(dev(Wq)), dev(s_w), want_acc=True)
    ref = qa.astype(np.int64) @ qw.T.astype(np.int64)
    assert ref[0, 0] == 1 << 23
    assert_bits(host(acc), ref.astype(np.int32), "acc")
    rY, _ = O.gemm(Aq, s_a, Wq, s_w, threads=THREADS)
    assert_y(host(Y), rY)


def test_empty_and_single_outputs():
    K = 128
    Wf = sq.weights_to_frag(dev(pack_codes(codes(0, K, 5))))
    assert Wf.shape == (1, 0, 1024)
    qa, qw = codes(4, K, 6), codes(8, K, 7)
    Wf = sq.weights_to_frag(dev(pack_codes(qw)))
    s_a, s_w = dev(np.ones(4, np.float32)), dev(np.full(8, 0.5, np.float32))
    _, acc = sq.w4a4_gemm_frag(dev(pack_codes(qa)), s_a, Wf, s_w, want_Y=False, want_acc=True)
    assert_bits(host(acc), (qa @ qw.T).astype(np.int32), "acc")
    Y = sq.w4a4_gemm_frag(dev(pack_codes(qa)), s_a, Wf, s_w)
    rY, _ = O.gemm(pack_codes(qa), np.ones(4, np.float32), pack_codes(qw), np.full(8, 0.5, np.float32))
    assert_y(host(Y), rY)
    Y0 = sq.w4a4_gemm_frag(dev(np.zeros((0, K // 2), np.uint8)), dev(np.ones(0, np.float32)), Wf, s_w)
    assert Y0.shape == (0, 8)


def codes8(R, K, seed):
    return np.random.default_rng(seed).integers(-128, 128, (R, K)).astype(np.int8)


@pytest.mark.parametrize("N,K", [(8, 64), (40, 320), (4104, 4160)])
def test_w8_conversion_bit_exact(N, K):
    Wq = codes8(N, K, N + K)
    got = host(sq.weights_to_frag(dev(Wq)))
    assert_bits(got, F.to_frag_q8(Wq, K), "fragment-ordered int8 weights")


def test_w8_gemm_on_oracle_ordered_weights():
    M, N, K = 20, 40, 320                        # two row tiles, a ragged group (int8: whole k steps)
    qa, qw = codes8(M, K, 1), codes8(N, K, 2)
    rng = np.random.default_rng(3)
    s_a = rng.uniform(0.01, 1, M).astype(np.float32)
    s_w = rng.uniform(1e-5, 1e-3, N).astype(np.float32)
    Wf = F.to_frag_q8(qw, K)
    Y, acc = sq.w8a8_gemm_frag(dev(qa), dev(s_a), dev(Wf), dev(s_w), want_acc=True)
    rY, racc = F.gemm_q8(qa, s_a, Wf, s_w, N, K)
    assert_bits(host(acc), racc, "acc")
    assert_y(host(Y), rY)


W8_SHAPES = [
    # short M (<= 48 tokens): wide, mid-width and narrow layers; LDS or L2 activations
    (1, 24576, 4096), (16, 12288, 4096), (33, 4096, 4096), (48, 4096, 12288), (5, 4104, 4160),
    (17, 16392, 8192), (1, 8, 64), (3, 24, 192), (40, 8200, 12288),
    # tiled plans: 64 x 64 with K splits, 64 x 128, 128 x 128, 256 x 128
    (49, 4104, 4160), (64, 12288, 4096), (300, 1032, 576), (1024, 4096, 4096), (1024, 4096, 12288),
    (2100, 4104, 3584), (4096, 12288, 4096), (4000, 4000, 4160),
    # 128 x 256 at 192 ... 511 of its tiles; 128 x 128 in two waves from 640 of its tiles (ragged M, N)
    (500, 12296, 4160), (1000, 12296, 4160), (520, 24576, 4096),
    # 128 x 128 in two k groups (an odd number of k steps; ragged M and N)
    (1000, 4000, 12352), (1024, 4096, 4096), (256, 12288, 4096),
]


@pytest.mark.parametrize("M,N,K", W8_SHAPES)
def test_w8_gemm_bit_exact(M, N, K):
    qa, qw = codes8(M, K, 10 + M), codes8(N, K, 20 + N)
    rng = np.random.default_rng(4)
    s_a = rng.uniform(0.01, 1, M).astype(np.float32)
    s_w = rng.uniform(1e-5, 1e-3, N).astype(np.float32)
    say(f"w8a8_gemm_frag M={M} N={N} K={K}")
    Wf = sq.weights_to_frag(dev(qw))
    Y, acc = sq.w8a8_gemm_frag(dev(qa), dev(s_a), Wf, dev(s_w), want_acc=True)
    Y, acc = host(Y), host(acc)
    rows = np.arange(M) if M * N * K <= 3e9 else np.unique(np.r_[0, M - 1, rng.choice(M, 24)])
    rY, racc = O.gemm_q8(qa[rows], s_a[rows], qw, s_w, threads=THREADS)
    assert_bits(acc[rows], racc, "acc")
    assert_y(Y[rows], rY)
    Y8, acc8 = sq.w8a8_gemm(dev(qa), dev(s_a), dev(qw), dev(s_w), want_acc=True)
    assert_bits(acc, host(acc8), "acc vs w8a8_gemm")
    assert_bits(Y, host(Y8), "Y vs w8a8_gemm")


@pytest.mark.parametrize("M", [3, 64])
def test_w8_gemm_at_the_largest_K(M):
    """K = 65536 with every product (-128)(-128) on row 0 / column 0: the sum 2^30."""
    K, N = 65536, 16
    qa, qw = codes8(M, K, 12), codes8(N, K, 13)
    qa[0, :] = -128
    qw[0, :] = -128
    s_a = np.ones(M, np.float32)
    s_w = np.full(N, 1e-9, np.float32)
    say(f"w8a8_gemm_frag largest K M={M}")
    Y, acc = sq.w8a8_gemm_frag(dev(qa), dev(s_a), sq.weights_to_frag(dev(qw)), dev(s_w), want_acc=True)
    ref = qa.astype(np.int64) @ qw.T.astype(np.int64)
    assert ref[0, 0] == 1 << 30
    assert_bits(host(acc), ref.astype(np.int32), "acc")
    rY, _ = O.gemm_q8(qa, s_a, qw, s_w, threads=THREADS)
    assert_y(host(Y), rY)
