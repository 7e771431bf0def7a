"""Pins of the TAC calibration oracle (App. C) against what the appendix and the
mathematics fix: the shrinkage end points, exact recovery of an affine
distortion, first- and second-moment matching, the diagonal closed form (with
and without the eigenvalue floor), the effect of full singular value
smoothing, a hand-computed one-channel case, and the fp16 rounding of the
stored parameters."""
from decimal import Decimal, getcontext

import numpy as np
import pytest

import synth
from oracle import tac_calib as T


def walsh(N, k):
    """+-1 Walsh function k over N = 2^n points: distinct k > 0 are orthogonal and zero-mean."""
    i = np.arange(N)
    return np.where(np.array([bin(x & k).count("1") % 2 for x in i]) == 0, 1.0, -1.0)


def diag_data(a, mu, N=64):
    """fp16 data whose block covariance is exactly diag(a^2) and mean exactly mu."""
    cols = [mu[j] + a[j] * walsh(N, j + 1) for j in range(len(a))]
    Z = np.stack(cols, axis=1).astype(np.float16)
    assert np.array_equal(Z.astype(np.float64), np.stack(cols, axis=1))    # exact in fp16
    return Z


def test_alpha_one_is_identity_and_mean_shift():
    zf, zq = synth.tac_calib_pair(500, 32, 8, synth.rng_for(900, synth.T_CALIB))
    M, d = T.calibrate(zf, zq, 8, alpha=1.0)
    assert np.array_equal(M, np.broadcast_to(np.eye(8), M.shape))
    mu_f = zf.astype(np.float64).mean(axis=0)
    mu_q = zq.astype(np.float64).mean(axis=0)
    np.testing.assert_allclose(d, mu_f - mu_q, rtol=0, atol=1e-12)


def test_identical_statistics_give_identity():
    zf, _ = synth.tac_calib_pair(800, 32, 16, synth.rng_for(901, synth.T_CALIB))
    M, d = T.calibrate(zf, zf, 16, rho=0.0, eta=0.0, alpha=0.0)
    np.testing.assert_allclose(M, np.broadcast_to(np.eye(16), M.shape), rtol=0, atol=1e-10)
    np.testing.assert_allclose(d, 0.0, atol=1e-10)


def test_affine_distortion_is_inverted_exactly():
    """Z_q = 2 Z_fp + 0.5: with no damping, smoothing or shrinkage, TAC(Z_q) = Z_fp."""
    rng = np.random.default_rng(3)
    g, N = 8, 512
    zf = (np.round(rng.normal(0, 1, (N, 4 * g)) * 64) / 64).astype(np.float16)
    zq = (2.0 * zf.astype(np.float64) + 0.5).astype(np.float16)
    assert np.array_equal(zq.astype(np.float64), 2.0 * zf.astype(np.float64) + 0.5)
    M, d = T.calibrate(zf, zq, g, rho=0.0, eta=0.0, alpha=0.0)
    np.testing.assert_allclose(M, np.broadcast_to(np.eye(g) / 2, M.shape), atol=1e-10)
    np.testing.assert_allclose(T.apply(zq, M, d, g), zf.astype(np.float64), atol=1e-9)


@pytest.mark.parametrize("eta,alpha,rho", [(0.15, 0.55, 3e-4), (0.0, 0.0, 3e-4), (0.5, 0.2, 1e-2)])
def test_compensated_mean_matches_full_precision(eta, alpha, rho):
    zf, zq = synth.tac_calib_pair(700, 64, 16, synth.rng_for(902, synth.T_CALIB))
    M, d = T.calibrate(zf, zq, 16, rho=rho, eta=eta, alpha=alpha)
    out = T.apply(zq, M, d, 16)
    np.testing.assert_allclose(out.mean(axis=0), zf.astype(np.float64).mean(axis=0), atol=1e-11)


def test_covariance_matching_without_stabilisers():
    zf, zq = synth.tac_calib_pair(2000, 32, 16, synth.rng_for(903, synth.T_CALIB))
    M, d = T.calibrate(zf, zq, 16, rho=0.0, eta=0.0, alpha=0.0)
    _, S_f = T.block_stats(zf, 16)
    _, S_out = T.block_stats(T.apply(zq, M, d, 16), 16)
    np.testing.assert_allclose(S_out, S_f, rtol=1e-9, atol=1e-11)


@pytest.mark.parametrize("eta,alpha", [(0.0, 0.0), (0.15, 0.55), (0.4, 0.1)])
def test_diagonal_closed_form(eta, alpha):
    """Exactly diagonal covariances: M = diag(a / sqrt(b^2 + lambda)), smoothing acts on
    the diagonal (the singular values of a positive diagonal matrix), then shrinkage."""
    a = np.array([0.5, 1.0, 1.5, 2.0, 0.75, 1.25, 0.25, 3.0])
    b = np.array([1.0, 0.5, 2.0, 1.5, 1.25, 0.75, 0.5, 2.5])
    mf = np.array([0.25, -0.5, 1.0, 0.0, -1.25, 0.5, 2.0, -0.75])
    mq = np.array([0.5, -0.25, 0.75, 0.25, -1.0, 0.0, 1.5, -0.5])
    zf, zq = diag_data(a, mf), diag_data(b, mq)
    M, d = T.calibrate(zf, zq, 8, rho=3e-4, eta=eta, alpha=alpha)
    lam = 3e-4 * max(np.mean(b ** 2), 1e-8)
    m = a / np.sqrt(b ** 2 + lam)
    m = (1 - eta) * m + eta * m.mean()
    Mf = (1 - alpha) * np.diag(m) + alpha * np.eye(8)
    np.testing.assert_allclose(M[0], Mf, atol=1e-12)
    np.testing.assert_allclose(d, mf - Mf @ mq, atol=1e-12)


def test_eigenvalue_floor_on_a_constant_channel():
    """A zero-variance full-precision channel: its eigenvalue is floored at 1e-12, so the
    square root contributes 1e-6 on that channel."""
    a = np.array([0.0, 1.0, 0.5, 2.0])
    b = np.array([1.0, 1.0, 1.0, 1.0])
    zf, zq = diag_data(a, np.zeros(4)), diag_data(b, np.zeros(4))
    M, _ = T.calibrate(zf, zq, 4, rho=0.0, eta=0.0, alpha=0.0)
    np.testing.assert_allclose(np.diag(M[0]), [1e-6, 1.0, 0.5, 2.0], rtol=1e-9)


def test_full_smoothing_equalises_singular_values():
    zf, zq = synth.tac_calib_pair(600, 16, 16, synth.rng_for(904, synth.T_CALIB))
    M0, _ = T.calibrate(zf, zq, 16, eta=0.0, alpha=0.0)
    M1, _ = T.calibrate(zf, zq, 16, eta=1.0, alpha=0.0)
    s0 = np.linalg.svd(M0[0], compute_uv=False)
    s1 = np.linalg.svd(M1[0], compute_uv=False)
    np.testing.assert_allclose(s1, s0.mean(), rtol=1e-12)
    # and the singular vectors are kept: M1 = mean(s0) x the orthogonal polar factor of M0
    U, _, Vt = np.linalg.svd(M0[0])
    np.testing.assert_allclose(M1[0], s0.mean() * U @ Vt, atol=1e-12)


def test_one_channel_by_hand():
    """g = 1, z_fp = (1, 3), z_q = (0, 4): mu = 2 and 2, variances 1 and 4."""
    getcontext().prec = 40
    zf = np.array([[1.0], [3.0]], np.float16)
    zq = np.array([[0.0], [4.0]], np.float16)
    M, d = T.calibrate(zf, zq, 1)
    lam = Decimal("3e-4") * Decimal(4)
    m = Decimal(1).sqrt() / (Decimal(4) + lam).sqrt()
    m_final = Decimal("0.45") * m + Decimal("0.55")       # smoothing is the identity for g = 1
    assert abs(M[0, 0, 0] - float(m_final)) < 1e-15
    assert abs(d[0] - float(Decimal(2) - m_final * 2)) < 1e-15


def test_fp16_rounding_of_parameters():
    """One RNE rounding from fp64: compared with a nearest-value search over all finite
    fp16 values, ties to the even code."""
    allh = np.arange(0, 0x7C00, dtype=np.uint16).view(np.float16).astype(np.float64)
    rng = np.random.default_rng(5)
    x = np.r_[rng.normal(0, 1, 2000), rng.normal(0, 1e-5, 500), (allh[1:300] + allh[:299]) / 2,
              (allh[20000:20300] + allh[20001:20301]) / 2]
    bits = T.to_fp16_bits(x)
    for v, h in zip(x, bits):
        k = np.searchsorted(allh, abs(v))
        cands = [c for c in (k - 1, k) if 0 <= c < len(allh)]
        dist = [abs(allh[c] - abs(v)) for c in cands]
        best = [c for c, dd in zip(cands, dist) if dd == min(dist)]
        want = best[0] if len(best) == 1 else [c for c in best if c % 2 == 0][0]
        want |= 0x8000 if (v < 0 and want) or (v < 0 and np.signbit(v)) else 0
        assert int(h) & 0x7FFF == want & 0x7FFF, (v, h, want)
        if want & 0x7FFF:
            assert (int(h) >> 15) == (1 if v < 0 else 0)
