"""GPU parity of the TAC closed-form calibration (App. C) through the C ABI.

The GPU evaluates the closed form in fp64 with Jacobi eigen- and singular value
decompositions; the oracle uses LAPACK.  Both are fp64 evaluations of the same
formulas, so they agree to rounding, not bit for bit: the unrounded parameters
are compared with a bound derived from that (see TOL), and the stored fp16
parameters must equal the oracle's except where the oracle's fp64 value lies
within that bound of an fp16 rounding midpoint.  The fp16 conversion itself is
checked exactly: the GPU's fp16 output must be the RNE rounding of the GPU's own
fp64 output."""
import numpy as np
import pytest
import torch

import paper_2606_04945_amd as sq
import synth
from oracle import tac_calib as T
from gpu_util import dev, host, say

pytestmark = pytest.mark.gpu

# Both sides round each of O(g) fp64 operations per output; the synthetic
# covariances are well conditioned (condition numbers below 1e3), so the two
# evaluations agree to ~1e-13 relative; 1e-9 (absolute, for values of order 1)
# leaves four orders of margin without admitting a wrong formula (a dropped
# term or a transposition moves values by 1e-3 or more).
TOL = 1e-9

CASES = [(1000, 64, 16), (257, 128, 1), (300, 128, 2), (17, 64, 4), (5000, 256, 8), (4096, 512, 32),
         (2000, 512, 64), (1500, 256, 128), (1, 64, 16), (20000, 4096, 16), (70000, 128, 16)]


def data(N, C, g, seed=0):
    zf, zq = synth.tac_calib_pair(N, C, g, synth.rng_for(950 + seed, synth.T_CALIB, N, C, g))
    return zf, zq


def fp16_midpoint_near(x, tol):
    """True where x is within tol (relative) of a point halfway between two fp16 values."""
    h = x.astype(np.float16)
    up = np.nextafter(h, np.float16(np.inf)).astype(np.float64)
    dn = np.nextafter(h, np.float16(-np.inf)).astype(np.float64)
    hv = h.astype(np.float64)
    mids = np.stack([(hv + up) / 2, (hv + dn) / 2])
    return (np.abs(mids - x[None]) <= tol * np.maximum(np.abs(x), 1e-30)[None]).any(axis=0)


def run(zf, zq, g, **kw):
    return sq.tac_calibrate(dev(zf), dev(zq), g, want_fp64=True, **kw)


@pytest.mark.parametrize("N,C,g", CASES, ids=[f"N{n}-C{c}-g{g}" for n, c, g in CASES])
def test_calibration_matches_oracle(N, C, g):
    say(f"tac_calibrate N={N} C={C} g={g} ws={sq.tac_calibrate_workspace_bytes(N, C, g)}")
    zf, zq = data(N, C, g)
    tM, td, M64, d64 = run(zf, zq, g)
    torch.cuda.synchronize()
    rM, rd = T.calibrate(zf, zq, g)
    M64, d64 = host(M64), host(d64)
    np.testing.assert_allclose(M64, rM, rtol=0, atol=TOL * max(1.0, np.abs(rM).max()))
    np.testing.assert_allclose(d64, rd, rtol=0, atol=TOL * max(1.0, np.abs(rd).max()))
    gM, gd = host(tM).view(np.uint16), host(td).view(np.uint16)
    # the GPU's fp16 parameters are the RNE rounding of its own fp64 values
    assert np.array_equal(gM, T.to_fp16_bits(M64))
    assert np.array_equal(gd, T.to_fp16_bits(d64))
    # and equal the oracle's away from fp16 midpoints
    for got, ref in ((gM.reshape(-1), rM.reshape(-1)), (gd, rd)):
        diff = got != T.to_fp16_bits(ref)
        assert not (diff & ~fp16_midpoint_near(ref, 1e-8)).any()


@pytest.mark.parametrize("eta,alpha,rho", [(0.0, 0.0, 3e-4), (1.0, 0.0, 3e-4), (0.3, 0.8, 1e-2), (0.15, 0.55, 0.0)])
def test_hyperparameters(eta, alpha, rho):
    zf, zq = data(3000, 256, 16, seed=1)
    _, _, M64, d64 = run(zf, zq, 16, eta=eta, alpha=alpha, rho=rho)
    rM, rd = T.calibrate(zf, zq, 16, rho=rho, eta=eta, alpha=alpha)
    np.testing.assert_allclose(host(M64), rM, atol=TOL * max(1.0, np.abs(rM).max()))
    np.testing.assert_allclose(host(d64), rd, atol=TOL * max(1.0, np.abs(rd).max()))


def test_alpha_one_gives_identity_exactly():
    zf, zq = data(800, 128, 8, seed=2)
    tM, td, M64, d64 = run(zf, zq, 8, alpha=1.0)
    assert np.array_equal(host(M64), np.broadcast_to(np.eye(8), (16, 8, 8)))
    mu = zf.astype(np.float64).mean(axis=0) - zq.astype(np.float64).mean(axis=0)
    np.testing.assert_allclose(host(d64), mu, atol=1e-12)


def test_identical_inputs_give_identity():
    zf, _ = data(4000, 128, 16, seed=3)
    _, _, M64, d64 = run(zf, zf, 16, rho=0.0, eta=0.0, alpha=0.0)
    np.testing.assert_allclose(host(M64), np.broadcast_to(np.eye(16), (8, 16, 16)), atol=1e-9)
    np.testing.assert_allclose(host(d64), 0.0, atol=1e-9)


def test_calibrated_tac_restores_the_mean():
    """Calibrate on the GPU, apply the fp16 parameters with tac_apply: the compensated
    mean is the full-precision mean up to the fp16 rounding of parameters and output."""
    zf, zq = data(8192, 512, 16, seed=4)
    tM, td = sq.tac_calibrate(dev(zf), dev(zq), 16)
    out = host(sq.tac_apply(dev(zq), tM, td, 16)).astype(np.float64)
    err = np.abs(out.mean(axis=0) - zf.astype(np.float64).mean(axis=0))
    assert err.max() < 5e-3
    # and the compensation helps: closer to the full-precision output than the raw input
    assert np.mean((out - zf) ** 2) < np.mean((zq.astype(np.float64) - zf) ** 2)


def test_deterministic():
    zf, zq = data(10000, 256, 32, seed=5)
    a = [host(x) for x in run(zf, zq, 32)]
    b = [host(x) for x in run(zf, zq, 32)]
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
