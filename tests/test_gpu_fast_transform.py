"""GPU checks of the matrix-core transform, stage by stage, through the C ABI.

* the basis split equals the reference bit for bit;
* the transform is within the rigorous bound of the exact product x P G_s
  (the gate is exact: gated columns are +0);
* quantising its output is bit-exact (the quantiser is the canonical one);
* codes differ from the fixed-order path only where the exact value lies within
  the two transforms' bounds (plus the scale difference) of a rounding
  boundary; the number of such flips is reported."""
import numpy as np
import pytest

import paper_2606_04945_amd as sq
import synth
from oracle import fast_transform as F
from oracle import oracle as O
from gpu_util import assert_bits, dev, host, say

pytestmark = pytest.mark.gpu
THREADS = 16


def case(M, K, seed, n_out=2):
    c = synth.small_case(seed, M, K, 8, n_out=n_out)
    return c["X"], c["state"], c["P"]


@pytest.mark.parametrize("K", [64, 512, 4096])
def test_split_basis_bit_exact(K):
    P = synth.orthogonal(K, synth.rng_for(1300, synth.T_P, K))
    Ps = host(sq.sgat_split_basis(dev(P))).view(np.uint16)
    assert_bits(Ps, F.split_basis(P), "Ps")


SHAPES = [(1, 64), (77, 192), (300, 512), (130, 1024), (1024, 4096), (33, 12288), (520, 4096), (385, 8192)]


@pytest.mark.parametrize("M,K", SHAPES)
@pytest.mark.parametrize("gated", [True, False], ids=["gated", "plain"])
def test_transform_within_bound(M, K, gated):
    X, st, P = case(M, K, 40 + K)
    dm, du = (K // 32, K // 32) if gated else (0, 0)
    say(f"transform_fast M={M} K={K} gated={gated}")
    Ps = sq.sgat_split_basis(dev(P))
    xp = host(sq.sgat_transform_fast(dev(X), dev(st) if gated else None, Ps, dm, du)).astype(np.float64)
    exact = F.exact_transform(X, st if gated else None, P, dm, du)
    bound = F.fast_bound(X, host(Ps).view(np.uint16), P)
    err = np.abs(xp - exact)
    assert (err <= bound).all(), f"max err {err.max()} vs bound {bound[err > bound].min()}"
    if gated:
        keep = F.gate_mask(st, K, dm, du)
        assert (xp[~keep] == 0).all() and not np.signbit(xp[~keep]).any()
    say(f"  max |err| {err.max():.3e}, max bound {bound.max():.3e}")


@pytest.mark.parametrize("M,K", [(300, 512), (1024, 4096)])
def test_quantised_codes_stage_exact_and_flips_explained(M, K):
    X, st, P = case(M, K, 70 + K, n_out=4)
    dm = du = K // 32
    Ps = sq.sgat_split_basis(dev(P))
    xp_d = sq.sgat_transform_fast(dev(X), dev(st), Ps, dm, du)
    Aq, s_a = sq.sgat_quantize(xp_d)
    xp = host(xp_d)
    # stage: the quantiser applied to this transform's output is bit-exact
    rq, rs, _ = O.quant_rows(xp)
    assert_bits(host(Aq), rq, "Aq")
    assert_bits(host(s_a), rs, "s_a")
    # against the fixed-order path: every differing code is explained by the bounds
    cq, cs = O.quant_act(X, st, P, dm, du, threads=THREADS)
    fq = O.unpack(host(Aq)).astype(np.int64)
    cqu = O.unpack(cq).astype(np.int64)
    exact = F.exact_transform(X, st, P, dm, du)
    slack = F.fast_bound(X, host(Ps).view(np.uint16), P) + F.canonical_bound(X, P)
    s_f, s_c = host(s_a).astype(np.float64), cs.astype(np.float64)
    diff = fq != cqu
    rows, cols = np.nonzero(diff)
    for i, j in zip(rows, cols):
        x = exact[i, j]
        n = np.floor(x / s_c[i])
        dist = min(abs(x - (n + 0.5) * s_c[i]), abs(x - (n - 0.5) * s_c[i]), abs(x - (n + 1.5) * s_c[i]))
        allow = 2 * (slack[i, j] + 7.5 * abs(s_f[i] - s_c[i]) + 8 * 2.0 ** -24 * s_c[i])
        assert dist <= allow, (i, j, x, s_c[i], dist, allow)
    say(f"  codes differing from the fixed-order path: {int(diff.sum())} of {diff.size}; "
        f"scales differing: {int((host(s_a) != cs).sum())} of {M}")
