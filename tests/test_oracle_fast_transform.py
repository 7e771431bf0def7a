"""Pins of the matrix-core transform reference: the split of the basis, and the
soundness and usefulness of the error bounds used to compare the fast
transform with the exact product and with the fixed-order transform."""
import numpy as np
import pytest

import synth
from oracle import fast_transform as F
from oracle import oracle as O


def basis(K, seed):
    return synth.orthogonal(K, synth.rng_for(1200 + seed, synth.T_P))


def test_split_residual_bound_and_exact_cases():
    P = basis(256, 0)
    Ps = F.split_basis(P).view(np.float16).astype(np.float64)
    v = P.T.astype(np.float64) * F.SCALE
    res = np.abs(v - Ps[:, :256] - Ps[:, 256:])
    assert (res <= 2.0 ** -22 * np.abs(v) + 2.0 ** -25).all()
    assert res.max() > 0                                   # the split is not trivially exact
    # exactly representable entries split with a zero low part
    Pi = np.eye(64, dtype=np.float32)
    Psi = F.split_basis(Pi).view(np.float16).astype(np.float64)
    assert np.array_equal(Psi[:, :64], np.eye(64) * 16384.0) and not Psi[:, 64:].any()
    # hi is the RNE fp16 of the scaled entry
    assert np.array_equal(F.split_basis(P)[:, :256], (P.T * np.float32(16384)).astype(np.float16).view(np.uint16))


def fast_emulated(X, Ps, order):
    """The fast transform in real fp32 arithmetic, in a given summation order."""
    x = X.astype(np.float32)
    ps = Ps.view(np.float16).astype(np.float32)
    K = x.shape[1]
    terms = np.concatenate([x, x], axis=1)[:, None, :] * ps[None, :, :]      # exact fp32 products
    if order == "sequential":
        acc = np.zeros(terms.shape[:2], np.float32)
        for k in range(2 * K):
            acc = (acc + terms[:, :, k]).astype(np.float32)
    elif order == "reversed":
        acc = np.zeros(terms.shape[:2], np.float32)
        for k in reversed(range(2 * K)):
            acc = (acc + terms[:, :, k]).astype(np.float32)
    elif order == "blocks32":
        acc = np.zeros(terms.shape[:2], np.float32)
        for k0 in range(0, 2 * K, 32):
            acc = (acc + terms[:, :, k0:k0 + 32].sum(axis=2, dtype=np.float32)).astype(np.float32)
    else:
        acc = terms.sum(axis=2, dtype=np.float32)                          # numpy pairwise
    return acc.astype(np.float64) / F.SCALE


@pytest.mark.parametrize("order", ["sequential", "reversed", "blocks32", "pairwise"])
def test_fast_bound_holds_for_any_order(order):
    K, M = 128, 6
    P = basis(K, 1)
    X = (np.random.default_rng(2).standard_normal((M, K)) * 3).astype(np.float16)
    X[0, :4] = 60.0                                        # outlier channels
    Ps = F.split_basis(P)
    exact = F.exact_transform(X, None, P, 0, 0)
    err = np.abs(fast_emulated(X, Ps, order) - exact)
    assert (err <= F.fast_bound(X, Ps, P)).all()


def test_fast_bound_is_tight_enough_to_see_a_dropped_term():
    K, M = 128, 6
    P = basis(K, 3)
    X = np.random.default_rng(4).standard_normal((M, K)).astype(np.float16)
    Ps = F.split_basis(P)
    bound = F.fast_bound(X, Ps, P)
    # the bound is small next to the values it guards
    assert bound.max() < 1e-4 * np.abs(F.exact_transform(X, None, P, 0, 0)).max()
    # dropping the low part of the split violates it
    no_lo = Ps.copy()
    no_lo[:, K:] = 0
    err = np.abs(fast_emulated(X, no_lo, "pairwise") - F.exact_transform(X, None, P, 0, 0))
    assert (err > bound).any()


def test_canonical_bound_holds_for_the_fixed_order_transform():
    K, M = 512, 5
    P = basis(K, 5)
    X = (np.random.default_rng(6).standard_normal((M, K)) * 2).astype(np.float16)
    st = np.array([0, 1, 0, 1, 1], np.uint8)
    xp = O.transform(X, st, P, K // 32, K // 32).astype(np.float64)
    exact = F.exact_transform(X, st, P, K // 32, K // 32)
    assert (np.abs(xp - exact) <= F.canonical_bound(X, P)).all()


def test_gate_mask_matches_the_band_layout():
    K, dm, du = 64, 4, 6
    m = F.gate_mask(np.array([0, 1], np.uint8), K, dm, du)
    assert not m[0, K - dm - du:K - du].any() and m[0, K - du:].all()        # unmasked drops the m band
    assert not m[1, K - du:].any() and m[1, K - dm - du:K - du].all()        # masked drops the u band
    assert m[:, :K - dm - du].all()
