"""Pins of the oracle's SGAT transform, weight preparation and GEMM against what the
paper fixes: Eq. 6 (transform-then-untransform equals X W^T), App. A (computation
consistency and the leakage term), Eq. 7-13 taken literally (split, explicit gated
bases, quantise, int GEMM, scatter), the gate special cases and brute force."""
import numpy as np
import pytest

import synth
from oracle import oracle as O

U = 2.0 ** -24


def _case(seed=0, M=24, K=128, N=40, state=None):
    return synth.small_case(seed, M, K, N, state=state)


# ------------------------------------------------------------------ transform

def test_identity_basis_is_exact_and_equals_no_basis():
    c = _case(1)
    K = c["X"].shape[1]
    dm, du = synth.default_band(K)
    I = np.eye(K, dtype=np.float32)
    a = O.transform(c["X"], c["state"], I, dm, du)
    b = O.transform(c["X"], c["state"], None, dm, du)
    assert a.tobytes() == b.tobytes()
    # with no gate the identity basis returns the fp16 input exactly
    c0 = O.transform(c["X"], None, I, 0, 0)
    assert (c0 == c["X"].astype(np.float32)).all()


def test_signed_permutation_basis_is_exact():
    c = _case(2)
    K = c["X"].shape[1]
    rng = np.random.default_rng(0)
    perm = rng.permutation(K)
    sign = rng.choice([-1.0, 1.0], K)
    P = np.zeros((K, K), np.float32)
    P[perm, np.arange(K)] = sign                       # x'_j = sign_j * x_perm[j]
    got = O.transform(c["X"], None, P, 0, 0)
    ref = c["X"].astype(np.float32)[:, perm] * sign.astype(np.float32)
    assert (got == ref).all()


def test_transform_error_bound_vs_fp64():
    """fp32 chunked-FMA result lies within the textbook dot-product error bound of
    the exact fp64 product: |err| <= (chunk + n_chunks) * u * sum|x||p| (1 + small)."""
    for K in (64, 512, 768):
        c = _case(3, M=16, K=K, N=8)
        got = O.transform(c["X"], None, c["P"], 0, 0).astype(np.float64)
        X64, P64 = c["X"].astype(np.float64), c["P"].astype(np.float64)
        ref = X64 @ P64
        bound = (min(K, 256) + (K + 255) // 256 + 2) * U * (np.abs(X64) @ np.abs(P64))
        assert (np.abs(got - ref) <= bound).all()
        # and it is much closer than the bound on average
        assert np.abs(got - ref).mean() < 0.05 * bound.mean()


def test_gate_zeroes_exactly_the_other_band():
    c = _case(4, M=32, K=256)
    K = 256
    dm, du = 8, 8
    full = O.transform(c["X"], None, c["P"], 0, 0)
    got = O.transform(c["X"], c["state"], c["P"], dm, du)
    for i, s in enumerate(c["state"]):
        keep = O.gate_vector(K, dm, du, bool(s)).astype(bool)
        assert (got[i, keep] == full[i, keep]).all()
        assert (got[i, ~keep] == 0).all() and not np.signbit(got[i, ~keep]).any()


def test_eq6_transform_untransform_identity():
    """(X P)(P^T W^T) = X W^T with quantisers off and no gate (Eq. 6)."""
    c = _case(5, M=16, K=512, N=24)
    xp = O.transform(c["X"], None, c["P"], 0, 0).astype(np.float64)
    wp = O.transform(c["W"], None, c["P"], 0, 0).astype(np.float64)    # rows of W P
    got = xp @ wp.T
    ref = O.fp64_linear(c["X"], c["W"])
    assert np.linalg.norm(got - ref) / np.linalg.norm(ref) < 1e-5
    # the fp64 closed form with the fp32-stored basis (orthogonal to fp32 accuracy)
    ref2 = O.fp64_sgat_noquant(c["X"], np.zeros(16, np.uint8), c["P"], c["W"], 0, 0)
    assert np.linalg.norm(ref2 - ref) / np.linalg.norm(ref) < 1e-5


def test_appA_consistency_when_inactive_component_is_zero():
    """App. A: if X^s P G_s^perp = 0 then X^s W^T = Phi_s(X^s) W~.  Build X^s = Z G_s P^T
    for random Z; the oracle's gated transform times the weight side must reproduce
    X W^T, while the wrong band (or P^T in place of P) would not."""
    K, N, M = 256, 32, 20
    rng = np.random.default_rng(6)
    P64 = synth.orthogonal(K, synth.rng_for(99, 0)).astype(np.float64)
    dm = du = K // 32
    state = (rng.random(M) < 0.5).astype(np.uint8)
    Z = rng.standard_normal((M, K))
    X = np.stack([Z[i] * O.gate_vector(K, dm, du, bool(state[i])) for i in range(M)]) @ P64.T
    X16 = X.astype(np.float16)
    W16 = (rng.standard_normal((N, K)) * 0.02).astype(np.float16)
    P32 = P64.astype(np.float32)
    xp = O.transform(X16, state, P32, dm, du).astype(np.float64)
    wp = O.transform(W16, None, P32, 0, 0).astype(np.float64)
    got = xp @ wp.T
    ref = O.fp64_linear(X16, W16)
    # X16 is X rounded to fp16, so its leakage into the gated band is ~2^-11 of X
    assert np.linalg.norm(got - ref) / np.linalg.norm(ref) < 2e-3
    # the opposite gate discards the band that carries the information
    wrong = O.transform(X16, 1 - state, P32, dm, du).astype(np.float64) @ wp.T
    assert np.linalg.norm(wrong - ref) / np.linalg.norm(ref) > 0.05


def test_appA_leakage_term():
    """Delta_s = X W^T - Phi_s(X) W~ equals X P G_s^perp P^T W^T (App. A)."""
    c = _case(7, M=24, K=512, N=16)
    K = 512
    dm, du = synth.default_band(K)
    xp = O.transform(c["X"], c["state"], c["P"], dm, du).astype(np.float64)
    wp = O.transform(c["W"], None, c["P"], 0, 0).astype(np.float64)
    delta = O.fp64_linear(c["X"], c["W"]) - xp @ wp.T
    ref = O.fp64_leakage(c["X"], c["state"], c["P"], c["W"], dm, du)
    assert np.linalg.norm(delta - ref) / np.linalg.norm(ref) < 1e-4


# ------------------------------------------------------------------ gate special cases

@pytest.mark.parametrize("kind", ["all_masked", "none_masked"])
def test_single_state_reduces_to_one_explicit_basis(kind):
    """All-masked input equals the ungated path with basis P G_m; none-masked with P G_u
    (Eq. 10), bit for bit."""
    c = _case(8, M=32, K=256, N=24)
    K = 256
    dm, du = synth.default_band(K)
    st = synth.state_edge(32, kind)
    masked = kind == "all_masked"
    Pg = (c["P"] * O.gate_vector(K, dm, du, masked)[None, :]).astype(np.float32)
    a = O.quant_act(c["X"], st, c["P"], dm, du)
    b = O.quant_act(c["X"], None, Pg, 0, 0)
    assert a[0].tobytes() == b[0].tobytes() and a[1].tobytes() == b[1].tobytes()


def test_token_permutation_equivariance_and_row_independence():
    c = _case(9, M=40, K=256, N=16)
    K = 256
    dm, du = synth.default_band(K)
    ref = O.sgat_linear(c["X"], c["state"], c["P"], c["W"], dm, du)
    perm = np.random.default_rng(1).permutation(40)
    got = O.sgat_linear(c["X"][perm], c["state"][perm], c["P"], c["W"], dm, du)
    assert got["Y"].tobytes() == ref["Y"][perm].tobytes()
    # flipping other rows' states leaves row 0 untouched
    st2 = c["state"].copy()
    st2[1:] ^= 1
    got2 = O.sgat_linear(c["X"], st2, c["P"], c["W"], dm, du)
    assert got2["Y"][0].tobytes() == ref["Y"][0].tobytes()
    assert got2["Aq"][0].tobytes() == ref["Aq"][0].tobytes()


# ------------------------------------------------------------------ paper-literal mode

@pytest.mark.parametrize("seed,M,K,N", [(10, 64, 256, 48), (11, 33, 512, 20), (12, 8, 64, 8)])
def test_canonical_matches_paper_literal(seed, M, K, N):
    """The per-row formulation equals the paper's split / gated-basis / quantise / GEMM /
    scatter sequence (Eq. 7-13) computed in fp64 with a searched quantiser: codes agree
    wherever the element is not within 1e-4 of a rounding midpoint, and outputs agree to
    the dequantisation rounding."""
    c = _case(seed, M=M, K=K, N=N)
    dm, du = synth.default_band(K)
    can = O.sgat_linear(c["X"], c["state"], c["P"], c["W"], dm, du)
    lit = O.paper_literal(c["X"], c["state"], c["P"], c["W"], dm, du)
    codes = O.unpack(can["Aq"])
    clear = lit["margin"] > 1e-4
    assert (codes[clear] == lit["codes"][clear]).all()
    assert np.abs(can["s_a"] / lit["s_a"] - 1).max() < 1e-6
    qw = O.unpack(can["Wq"])
    assert (qw == lit["qw"]).mean() > 0.999
    # rows whose codes all agree produce the same output up to fp16 rounding
    rows = np.all(codes == lit["codes"], axis=1) & np.all(qw == lit["qw"], axis=1).all()
    if rows.any():
        y = can["Y"].astype(np.float64)[rows]
        ref = lit["Y"][rows]
        assert np.all(np.abs(y - ref) <= 2 ** -10 * np.abs(ref) + 1e-7)


def test_brute_force_tiny_exhaustive_states():
    """M = 4, K = 64, N = 4, all 16 state vectors: canonical vs paper-literal."""
    K, N, M = 64, 4, 4
    base = _case(13, M=M, K=K, N=N)
    dm, du = synth.default_band(K)
    for bits in range(16):
        st = np.array([(bits >> i) & 1 for i in range(M)], np.uint8)
        can = O.sgat_linear(base["X"], st, base["P"], base["W"], dm, du)
        lit = O.paper_literal(base["X"], st, base["P"], base["W"], dm, du)
        codes = O.unpack(can["Aq"])
        clear = lit["margin"] > 1e-4
        assert (codes[clear] == lit["codes"][clear]).all()
        # int GEMM equals the int64 product of the unpacked codes
        acc = codes.astype(np.int64) @ O.unpack(can["Wq"]).astype(np.int64).T
        assert (acc == can["acc"]).all()


# ------------------------------------------------------------------ GEMM

def test_gemm_int_exact_and_dequant_rounding():
    rng = np.random.default_rng(14)
    M, N, K = 17, 23, 320
    qa = rng.integers(-7, 8, (M, K))
    qw = rng.integers(-7, 8, (N, K))
    Aq = ((qa[:, 0::2] & 15) | ((qa[:, 1::2] & 15) << 4)).astype(np.uint8)
    Wq = ((qw[:, 0::2] & 15) | ((qw[:, 1::2] & 15) << 4)).astype(np.uint8)
    s_a = rng.uniform(0.01, 2, M).astype(np.float32)
    s_w = rng.uniform(1e-4, 1e-2, N).astype(np.float32)
    Y, acc = O.gemm(Aq, s_a, Wq, s_w)
    assert (acc == qa @ qw.T).all()
    ref = (qa @ qw.T) * s_a[:, None].astype(np.float64) * s_w[None, :].astype(np.float64)
    # two fp32 roundings then one fp16 rounding
    assert np.all(np.abs(Y.astype(np.float64) - ref) <= np.abs(ref) * (2 ** -11 + 2 ** -22) + 2 ** -25)


def test_gemm_extreme_codes_fit_int32():
    K = 18944
    Aq = np.full((1, K // 2), 0x99, np.uint8)        # all codes -7
    Wq = np.full((2, K // 2), 0x99, np.uint8)
    Wq[1] = 0x77                                      # all codes +7
    Y, acc = O.gemm(Aq, np.ones(1, np.float32), Wq, np.ones(2, np.float32))
    assert acc.tolist() == [[49 * K, -49 * K]]


def test_w4a4_close_to_fp_linear():
    """Sanity: the quantised linear approximates X W^T (W4A4 error is large but bounded)."""
    c = _case(15, M=64, K=512, N=64)
    dm, du = synth.default_band(512)
    out = O.sgat_linear(c["X"], c["state"], c["P"], c["W"], dm, du)
    ref = O.fp64_linear(c["X"], c["W"])
    rel = np.linalg.norm(out["Y"].astype(np.float64) - ref) / np.linalg.norm(ref)
    assert rel < 0.35
