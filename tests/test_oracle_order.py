"""Pins of the order conventions the paper leaves open (T3 chunked transform, R2
TAC bias last, G1 dequantisation order): hand-built inputs on which the chosen
convention and a plausible other one give different bits (tests/order_cases.py
works them out).  Each expected value is first re-derived here with exact
rational arithmetic, for the chosen order and for the other one, and then
required of the oracle."""
from fractions import Fraction as F

import numpy as np

import order_cases as C
from oracle import oracle as O


def test_t3_rational_derivation():
    X, P = C.t3_inputs()
    x = [F(float(v)) for v in X[0].astype(np.float32)]

    def chunked(col, kc):
        tot = F(0)
        for c0 in range(0, C.T3_K, kc):
            acc = F(0)
            for k in range(c0, min(C.T3_K, c0 + kc)):
                acc = C.f32(acc + x[k] * F(float(P[k, col])))   # a fused multiply-add: one rounding
            tot = C.f32(tot + acc)
        return tot

    assert chunked(0, 256) == C.T3_COL0 and chunked(1, 256) == C.T3_COL1
    assert chunked(0, C.T3_K) == C.T3_FLAT_COL0 != C.T3_COL0          # a flat chain differs
    assert chunked(1, 128) == C.T3_C128_COL1 != C.T3_COL1             # chunks of 128 differ


def test_t3_oracle_uses_chunks_of_256():
    X, P = C.t3_inputs()
    xp = O.transform(X, None, P, 0, 0)
    assert xp[0, 0] == C.T3_COL0 and xp[0, 1] == C.T3_COL1
    assert (xp[0, 2:] == 0).all() and not np.signbit(xp[0, 2:]).any()


def test_r2_rational_derivation():
    Z, Mb, d = C.r2_inputs()
    z = [F(float(v)) for v in Z[0, :2].astype(np.float32)]
    m = [F(float(v)) for v in Mb[0, 0].astype(np.float32)]
    dd = F(float(d[0]))
    last = F(0)
    for c in range(2):
        last = C.f32(last + m[c] * z[c])
    last = C.f16(C.f32(last + dd))
    first = dd
    for c in range(2):
        first = C.f32(first + m[c] * z[c])
    first = C.f16(first)
    assert last == C.R2_OUT0 and first == C.R2_BIAS_FIRST_OUT0


def test_r2_oracle_adds_the_bias_last():
    Z, Mb, d = C.r2_inputs()
    out = O.tac(Z, Mb, d, C.R2_G)
    assert float(out[0, 0]) == C.R2_OUT0
    assert float(out[0, 1]) == 2.0 ** -6 and (out[0, 2:] == 0).all()


def test_g1_rational_derivation():
    _, s_a, _, s_w = C.g1_inputs()
    a, w, acc = F(float(s_a[0])), F(float(s_w[0])), F(C.G1_ACC)
    g1 = C.f16(C.f32(C.f32(acc * a) * w))
    other = C.f16(C.f32(acc * C.f32(a * w)))
    assert g1 == C.G1_Y and other == C.G1_OTHER_Y


def test_g1_oracle_dequantises_acc_times_sa_then_sw():
    Aq, s_a, Wq, s_w = C.g1_inputs()
    Y, acc = O.gemm(Aq, s_a, Wq, s_w)
    assert acc[0, 0] == C.G1_ACC
    assert float(Y[0, 0]) == C.G1_Y
