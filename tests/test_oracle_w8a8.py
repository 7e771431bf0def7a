"""Pins of the oracle's W8A8 variant (App. D: the same method at 8 bits):
symmetric per-row 8-bit quantiser s = absmax/127 and the int8 GEMM."""
import numpy as np
import pytest

import synth
from oracle import oracle as O


def test_hand_example():
    # absmax 127 -> s = 1: codes are the half-even roundings: 0.5 -> 0, 1.5 -> 2, -2.5 -> -2, 126.5 -> 126
    x = np.array([[127, -127, 0.5, 1.5, -2.5, 126.5, 3.25, -0.75]], np.float32)
    q, s = O.quant_rows_q8(x)
    assert s[0] == 1.0
    assert q.tolist() == [[127, -127, 0, 2, -2, 126, 3, -1]]


@pytest.mark.parametrize("amax", [1.0, 127.0, 0.3, 65504.0, 2.0e-3])
def test_exhaustive_fp16_values_vs_search(amax):
    h = np.arange(65536, dtype=np.uint16)
    v = h.view(np.float16).astype(np.float32)
    v = v[np.isfinite(v) & (np.abs(v) <= amax)]
    row = np.concatenate([[np.float32(amax)], v]).astype(np.float32)
    q, s = O.quant_rows_q8(row[None, :])
    s32 = np.float32(amax) / np.float32(127.0)
    assert s[0] == s32
    ratio = (row / s32).astype(np.float32)
    assert (q[0] == O.nearest_code(ratio, -128, 127)).all()


def test_invariants():
    rng = np.random.default_rng(4)
    x = (rng.standard_normal((200, 640)) * rng.uniform(1e-3, 1e3, (200, 1))).astype(np.float32)
    q, s = O.quant_rows_q8(x)
    assert q.min() >= -127 and q.max() <= 127
    assert (np.abs(q.astype(np.int32)).max(axis=1) == 127).all()
    err = np.abs(x.astype(np.float64) - s[:, None].astype(np.float64) * q)
    assert (err <= s[:, None] * (0.5 + 2.0 ** -17)).all()
    z, sz = O.quant_rows_q8(np.zeros((1, 64), np.float32))
    assert sz[0] == 0 and (z == 0).all()


def test_gemm_q8_int_exact():
    rng = np.random.default_rng(5)
    qa = rng.integers(-128, 128, (9, 320)).astype(np.int8)
    qw = rng.integers(-128, 128, (11, 320)).astype(np.int8)
    s_a = rng.uniform(0.01, 1, 9).astype(np.float32)
    s_w = rng.uniform(1e-4, 1e-2, 11).astype(np.float32)
    Y, acc = O.gemm_q8(qa, s_a, qw, s_w)
    assert (acc == qa.astype(np.int64) @ qw.astype(np.int64).T).all()
    ref = acc * s_a[:, None].astype(np.float64) * s_w[None, :].astype(np.float64)
    assert np.all(np.abs(Y.astype(np.float64) - ref) <= np.abs(ref) * (2 ** -11 + 2 ** -22) + 2 ** -25)


def test_w8a8_closer_than_w4a4():
    """W8A8 reproduces the unquantised SGAT projection (App. A, quantisers off) much
    more closely than W4A4 on the same layer (with a random basis the gate itself
    drops the other band, so the reference is the gated fp64 output)."""
    c = synth.small_case(16, 64, 512, 64)
    dm, du = synth.default_band(512)
    ref = O.fp64_sgat_noquant(c["X"], c["state"], c["P"], c["W"], dm, du)
    Aq, s_a = O.quant_act_q8(c["X"], c["state"], c["P"], dm, du)
    Wq, s_w = O.prepare_weights_q8(c["W"], c["P"])
    Y8, _ = O.gemm_q8(Aq, s_a, Wq, s_w)
    Y4 = O.sgat_linear(c["X"], c["state"], c["P"], c["W"], dm, du)["Y"]
    e8 = np.linalg.norm(Y8.astype(np.float64) - ref) / np.linalg.norm(ref)
    e4 = np.linalg.norm(Y4.astype(np.float64) - ref) / np.linalg.norm(ref)
    assert e8 < 0.05 and e8 < e4 / 5


def test_q8_paper_literal_agreement():
    """8-bit codes of the canonical path match an fp64 split/gated-basis formulation
    away from rounding midpoints (the W8A8 counterpart of the Eq. 7-13 check)."""
    c = synth.small_case(17, 40, 256, 8)
    K = 256
    dm, du = synth.default_band(K)
    Aq, s_a = O.quant_act_q8(c["X"], c["state"], c["P"], dm, du)
    X64, P64 = c["X"].astype(np.float64), c["P"].astype(np.float64)
    for i in range(40):
        phi = X64[i] @ P64 @ np.diag(O.gate_vector(K, dm, du, bool(c["state"][i])))
        s = np.abs(phi).max() / 127.0
        ratio = phi / s
        clear = np.abs(np.abs(ratio - np.floor(ratio)) - 0.5) > 1e-3
        assert abs(s_a[i] / s - 1) < 1e-6
        assert (Aq[i][clear] == O.nearest_code(ratio[clear], -128, 127)).all()
