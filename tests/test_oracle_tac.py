"""Pins of the oracle's TAC (Eq. 17, App. C row-major form Z_b M_b^T + 1 d_b^T)."""
import numpy as np
import pytest

import synth
from oracle import oracle as O


def _z(M, C, seed=0):
    return (np.random.default_rng(seed).standard_normal((M, C)) * 3).astype(np.float16)


@pytest.mark.parametrize("g", [4, 16, 128])
def test_identity_blocks_are_a_no_op(g):
    Z = _z(32, 512)
    Z[0, :8] = np.float16(-0.0)
    Mb, d = synth.tac_params(512, g, None, identity=True)
    out = O.tac(Z, Mb, d, g)
    # bit-exact except that -0 inputs may come back as +0
    same = (out.view(np.uint16) == Z.view(np.uint16)) | ((out == 0) & (Z == 0))
    assert same.all()


def test_power_of_two_scaling_is_exact():
    Z = _z(16, 256, 1)
    g = 16
    Mb, d = synth.tac_params(256, g, None, identity=True)
    out = O.tac(Z, (Mb.astype(np.float32) * 4).astype(np.float16), d, g)
    assert (out.astype(np.float32) == Z.astype(np.float32) * 4).all()


def test_bias_only_and_hand_block():
    # g = 2, one token: M_0 = [[1, 2], [3, 4]], d = [0.5, -1]; z = [1, -1]
    # z'_0 = 1*1 + 2*(-1) + 0.5 = -0.5 ; z'_1 = 3*1 + 4*(-1) - 1 = -2
    Z = np.array([[1, -1]], np.float16)
    Mb = np.array([[[1, 2], [3, 4]]], np.float16)
    d = np.array([0.5, -1], np.float16)
    assert O.tac(Z, Mb, d, 2).tolist() == [[-0.5, -2.0]]


@pytest.mark.parametrize("g", [8, 16, 64, 128])
def test_close_to_fp64_and_rounded_once(g):
    """Each output is within one fp16 ulp of the fp64 affine map, and equals its RNE
    rounding wherever the fp32 accumulation error bound cannot reach an fp16 midpoint."""
    C = 512
    Z = _z(24, C, 2)
    Mb, d = synth.tac_params(C, g, synth.rng_for(77, g))
    out = O.tac(Z, Mb, d, g).astype(np.float64)
    Z64 = Z.astype(np.float64).reshape(24, C // g, g)
    ref = np.einsum("ibc,brc->ibr", Z64, Mb.astype(np.float64)).reshape(24, C) + d.astype(np.float64)
    rn = ref.astype(np.float16).astype(np.float64)
    ulp = np.spacing(np.abs(ref).astype(np.float16)).astype(np.float64)
    assert np.all(np.abs(out - ref) <= ulp)
    # away from fp16 midpoints the result is the correctly rounded one
    frac = np.abs(ref - rn) / ulp                   # 0.5 at an fp16 midpoint
    absmag = np.einsum("ibc,brc->ibr", np.abs(Z64), np.abs(Mb.astype(np.float64))).reshape(24, C)
    fp32_err = (g + 2) * 2.0 ** -24 * (absmag + np.abs(d.astype(np.float64)))
    clear = np.abs(frac - 0.5) * ulp > fp32_err
    assert clear.mean() > 0.9
    assert np.all(out[clear] == rn[clear])


def test_blocks_are_independent():
    C, g = 256, 16
    Z = _z(8, C, 3)
    Mb, d = synth.tac_params(C, g, synth.rng_for(78, 0))
    base = O.tac(Z, Mb, d, g)
    Mb2 = Mb.copy()
    Mb2[5] = (Mb2[5].astype(np.float32) * 1.5).astype(np.float16)
    pert = O.tac(Z, Mb2, d, g)
    changed = np.any(pert != base, axis=0)
    assert changed[5 * g:6 * g].any()
    assert not changed[:5 * g].any() and not changed[6 * g:].any()


def test_default_block_rule():
    """g = 16, else the largest g <= 16 dividing C (App. C)."""
    assert synth.default_tac_block(4096) == 16
    assert synth.default_tac_block(3584) == 16
    assert synth.default_tac_block(360) == 15
    assert synth.default_tac_block(98) == 14
    assert synth.default_tac_block(17) == 1


def test_gate_vector_matches_eq9():
    # K = 64, d_m = d_u = 2: G_m = diag(1_60, 1_2, 0_2), G_u = diag(1_60, 0_2, 1_2)
    gm = O.gate_vector(64, 2, 2, True)
    gu = O.gate_vector(64, 2, 2, False)
    assert gm.tolist() == [1.0] * 60 + [1.0, 1.0] + [0.0, 0.0]
    assert gu.tolist() == [1.0] * 60 + [0.0, 0.0] + [1.0, 1.0]


def test_tac_then_quant_act_equals_fused_composition():
    """TAC materialised as fp16 then quantised equals the oracle's quant_act with TAC."""
    c = synth.small_case(20, 16, 256, 8, g=16)
    K = 256
    dm, du = synth.default_band(K)
    z = O.tac(c["X"], c["tac_M"], c["tac_d"], 16)
    a = O.quant_act(z, c["state"], c["P"], dm, du)
    b = O.quant_act(c["X"], c["state"], c["P"], dm, du, c["tac_M"], c["tac_d"], 16)
    assert a[0].tobytes() == b[0].tobytes() and a[1].tobytes() == b[1].tobytes()
