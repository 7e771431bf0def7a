"""GPU parity: every entry point of libstarquant against the CPU oracle on the same
seeded inputs.  Codes, scales, transformed rows and int32 accumulators must be
bit-identical; fp16 outputs within 1e-3 rel / 1e-2 abs and in fact bit-identical."""
import glob
import json
import os

import numpy as np
import pytest
import torch

import paper_2606_04945_amd as sq
import synth
from oracle import oracle as O
from gpu_util import assert_bits, assert_y, dev, host, pack_codes, say

pytestmark = pytest.mark.gpu
THREADS = min(16, os.cpu_count() or 1)


def _x(M, K, seed, state=None, n_out=2):
    st = state if state is not None else (np.random.default_rng(seed).random(M) < 0.5).astype(np.uint8)
    rng = synth.rng_for(500 + seed, 0)
    m_idx, u_idx = synth.outlier_channels(K, n_out, rng)
    return synth.activations(M, K, st, m_idx, u_idx, rng), st


# ------------------------------------------------------------------ quantiser

@pytest.mark.parametrize("amax", [1.0, 7.0, 0.3, 1234.5, 3.0e-3, 65504.0])
def test_quantiser_exhaustive_fp16(amax):
    """Every finite fp16 value |v| <= amax in rows with absmax amax: GPU division,
    rint and packing agree with the oracle bit for bit."""
    h = np.arange(65536, dtype=np.uint16)
    v = h.view(np.float16)
    v = v[np.isfinite(v) & (np.abs(v.astype(np.float32)) <= amax)]
    K = 4096
    n = (len(v) + K - 2) // (K - 1)
    rows = np.zeros((n, K), np.float16)
    rows[:, 0] = np.float16(amax)
    flat = np.zeros(n * (K - 1), np.float16)
    flat[:len(v)] = v
    rows[:, 1:] = flat.reshape(n, K - 1)
    say(f"quantiser exhaustive amax={amax} rows={n}")
    Aq, s = sq.sgat_quant_act(dev(rows), None, None, 0, 0)
    ref_q, ref_s = O.quant_act(rows, None, None, 0, 0)
    assert_bits(host(s), ref_s, "s_a")
    assert_bits(host(Aq), ref_q, "Aq")
    # the same rows through the fp32 entry point
    Aq2, s2 = sq.sgat_quantize(dev(rows.astype(np.float32)))
    assert_bits(host(s2), ref_s, "s (fp32 path)")
    assert_bits(host(Aq2), ref_q, "Aq (fp32 path)")


def test_zero_rows_and_tiny_scales():
    K = 256
    x = np.zeros((4, K), np.float32)
    x[1, 3] = 1e-45                 # scale underflows to 0 -> all codes 0
    x[2, :] = 1e-40                 # subnormal rows
    x[3, 7] = -3e-39
    Aq, s = sq.sgat_quantize(dev(x))
    rq, rs, _ = O.quant_rows(x)
    assert_bits(host(s), rs, "s")
    assert_bits(host(Aq), rq, "Aq")


# ------------------------------------------------------------------ folded basis (P = NULL)

# while rows x vectors per lane <= 768 a row spans one workgroup per vector of
# a lane: (77, 4096), (130, 3584), (5, 6144), (16, 12288), (64, 18944);
# (129, 12288) takes one workgroup per row
@pytest.mark.parametrize("M,K", [(1, 64), (3, 512), (77, 4096), (130, 3584), (5, 6144), (16, 12288),
                                 (129, 12288), (64, 18944), (3, 131072)])
@pytest.mark.parametrize("layout", ["random", "all_masked", "none_masked", "alternating"])
def test_quant_act_folded(M, K, layout):
    st = None if layout == "random" else synth.state_edge(M, layout)
    X, st = _x(M, K, 1, st)
    dm, du = synth.default_band(K)
    say(f"quant_act folded M={M} K={K} {layout}")
    Aq, s = sq.sgat_quant_act(dev(X), dev(st), None, dm, du)
    ref_q, ref_s = O.quant_act(X, st, None, dm, du)
    assert_bits(host(s), ref_s, "s_a")
    assert_bits(host(Aq), ref_q, "Aq")


@pytest.mark.parametrize("K", [24576, 32768, 131072])
def test_quantize_rows_longer_than_the_register_tile(K):
    """Rows above 12 x 256 vectors of 8 are read twice instead of held (the reload path)."""
    x = np.random.default_rng(K).standard_normal((3, K)).astype(np.float32)
    x[1, 5] = 40.0
    Aq, s = sq.sgat_quantize(dev(x))
    rq, rs, _ = O.quant_rows(x)
    assert_bits(host(s), rs, "s")
    assert_bits(host(Aq), rq, "Aq")
    Aq8, s8 = sq.sgat_quantize_w8(dev(x))
    rq8, rs8 = O.quant_rows_q8(x)
    assert_bits(host(s8), rs8, "s8")
    assert_bits(host(Aq8), rq8, "Aq8")


def test_quant_act_folded_no_gate_and_custom_bands():
    X, st = _x(50, 512, 2)
    for dm, du in [(0, 0), (16, 0), (0, 48), (100, 200)]:
        Aq, s = sq.sgat_quant_act(dev(X), dev(st), None, dm, du)
        ref_q, ref_s = O.quant_act(X, st, None, dm, du)
        assert_bits(host(s), ref_s, f"s_a bands {dm},{du}")
        assert_bits(host(Aq), ref_q, f"Aq bands {dm},{du}")


# ------------------------------------------------------------------ dense transform

@pytest.mark.parametrize("M,K", [(1, 64), (5, 192), (130, 512), (257, 1024), (33, 4096), (2100, 4096), (2000, 4160)])
def test_transform_bit_exact(M, K):
    X, st = _x(M, K, 3)
    P = synth.orthogonal(K, synth.rng_for(600, K))
    dm, du = synth.default_band(K)
    say(f"transform M={M} K={K}")
    xp = sq.sgat_transform(dev(X), dev(st), dev(P), dm, du)
    ref = O.transform(X, st, P, dm, du, threads=THREADS)
    assert_bits(host(xp), ref, "x'")
    xp0 = sq.sgat_transform(dev(X), None, dev(P))
    assert_bits(host(xp0), O.transform(X, None, P, 0, 0, threads=THREADS), "x' ungated")


@pytest.mark.parametrize("M,K,dm,du", [(300, 1024, 256, 384), (1000, 4096, 128, 128), (70, 4096, 128, 128),
                                        (513, 1024, 0, 384), (260, 1024, 256, 0), (2100, 4096, 128, 128)])
@pytest.mark.parametrize("layout", ["random", "all_masked", "none_masked", "alternating", "blocks"])
def test_transform_rows_grouped_by_state(M, K, dm, du, layout):
    """Bands that hold whole 128-column tiles: rows are taken grouped by state and
    row tiles of one state skip the tiles of the band they drop; the result is
    the oracle's bit for bit, the dropped columns +0."""
    rng = np.random.default_rng(M + K + dm)
    st = {"random": (rng.random(M) < 0.4), "all_masked": np.ones(M, bool), "none_masked": np.zeros(M, bool),
          "alternating": np.arange(M) % 2 == 1, "blocks": (np.arange(M) // 37) % 3 == 0}[layout].astype(np.uint8)
    X, _ = _x(M, K, 9, state=st)
    P = synth.orthogonal(K, synth.rng_for(604, K))
    say(f"transform grouped M={M} K={K} dm={dm} du={du} {layout}")
    xp = host(sq.sgat_transform(dev(X), dev(st), dev(P), dm, du))
    ref = O.transform(X, st, P, dm, du, threads=THREADS)
    assert_bits(xp, ref, "x'")
    dropped_u = st.astype(bool)[:, None] & (np.arange(K) >= K - du)[None, :]
    dropped_m = ~st.astype(bool)[:, None] & ((np.arange(K) >= K - dm - du) & (np.arange(K) < K - du))[None, :]
    gone = xp[dropped_u | dropped_m]
    assert (gone == 0).all() and not np.signbit(gone).any()


def test_transform_subnormal_products_and_signed_zeros():
    """A basis of subnormal and zero entries: products, chunk sums and totals are
    fp32 subnormals or signed zeros, kept (not flushed) and summed exactly as the
    oracle's IEEE chain does; zero columns give +0 for every row."""
    M, K = 200, 512
    X, st = _x(M, K, 12)
    P = synth.orthogonal(K, synth.rng_for(606, K)) * np.float32(2.0 ** -136)   # entries around 2^-140
    P[:, 5::7] = 0.0
    P[:, 6::7] = -0.0
    P = P.astype(np.float32)
    assert (np.abs(P[P != 0]) < np.float32(2.0 ** -126)).all()
    say(f"transform subnormal basis M={M} K={K}")
    for M_ in (M, 20):   # the pipelined kernel and the one for up to 32 rows
        xp = host(sq.sgat_transform(dev(X[:M_]), None, dev(P)))
        ref = O.transform(X[:M_], None, P, 0, 0, threads=THREADS)
        assert (ref != 0).any() and (np.abs(ref[ref != 0]) < np.float32(2.0 ** -126)).any()
        assert_bits(xp, ref, f"x' (subnormal basis, {M_} rows)")


def test_transform_identity_basis_equals_folded():
    X, st = _x(40, 512, 4)
    dm, du = synth.default_band(512)
    a = sq.sgat_transform(dev(X), dev(st), dev(np.eye(512, dtype=np.float32)), dm, du)
    b = sq.sgat_transform(dev(X), dev(st), None, dm, du)
    assert_bits(host(a), host(b), "P = I vs P = NULL")
    assert_bits(host(b), O.transform(X, st, None, dm, du), "P = NULL")


@pytest.mark.parametrize("M,K", [(7, 256), (200, 1024), (129, 4096)])
def test_quant_act_dense(M, K):
    X, st = _x(M, K, 5)
    P = synth.orthogonal(K, synth.rng_for(601, K))
    dm, du = synth.default_band(K)
    say(f"quant_act dense M={M} K={K}")
    Aq, s = sq.sgat_quant_act(dev(X), dev(st), dev(P), dm, du)
    ref_q, ref_s = O.quant_act(X, st, P, dm, du, threads=THREADS)
    assert_bits(host(s), ref_s, "s_a")
    assert_bits(host(Aq), ref_q, "Aq")


@pytest.mark.parametrize("N,K,withP", [(24, 512, True), (200, 1024, True), (64, 4096, False), (8, 64, True)])
def test_prepare_weights(N, K, withP):
    W = synth.weights(N, K, synth.rng_for(602, N, K))
    P = synth.orthogonal(K, synth.rng_for(603, K)) if withP else None
    say(f"prepare_weights N={N} K={K} P={withP}")
    Wq, s_w = sq.sgat_prepare_weights(dev(W), dev(P) if withP else None)
    if withP:
        rq, rs = O.prepare_weights(W, P, threads=THREADS)
    else:
        rq, rs = O.quant_act(W, None, None, 0, 0)
    assert_bits(host(s_w), rs, "s_w")
    assert_bits(host(Wq), rq, "Wq")


# ------------------------------------------------------------------ GEMM

def _codes(M, K, seed, lo=-7, hi=7):
    q = np.random.default_rng(seed).integers(lo, hi + 1, (M, K))
    return pack_codes(q)


# every launch plan: short M, 1 to 3 row tiles of 16 (activations shared in LDS for
# wide 4-bit layers, expanded once for one row tile, per wave for more; a half
# last k step and a partial last workgroup; K split inside the workgroup 1, 2, 4
# or 8 ways), the tiled shapes with ragged last tiles and the split-K path
GEMM_SHAPES = [(1, 8, 64), (16, 4096, 4096), (5, 4104, 4096), (9, 136, 192), (16, 24, 18944),
               (16, 12288, 4096), (16, 4096, 12288), (9, 16392, 192), (16, 32768, 256), (33, 520, 1024),
               (16, 24576, 4096), (7, 37888, 3584), (3, 12304, 4032), (1, 12288, 64), (16, 16392, 8192),
               (11, 2056, 4160), (4096, 8200, 192), (4096, 8200, 4160),
               (64, 24576, 4096), (48, 12304, 4032), (20, 16384, 8192), (64, 16392, 8192), (40, 4104, 12288),
               (77, 200, 192), (128, 256, 512), (300, 136, 4096), (300, 16384, 64), (1024, 1024, 1024),
               (1000, 8200, 64), (2100, 12296, 64), (513, 4104, 3584), (64, 512, 18944),
               (4096, 4096, 192), (4000, 4000, 4160), (1000, 12296, 4160),
               # two k groups per tile: ragged M and N, an odd number of k steps (half a last step at 4 bits)
               (1000, 4000, 12352), (1024, 3584, 18944), (1000, 3584, 19008)]


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
def test_gemm_bit_exact(M, N, K):
    Aq = _codes(M, K, 1)
    Wq = _codes(N, K, 2)
    rng = np.random.default_rng(3)
    s_a = rng.uniform(0.05, 3, M).astype(np.float32)
    s_w = rng.uniform(1e-4, 5e-3, N).astype(np.float32)
    say(f"gemm M={M} N={N} K={K} ws={sq.gemm_workspace_bytes(M, N, K)}")
    Y, acc = sq.w4a4_gemm(dev(Aq), dev(s_a), dev(Wq), dev(s_w), want_acc=True)
    Y, acc = host(Y), host(acc)
    rows = np.arange(M) if M * N * K <= 3e9 else np.unique(np.r_[0, M - 1, np.random.default_rng(4).choice(M, 24)])
    rY, racc = O.gemm(Aq[rows], s_a[rows], Wq, s_w, threads=THREADS)
    assert_bits(acc[rows], racc, "acc")
    assert_y(Y[rows], rY)


def test_gemm_extreme_codes():
    """All codes -8 or +7 at the largest config K: the scaled int8 sums stay exact."""
    K, M, N = 18944, 8, 16
    q = np.random.default_rng(5).choice([-8, 7], (M, K))
    w = np.random.default_rng(6).choice([-8, 7], (N, K))
    Aq, Wq = pack_codes(q), pack_codes(w)
    s_a = np.ones(M, np.float32)
    s_w = np.full(N, 1e-3, np.float32)
    Y, acc = sq.w4a4_gemm(dev(Aq), dev(s_a), dev(Wq), dev(s_w), want_acc=True)
    assert_bits(host(acc), (q @ w.T).astype(np.int32), "acc")
    rY, _ = O.gemm(Aq, s_a, Wq, s_w)
    assert_y(host(Y), rY)


@pytest.mark.parametrize("M,N", [(1, 8), (3, 16), (130, 136)])
def test_gemm_at_the_largest_K(M, N):
    """K = 131072: random codes, and the one extreme sum (every product (-8)(-8), so
    the dot product is 2^23 and its x256 scaled form is 2^31) on row 0 / column 0."""
    K = 131072
    rng = np.random.default_rng(11 + M)
    q = rng.integers(-8, 8, (M, K))
    w = rng.integers(-8, 8, (N, K))
    q[0, :] = -8
    w[0, :] = -8
    Aq, Wq = pack_codes(q), pack_codes(w)
    s_a = rng.uniform(0.5, 1, M).astype(np.float32)
    s_w = rng.uniform(1e-8, 1e-7, N).astype(np.float32)
    say(f"gemm largest K M={M} N={N} ws={sq.gemm_workspace_bytes(M, N, K)}")
    Y, acc = sq.w4a4_gemm(dev(Aq), dev(s_a), dev(Wq), dev(s_w), want_acc=True)
    ref = q.astype(np.int64) @ w.T.astype(np.int64)
    assert ref[0, 0] == 1 << 23
    assert_bits(host(acc), ref.astype(np.int32), "acc")
    rY, racc = O.gemm(Aq, s_a, Wq, s_w, threads=THREADS)
    assert_bits(racc, ref.astype(np.int32), "oracle acc")
    assert_y(host(Y), rY)


def test_w8a8_gemm_at_the_largest_K():
    K, M, N = 65536, 3, 16
    q = np.full((M, K), -128, np.int8)
    w = np.full((N, K), -128, np.int8)
    q[1:] = np.random.default_rng(12).integers(-128, 128, (M - 1, K))
    s_a = np.ones(M, np.float32)
    s_w = np.full(N, 1e-9, np.float32)
    Y, acc = sq.w8a8_gemm(dev(q), dev(s_a), dev(w), dev(s_w), want_acc=True)
    ref = q.astype(np.int64) @ w.T.astype(np.int64)
    assert ref[0, 0] == 1 << 30
    assert_bits(host(acc), ref.astype(np.int32), "acc")


def test_gemm_split_and_unsplit_agree():
    """Rows computed through the split-K path (few tiles) and through the short-M
    kernels equal the same rows inside a tall M that takes the single-pass path."""
    K, N = 12288, 4096
    Aq = _codes(2048, K, 7)
    Wq = _codes(N, K, 8)
    s_a = np.random.default_rng(9).uniform(0.1, 2, 2048).astype(np.float32)
    s_w = np.random.default_rng(10).uniform(1e-3, 2e-3, N).astype(np.float32)
    assert sq.gemm_workspace_bytes(96, N, K) > 0 and sq.gemm_workspace_bytes(2048, N, K) == 0
    big = host(sq.w4a4_gemm(dev(Aq), dev(s_a), dev(Wq), dev(s_w)))
    for m in (96, 48, 16):
        small = host(sq.w4a4_gemm(dev(Aq[:m]), dev(s_a[:m]), dev(Wq), dev(s_w)))
        assert_bits(small, big[:m], f"{m} rows vs the single-pass rows")


# ------------------------------------------------------------------ TAC

@pytest.mark.parametrize("g", [1, 2, 4, 8, 16, 32, 64, 128])
@pytest.mark.parametrize("M,C", [(1, 128), (100, 512), (257, 4096), (1000, 3584)])
def test_tac_bit_exact(g, M, C):
    Z = (np.random.default_rng(g + M).standard_normal((M, C)) * 2).astype(np.float16)
    Mb, d = synth.tac_params(C, g, synth.rng_for(700, g, C))
    say(f"tac g={g} M={M} C={C}")
    out = host(sq.tac_apply(dev(Z), dev(Mb), dev(d), g))
    assert_bits(out, O.tac(Z, Mb, d, g, threads=THREADS), "tac")


@pytest.mark.parametrize("g", [1, 2, 4, 8, 16, 32, 64])
@pytest.mark.parametrize("M,C", [(70, 192), (300, 320)])
def test_tac_bit_exact_widths_off_the_tile(g, M, C):
    """Widths that are not a multiple of 128 channels take the VALU kernel."""
    Z = (np.random.default_rng(g + M + 1).standard_normal((M, C)) * 2).astype(np.float16)
    Mb, d = synth.tac_params(C, g, synth.rng_for(704, g, C))
    say(f"tac g={g} M={M} C={C}")
    out = host(sq.tac_apply(dev(Z), dev(Mb), dev(d), g))
    assert_bits(out, O.tac(Z, Mb, d, g, threads=THREADS), "tac")


@pytest.mark.parametrize("g", [16, 128])
def test_tac_identity_is_a_no_op(g):
    Z = (np.random.default_rng(1).standard_normal((64, 4096)) * 4).astype(np.float16)
    Mb, d = synth.tac_params(4096, g, None, identity=True)
    out = host(sq.tac_apply(dev(Z), dev(Mb), dev(d), g))
    same = (out.view(np.uint16) == Z.view(np.uint16)) | ((out == 0) & (Z == 0))
    assert same.all()


@pytest.mark.parametrize("withP", [False, True])
@pytest.mark.parametrize("g", [16, 128])
def test_quant_act_with_tac(withP, g):
    M, K = 150, 1024
    X, st = _x(M, K, 6)
    Mb, d = synth.tac_params(K, g, synth.rng_for(701, g))
    P = synth.orthogonal(K, synth.rng_for(702, K)) if withP else None
    dm, du = synth.default_band(K)
    say(f"quant_act + tac g={g} P={withP}")
    Aq, s = sq.sgat_quant_act(dev(X), dev(st), dev(P) if withP else None, dm, du, dev(Mb), dev(d), g)
    rq, rs = O.quant_act(X, st, P, dm, du, Mb, d, g, threads=THREADS)
    assert_bits(host(s), rs, "s_a")
    assert_bits(host(Aq), rq, "Aq")


@pytest.mark.parametrize("g", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("M,K", [(1, 64), (37, 512), (300, 3584), (129, 4096), (20, 8192), (1025, 1024),
                                 (2100, 3584), (4100, 3584), (5000, 4096), (33000, 512)])
def test_quant_act_tac_folded_fused(g, M, K):
    """TAC fused with the gate and quantiser (folded basis, g <= 16, K <= 4096; wider
    rows take the staged path): bit-exact with the oracle's TAC-then-quantise.  The
    larger M give each workgroup a run of 2 ... 64 rows (a ragged last run
    included), which streams through the ring of row slots."""
    X, st = _x(M, K, 8)
    Mb, d = synth.tac_params(K, g, synth.rng_for(703, g, K))
    dm, du = synth.default_band(K)
    say(f"quant_act + fused tac g={g} M={M} K={K}")
    Aq, s = sq.sgat_quant_act(dev(X), dev(st), None, dm, du, dev(Mb), dev(d), g)
    rq, rs = O.quant_act(X, st, None, dm, du, Mb, d, g, threads=THREADS)
    assert_bits(host(s), rs, "s_a")
    assert_bits(host(Aq), rq, "Aq")
    # no gate
    Aq, s = sq.sgat_quant_act(dev(X), None, None, 0, 0, dev(Mb), dev(d), g)
    rq, rs = O.quant_act(X, None, None, 0, 0, Mb, d, g, threads=THREADS)
    assert_bits(host(s), rs, "s_a (no gate)")
    assert_bits(host(Aq), rq, "Aq (no gate)")


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("M,K,dm,du", [(4100, 3584, 112, 112), (4100, 3584, 40, 24), (4096, 4096, 1000, 600),
                                       (8200, 4096, 0, 0), (4111, 2048, 8, 520)])
def test_quant_act_tac_fused_matrix_cores_bands(bits, M, K, dm, du):
    """The matrix-core form of the fused TAC pass (g = 16, >= 4096 tokens, rows
    of four to eight 512-channel parts): band edges inside a 16-channel
    block, bands spanning several waves, no band, a ragged last 16-token tile,
    several tiles per workgroup (8200 tokens), 4- and 8-bit codes."""
    X, st = _x(M, K, 12)
    Mb, d = synth.tac_params(K, 16, synth.rng_for(707, K, dm))
    say(f"quant_act + fused tac (matrix cores) M={M} K={K} bands={dm},{du} bits={bits}")
    qa, oq = (sq.sgat_quant_act, O.quant_act) if bits == 4 else (sq.sgat_quant_act_w8, O.quant_act_q8)
    Aq, s = qa(dev(X), dev(st), None, dm, du, dev(Mb), dev(d), 16)
    rq, rs = oq(X, st, None, dm, du, Mb, d, 16, threads=THREADS)
    assert_bits(host(s), rs, "s_a")
    assert_bits(host(Aq), rq, "Aq")


# ------------------------------------------------------------------ end to end

def test_config0_end_to_end():
    """The small configuration in full: 128 tokens, K = N = 512, dense P."""
    st = synth.config_state(synth.SINGLE_LINEAR)
    t = synth.site_tensors(synth.SINGLE_LINEAR, 0, st)
    say("config 0 end to end")
    Xd, Pd = dev(t.X), dev(t.P)
    Wq, s_w = sq.sgat_prepare_weights(dev(t.W), Pd)
    Aq, s_a = sq.sgat_quant_act(Xd, dev(st), Pd, t.dm, t.du)
    Y, acc = sq.w4a4_gemm(Aq, s_a, Wq, s_w, want_acc=True)
    ref = O.sgat_linear(t.X, st, t.P, t.W, t.dm, t.du, threads=THREADS)
    for k, v in dict(Aq=Aq, s_a=s_a, Wq=Wq, s_w=s_w, acc=acc).items():
        assert_bits(host(v), ref[k], k)
    assert_y(host(Y), ref["Y"])
    # determinism: a second run is bitwise identical
    Y2 = sq.w4a4_gemm(*sq.sgat_quant_act(Xd, dev(st), Pd, t.dm, t.du), Wq, s_w)
    assert_bits(host(Y2), host(Y), "repeat")


GOLD = sorted(glob.glob(os.path.join(os.path.dirname(__file__), "golden", "*.json")))


@pytest.mark.parametrize("path", GOLD, ids=[os.path.basename(p) for p in GOLD])
def test_golden_fixtures(path):
    from test_oracle_golden import load
    d, ins, outs = load(path)
    g = d["g"]
    say(f"golden {os.path.basename(path)}")
    P = dev(ins["P"]) if d["has_P"] else None
    Aq, s_a = sq.sgat_quant_act(dev(ins["X"]), dev(ins["state"]), P, d["dm"], d["du"],
                                dev(ins["tac_M"]) if g else None, dev(ins["tac_d"]) if g else None, g)
    Wq, s_w = sq.sgat_prepare_weights(dev(ins["W"]), P)
    Y, acc = sq.w4a4_gemm(Aq, s_a, Wq, s_w, want_acc=True)
    for k, v in dict(Aq=Aq, s_a=s_a, Wq=Wq, s_w=s_w, acc=acc, Y=Y).items():
        assert_bits(host(v), outs[k], k)


def test_empty_inputs_leave_outputs_untouched():
    Aq = torch.full((0, 32), 7, dtype=torch.uint8, device="cuda")
    s = torch.empty((0,), dtype=torch.float32, device="cuda")
    sq.sgat_quant_act(torch.empty((0, 64), dtype=torch.float16, device="cuda"), None, None, 2, 2, Aq=Aq, s_a=s)
    Y = torch.full((4, 16), 3.0, dtype=torch.float16, device="cuda")
    sq.w4a4_gemm(torch.empty((4, 32), dtype=torch.uint8, device="cuda")[:0], s,
                 torch.zeros((16, 32), dtype=torch.uint8, device="cuda"),
                 torch.ones(16, dtype=torch.float32, device="cuda"), Y=Y[:0])
    torch.cuda.synchronize()
    assert (host(Y) == 3.0).all()


# ------------------------------------------------------------------ W8A8 (App. D)

@pytest.mark.parametrize("amax", [1.0, 127.0, 0.3, 65504.0])
def test_w8_quantiser_exhaustive_fp16(amax):
    h = np.arange(65536, dtype=np.uint16)
    v = h.view(np.float16)
    v = v[np.isfinite(v) & (np.abs(v.astype(np.float32)) <= amax)]
    K = 4096
    n = (len(v) + K - 2) // (K - 1)
    rows = np.zeros((n, K), np.float16)
    rows[:, 0] = np.float16(amax)
    flat = np.zeros(n * (K - 1), np.float16)
    flat[:len(v)] = v
    rows[:, 1:] = flat.reshape(n, K - 1)
    say(f"w8 quantiser exhaustive amax={amax}")
    Aq, s = sq.sgat_quant_act_w8(dev(rows), None, None, 0, 0)
    rq, rs = O.quant_act_q8(rows, None, None, 0, 0)
    assert_bits(host(s), rs, "s_a")
    assert_bits(host(Aq), rq, "Aq")
    Aq2, s2 = sq.sgat_quantize_w8(dev(rows.astype(np.float32)))
    assert_bits(host(Aq2), rq, "Aq (fp32 path)")


@pytest.mark.parametrize("M,K", [(16, 12288), (3, 6144), (384, 4096), (385, 4096)])
def test_w8_quant_act_short_batches(M, K):
    """8-bit codes on the row-split path (rows x vectors per lane <= 768) and
    just past it, fp16 and fp32 inputs."""
    X, st = _x(M, K, 10)
    dm, du = synth.default_band(K)
    say(f"w8 quant_act short M={M} K={K}")
    Aq, s = sq.sgat_quant_act_w8(dev(X), dev(st), None, dm, du)
    rq, rs = O.quant_act_q8(X, st, None, dm, du)
    assert_bits(host(s), rs, "s_a")
    assert_bits(host(Aq), rq, "Aq")
    x32 = X.astype(np.float32)
    Aq2, s2 = sq.sgat_quantize_w8(dev(x32))
    rq2, rs2 = O.quant_rows_q8(x32)
    assert_bits(host(s2), rs2, "s (fp32 path)")
    assert_bits(host(Aq2), rq2, "Aq (fp32 path)")


@pytest.mark.parametrize("withP,g", [(False, 0), (True, 0), (False, 16), (False, 128), (True, 16)])
def test_w8_quant_act(withP, g):
    M, K = 150, 1024
    X, st = _x(M, K, 9)
    P = synth.orthogonal(K, synth.rng_for(704, K)) if withP else None
    dm, du = synth.default_band(K)
    Mb, d = synth.tac_params(K, g, synth.rng_for(705, g)) if g else (None, None)
    say(f"w8 quant_act P={withP} g={g}")
    Aq, s = sq.sgat_quant_act_w8(dev(X), dev(st), dev(P) if withP else None, dm, du,
                                 dev(Mb) if g else None, dev(d) if g else None, g)
    rq, rs = O.quant_act_q8(X, st, P, dm, du, Mb, d, g, threads=THREADS)
    assert_bits(host(s), rs, "s_a")
    assert_bits(host(Aq), rq, "Aq")


@pytest.mark.parametrize("M,K", [(2100, 3584), (17, 4096), (4100, 3584)])
def test_w8_quant_act_tac_fused(M, K):
    """8-bit codes from the fused TAC pass (g = 16, folded basis) on several
    16-token tiles and a ragged last one."""
    X, st = _x(M, K, 10)
    dm, du = synth.default_band(K)
    Mb, d = synth.tac_params(K, 16, synth.rng_for(706, K))
    say(f"w8 quant_act fused tac M={M} K={K}")
    Aq, s = sq.sgat_quant_act_w8(dev(X), dev(st), None, dm, du, dev(Mb), dev(d), 16)
    rq, rs = O.quant_act_q8(X, st, None, dm, du, Mb, d, 16, threads=THREADS)
    assert_bits(host(s), rs, "s_a")
    assert_bits(host(Aq), rq, "Aq")


@pytest.mark.parametrize("withP", [True, False])
def test_w8_prepare_weights(withP):
    N, K = 200, 1024
    W = synth.weights(N, K, synth.rng_for(706, N))
    P = synth.orthogonal(K, synth.rng_for(707, K)) if withP else None
    Wq, s_w = sq.sgat_prepare_weights_w8(dev(W), dev(P) if withP else None)
    rq, rs = (O.prepare_weights_q8(W, P, threads=THREADS) if withP else O.quant_act_q8(W, None, None, 0, 0))
    assert_bits(host(s_w), rs, "s_w")
    assert_bits(host(Wq), rq, "Wq")


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
def test_w8a8_gemm_bit_exact(M, N, K):
    rng = np.random.default_rng(10)
    Aq = rng.integers(-128, 128, (M, K)).astype(np.int8)
    Wq = rng.integers(-128, 128, (N, K)).astype(np.int8)
    s_a = rng.uniform(0.01, 1, M).astype(np.float32)
    s_w = rng.uniform(1e-5, 1e-3, N).astype(np.float32)
    say(f"w8a8 gemm M={M} N={N} K={K}")
    Y, acc = sq.w8a8_gemm(dev(Aq), dev(s_a), dev(Wq), dev(s_w), want_acc=True)
    Y, acc = host(Y), host(acc)
    rows = np.arange(M) if M * N * K <= 3e9 else np.unique(np.r_[0, M - 1, rng.choice(M, 24)])
    rY, racc = O.gemm_q8(Aq[rows], s_a[rows], Wq, s_w, threads=THREADS)
    assert_bits(acc[rows], racc, "acc")
    assert_y(Y[rows], rY)


def test_w8a8_config0_end_to_end():
    st = synth.config_state(synth.SINGLE_LINEAR)
    t = synth.site_tensors(synth.SINGLE_LINEAR, 0, st)
    Pd = dev(t.P)
    Wq, s_w = sq.sgat_prepare_weights_w8(dev(t.W), Pd)
    Aq, s_a = sq.sgat_quant_act_w8(dev(t.X), dev(st), Pd, t.dm, t.du)
    Y, acc = sq.w8a8_gemm(Aq, s_a, Wq, s_w, want_acc=True)
    rA, rs = O.quant_act_q8(t.X, st, t.P, t.dm, t.du, threads=THREADS)
    rW, rsw = O.prepare_weights_q8(t.W, t.P, threads=THREADS)
    rY, racc = O.gemm_q8(rA, rs, rW, rsw, threads=THREADS)
    for name, got, ref in (("Aq", Aq, rA), ("s_a", s_a, rs), ("Wq", Wq, rW), ("s_w", s_w, rsw), ("acc", acc, racc)):
        assert_bits(host(got), ref, name)
    assert_y(host(Y), rY)
