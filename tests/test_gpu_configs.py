"""GPU parity at the full workload sizes, in the launch configurations the benchmark
uses: every linear of the LLaDA- and Dream-shaped layer sets, the TAC + O-projection
workload (g = 128, 16384 tokens), and the denoising-step sweep over token counts.

The GPU runs each whole layer, with fragment-ordered weights (the benchmark's
launch) and row-major weights, which must agree on every output; the oracle
recomputes 64 sampled token rows (first and last, first and last of each state,
random) one by one (rows are independent) against every output channel where
the basis is folded (the oracle's weights are then cheap) and 256 sampled
channels (every 128-column tile edge among them) with the dense basis, and
those must match bit for bit.  Properties that hold at any size are checked on
every row."""
import os

import numpy as np
import pytest
import torch

import paper_2606_04945_amd as sq
import synth
from oracle import oracle as O
from gpu_util import assert_bits, assert_y, dev, host, say

pytestmark = [pytest.mark.gpu, pytest.mark.slow]
THREADS = min(16, os.cpu_count() or 1)


def sample_rows(state, n, seed):
    """First, last, first masked, first unmasked, and random rows."""
    M = len(state)
    rng = np.random.default_rng(seed)
    pick = [0, M - 1]
    for s in (0, 1):
        idx = np.nonzero(state == s)[0]
        if len(idx):
            pick += [int(idx[0]), int(idx[-1])]
    pick += list(rng.choice(M, size=min(n, M), replace=False))
    return np.unique(np.array(pick))


def check_codes_all_rows(Aq, s_a):
    """Every row with a non-zero scale has codes in [-7, 7] and max |code| = 7."""
    a = host(Aq)
    lo = (a & 15).astype(np.int8)
    hi = (a >> 4).astype(np.int8)
    lo = np.where(lo >= 8, lo - 16, lo)
    hi = np.where(hi >= 8, hi - 16, hi)
    mx = np.maximum(np.abs(lo).max(axis=1), np.abs(hi).max(axis=1))
    mn = np.minimum(lo.min(axis=1), hi.min(axis=1))
    s = host(s_a)
    assert (mn >= -7).all()
    assert (mx[s > 0] == 7).all() and (mx[s == 0] == 0).all()


def sample_cols(N, n, seed):
    """First and last columns, both sides of every 128- and 256-column tile edge
    up to n / 4 of them, and random columns: n in all (every column if N <= n)."""
    if N <= n:
        return np.arange(N)
    edges = np.arange(128, N, 128)
    edges = edges[np.linspace(0, len(edges) - 1, min(len(edges), n // 8)).astype(int)] if len(edges) else edges
    pick = np.unique(np.r_[0, N - 1, edges - 1, edges])
    rest = np.setdiff1d(np.arange(N), pick)
    extra = np.random.default_rng(seed).choice(rest, size=max(0, n - len(pick)), replace=False)
    return np.unique(np.r_[pick, extra])


def run_site(cid, si, state, *, g=None, folded=False, n_rows=64, n_cols=None, tac_identity=False):
    """One linear of workload `cid` on the GPU, whole, in the benchmark's launch
    (fragment-ordered weights) and with row-major weights (equal bit for bit);
    then the oracle recomputes n_rows sampled token rows against n_cols sampled
    output channels (every channel when n_cols is None: the default for a folded
    basis, whose oracle weights are cheap), bit for bit."""
    t = synth.site_tensors(cid, si, state, tac_identity=tac_identity, g=g, with_P=not folded)
    K, N, M = t.site.K, t.site.N, len(state)
    if n_cols is None and not folded:
        n_cols = 256
    say(f"config {cid} site {t.site.name} M={M} K={K} N={N} tac={t.g} folded={folded} rows={n_rows} "
        f"cols={'all' if n_cols is None else n_cols}")
    Xd, Wd = dev(t.X), dev(t.W)
    Pd = None if folded else dev(t.P)
    tM = dev(t.tac_M) if t.tac_M is not None else None
    td = dev(t.tac_d) if t.tac_d is not None else None
    Wq, s_w = sq.sgat_prepare_weights(Wd, Pd)
    Aq, s_a = sq.sgat_quant_act(Xd, dev(state), Pd, t.dm, t.du, tM, td, t.g)
    Y, acc = sq.w4a4_gemm_frag(Aq, s_a, sq.weights_to_frag(Wq), s_w, want_acc=True)
    Yr, accr = sq.w4a4_gemm(Aq, s_a, Wq, s_w, want_acc=True)
    assert torch.equal(acc, accr) and torch.equal(Y, Yr), "fragment-ordered and row-major weights differ"
    del Yr, accr
    torch.cuda.synchronize()
    rows = sample_rows(state, n_rows, 1000 + si)
    cols = np.arange(N) if n_cols is None else sample_cols(N, n_cols, 2000 + si)
    P = None if folded else t.P
    rq, rs = O.quant_act(t.X[rows], state[rows], P, t.dm, t.du, t.tac_M, t.tac_d, t.g, threads=THREADS)
    if folded:
        wq, ws = O.quant_act(t.W[cols], None, None, 0, 0, threads=THREADS)
    else:
        wq, ws = O.prepare_weights(t.W[cols], P, threads=THREADS)
    ry, racc = O.gemm(rq, rs, wq, ws, threads=THREADS)
    assert_bits(host(s_a)[rows], rs, "s_a rows")
    assert_bits(host(Aq)[rows], rq, "Aq rows")
    assert_bits(host(s_w)[cols], ws, "s_w rows")
    assert_bits(host(Wq)[cols], wq, "Wq rows")
    ri = torch.from_numpy(rows).cuda()
    ci = torch.from_numpy(cols).cuda()
    assert_bits(host(acc.index_select(0, ri).index_select(1, ci)), racc, "acc samples")
    assert_y(host(Y.index_select(0, ri).index_select(1, ci)), ry)
    check_codes_all_rows(Aq, s_a)
    check_codes_all_rows(Wq, s_w)
    del Wq, s_w, Y, acc, Xd, Wd, Pd
    return dict(Aq=Aq, s_a=s_a)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("si", range(4), ids=[s.name for s in synth.CONFIGS[synth.LLADA].sites])
@pytest.mark.parametrize("folded", [False, True], ids=["denseP", "foldedP"])
def test_llada_layer_set(si, folded):
    run_site(synth.LLADA, si, synth.config_state(synth.LLADA), folded=folded)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("si", range(4), ids=[s.name for s in synth.CONFIGS[synth.DREAM].sites])
def test_dream_layer_set(si):
    run_site(synth.DREAM, si, synth.config_state(synth.DREAM))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("si", [1, 2], ids=["o_tac_fused", "gate_up"])
def test_dream_layer_set_folded(si):
    """Folded P at 8 x 2048 tokens: the O projection runs TAC (g = 16) fused into the
    quantiser; gate+up is the widest GEMM of the set."""
    run_site(synth.DREAM, si, synth.config_state(synth.DREAM), folded=True)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("si", range(4), ids=[s.name for s in synth.CONFIGS[synth.LLADA].sites])
def test_llada_layer_set_w8a8(si):
    """The W8A8 variant (App. D) of every linear of the LLaDA-shaped set, folded P."""
    st = synth.config_state(synth.LLADA)
    t = synth.site_tensors(synth.LLADA, si, st, with_P=False)
    K, N, M = t.site.K, t.site.N, len(st)
    say(f"w8a8 config 1 site {t.site.name} M={M} K={K} N={N}")
    tM = dev(t.tac_M) if t.tac_M is not None else None
    td = dev(t.tac_d) if t.tac_d is not None else None
    Wq, s_w = sq.sgat_prepare_weights_w8(dev(t.W), None)
    Aq, s_a = sq.sgat_quant_act_w8(dev(t.X), dev(st), None, t.dm, t.du, tM, td, t.g)
    Y, acc = sq.w8a8_gemm(Aq, s_a, Wq, s_w, want_acc=True)
    torch.cuda.synchronize()
    rows = sample_rows(st, 64, 3000 + si)
    cols = np.arange(N)
    rq, rs = O.quant_act_q8(t.X[rows], st[rows], None, t.dm, t.du, t.tac_M, t.tac_d, t.g, threads=THREADS)
    wq, ws = O.prepare_weights_q8(t.W[cols], None, threads=THREADS)
    ry, racc = O.gemm_q8(rq, rs, wq, ws, threads=THREADS)
    assert_bits(host(s_a)[rows], rs, "s_a rows")
    assert_bits(host(Aq)[rows], rq, "Aq rows")
    assert_bits(host(Wq)[cols], wq, "Wq rows")
    ri = torch.from_numpy(rows).cuda()
    ci = torch.from_numpy(cols).cuda()
    assert_bits(host(acc.index_select(0, ri).index_select(1, ci)), racc, "acc samples")
    assert_y(host(Y.index_select(0, ri).index_select(1, ci)), ry)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("folded", [True, False], ids=["foldedP", "denseP"])
def test_tac_oproj_g128(folded):
    """TAC (32 blocks of 128) on 8 x 2048 tokens, then SGAT quantise, then the
    4096 -> 4096 GEMM."""
    run_site(synth.TAC_OPROJ, 0, synth.config_state(synth.TAC_OPROJ), folded=folded)


@pytest.mark.timeout(600)
def test_tac_oproj_identity_blocks_is_plain_sgat():
    """With identity blocks and zero bias the TAC + O-projection equals the same layer
    without TAC, bit for bit."""
    st = synth.config_state(synth.TAC_OPROJ)
    t = synth.site_tensors(synth.TAC_OPROJ, 0, st, tac_identity=True, with_W=False, with_P=False)
    Xd = dev(t.X)
    a = sq.sgat_quant_act(Xd, dev(st), None, t.dm, t.du, dev(t.tac_M), dev(t.tac_d), t.g)
    b = sq.sgat_quant_act(Xd, dev(st), None, t.dm, t.du)
    assert_bits(host(a[0]), host(b[0]), "Aq")
    assert_bits(host(a[1]), host(b[1]), "s_a")


SWEEP = [16, 32, 64, 256, 1024, 4096, 16384]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("M", SWEEP)
def test_denoise_sweep_token_counts(M):
    """Denoising-step sweep: each token count through every linear of the LLaDA set
    (folded P, the per-step GEMM path), at step t = 32, sampled rows vs the oracle."""
    st = synth.config_state(synth.LLADA_SWEEP, M=M, t=32)
    for si in range(4):
        run_site(synth.LLADA_SWEEP, si, st, folded=True)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("layout", ["t0", "t64", "all_masked", "none_masked", "alternating"])
def test_denoise_sweep_layouts(layout):
    """Step layouts (t = 0, all generation tokens masked; t = 64, none) and the edge
    layouts at 1024 tokens through the dense-P QKV and down linears."""
    M = 1024
    if layout in ("t0", "t64"):
        st = synth.config_state(synth.LLADA_SWEEP, M=M, t=int(layout[1:]))
    else:
        st = synth.state_edge(M, layout)
    for si in (0, 3):
        run_site(synth.LLADA_SWEEP, si, st, n_rows=16, n_cols=64)


def test_transform_beyond_2gib_of_activations():
    """A call whose X exceeds 2 GiB (65608 x 16384 fp16) runs as chunks of rows;
    sampled rows on both sides of the chunk edge match the oracle bit for bit and
    every other row (all zero on input) is zero."""
    M, K = 65408 + 200, 16384
    rng = np.random.default_rng(16384)
    st = (rng.random(M) < 0.5).astype(np.uint8)
    rows = np.unique(np.array([0, 1, 65407, 65408, 65409, M - 1] + list(rng.choice(M, 4, replace=False))))
    Xs = (rng.standard_normal((len(rows), K)) * 2.0).astype(np.float16)
    P = synth.orthogonal(K, synth.rng_for(605, K))
    dm, du = synth.default_band(K)
    say(f"transform beyond 2 GiB: M={M} K={K}")
    X = torch.zeros((M, K), dtype=torch.float16, device="cuda")
    X[torch.from_numpy(rows).cuda()] = dev(Xs)
    xp = sq.sgat_transform(X, dev(st), dev(P), dm, du)
    ref = O.transform(Xs, st[rows], P, dm, du, threads=THREADS)
    assert_bits(host(xp[torch.from_numpy(rows).cuda()]), ref, "x' sampled rows")
    others = torch.ones(M, dtype=torch.bool, device="cuda")
    others[torch.from_numpy(rows).cuda()] = False
    assert bool((xp[others] == 0).all())
