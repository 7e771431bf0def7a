"""Linear-layer steps captured in a HIP graph and replayed: every replay gives
the eager call's bytes (codes, scales, accumulators and fp16 outputs).

Each case captures the calls once, replays the graph three times with eager
work on the same buffers in between (the outputs are overwritten by an eager
call on other inputs before every replay), and compares each replay with the
eager result, so a graph node that reads stale state or writes past its
buffers would show.  Covered: the folded quantiser with TAC fused, the
fragment-order GEMM on its short-M, k-group and K-split plans (the split plan
with its reduction pass), the dense transform with TAC ahead of it, and the
8-bit GEMM."""
import numpy as np
import pytest
import torch

import paper_2606_04945_amd as sq
import synth
from gpu_util import assert_bits, dev, host, say

pytestmark = pytest.mark.gpu
REPLAYS = 3


def capture(fn):
    fn()                                    # eager warm-up: one-time set-up stays outside the graph
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            fn()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    return g


def check_replays(g, outs, want, scramble):
    for r in range(REPLAYS):
        scramble()                          # eager work that overwrites every output
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, t in outs.items():
            assert_bits(host(t), want[name], f"{name}, replay {r}")


@pytest.mark.parametrize("M,K,N", [(64, 1024, 2048), (300, 4096, 1032), (1024, 3584, 18944)])
def test_folded_step_graph(M, K, N):
    """TAC-fused quantiser + fragment-order GEMM: the short-M four-tile plan at
    64 tokens, the K-split plan and its reduction pass at 300 tokens
    (300 x 1032 x 4096: four splits), the tiled plan at 1024 tokens."""
    c = synth.small_case(40 + M, M, K, N, g=16)
    dm, du = synth.default_band(K)
    X, st = dev(c["X"]), dev(c["state"])
    tM, td = dev(c["tac_M"]), dev(c["tac_d"])
    Wq, s_w = sq.sgat_prepare_weights(dev(c["W"]), None)
    Wf = sq.weights_to_frag(Wq)
    Aq = torch.empty((M, K // 2), dtype=torch.uint8, device="cuda")
    s_a = torch.empty(M, dtype=torch.float32, device="cuda")
    Y = torch.empty((M, N), dtype=torch.float16, device="cuda")
    acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
    qws = torch.empty(max(sq.quant_act_workspace_bytes(M, K, False, True), 1), dtype=torch.uint8, device="cuda")
    gws = torch.empty(max(sq.gemm_workspace_bytes(M, N, K), 1), dtype=torch.uint8, device="cuda")
    say(f"graph folded M={M} K={K} N={N}")

    def step():
        sq.sgat_quant_act(X, st, None, dm, du, tM, td, 16, Aq=Aq, s_a=s_a, ws=qws)
        sq.w4a4_gemm_frag(Aq, s_a, Wf, s_w, Y=Y, acc=acc, want_acc=True, ws=gws)
    step()
    want = {"Aq": host(Aq), "s_a": host(s_a), "Y": host(Y), "acc": host(acc)}
    g = capture(step)
    X2 = X.flip(0).contiguous()

    def scramble():
        sq.sgat_quant_act(X2, st, None, dm, du, tM, td, 16, Aq=Aq, s_a=s_a, ws=qws)
        sq.w4a4_gemm_frag(Aq, s_a, Wf, s_w, Y=Y, acc=acc, want_acc=True, ws=gws)
    check_replays(g, {"Aq": Aq, "s_a": s_a, "Y": Y, "acc": acc}, want, scramble)


@pytest.mark.parametrize("bits", [4, 8])
def test_deep_k_gemm_graph(bits):
    """The k-group plan (1024 x 3584 x 18944: 224 tiles of 128 x 128)."""
    M, N, K = 1024, 3584, 18944
    rng = np.random.default_rng(bits)
    if bits == 4:
        Aq = dev(rng.integers(0, 256, (M, K // 2), dtype=np.uint8))
        Wq = dev(rng.integers(0, 256, (N, K // 2), dtype=np.uint8))
    else:
        Aq = dev(rng.integers(-128, 128, (M, K), dtype=np.int8))
        Wq = dev(rng.integers(-128, 128, (N, K), dtype=np.int8))
    s_a = dev(rng.uniform(0.01, 1, M).astype(np.float32))
    s_w = dev(rng.uniform(1e-5, 1e-3, N).astype(np.float32))
    Wf = sq.weights_to_frag(Wq)
    Y = torch.empty((M, N), dtype=torch.float16, device="cuda")
    acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
    gws = torch.empty(max(sq.gemm_workspace_bytes(M, N, K, bits), 1), dtype=torch.uint8, device="cuda")
    say(f"graph deep-K gemm bits={bits}")

    def step():
        sq.w4a4_gemm_frag(Aq, s_a, Wf, s_w, Y=Y, acc=acc, want_acc=True, ws=gws, bits=bits)
    step()
    want = {"Y": host(Y), "acc": host(acc)}
    # and equal to the row-major GEMM on the same codes
    Y2, acc2 = sq.w4a4_gemm(Aq, s_a, Wq, s_w, want_acc=True, bits=bits)
    assert_bits(want["acc"], host(acc2), "acc vs row-major")
    g = capture(step)
    s_a2 = s_a.flip(0).contiguous()

    def scramble():
        sq.w4a4_gemm_frag(Aq, s_a2, Wf, s_w, Y=Y, acc=acc, want_acc=True, ws=gws, bits=bits)
    check_replays(g, {"Y": Y, "acc": acc}, want, scramble)


def test_dense_step_graph():
    """TAC (its own pass ahead of the dense transform), transform + gate +
    quantiser with a dense P, and the row-major GEMM."""
    M, K, N = 128, 512, 256
    c = synth.small_case(77, M, K, N, g=16)
    dm, du = synth.default_band(K)
    X, st, P = dev(c["X"]), dev(c["state"]), dev(c["P"])
    tM, td = dev(c["tac_M"]), dev(c["tac_d"])
    Wq, s_w = sq.sgat_prepare_weights(dev(c["W"]), P)
    Aq = torch.empty((M, K // 2), dtype=torch.uint8, device="cuda")
    s_a = torch.empty(M, dtype=torch.float32, device="cuda")
    Y = torch.empty((M, N), dtype=torch.float16, device="cuda")
    qws = torch.empty(max(sq.quant_act_workspace_bytes(M, K, True, True), 1), dtype=torch.uint8, device="cuda")
    gws = torch.empty(max(sq.gemm_workspace_bytes(M, N, K), 1), dtype=torch.uint8, device="cuda")
    say("graph dense step")

    def step():
        sq.sgat_quant_act(X, st, P, dm, du, tM, td, 16, Aq=Aq, s_a=s_a, ws=qws)
        sq.w4a4_gemm(Aq, s_a, Wq, s_w, Y=Y, ws=gws)
    step()
    want = {"Aq": host(Aq), "s_a": host(s_a), "Y": host(Y)}
    g = capture(step)
    st2 = (1 - st).contiguous()

    def scramble():
        sq.sgat_quant_act(X, st2, P, dm, du, tM, td, 16, Aq=Aq, s_a=s_a, ws=qws)
        sq.w4a4_gemm(Aq, s_a, Wq, s_w, Y=Y, ws=gws)
    check_replays(g, {"Aq": Aq, "s_a": s_a, "Y": Y}, want, scramble)
