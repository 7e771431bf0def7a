"""w4a4_gemm_frag_noalloc, the GEMM entry point that allocates nothing: called
through the C ABI and compared bit for bit with w4a4_gemm_frag (caller-given
workspace) and with the oracle, on two calls in a row, the second smaller, so
that the library's scratch array is reused with a smaller shape."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2606_04945_amd as sq
from paper_2606_04945_amd import _lib as L
from oracle import oracle as O
from gpu_util import assert_bits, assert_y, dev, host, say

pytestmark = pytest.mark.gpu


def _case(seed, M, N, K):
    rng = np.random.default_rng(seed)
    Aq = rng.integers(0, 256, (M, K // 2), dtype=np.uint8)
    Wq = rng.integers(0, 256, (N, K // 2), dtype=np.uint8)
    s_a = (rng.random(M) * 0.5 + 0.25).astype(np.float32)
    s_w = (rng.random(N) * 0.01 + 0.001).astype(np.float32)
    return Aq, s_a, Wq, s_w


def _noalloc(Aq, s_a, Wf, s_w, M, N, K, stream=None):
    Y = torch.empty((M, N), dtype=torch.float16, device="cuda")
    acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream() if stream is None else stream
    rc = L.lib().w4a4_gemm_frag_noalloc(Aq.data_ptr(), s_a.data_ptr(), Wf.data_ptr(), s_w.data_ptr(), M, N, K,
                                        Y.data_ptr(), acc.data_ptr(), ctypes.c_void_p(s.cuda_stream))
    L.check(rc)
    return Y, acc


# (M, N, K): the first two split K across workgroups (the scratch holds the
# partial sums), the second smaller than the first; then a short-M and a tiled
# shape that need no scratch
SHAPES = [(100, 520, 4096), (70, 264, 2048), (16, 4096, 4096), (300, 1024, 512)]


def test_noalloc_matches_workspace_entry_point():
    assert sq.gemm_workspace_bytes(*SHAPES[0]) > sq.gemm_workspace_bytes(*SHAPES[1]) > 0
    assert sq.gemm_workspace_bytes(*SHAPES[0]) <= 16 << 20
    for i, (M, N, K) in enumerate(SHAPES):
        say(f"noalloc: call {i}, M={M} N={N} K={K}, ws={sq.gemm_workspace_bytes(M, N, K)}")
        Aq, s_a, Wq, s_w = _case(100 + i, M, N, K)
        dA, dsa, dW, dsw = dev(Aq), dev(s_a), dev(Wq), dev(s_w)
        Wf = sq.weights_to_frag(dW)
        Y0, acc0 = sq.w4a4_gemm_frag(dA, dsa, Wf, dsw, want_acc=True)
        Y1, acc1 = _noalloc(dA, dsa, Wf, dsw, M, N, K)
        ref_Y, ref_acc = O.gemm(Aq, s_a, Wq, s_w, threads=8)
        assert_bits(host(acc1), host(acc0), f"acc vs w4a4_gemm_frag, call {i}")
        assert_bits(host(Y1), host(Y0), f"Y vs w4a4_gemm_frag, call {i}")
        assert_bits(host(acc1), ref_acc, f"acc vs oracle, call {i}")
        assert_y(host(Y1), ref_Y, f"Y vs oracle, call {i}")


def test_noalloc_on_a_side_stream():
    M, N, K = SHAPES[0]
    Aq, s_a, Wq, s_w = _case(7, M, N, K)
    dA, dsa, dW, dsw = dev(Aq), dev(s_a), dev(Wq), dev(s_w)
    Wf = sq.weights_to_frag(dW)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        Y1, acc1 = _noalloc(dA, dsa, Wf, dsw, M, N, K, stream=s)
    s.synchronize()
    _, ref_acc = O.gemm(Aq, s_a, Wq, s_w, threads=8)
    assert_bits(host(acc1), ref_acc, "acc on a side stream")


def test_noalloc_empty_is_noop():
    assert L.lib().w4a4_gemm_frag_noalloc(None, None, None, None, 0, 64, 128, None, None, None) == L.SQ_OK
