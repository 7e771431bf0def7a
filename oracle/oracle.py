"""CPU oracle for the STaR-Quant W4A4 hot path.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this module.  It shares no code with the HIP library.

Two layers:

* ``canonical``: numpy wrappers around ``sq_oracle.c`` (plain scalar C).  This
  is the definition the GPU results are compared with, bit for bit: the
  arithmetic order and rounding of every step is fixed there (see the C file's
  header for the readings of the points the paper leaves open).
* ``fp64`` / ``paper_literal``: independent formulations in numpy, used only to
  pin the canonical layer (Eq. 6, App. A closed forms, the paper's
  split-transform-quantise-scatter order of Eq. 7-13).
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Optional, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsq_oracle.so")

_lib = None
_lock = threading.Lock()

_p = ctypes.c_void_p
_i64 = ctypes.c_int64
_i32 = ctypes.c_int


def lib():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                from oracle.build import build as _build
                _build()
            L = ctypes.CDLL(LIB_PATH)
            L.sqo_h2f_array.argtypes = [_p, _p, _i64]
            L.sqo_f2h_array.argtypes = [_p, _p, _i64]
            L.sqo_tac.argtypes = [_p, _p, _p, _i64, _i32, _i32, _p]
            L.sqo_transform.argtypes = [_p, _p, _p, _i64, _i32, _i32, _i32, _p]
            L.sqo_quant_rows.argtypes = [_p, _i64, _i32, _p, _p, _p]
            L.sqo_unpack.argtypes = [_p, _i64, _i32, _p]
            L.sqo_quant_act.argtypes = [_p, _p, _p, _i64, _i32, _i32, _i32, _p, _p, _i32, _p, _p]
            L.sqo_prepare_weights.argtypes = [_p, _p, _i64, _i32, _p, _p]
            L.sqo_gemm.argtypes = [_p, _p, _p, _p, _i64, _i64, _i32, _p, _p]
            L.sqo_gemm.restype = _i32
            L.sqo_quant_rows_q8.argtypes = [_p, _i64, _i32, _p, _p]
            L.sqo_quant_act_q8.argtypes = [_p, _p, _p, _i64, _i32, _i32, _i32, _p, _p, _i32, _p, _p]
            L.sqo_prepare_weights_q8.argtypes = [_p, _p, _i64, _i32, _p, _p]
            L.sqo_gemm_q8.argtypes = [_p, _p, _p, _p, _i64, _i64, _i32, _p, _p]
            L.sqo_gemm_q8.restype = _i32
            _lib = L
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def _rows_parallel(fn, M: int, threads: int):
    """Run fn(r0, r1) over row ranges on `threads` threads (ctypes drops the GIL)."""
    threads = max(1, min(threads, M))
    if threads == 1:
        fn(0, M)
        return
    bounds = np.linspace(0, M, threads + 1).astype(int)
    ts = [threading.Thread(target=fn, args=(int(bounds[t]), int(bounds[t + 1])))
          for t in range(threads) if bounds[t + 1] > bounds[t]]
    for t in ts:
        t.start()
    for t in ts:
        t.join()


# ============================================================ canonical layer

def h2f(h: np.ndarray) -> np.ndarray:
    h = _c(h, np.uint16)
    out = np.empty(h.shape, np.float32)
    lib().sqo_h2f_array(_ptr(h), _ptr(out), h.size)
    return out


def f2h(f: np.ndarray) -> np.ndarray:
    f = _c(f, np.float32)
    out = np.empty(f.shape, np.uint16)
    lib().sqo_f2h_array(_ptr(f), _ptr(out), f.size)
    return out


def tac(Z: np.ndarray, Mb: np.ndarray, d: np.ndarray, g: int, threads: int = 1) -> np.ndarray:
    """Eq. 17 (App. C row-major form); fp16 in, fp16 out (as uint16 bits)."""
    Z = _c(Z.view(np.uint16) if Z.dtype == np.float16 else Z, np.uint16)
    Mb = _c(Mb.view(np.uint16) if Mb.dtype == np.float16 else Mb, np.uint16)
    d = _c(d.view(np.uint16) if d.dtype == np.float16 else d, np.uint16)
    M, C = Z.shape
    out = np.empty((M, C), np.uint16)

    def run(r0, r1):
        lib().sqo_tac(_ptr(Z[r0:]), _ptr(Mb), _ptr(d), r1 - r0, C, g, _ptr(out[r0:]))
    _rows_parallel(run, M, threads)
    return out.view(np.float16)


def transform(X: np.ndarray, state: Optional[np.ndarray], P: Optional[np.ndarray],
              dm: int, du: int, threads: int = 1) -> np.ndarray:
    """x' = x P G_s (Eq. 11), canonical fp32; P None = input already in the P basis."""
    X = _c(X.view(np.uint16), np.uint16)
    M, K = X.shape
    P = _c(P, np.float32)
    state = _c(state, np.uint8)
    out = np.empty((M, K), np.float32)

    def run(r0, r1):
        lib().sqo_transform(_ptr(X[r0:]), None if state is None else _ptr(state[r0:]), _ptr(P),
                            r1 - r0, K, dm, du, _ptr(out[r0:]))
    _rows_parallel(run, M, threads)
    return out


def quant_rows(x: np.ndarray):
    """Per-row symmetric int4 quantisation: (packed [M][K/2] uint8, scale [M] fp32, codes int8)."""
    x = _c(x, np.float32)
    M, K = x.shape
    packed = np.empty((M, K // 2), np.uint8)
    scale = np.empty(M, np.float32)
    codes = np.empty((M, K), np.int8)
    lib().sqo_quant_rows(_ptr(x), M, K, _ptr(packed), _ptr(scale), _ptr(codes))
    return packed, scale, codes


def unpack(packed: np.ndarray) -> np.ndarray:
    packed = _c(packed, np.uint8)
    M, Kh = packed.shape
    out = np.empty((M, 2 * Kh), np.int8)
    lib().sqo_unpack(_ptr(packed), M, 2 * Kh, _ptr(out))
    return out


def quant_act(X, state, P, dm: int, du: int, tac_M=None, tac_d=None, g: int = 0,
              threads: int = 1):
    """Activation side of one SGAT linear: [TAC] -> x P G_s -> Q_a.  Returns (Aq, s_a)."""
    X = _c(X.view(np.uint16), np.uint16)
    M, K = X.shape
    P = _c(P, np.float32)
    state = _c(state, np.uint8)
    tM = None if tac_M is None else _c(tac_M.view(np.uint16), np.uint16)
    td = None if tac_d is None else _c(tac_d.view(np.uint16), np.uint16)
    Aq = np.empty((M, K // 2), np.uint8)
    s_a = np.empty(M, np.float32)

    def run(r0, r1):
        lib().sqo_quant_act(_ptr(X[r0:]), None if state is None else _ptr(state[r0:]), _ptr(P),
                            r1 - r0, K, dm, du, _ptr(tM), _ptr(td), g,
                            _ptr(Aq[r0:]), _ptr(s_a[r0:]))
    _rows_parallel(run, M, threads)
    return Aq, s_a


def prepare_weights(W, P, threads: int = 1):
    """W~ = Q_w(P^T W^T), stored as [N][K/2] codes of the rows of W P, and s_w [N]."""
    W = _c(W.view(np.uint16), np.uint16)
    N, K = W.shape
    P = _c(P, np.float32)
    Wq = np.empty((N, K // 2), np.uint8)
    s_w = np.empty(N, np.float32)

    def run(r0, r1):
        lib().sqo_prepare_weights(_ptr(W[r0:]), _ptr(P), r1 - r0, K, _ptr(Wq[r0:]), _ptr(s_w[r0:]))
    _rows_parallel(run, N, threads)
    return Wq, s_w


def gemm(Aq, s_a, Wq, s_w, threads: int = 1):
    """Eq. 13 / Eq. 5: (Y fp16 [M][N], acc int32 [M][N])."""
    Aq = _c(Aq, np.uint8)
    Wq = _c(Wq, np.uint8)
    s_a = _c(s_a, np.float32)
    s_w = _c(s_w, np.float32)
    M, Kh = Aq.shape
    N = Wq.shape[0]
    Y = np.empty((M, N), np.uint16)
    acc = np.empty((M, N), np.int32)
    bad = [0]

    def run(r0, r1):
        bad[0] |= lib().sqo_gemm(_ptr(Aq[r0:]), _ptr(s_a[r0:]), _ptr(Wq), _ptr(s_w),
                                 r1 - r0, N, 2 * Kh, _ptr(Y[r0:]), _ptr(acc[r0:]))
    _rows_parallel(run, M, threads)
    if bad[0]:
        raise OverflowError("int32 accumulator overflow")
    return Y.view(np.float16), acc


def sgat_linear(X, state, P, W, dm, du, tac_M=None, tac_d=None, g=0, threads: int = 1):
    """The whole quantised SGAT linear: returns dict with Aq, s_a, Wq, s_w, Y, acc."""
    Aq, s_a = quant_act(X, state, P, dm, du, tac_M, tac_d, g, threads)
    Wq, s_w = prepare_weights(W, P, threads)
    Y, acc = gemm(Aq, s_a, Wq, s_w, threads)
    return dict(Aq=Aq, s_a=s_a, Wq=Wq, s_w=s_w, Y=Y, acc=acc)


# ------------------------------------------------------------ W8A8 (App. D)

def quant_rows_q8(x: np.ndarray):
    """Per-row symmetric 8-bit quantisation: (codes int8 [M][K], scale [M] fp32)."""
    x = _c(x, np.float32)
    M, K = x.shape
    codes = np.empty((M, K), np.int8)
    scale = np.empty(M, np.float32)
    lib().sqo_quant_rows_q8(_ptr(x), M, K, _ptr(codes), _ptr(scale))
    return codes, scale


def quant_act_q8(X, state, P, dm: int, du: int, tac_M=None, tac_d=None, g: int = 0, threads: int = 1):
    """W8A8 activation side: [TAC] -> x P G_s -> 8-bit per token.  Returns (Aq int8, s_a)."""
    X = _c(X.view(np.uint16), np.uint16)
    M, K = X.shape
    P = _c(P, np.float32)
    state = _c(state, np.uint8)
    tM = None if tac_M is None else _c(tac_M.view(np.uint16), np.uint16)
    td = None if tac_d is None else _c(tac_d.view(np.uint16), np.uint16)
    Aq = np.empty((M, K), np.int8)
    s_a = np.empty(M, np.float32)

    def run(r0, r1):
        lib().sqo_quant_act_q8(_ptr(X[r0:]), None if state is None else _ptr(state[r0:]), _ptr(P),
                               r1 - r0, K, dm, du, _ptr(tM), _ptr(td), g, _ptr(Aq[r0:]), _ptr(s_a[r0:]))
    _rows_parallel(run, M, threads)
    return Aq, s_a


def prepare_weights_q8(W, P, threads: int = 1):
    W = _c(W.view(np.uint16), np.uint16)
    N, K = W.shape
    P = _c(P, np.float32)
    Wq = np.empty((N, K), np.int8)
    s_w = np.empty(N, np.float32)

    def run(r0, r1):
        lib().sqo_prepare_weights_q8(_ptr(W[r0:]), _ptr(P), r1 - r0, K, _ptr(Wq[r0:]), _ptr(s_w[r0:]))
    _rows_parallel(run, N, threads)
    return Wq, s_w


def gemm_q8(Aq, s_a, Wq, s_w, threads: int = 1):
    Aq = _c(Aq, np.int8)
    Wq = _c(Wq, np.int8)
    s_a = _c(s_a, np.float32)
    s_w = _c(s_w, np.float32)
    M, K = Aq.shape
    N = Wq.shape[0]
    Y = np.empty((M, N), np.uint16)
    acc = np.empty((M, N), np.int32)
    bad = [0]

    def run(r0, r1):
        bad[0] |= lib().sqo_gemm_q8(_ptr(Aq[r0:]), _ptr(s_a[r0:]), _ptr(Wq), _ptr(s_w), r1 - r0, N, K,
                                    _ptr(Y[r0:]), _ptr(acc[r0:]))
    _rows_parallel(run, M, threads)
    if bad[0]:
        raise OverflowError("int32 accumulator overflow")
    return Y.view(np.float16), acc


# ============================================================ fp64 / paper-literal layer

def gate_vector(K: int, dm: int, du: int, masked: bool) -> np.ndarray:
    """Diagonal of G_m or G_u (Eq. 9) over columns ordered [U_sh, U_m, U_u] (Eq. 8)."""
    dsh = K - dm - du
    g = np.zeros(K)
    g[:dsh] = 1.0
    if masked:
        g[dsh:dsh + dm] = 1.0
    else:
        g[dsh + dm:] = 1.0
    return g


def fp64_linear(X, W) -> np.ndarray:
    """Y = X W^T (Eq. 1) in fp64."""
    return X.astype(np.float64) @ W.astype(np.float64).T


def fp64_sgat_noquant(X, state, P, W, dm, du) -> np.ndarray:
    """Phi_s(X^s) W~ with quantisers disabled (App. A), fp64, row by row state."""
    X64 = X.astype(np.float64)
    P64 = P.astype(np.float64)
    Wt = P64.T @ W.astype(np.float64).T                  # P^T W^T (Eq. 12, no Q_w)
    K = X.shape[1]
    out = np.empty((X.shape[0], W.shape[0]))
    for s in (0, 1):
        rows = np.nonzero(state == s)[0]
        if len(rows):
            G = np.diag(gate_vector(K, dm, du, bool(s)))
            out[rows] = X64[rows] @ P64 @ G @ Wt
    return out


def fp64_leakage(X, state, P, W, dm, du) -> np.ndarray:
    """Delta_s = X^s P G_s^perp P^T W^T (App. A)."""
    X64 = X.astype(np.float64)
    P64 = P.astype(np.float64)
    K = X.shape[1]
    out = np.empty((X.shape[0], W.shape[0]))
    for s in (0, 1):
        rows = np.nonzero(state == s)[0]
        if len(rows):
            Gp = np.diag(1.0 - gate_vector(K, dm, du, bool(s)))
            out[rows] = X64[rows] @ P64 @ Gp @ P64.T @ W.astype(np.float64).T
    return out


def nearest_code(v: np.ndarray, lo: int = -8, hi: int = 7) -> np.ndarray:
    """Brute-force search of the integer code in [lo, hi] nearest to v, ties to even."""
    cands = np.arange(lo, hi + 1, dtype=np.float64)
    v = np.asarray(v, np.float64)[..., None]
    dist = np.abs(v - cands)
    best = dist.min(axis=-1, keepdims=True)
    tie = dist == best
    # among equally near candidates prefer the even one
    pref = tie & (np.mod(cands, 2) == 0)
    pick = np.where(pref.any(axis=-1, keepdims=True), pref, tie)
    return cands[np.argmax(pick, axis=-1)].astype(np.int8)


def paper_literal(X, state, P, W, dm, du):
    """Eq. 7-13 taken literally, in fp64: split tokens by state, transform each group
    with its explicit gated basis P_s = P G_s, quantise per token (s = absmax/7, nearest
    code by search), multiply with the shared Q_w(P^T W^T) in int64, dequantise, and
    scatter back to token order.  Also returns each activation element's distance to
    the nearest rounding midpoint so callers can set aside near-ties."""
    X64 = X.astype(np.float64)
    P64 = P.astype(np.float64)
    K = X.shape[1]
    M, N = X.shape[0], W.shape[0]
    # shared weight side, Eq. 12: rows of W P, per-output-channel quantiser
    Wp = W.astype(np.float64) @ P64
    s_w = np.abs(Wp).max(axis=1) / 7.0
    qw = nearest_code(np.where(s_w[:, None] > 0, Wp / np.where(s_w > 0, s_w, 1)[:, None], 0))
    codes = np.zeros((M, K), np.int8)
    s_a = np.zeros(M)
    margin = np.full((M, K), np.inf)
    Y = np.zeros((M, N))
    for s in (1, 0):                                       # m, u
        idx = np.nonzero(state == s)[0]                    # I_s (Eq. 7)
        if not len(idx):
            continue
        Ps = P64 @ np.diag(gate_vector(K, dm, du, bool(s)))   # Eq. 10
        Phi = X64[idx] @ Ps                                 # Eq. 11
        ss = np.abs(Phi).max(axis=1) / 7.0
        ratio = Phi / np.where(ss > 0, ss, 1)[:, None]
        q = nearest_code(np.where(ss[:, None] > 0, ratio, 0))
        acc = q.astype(np.int64) @ qw.astype(np.int64).T
        Ys = acc * ss[:, None] * s_w[None, :]               # Eq. 13, dequantised
        codes[idx] = q                                      # scatter back
        s_a[idx] = ss
        margin[idx] = np.abs(np.abs(ratio - np.floor(ratio)) - 0.5)
        Y[idx] = Ys
    return dict(codes=codes, s_a=s_a, qw=qw, s_w=s_w, Y=Y, margin=margin)
