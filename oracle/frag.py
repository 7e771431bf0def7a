"""Reference for fragment-ordered int4 weights.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this module.  It shares no code with the HIP library.

The W4A4 GEMM of Eq. 5 / Eq. 13 does not depend on where the weight bytes are
kept.  The weights W~ are fixed once prepared (Eq. 12), so they may be stored
in the order the GEMM reads them.  This module defines that order:

* the packed int4 weights Wq [N][K/2] (two codes per byte) are padded with zero
  rows to a multiple of 16 rows and with zero bytes to a multiple of 64 bytes
  (128 codes) per row;
* block (g, t) holds rows 16 g .. 16 g + 15 and bytes 64 t .. 64 t + 63 of
  those rows, 1024 bytes, at offset (t G + g) 1024 with G = ceil(N / 16) (the
  blocks of one k step side by side);
* inside a block, unit u = 16 j + r (16 bytes at 16 u) holds bytes
  64 t + 16 j .. 64 t + 16 j + 15 of row 16 g + r (j = 0..3, r = 0..15).

``gemm`` is then by definition the int4 GEMM of the weights this layout holds.

The W8A8 variant (App. D) keeps one signed byte per code, rows of K bytes.  Its
layout is the one above applied to those bytes, a row of K int8 codes being
stored exactly as a packed row of 2 K int4 codes (so a k step holds 64 int8
codes); ``gemm_q8`` is the int8 GEMM of the weights it holds.
"""
from __future__ import annotations

import numpy as np

from . import oracle as O

ROWS = 16          # rows per group
STEP = 64          # bytes of a row per k step (128 codes)
UNIT = 16          # bytes per unit


def _dims(N: int, K: int):
    assert K % 64 == 0 and K > 0 and N >= 0
    return (N + ROWS - 1) // ROWS, (K // 2 + STEP - 1) // STEP


def frag_bytes(N: int, K: int) -> int:
    G, T = _dims(N, K)
    return G * T * ROWS * STEP


def to_frag(Wq: np.ndarray, K: int) -> np.ndarray:
    """Wq [N][K/2] (any dtype) -> the fragment order, shape [T][G][1024]."""
    Wq = np.asarray(Wq)
    N = Wq.shape[0]
    assert Wq.shape[1] == K // 2
    G, T = _dims(N, K)
    padded = np.zeros((G * ROWS, T * STEP), Wq.dtype)
    padded[:N, :K // 2] = Wq
    # [g][r][t][j][b] -> [t][g][j][r][b]: block (g, t) at t G + g, inside it unit 16 j + r
    units = padded.reshape(G, ROWS, T, STEP // UNIT, UNIT).transpose(2, 0, 3, 1, 4)
    return np.ascontiguousarray(units).reshape(T, G, ROWS * STEP)


def from_frag(Wf: np.ndarray, N: int, K: int) -> np.ndarray:
    """The inverse of to_frag; raises if a padding byte is not zero."""
    G, T = _dims(N, K)
    Wf = np.asarray(Wf)
    assert Wf.size == G * T * ROWS * STEP
    units = Wf.reshape(T, G, STEP // UNIT, ROWS, UNIT).transpose(1, 3, 0, 2, 4)
    padded = np.ascontiguousarray(units).reshape(G * ROWS, T * STEP)
    if padded[N:].any() or padded[:, K // 2:].any():
        raise ValueError("padding of fragment-ordered weights is not zero")
    return np.ascontiguousarray(padded[:N, :K // 2])


def gemm(Aq, s_a, Wf, s_w, N: int, K: int, threads: int = 1):
    """Eq. 13 / Eq. 5 with fragment-ordered weights: the int4 GEMM of the
    weights they hold."""
    return O.gemm(Aq, s_a, from_frag(Wf, N, K).astype(np.uint8), s_w, threads=threads)


def to_frag_q8(Wq: np.ndarray, K: int) -> np.ndarray:
    """int8 weights [N][K] -> the fragment order of their bytes, [ceil(K/64)][G][1024] uint8."""
    Wq = np.ascontiguousarray(Wq, dtype=np.int8)
    assert Wq.shape[1] == K
    return to_frag(Wq.view(np.uint8), 2 * K)


def gemm_q8(Aq, s_a, Wf, s_w, N: int, K: int, threads: int = 1):
    """App. D's int8 GEMM with fragment-ordered weights: the int8 GEMM of the
    weights they hold."""
    return O.gemm_q8(Aq, s_a, from_frag(Wf, N, 2 * K).view(np.int8), s_w, threads=threads)
