"""Reference for int4 codes carried on the FP6 matrix cores.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this module.  It shares no code with the HIP library.

The W4A4 GEMM of Eq. 5 / Eq. 13 multiplies int4 codes.  The FP6 path stores the
same codes as 6-bit floats in the e3m2 format (OCP Microscaling Formats v1.0,
FP6 E3M2: sign bit, 3 exponent bits with bias 3, 2 mantissa bits, subnormals
at exponent field 0, no infinities or NaNs), in which every integer -8..7 is
exact, and multiplies them on the matrix cores.  This module defines:

* ``e3m2_value``: the value of a 6-bit pattern, from the format definition;
* ``encode``: the pattern of an integer code, found by searching all 64 patterns
  (no formula shared with the GPU encoder);
* ``to_fp6`` / ``from_fp6``: the operand layout.  Per row, K codes padded with
  zero codes to whole blocks of 128; block b takes 96 bytes at offset 96 b;
  chunk c of the block (codes 128 b + 32 c .. 128 b + 32 c + 31) is the 192-bit
  little-endian string with code j in bits 6 j .. 6 j + 5, whose bytes 0..15 are
  stored at 96 b + 16 c and bytes 16..23 at 96 b + 64 + 8 c;
* ``gemm``: the product on such operands, which by definition is the int4 GEMM
  of the decoded codes (Eq. 5 / Eq. 13 epilogue unchanged).
"""
from __future__ import annotations

import numpy as np

from . import oracle as O

BLOCK = 128            # codes per block
BLOCK_BYTES = 96       # 128 x 6 bits
CHUNK = 32             # codes per chunk (one MFMA lane group's k range)


def e3m2_value(bits: int) -> float:
    """Value of a 6-bit e3m2 pattern: (-1)^s 2^(e-3) (1 + m/4), or (-1)^s 2^-2 (m/4) for e = 0."""
    bits = int(bits)
    assert 0 <= bits < 64
    s = (bits >> 5) & 1
    e = (bits >> 2) & 7
    m = bits & 3
    mag = (m / 4.0) * 2.0 ** (1 - 3) if e == 0 else (1.0 + m / 4.0) * 2.0 ** (e - 3)
    return -mag if s else mag


def encode(q: int) -> int:
    """The 6-bit pattern whose value is exactly the integer q (positive zero for 0)."""
    hits = [b for b in range(64) if e3m2_value(b) == q and not (q == 0 and b >> 5)]
    if len(hits) != 1:
        raise ValueError(f"{q} is not exactly representable once in e3m2")
    return hits[0]


_ENC = {q: encode(q) for q in range(-8, 8)}
_DEC = {b: e3m2_value(b) for b in range(64)}


def row_bytes(K: int) -> int:
    return BLOCK_BYTES * ((K + BLOCK - 1) // BLOCK)


def to_fp6(codes: np.ndarray) -> np.ndarray:
    """int codes [R][K] in -8..7 -> operand bytes [R][row_bytes(K)]."""
    codes = np.asarray(codes)
    R, K = codes.shape
    nblk = (K + BLOCK - 1) // BLOCK
    out = np.zeros((R, nblk * BLOCK_BYTES), np.uint8)
    for r in range(R):
        for b in range(nblk):
            for c in range(4):
                k0 = b * BLOCK + c * CHUNK
                word = 0
                for j in range(CHUNK):
                    q = int(codes[r, k0 + j]) if k0 + j < K else 0
                    word |= _ENC[q] << (6 * j)
                frag = word.to_bytes(24, "little")
                out[r, b * 96 + 16 * c: b * 96 + 16 * c + 16] = np.frombuffer(frag[:16], np.uint8)
                out[r, b * 96 + 64 + 8 * c: b * 96 + 64 + 8 * c + 8] = np.frombuffer(frag[16:], np.uint8)
    return out


def from_fp6(data: np.ndarray, K: int) -> np.ndarray:
    """Operand bytes [R][row_bytes(K)] -> values [R][K] (float64; integers for valid data)."""
    data = np.asarray(data, np.uint8)
    R = data.shape[0]
    nblk = (K + BLOCK - 1) // BLOCK
    assert data.shape[1] == nblk * BLOCK_BYTES
    out = np.zeros((R, K), np.float64)
    for r in range(R):
        for b in range(nblk):
            for c in range(4):
                frag = bytes(data[r, b * 96 + 16 * c: b * 96 + 16 * c + 16]) + \
                    bytes(data[r, b * 96 + 64 + 8 * c: b * 96 + 64 + 8 * c + 8])
                word = int.from_bytes(frag, "little")
                for j in range(CHUNK):
                    k = b * BLOCK + c * CHUNK + j
                    if k < K:
                        out[r, k] = _DEC[(word >> (6 * j)) & 63]
    return out


def pack_int4(codes: np.ndarray) -> np.ndarray:
    """int codes [R][K] -> the packed int4 layout of the W4A4 path (two's complement
    nibbles, code 2t in the low nibble of byte t)."""
    c = (np.asarray(codes).astype(np.int64) & 15).astype(np.uint8)
    return (c[:, 0::2] | (c[:, 1::2] << 4)).astype(np.uint8)


def codes_to_fp6(packed: np.ndarray) -> np.ndarray:
    """The conversion the library offers: packed int4 [R][K/2] -> operand bytes."""
    return to_fp6(O.unpack(packed))


def gemm(A6, s_a, W6, s_w, K: int, threads: int = 1):
    """Eq. 13 / Eq. 5 on FP6 operands: the canonical int4 GEMM of the decoded codes."""
    qa = from_fp6(A6, K)
    qw = from_fp6(W6, K)
    for q in (qa, qw):
        if not (np.all(q == np.round(q)) and q.min() >= -8 and q.max() <= 7):
            raise ValueError("operands do not hold int4 codes")
    return O.gemm(pack_int4(qa.astype(np.int64)), s_a, pack_int4(qw.astype(np.int64)), s_w, threads=threads)
