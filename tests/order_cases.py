"""Hand-built inputs on which the order conventions of the fixed arithmetic
change the result, shared by the oracle pins (CPU) and the kernel checks (GPU).

Each case states its inputs, the value the convention gives, and the value a
plausible other convention would give, worked out by hand below.  The tests
re-derive both with exact rational arithmetic (fractions.Fraction and an
explicit round-to-nearest-even), independently of the oracle's C code.

T3, the transform's k chunks of 256 (Eq. 11 read with a fixed order):
  x = 512 ones; column 0 of P holds 2^24 at k = 0 and 1.0 at k = 256..511;
  column 1 holds 2^24 at k = 0 and 1.0 at k = 128..255; all else 0.
  * Chunks of 256: column 0 = 2^24 + (256 ones summed from +0 = 256) =
    16777472; column 1: every 1.0 is added to 2^24 inside chunk 0, and
    2^24 + 1 is a tie between 2^24 and 2^24 + 2 that rounds to the even
    2^24, so column 1 = 16777216.
  * One flat chain would give column 0 = 16777216 (each 1.0 lost the same
    way); chunks of 128 would give column 1 = 2^24 + 128 = 16777344.

R2, the TAC bias added last (Eq. 17 read with a fixed order), g = 2:
  z = (64, 2^-6), M_0 row 0 = (32, 2^-7), d_0 = -1023.5 (all fp16-exact).
  * Bias last: 32 * 64 = 2048, then 2048 + 2^-13 is a tie at fp32 spacing
    2^-12 that rounds to the even 2048; 2048 - 1023.5 = 1024.5 exactly, a
    tie between the fp16 values 1024 and 1025 that rounds to the even 1024.
  * Bias first: -1023.5 + 2048 = 1024.5, then + 2^-13 = 1024.5 + 2^-13
    (exact: fp32 spacing at 1024 is 2^-13), above the tie: fp16 1025.

G1, the dequantisation order Y = fp16((float(acc) * s_a) * s_w) (Eq. 13):
  acc = 3, s_a = 0x3EAABFFE (0.33349603...), s_w = 0x3F800002 (1 + 2^-22).
  * (acc * s_a) * s_w rounds to exactly 1 + 2^-11, the midpoint between the
    fp16 values 1 and 1 + 2^-10, which rounds to the even 1.0.
  * acc * (s_a * s_w) rounds to 1 + 2^-11 + 2^-23, above the midpoint: fp16
    1 + 2^-10.
"""
import numpy as np

# ---- T3
T3_K = 512
T3_COL0, T3_COL1 = 16777472.0, 16777216.0          # chunks of 256
T3_FLAT_COL0, T3_C128_COL1 = 16777216.0, 16777344.0  # the other orders


def t3_inputs():
    X = np.ones((1, T3_K), np.float16)
    P = np.zeros((T3_K, T3_K), np.float32)
    P[0, 0] = 2.0 ** 24
    P[256:, 0] = 1.0
    P[0, 1] = 2.0 ** 24
    P[128:256, 1] = 1.0
    return X, P


# ---- R2
R2_C, R2_G = 64, 2
R2_OUT0 = 1024.0             # bias last
R2_BIAS_FIRST_OUT0 = 1025.0  # bias first


def r2_inputs():
    Z = np.zeros((1, R2_C), np.float16)
    Z[0, 0], Z[0, 1] = 64.0, 2.0 ** -6
    Mb = np.zeros((R2_C // R2_G, R2_G, R2_G), np.float16)
    Mb[:, 0, 0] = 1.0
    Mb[:, 1, 1] = 1.0
    Mb[0, 0, 0], Mb[0, 0, 1] = 32.0, 2.0 ** -7
    d = np.zeros(R2_C, np.float16)
    d[0] = -1023.5
    return Z, Mb, d


# ---- G1
G1_ACC = 3
G1_SA_BITS, G1_SW_BITS = 0x3EAABFFE, 0x3F800002
G1_Y = 1.0                       # (acc * s_a) * s_w
G1_OTHER_Y = 1.0 + 2.0 ** -10    # acc * (s_a * s_w)


def g1_inputs(K=64, N=8):
    """Codes whose dot product is 3 in row 0 / column 0, scales as above."""
    qa = np.zeros((1, K), np.int64)
    qw = np.zeros((N, K), np.int64)
    qa[0, :3] = 1
    qw[0, :3] = 1
    pack = lambda q: ((q[:, 0::2] & 15) | ((q[:, 1::2] & 15) << 4)).astype(np.uint8)   # noqa: E731
    s_a = np.array([G1_SA_BITS], np.uint32).view(np.float32)
    s_w = np.full(N, G1_SW_BITS, np.uint32).view(np.float32)
    return pack(qa), s_a, pack(qw), s_w


# ---- exact re-derivation (rationals + round to nearest even)

def rne(x, mant_bits, min_exp):
    """Round a Fraction to the nearest number with `mant_bits` bits after the
    leading one (ties to even), normals only down to 2^min_exp; returns a
    Fraction."""
    from fractions import Fraction
    if x == 0:
        return Fraction(0)
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = 0
    while a >= 2:
        a /= 2
        e += 1
    while a < 1:
        a *= 2
        e -= 1
    e = max(e, min_exp)
    q = abs(x) / Fraction(2) ** (e - mant_bits)       # in units of the spacing
    n = q.numerator // q.denominator
    r = q - n
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return sign * Fraction(n) * Fraction(2) ** (e - mant_bits)


def f32(x):
    return rne(x, 23, -126)


def f16(x):
    return rne(x, 10, -14)
