"""Reference for the matrix-core activation transform.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this module.  It shares no code with the HIP library.

The fast transform computes x' = x P G_s (Eq. 11) as an fp16 GEMM: the basis is
split once as v = 2^14 P (exact), hi = fp16(v), lo = fp16(v - hi), and
2^14 x' = sum_k x_k hi_kj + sum_k x_k lo_kj with fp32 accumulation.  It is not
the fixed-order transform that defines the codes, so it is checked stage by
stage:

* ``split_basis``: the split itself, in numpy (fp32 scaling, RNE narrowing);
* ``exact_transform``: x P G_s in fp64 (the value both transforms approximate);
* ``fast_bound``: a rigorous per-element bound on |fast - exact|, from the
  split residual and the fp32 accumulation of 2K exact products:
      2^-14 ( sum_k |x_k| |v_kj - hi_kj - lo_kj|
              + gamma_2K sum_k |x_k| (|hi_kj| + |lo_kj|) ),
  gamma_n = n u / (1 - n u) with u = 2^-23, which holds for any summation order
  and either rounding mode of the additions;
* ``canonical_bound``: the same kind of bound for the fixed-order fp32 chain
  (u = 2^-24, K products with one rounding each plus the K/256 chunk sums), used
  to explain where codes from the two transforms may differ.
"""
from __future__ import annotations

import numpy as np

SCALE = 2.0 ** 14


def _f16(a):
    a = np.asarray(a)
    return a.view(np.float16) if a.dtype == np.uint16 else a.astype(np.float16)


def split_basis(P: np.ndarray) -> np.ndarray:
    """Ps [K][2K] as fp16 bits: Ps[j][k] = hi(2^14 P[k][j]), Ps[j][K + k] = lo."""
    v = np.asarray(P, np.float32).T * np.float32(SCALE)           # exact scaling
    hi = v.astype(np.float16)
    lo = (v - hi.astype(np.float32)).astype(np.float16)            # v - hi exact in fp32
    return np.ascontiguousarray(np.concatenate([hi, lo], axis=1)).view(np.uint16)


def gate_mask(state, K: int, dm: int, du: int) -> np.ndarray:
    """[M][K] booleans: column kept for the row's state (Eq. 9-10 band layout)."""
    j = np.arange(K)
    m_band = (j >= K - dm - du) & (j < K - du)
    u_band = j >= K - du
    st = np.asarray(state).astype(bool)[:, None]
    return np.where(st, ~u_band[None, :], ~m_band[None, :])


def exact_transform(X, state, P, dm: int, du: int) -> np.ndarray:
    x = _f16(X).astype(np.float64) @ np.asarray(P, np.float64)
    if state is not None:
        x = np.where(gate_mask(state, x.shape[1], dm, du), x, 0.0)
    return x


def fast_bound(X, Ps, P) -> np.ndarray:
    K = np.asarray(P).shape[0]
    v = np.asarray(P, np.float32).T.astype(np.float64) * SCALE
    ps = _f16(Ps).astype(np.float64)
    hi, lo = ps[:, :K], ps[:, K:]
    delta = np.abs(v - hi - lo)                                    # exact in fp64
    ax = np.abs(_f16(X).astype(np.float64))
    n = 2 * K
    u = 2.0 ** -23
    gamma = n * u / (1 - n * u)
    b = (ax @ delta.T + gamma * (ax @ (np.abs(hi) + np.abs(lo)).T)) / SCALE
    return b * (1 + 1e-9)                                          # room for this fp64 evaluation


def canonical_bound(X, P) -> np.ndarray:
    K = np.asarray(P).shape[0]
    n = K + K // 256
    u = 2.0 ** -24
    gamma = n * u / (1 - n * u)
    ax = np.abs(_f16(X).astype(np.float64))
    return gamma * (ax @ np.abs(np.asarray(P, np.float64))) * (1 + 1e-9)
