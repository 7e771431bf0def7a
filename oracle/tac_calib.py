"""CPU oracle for the TAC closed-form calibration (App. C).  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this module.  It shares no code with the HIP library.

Plain numpy in fp64, in the order the appendix gives the steps:

1. block statistics: per block of g channels, the population mean
   mu_b = (1/N) sum_i z_i and covariance Sigma_b = (1/N) sum_i z_i z_i^T - mu_b mu_b^T,
   for the full-precision and for the quantised attention output;
2. damped covariance matching: lambda_b = rho max(Tr(Sigma_b^Q) / g, eps),
   M_b = (Sigma_b^FP)^(1/2) (Sigma_b^Q + lambda_b I)^(-1/2), every matrix power
   taken through a symmetric eigendecomposition with eigenvalues clamped
   below at 1e-12;
3. singular value smoothing: M_b = U diag(sigma) V^T, sigma' = (1 - eta) sigma +
   eta mean(sigma), M_b^sv = U diag(sigma') V^T;
4. identity shrinkage: M_b^final = (1 - alpha) M_b^sv + alpha I;
5. bias: d_b = mu_b^FP - M_b^final mu_b^Q.

Stored parameters are M_b^final[r][c] and d_b, each rounded once from fp64 to
fp16 (round to nearest even), in the layout the TAC kernels read
([C/g][g][g] and [C]).  Library primitives used: numpy's batched matmul,
``eigh`` and ``svd``.  Defaults are the appendix's: rho = 3e-4, eps = 1e-8,
eta = 0.15, alpha = 0.55.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np

RHO = 3e-4
EPS = 1e-8
ETA = 0.15
ALPHA = 0.55
EIG_FLOOR = 1e-12


def block_stats(Z: np.ndarray, g: int) -> Tuple[np.ndarray, np.ndarray]:
    """App. C, block-wise statistics: (mu [B][g], Sigma [B][g][g]) in fp64."""
    Z = np.asarray(Z)
    if Z.dtype == np.uint16:
        Z = Z.view(np.float16)
    Z = Z.astype(np.float64)
    N, C = Z.shape
    B = C // g
    Zb = Z.reshape(N, B, g).transpose(1, 0, 2)             # [B][N][g]
    mu = Zb.sum(axis=1) / N
    second = np.matmul(Zb.transpose(0, 2, 1), Zb) / N       # (1/N) sum_i z_i z_i^T
    return mu, second - mu[:, :, None] * mu[:, None, :]


def mat_power(A: np.ndarray, p: float) -> np.ndarray:
    """App. C: A^p = Q diag(max(lambda_i, 1e-12)^p) Q^T, A = Q diag(lambda) Q^T."""
    lam, Q = np.linalg.eigh(A)
    return (Q * np.maximum(lam, EIG_FLOOR) ** p) @ Q.T


def calibrate_block(mu_f, S_f, mu_q, S_q, rho=RHO, eps=EPS, eta=ETA, alpha=ALPHA):
    """Steps 2-5 for one block: (M_final [g][g], d [g]) in fp64."""
    g = len(mu_f)
    I = np.eye(g)
    lam = rho * max(np.trace(S_q) / g, eps)                 # damping
    M = mat_power(S_f, 0.5) @ mat_power(S_q + lam * I, -0.5)  # covariance matching
    U, sig, Vt = np.linalg.svd(M)                           # singular value smoothing
    sig_s = (1.0 - eta) * sig + eta * sig.mean()
    M_sv = (U * sig_s) @ Vt
    M_final = (1.0 - alpha) * M_sv + alpha * I              # identity shrinkage
    d = mu_f - M_final @ mu_q                               # bias
    return M_final, d


def calibrate(Z_fp, Z_q, g: int, rho=RHO, eps=EPS, eta=ETA, alpha=ALPHA):
    """Whole calibration: (M [C/g][g][g] fp64, d [C] fp64)."""
    mu_f, S_f = block_stats(Z_fp, g)
    mu_q, S_q = block_stats(Z_q, g)
    B = mu_f.shape[0]
    M = np.empty((B, g, g))
    d = np.empty((B, g))
    for b in range(B):
        M[b], d[b] = calibrate_block(mu_f[b], S_f[b], mu_q[b], S_q[b], rho, eps, eta, alpha)
    return M, d.reshape(-1)


def to_fp16_bits(x: np.ndarray) -> np.ndarray:
    """One RNE rounding from fp64 to fp16, as IEEE bits (uint16)."""
    return np.asarray(x, np.float64).astype(np.float16).view(np.uint16)


def apply(Z, M, d, g: int) -> np.ndarray:
    """Z^TAC_b = Z_b M_b^T + 1 d_b^T in fp64 (used by the pins only)."""
    Z = np.asarray(Z)
    if Z.dtype == np.uint16:
        Z = Z.view(np.float16)
    Z = Z.astype(np.float64)
    N, C = Z.shape
    B = C // g
    Zb = Z.reshape(N, B, g).transpose(1, 0, 2)
    out = np.matmul(Zb, np.asarray(M).transpose(0, 2, 1)) + np.asarray(d).reshape(B, 1, g)
    return out.transpose(1, 0, 2).reshape(N, C)
