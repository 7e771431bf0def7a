"""Seeded synthetic inputs for the STaR-Quant W4A4 hot path.

This package generates inputs only: activations, token mask states, weights,
the orthogonal SGAT basis and the TAC parameters.  It holds none of the
method's arithmetic (no transform, quantisation, GEMM or TAC), so that both the
CPU oracle and the HIP path can be fed the identical bytes from here.
"""
from .gen import *  # noqa: F401,F403
