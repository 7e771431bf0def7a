"""STaR-Quant W4A4 hot path on MI355X (gfx950): thin torch binding of libstarquant.

Every function here only checks and marshals arguments (device pointers, sizes,
the current HIP stream) and calls the C ABI declared in include/starquant.h;
all arithmetic runs in the library's HIP kernels.  torch provides device memory
and streams.  Outputs and workspaces are allocated with torch when not given.

    Aq, s_a = sgat_quant_act(X, state, P)            # Eq. 11 + per-token int4
    Wq, s_w = sgat_prepare_weights(W, P)             # Eq. 12, offline
    Y = w4a4_gemm(Aq, s_a, Wq, s_w)                  # Eq. 13
    Zc = tac_apply(Z, tac_M, tac_d, g)               # Eq. 17
"""
from __future__ import annotations

import functools
from typing import Optional, Tuple

import torch

from ._lib import SQ_OK, StarQuantError, check, lib  # noqa: F401

__all__ = ["sgat_prepare_weights", "sgat_transform", "sgat_quantize", "sgat_quant_act", "w4a4_gemm", "tac_apply",
           "tac_default_block", "default_band", "quant_act_workspace_bytes", "gemm_workspace_bytes",
           "prepare_weights_workspace_bytes", "StarQuantError", "lib",
           "sgat_prepare_weights_w8", "sgat_quantize_w8", "sgat_quant_act_w8", "w8a8_gemm",
           "tac_calibrate", "tac_calibrate_workspace_bytes", "sgat_split_basis", "sgat_transform_fast",
           "fp6_row_bytes", "codes_to_fp6", "w4a4_gemm_fp6",
           "frag_weight_bytes", "weights_to_frag", "w4a4_gemm_frag", "w8a8_gemm_frag"]


def _on_stream(fn):
    """Runs a binding call with `stream` (when given) as torch's current stream,
    so that every tensor the call allocates (outputs, workspaces) belongs to the
    stream its kernels run on and the caching allocator cannot hand that memory
    to other work while they use it.  A raw HIP stream handle is wrapped as an
    external stream."""
    @functools.wraps(fn)
    def wrapper(*args, stream=None, **kw):
        if stream is None:
            return fn(*args, stream=None, **kw)
        s = stream if isinstance(stream, torch.cuda.Stream) else torch.cuda.ExternalStream(int(stream))
        with torch.cuda.stream(s):
            return fn(*args, stream=s, **kw)
    return wrapper


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _need(t: Optional[torch.Tensor], name: str, dtype, shape=None, optional=False):
    if t is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def _ws(nbytes: int, ws: Optional[torch.Tensor], device) -> Tuple[Optional[torch.Tensor], int]:
    if nbytes == 0:
        return ws, (ws.numel() if ws is not None else 0)
    if ws is None:
        ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return ws, ws.numel() * ws.element_size()


def tac_default_block(C: int) -> int:
    return int(lib().sq_tac_default_block(int(C)))


def default_band(K: int) -> Tuple[int, int]:
    """d_m = d_u = K/32 (App. B default subspace allocation)."""
    return K // 32, K // 32


def quant_act_workspace_bytes(M: int, K: int, has_P: bool, has_tac: bool) -> int:
    return int(lib().sq_quant_act_workspace_bytes(M, K, int(has_P), int(has_tac)))


def prepare_weights_workspace_bytes(N: int, K: int, has_P: bool) -> int:
    return int(lib().sq_prepare_weights_workspace_bytes(N, K, int(has_P)))


def gemm_workspace_bytes(M: int, N: int, K: int, bits: int = 4) -> int:
    f = lib().sq_gemm_w8_workspace_bytes if bits == 8 else lib().sq_gemm_workspace_bytes
    return int(f(M, N, K))


def _codes_spec(bits: int, K: int):
    """(dtype, row width) of a code tensor: packed int4 uint8 [K/2] or int8 [K]."""
    return (torch.int8, K) if bits == 8 else (torch.uint8, K // 2)


@_on_stream
def sgat_prepare_weights(W: torch.Tensor, P: Optional[torch.Tensor] = None, *, Wq=None, s_w=None, ws=None,
                         stream=None, bits: int = 4):
    """W~ = Q_w(P^T W^T) as rows of W P: returns (Wq, s_w [N] fp32); Wq is [N][K/2]
    packed int4 (bits=4) or [N][K] int8 (bits=8, App. D)."""
    N, K = W.shape
    dt, kw = _codes_spec(bits, K)
    _need(W, "W", torch.float16)
    _need(P, "P", torch.float32, (K, K), optional=True)
    if Wq is None:
        Wq = torch.empty((N, kw), dtype=dt, device=W.device)
    if s_w is None:
        s_w = torch.empty((N,), dtype=torch.float32, device=W.device)
    _need(Wq, "Wq", dt, (N, kw))
    _need(s_w, "s_w", torch.float32, (N,))
    ws, wsb = _ws(prepare_weights_workspace_bytes(N, K, P is not None), ws, W.device)
    f = lib().sgat_prepare_weights_w8 if bits == 8 else lib().sgat_prepare_weights
    check(f(_ptr(W), _ptr(P), N, K, _ptr(Wq), _ptr(s_w), _ptr(ws), wsb, _stream(stream)))
    return Wq, s_w


def sgat_prepare_weights_w8(W, P=None, **kw):
    return sgat_prepare_weights(W, P, bits=8, **kw)


@_on_stream
def sgat_transform(X: torch.Tensor, state: Optional[torch.Tensor], P: Optional[torch.Tensor],
                   d_m: Optional[int] = None, d_u: Optional[int] = None, *, out=None, stream=None):
    """x'_i = x_i P G_{s_i} (Eq. 11), fp32 [M][K]."""
    M, K = X.shape
    dm0, du0 = default_band(K)
    d_m = dm0 if d_m is None else d_m
    d_u = du0 if d_u is None else d_u
    _need(X, "X", torch.float16)
    _need(state, "state", torch.uint8, (M,), optional=True)
    _need(P, "P", torch.float32, (K, K), optional=True)
    if out is None:
        out = torch.empty((M, K), dtype=torch.float32, device=X.device)
    _need(out, "out", torch.float32, (M, K))
    check(lib().sgat_transform(_ptr(X), _ptr(state), _ptr(P), M, K, d_m, d_u, _ptr(out), _stream(stream)))
    return out


@_on_stream
def sgat_quantize(Xp: torch.Tensor, *, Aq=None, s=None, stream=None, bits: int = 4):
    """Per-row symmetric quantisation of fp32 rows (Eq. 2, z = 0): returns (Aq, s [M] fp32)."""
    M, K = Xp.shape
    dt, kw = _codes_spec(bits, K)
    _need(Xp, "Xp", torch.float32)
    if Aq is None:
        Aq = torch.empty((M, kw), dtype=dt, device=Xp.device)
    if s is None:
        s = torch.empty((M,), dtype=torch.float32, device=Xp.device)
    _need(Aq, "Aq", dt, (M, kw))
    _need(s, "s", torch.float32, (M,))
    f = lib().sgat_quantize_w8 if bits == 8 else lib().sgat_quantize
    check(f(_ptr(Xp), M, K, _ptr(Aq), _ptr(s), _stream(stream)))
    return Aq, s


def sgat_quantize_w8(Xp, **kw):
    return sgat_quantize(Xp, bits=8, **kw)


@_on_stream
def sgat_quant_act(X: torch.Tensor, state: Optional[torch.Tensor], P: Optional[torch.Tensor] = None,
                   d_m: Optional[int] = None, d_u: Optional[int] = None, tac_M: Optional[torch.Tensor] = None,
                   tac_d: Optional[torch.Tensor] = None, g: int = 0, *, Aq=None, s_a=None, ws=None, stream=None,
                   bits: int = 4):
    """[TAC] -> x P G_s -> per-token codes: returns (Aq, s_a [M] fp32), Aq packed int4
    [M][K/2] uint8 (bits=4) or int8 [M][K] (bits=8)."""
    M, K = X.shape
    dt, kw = _codes_spec(bits, K)
    dm0, du0 = default_band(K)
    d_m = dm0 if d_m is None else d_m
    d_u = du0 if d_u is None else d_u
    _need(X, "X", torch.float16)
    _need(state, "state", torch.uint8, (M,), optional=True)
    _need(P, "P", torch.float32, (K, K), optional=True)
    if tac_M is not None:
        _need(tac_M, "tac_M", torch.float16, (K // g, g, g))
        _need(tac_d, "tac_d", torch.float16, (K,))
    if Aq is None:
        Aq = torch.empty((M, kw), dtype=dt, device=X.device)
    if s_a is None:
        s_a = torch.empty((M,), dtype=torch.float32, device=X.device)
    _need(Aq, "Aq", dt, (M, kw))
    _need(s_a, "s_a", torch.float32, (M,))
    ws, wsb = _ws(quant_act_workspace_bytes(M, K, P is not None, tac_M is not None), ws, X.device)
    f = lib().sgat_quant_act_w8 if bits == 8 else lib().sgat_quant_act
    check(f(_ptr(X), _ptr(state), _ptr(P), M, K, d_m, d_u, _ptr(tac_M), _ptr(tac_d), g,
            _ptr(Aq), _ptr(s_a), _ptr(ws), wsb, _stream(stream)))
    return Aq, s_a


def sgat_quant_act_w8(X, state, P=None, d_m=None, d_u=None, tac_M=None, tac_d=None, g=0, **kw):
    return sgat_quant_act(X, state, P, d_m, d_u, tac_M, tac_d, g, bits=8, **kw)


@_on_stream
def w4a4_gemm(Aq: torch.Tensor, s_a: torch.Tensor, Wq: torch.Tensor, s_w: torch.Tensor, *, Y=None, acc=None,
              want_Y: bool = True, want_acc: bool = False, ws=None, stream=None, bits: int = 4):
    """Y = fp16((acc * s_a) * s_w) with acc = Aq . Wq^T exact (Eq. 13).  Returns Y, or (Y, acc).
    bits=8 takes int8 codes (App. D)."""
    M, Kc = Aq.shape
    N = Wq.shape[0]
    dt = torch.int8 if bits == 8 else torch.uint8
    K = Kc if bits == 8 else 2 * Kc
    _need(Aq, "Aq", dt)
    _need(Wq, "Wq", dt, (N, Kc))
    _need(s_a, "s_a", torch.float32, (M,))
    _need(s_w, "s_w", torch.float32, (N,))
    if Y is None and want_Y:
        Y = torch.empty((M, N), dtype=torch.float16, device=Aq.device)
    if acc is None and want_acc:
        acc = torch.empty((M, N), dtype=torch.int32, device=Aq.device)
    _need(Y, "Y", torch.float16, (M, N), optional=True)
    _need(acc, "acc", torch.int32, (M, N), optional=True)
    ws, wsb = _ws(gemm_workspace_bytes(M, N, K, bits), ws, Aq.device)
    f = lib().w8a8_gemm if bits == 8 else lib().w4a4_gemm
    check(f(_ptr(Aq), _ptr(s_a), _ptr(Wq), _ptr(s_w), M, N, K, _ptr(Y), _ptr(acc), _ptr(ws), wsb, _stream(stream)))
    return (Y, acc) if want_acc else Y


def w8a8_gemm(Aq, s_a, Wq, s_w, **kw):
    return w4a4_gemm(Aq, s_a, Wq, s_w, bits=8, **kw)


def fp6_row_bytes(K: int) -> int:
    """Bytes per row of an FP6 operand of K codes (96 per block of 128)."""
    n = int(lib().sq_fp6_row_bytes(K))
    if n == 0:
        raise ValueError(f"K={K}: need 64 <= K <= 131072 and K % 64 == 0")
    return n


@_on_stream
def codes_to_fp6(codes: torch.Tensor, *, out=None, stream=None):
    """Packed int4 codes [R, K/2] -> the FP6 (e3m2) operand layout [R, fp6_row_bytes(K)]."""
    R, Kh = codes.shape
    K = 2 * Kh
    _need(codes, "codes", torch.uint8)
    rb = fp6_row_bytes(K)
    if out is None:
        out = torch.empty((R, rb), dtype=torch.uint8, device=codes.device)
    _need(out, "out", torch.uint8, (R, rb))
    check(lib().sq_codes_to_fp6(_ptr(codes), R, K, _ptr(out), _stream(stream)))
    return out


@_on_stream
def w4a4_gemm_fp6(A6: torch.Tensor, s_a: torch.Tensor, W6: torch.Tensor, s_w: torch.Tensor, K: int, *, Y=None,
                  acc=None, want_Y: bool = True, want_acc: bool = False, stream=None):
    """The W4A4 GEMM (Eq. 13) on FP6 operands (codes_to_fp6 layout) and the FP6
    matrix cores; bit-identical to w4a4_gemm.  Returns Y, or (Y, acc)."""
    M, N = A6.shape[0], W6.shape[0]
    rb = fp6_row_bytes(K)
    _need(A6, "A6", torch.uint8, (M, rb))
    _need(W6, "W6", torch.uint8, (N, rb))
    _need(s_a, "s_a", torch.float32, (M,))
    _need(s_w, "s_w", torch.float32, (N,))
    if Y is None and want_Y:
        Y = torch.empty((M, N), dtype=torch.float16, device=A6.device)
    if acc is None and want_acc:
        acc = torch.empty((M, N), dtype=torch.int32, device=A6.device)
    _need(Y, "Y", torch.float16, (M, N), optional=True)
    _need(acc, "acc", torch.int32, (M, N), optional=True)
    check(lib().w4a4_gemm_fp6(_ptr(A6), _ptr(s_a), _ptr(W6), _ptr(s_w), M, N, K, _ptr(Y), _ptr(acc),
                              _stream(stream)))
    return (Y, acc) if want_acc else Y


def frag_weight_bytes(N: int, K: int, bits: int = 4) -> int:
    """Bytes of the fragment-ordered weights of an N x K code matrix (1 KB per
    16 rows and k step of 64 bytes: 128 int4 or 64 int8 codes)."""
    n = int(lib().sq_frag_weight_w8_bytes(N, K) if bits == 8 else lib().sq_frag_weight_bytes(N, K))
    if n == 0 and N > 0:
        kmax = 65536 if bits == 8 else 131072
        raise ValueError(f"K={K}: need 64 <= K <= {kmax} and K % 64 == 0")
    return n


def _frag_shape(N: int, K: int, bits: int):
    step = 64 if bits == 8 else 128
    return ((K + step - 1) // step, (N + 15) // 16, 1024)


@_on_stream
def weights_to_frag(Wq: torch.Tensor, *, out=None, stream=None):
    """Code matrix -> fragment order [k steps, ceil(N/16), 1024] (uint8): packed
    int4 weights [N, K/2] (uint8, 128 codes a k step) or int8 weights [N, K]
    (int8, 64 codes a k step)."""
    N, Kc = Wq.shape
    bits = 8 if Wq.dtype == torch.int8 else 4
    K = Kc if bits == 8 else 2 * Kc
    _need(Wq, "Wq", torch.int8 if bits == 8 else torch.uint8)
    shape = _frag_shape(N, K, bits)
    frag_weight_bytes(N, K, bits)
    if out is None:
        out = torch.empty(shape, dtype=torch.uint8, device=Wq.device)
    _need(out, "out", torch.uint8, shape)
    f = lib().sq_weights_to_frag_w8 if bits == 8 else lib().sq_weights_to_frag
    check(f(_ptr(Wq), N, K, _ptr(out), _stream(stream)))
    return out


@_on_stream
def w4a4_gemm_frag(Aq: torch.Tensor, s_a: torch.Tensor, Wf: torch.Tensor, s_w: torch.Tensor, *, Y=None, acc=None,
                   want_Y: bool = True, want_acc: bool = False, ws=None, stream=None, bits: int = 4):
    """w4a4_gemm (Eq. 13) with the weights in fragment order (weights_to_frag);
    N is s_w's length.  Bit-identical to w4a4_gemm.  bits=8 takes int8
    activation codes and the fragment order of int8 weights (App. D),
    bit-identical to w8a8_gemm.  Returns Y, or (Y, acc)."""
    M, Kc = Aq.shape
    N = s_w.shape[0]
    K = Kc if bits == 8 else 2 * Kc
    _need(Aq, "Aq", torch.int8 if bits == 8 else torch.uint8)
    _need(Wf, "Wf", torch.uint8, _frag_shape(N, K, bits))
    _need(s_a, "s_a", torch.float32, (M,))
    _need(s_w, "s_w", torch.float32, (N,))
    if Y is None and want_Y:
        Y = torch.empty((M, N), dtype=torch.float16, device=Aq.device)
    if acc is None and want_acc:
        acc = torch.empty((M, N), dtype=torch.int32, device=Aq.device)
    _need(Y, "Y", torch.float16, (M, N), optional=True)
    _need(acc, "acc", torch.int32, (M, N), optional=True)
    ws, wsb = _ws(gemm_workspace_bytes(M, N, K, bits), ws, Aq.device)
    f = lib().w8a8_gemm_frag if bits == 8 else lib().w4a4_gemm_frag
    check(f(_ptr(Aq), _ptr(s_a), _ptr(Wf), _ptr(s_w), M, N, K, _ptr(Y), _ptr(acc), _ptr(ws), wsb, _stream(stream)))
    return (Y, acc) if want_acc else Y


def w8a8_gemm_frag(Aq, s_a, Wf, s_w, **kw):
    return w4a4_gemm_frag(Aq, s_a, Wf, s_w, bits=8, **kw)


@_on_stream
def tac_apply(Z: torch.Tensor, tac_M: torch.Tensor, tac_d: torch.Tensor, g: int, *, out=None, stream=None):
    """Z_b M_b^T + 1 d_b^T per block of g channels (Eq. 17), fp16 out."""
    M, C = Z.shape
    _need(Z, "Z", torch.float16)
    _need(tac_M, "tac_M", torch.float16, (C // g, g, g))
    _need(tac_d, "tac_d", torch.float16, (C,))
    if out is None:
        out = torch.empty_like(Z)
    _need(out, "out", torch.float16, (M, C))
    check(lib().tac_apply(_ptr(Z), _ptr(tac_M), _ptr(tac_d), M, C, g, _ptr(out), _stream(stream)))
    return out


TAC_RHO, TAC_EPS, TAC_ETA, TAC_ALPHA = 3e-4, 1e-8, 0.15, 0.55   # App. C defaults


def tac_calibrate_workspace_bytes(N: int, C: int, g: int) -> int:
    return int(lib().sq_tac_calibrate_workspace_bytes(N, C, g))


@_on_stream
def tac_calibrate(Z_fp: torch.Tensor, Z_q: torch.Tensor, g: int, *, rho: float = TAC_RHO, eps: float = TAC_EPS,
                  eta: float = TAC_ETA, alpha: float = TAC_ALPHA, want_fp64: bool = False, tac_M=None, tac_d=None,
                  ws=None, stream=None):
    """Closed-form TAC parameters (App. C) from paired full-precision / quantised
    attention outputs: (tac_M fp16 [C/g, g, g], tac_d fp16 [C]) and, with
    want_fp64, also the unrounded fp64 (M, d)."""
    N, C = Z_fp.shape
    _need(Z_fp, "Z_fp", torch.float16)
    _need(Z_q, "Z_q", torch.float16, (N, C))
    dev = Z_fp.device
    if tac_M is None:
        tac_M = torch.empty((C // g, g, g), dtype=torch.float16, device=dev)
    if tac_d is None:
        tac_d = torch.empty((C,), dtype=torch.float16, device=dev)
    _need(tac_M, "tac_M", torch.float16, (C // g, g, g))
    _need(tac_d, "tac_d", torch.float16, (C,))
    M64 = torch.empty((C // g, g, g), dtype=torch.float64, device=dev) if want_fp64 else None
    d64 = torch.empty((C,), dtype=torch.float64, device=dev) if want_fp64 else None
    ws, wsb = _ws(tac_calibrate_workspace_bytes(N, C, g), ws, dev)
    check(lib().tac_calibrate(_ptr(Z_fp), _ptr(Z_q), N, C, g, rho, eps, eta, alpha, _ptr(tac_M), _ptr(tac_d),
                              _ptr(M64), _ptr(d64), _ptr(ws), wsb, _stream(stream)))
    return (tac_M, tac_d, M64, d64) if want_fp64 else (tac_M, tac_d)


@_on_stream
def sgat_split_basis(P: torch.Tensor, *, out=None, stream=None):
    """fp16 hi / lo split of 2^14 P, transposed: Ps [K, 2K] for sgat_transform_fast."""
    K = P.shape[0]
    _need(P, "P", torch.float32, (K, K))
    if out is None:
        out = torch.empty((K, 2 * K), dtype=torch.float16, device=P.device)
    _need(out, "out", torch.float16, (K, 2 * K))
    check(lib().sgat_split_basis(_ptr(P), K, _ptr(out), _stream(stream)))
    return out


@_on_stream
def sgat_transform_fast(X: torch.Tensor, state: Optional[torch.Tensor], Ps: torch.Tensor,
                        d_m: Optional[int] = None, d_u: Optional[int] = None, *, out=None, stream=None):
    """x' = x P G_s on the fp16 matrix cores (within a stated bound of the exact
    product; not bit-identical to sgat_transform).  fp32 out."""
    M, K = X.shape
    _need(X, "X", torch.float16)
    _need(state, "state", torch.uint8, (M,), optional=True)
    _need(Ps, "Ps", torch.float16, (K, 2 * K))
    dm0, du0 = default_band(K)
    d_m = dm0 if d_m is None else d_m
    d_u = du0 if d_u is None else d_u
    if out is None:
        out = torch.empty((M, K), dtype=torch.float32, device=X.device)
    _need(out, "out", torch.float32, (M, K))
    check(lib().sgat_transform_fast(_ptr(X), _ptr(state), _ptr(Ps), M, K, d_m, d_u, _ptr(out), _stream(stream)))
    return out
