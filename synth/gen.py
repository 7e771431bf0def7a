"""Seeded synthetic tensors with the shapes and value structure of the workloads.

Recipe (every draw is fp64 from a Philox stream keyed by
``SeedSequence([SEED, config_id, tensor_id, ...])``, then cast RNE to the
stored dtype):

* activations X, fp16 [M][K]: N(0, 1) everywhere; each token state owns a
  disjoint, seeded set of outlier channels in the input basis, multiplied by
  16 on masked tokens and by 8 on unmasked tokens (state-dependent outliers,
  as in the paper's Fig. 1 motivation);
* weights W, fp16 [N][K]: N(0, 0.02);
* SGAT basis P, fp32 [K][K]: a Gaussian matrix orthogonalised by QR with the
  signs of diag(R) folded in (the initialisation of App. B).  For K > 512 the
  basis is (A kron B) Pi (C kron D), with A, B, C, D such factors of sizes K/b
  and b (b = 128, or 64) and Pi a random permutation: dense, orthogonal and
  free of a Kronecker structure, built in seconds (a full K x K QR at K =
  18944 takes many minutes on the host), in fp64 and stored as fp32;
* TAC parameters: M_b = I + N(0, 0.01) per g x g block and d ~ N(0, 0.01),
  both fp16 (Eq. 17); the identity case is M_b = I, d = 0;
* token states, uint8 [M]: 0 = unmasked, 1 = masked, with the layouts below;
* TAC calibration pairs (App. C), fp16 [N][C] each: a "full-precision"
  attention output with a per-block mean and a per-block correlated covariance
  (z = mu_b + xi L_b^T, xi ~ N(0, I), L_b lower triangular with diagonal in
  [0.5, 1.5] and N(0, 0.5^2 / g) below it, which keeps the covariance well
  conditioned at every g), and a "quantised" counterpart drawn as a
  generic perturbation of it: a per-channel gain 1 + N(0, 0.05), additive
  N(0, 0.1^2) noise and a per-channel offset N(0, 0.05).

Nothing here transforms, quantises or multiplies the method's operands.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

SEED = 260604945

# tensor ids (third SeedSequence word)
T_STATE = 1
T_OUTLIER = 2
T_X = 3
T_W = 4
T_P = 5
T_TAC = 6
T_CALIB = 7


def rng_for(config_id: int, tensor_id: int, *extra: int) -> np.random.Generator:
    return np.random.Generator(
        np.random.Philox(np.random.SeedSequence([SEED, int(config_id), int(tensor_id), *map(int, extra)])))


# ----------------------------------------------------------------------------- states

def state_prompt_then_random(M: int, n_prompt: int, n_masked: int, rng) -> np.ndarray:
    """Rows [0, n_prompt) unmasked; n_masked of the remaining rows masked at random."""
    s = np.zeros(M, np.uint8)
    pos = rng.choice(M - n_prompt, size=n_masked, replace=False)
    s[n_prompt + pos] = 1
    return s


def state_prompt_then_blocks(M: int, n_prompt: int, block: int, n_blocks_masked: int, rng) -> np.ndarray:
    """Rows [0, n_prompt) unmasked; the rest split in blocks, n of them masked."""
    s = np.zeros(M, np.uint8)
    nb = (M - n_prompt) // block
    for b in rng.choice(nb, size=n_blocks_masked, replace=False):
        s[n_prompt + b * block: n_prompt + (b + 1) * block] = 1
    return s


def state_uniform_fraction(batch: int, seq: int, lo: float, hi: float, rng) -> np.ndarray:
    """Per sequence, a mask fraction f ~ U[lo, hi] and round(f*seq) masked positions."""
    s = np.zeros((batch, seq), np.uint8)
    for b in range(batch):
        f = rng.uniform(lo, hi)
        n = int(round(f * seq))
        s[b, rng.choice(seq, size=n, replace=False)] = 1
    return s.reshape(-1)


def state_denoise_step(M: int, t: int, rng_order, n_prompt: int = 512, n_gen: int = 256,
                       steps: int = 64) -> np.ndarray:
    """Denoising-step layout: after step t, n_gen - t*n_gen/steps generation positions
    are still masked (unmasked in a seeded order); token i takes the state of
    position (n_prompt + i) mod (n_prompt + n_gen)."""
    L = n_prompt + n_gen
    order = rng_order.permutation(n_gen)
    masked = np.zeros(L, np.uint8)
    masked[n_prompt:] = 1
    n_unmasked = (t * n_gen) // steps
    masked[n_prompt + order[:n_unmasked]] = 0
    return masked[(n_prompt + np.arange(M)) % L].astype(np.uint8)


def state_edge(M: int, kind: str) -> np.ndarray:
    if kind == "all_masked":
        return np.ones(M, np.uint8)
    if kind == "none_masked":
        return np.zeros(M, np.uint8)
    if kind == "alternating":
        return (np.arange(M) & 1).astype(np.uint8)
    raise ValueError(kind)


# ----------------------------------------------------------------------------- tensors

def outlier_channels(K: int, n_per_state: int, rng) -> Tuple[np.ndarray, np.ndarray]:
    idx = rng.choice(K, size=2 * n_per_state, replace=False)
    return np.sort(idx[:n_per_state]), np.sort(idx[n_per_state:])


def activations(M: int, K: int, state: np.ndarray, m_idx, u_idx, rng,
                mult_m: float = 16.0, mult_u: float = 8.0) -> np.ndarray:
    x = rng.standard_normal((M, K))
    masked = state.astype(bool)
    if len(m_idx):
        x[np.ix_(masked, m_idx)] *= mult_m
    if len(u_idx):
        x[np.ix_(~masked, u_idx)] *= mult_u
    return x.astype(np.float16)


def weights(N: int, K: int, rng, std: float = 0.02) -> np.ndarray:
    out = np.empty((N, K), np.float16)
    step = max(1, (1 << 24) // max(K, 1))
    for r0 in range(0, N, step):
        r1 = min(N, r0 + step)
        out[r0:r1] = (rng.standard_normal((r1 - r0, K)) * std).astype(np.float16)
    return out


def _gaussian_orthogonal(n: int, rng) -> np.ndarray:
    q, r = np.linalg.qr(rng.standard_normal((n, n)))
    return q * np.sign(np.diag(r))[None, :]


def orthogonal(K: int, rng) -> np.ndarray:
    """Dense orthogonal fp32 [K][K] (see the module docstring)."""
    if K <= 512:
        return _gaussian_orthogonal(K, rng).astype(np.float32)
    b = 128 if K % 128 == 0 else 64
    if K % b:
        raise ValueError("K must be a multiple of 64")
    a = K // b
    A, B = _gaussian_orthogonal(a, rng), _gaussian_orthogonal(b, rng)
    C, D = _gaussian_orthogonal(a, rng), _gaussian_orthogonal(b, rng)
    perm = rng.permutation(K)
    # Y = Pi (C kron D): row p is row perm[p] of the Kronecker product,
    # kron(C, D)[ia b + ib, :] = kron(C[ia], D[ib]); viewed as [a][b][K]
    Y = (C[perm // b][:, :, None] * D[perm % b][:, None, :]).reshape(a, b, K)
    # (A kron B) Y: B on the second index, then A on the first
    Y = np.matmul(B, Y)
    out = np.tensordot(A, Y, axes=(1, 0)).reshape(K, K)
    return out.astype(np.float32)


def tac_params(C: int, g: int, rng, std: float = 0.01, identity: bool = False):
    """TAC block matrices fp16 [C/g][g][g] (row r, column c of M_b) and bias fp16 [C]."""
    nb = C // g
    if identity:
        Mb = np.broadcast_to(np.eye(g), (nb, g, g)).astype(np.float16)
        d = np.zeros(C, np.float16)
        return np.ascontiguousarray(Mb), d
    Mb = (np.eye(g)[None] + rng.standard_normal((nb, g, g)) * std).astype(np.float16)
    d = (rng.standard_normal(C) * std).astype(np.float16)
    return Mb, d


def tac_calib_pair(N: int, C: int, g: int, rng) -> Tuple[np.ndarray, np.ndarray]:
    """Paired (full-precision, quantised) attention outputs for TAC calibration,
    fp16 [N][C] each; blocks of g channels are correlated within, independent
    across."""
    B = C // g
    mu = rng.normal(0.0, 0.5, size=(B, g))
    L = np.tril(rng.normal(0.0, 0.5 / np.sqrt(g), size=(B, g, g)), -1)
    idx = np.arange(g)
    L[:, idx, idx] = rng.uniform(0.5, 1.5, size=(B, g))
    xi = rng.standard_normal((B, N, g))
    zf = (mu[:, None, :] + np.matmul(xi, L.transpose(0, 2, 1))).transpose(1, 0, 2).reshape(N, C)
    gain = 1.0 + rng.normal(0.0, 0.05, size=C)
    off = rng.normal(0.0, 0.05, size=C)
    zq = zf * gain[None] + rng.normal(0.0, 0.1, size=(N, C)) + off[None]
    return zf.astype(np.float16), zq.astype(np.float16)


def default_band(K: int) -> Tuple[int, int]:
    """d_m = d_u = d/32 (the paper's default subspace allocation)."""
    return K // 32, K // 32


def default_tac_block(C: int) -> int:
    """g = 16, or the largest g <= 16 dividing C."""
    for g in range(16, 0, -1):
        if C % g == 0:
            return g
    return 1


# ----------------------------------------------------------------------------- configs

@dataclasses.dataclass(frozen=True)
class Site:
    name: str
    K: int
    N: int
    tac: bool = False          # TAC ahead of this linear (the O-projection)


@dataclasses.dataclass(frozen=True)
class Config:
    cid: int
    name: str
    M: int
    sites: Tuple[Site, ...]
    outliers: Optional[int]    # outlier channels per state; None = round(K/100)
    tac_g: Optional[int] = None

    def n_outliers(self, K: int) -> int:
        return self.outliers if self.outliers is not None else int(round(K / 100))


LLADA_SITES = (Site("qkv", 4096, 12288), Site("o", 4096, 4096, tac=True),
               Site("gate_up", 4096, 24576), Site("down", 12288, 4096))
DREAM_SITES = (Site("qkv", 3584, 4608), Site("o", 3584, 3584, tac=True),
               Site("gate_up", 3584, 37888), Site("down", 18944, 3584))

# workload ids (each id also keys its seeded generators)
SINGLE_LINEAR, LLADA, DREAM, TAC_OPROJ, LLADA_SWEEP = 0, 1, 2, 3, 4

CONFIGS: Dict[int, Config] = {
    0: Config(0, "single SGAT W4A4 linear, 128 tokens, K=N=512", 128,
              (Site("linear", 512, 512),), outliers=4),
    1: Config(1, "LLaDA-8B-shaped layer set, 1024 tokens", 1024, LLADA_SITES, outliers=None),
    2: Config(2, "Dream-7B-shaped layer set, 8x2048 tokens", 16384, DREAM_SITES, outliers=None),
    3: Config(3, "TAC g=128 + O-proj 4096->4096, 8x2048 tokens", 16384,
              (Site("o", 4096, 4096, tac=True),), outliers=None, tac_g=128),
    4: Config(4, "LLaDA-8B-shaped layer set, denoising-step sweep", 1024, LLADA_SITES, outliers=None),
}

SWEEP_M = tuple(16 << i for i in range(11))     # 16 .. 16384


def config_state(cid: int, M: Optional[int] = None, t: Optional[int] = None) -> np.ndarray:
    rng = rng_for(cid, T_STATE)
    if cid == 0:
        return state_prompt_then_random(128, 64, 32, rng)
    if cid == 1:
        return state_prompt_then_blocks(1024, 512, 32, 8, rng)
    if cid in (2, 3):
        return state_uniform_fraction(8, 2048, 0.1, 0.9, rng)
    if cid == 4:
        return state_denoise_step(M if M is not None else 1024, 0 if t is None else t, rng)
    raise ValueError(cid)


@dataclasses.dataclass
class SiteTensors:
    site: Site
    X: np.ndarray               # fp16 [M][K]
    W: np.ndarray               # fp16 [N][K]
    P: np.ndarray               # fp32 [K][K]
    dm: int
    du: int
    tac_M: Optional[np.ndarray] = None
    tac_d: Optional[np.ndarray] = None
    g: int = 0


def site_tensors(cid: int, si: int, state: np.ndarray, *, with_W: bool = True, with_P: bool = True,
                 tac_identity: bool = False, g: Optional[int] = None) -> SiteTensors:
    cfg = CONFIGS[cid]
    site = cfg.sites[si]
    K, N, M = site.K, site.N, len(state)
    m_idx, u_idx = outlier_channels(K, cfg.n_outliers(K), rng_for(cid, T_OUTLIER, si))
    X = activations(M, K, state, m_idx, u_idx, rng_for(cid, T_X, si))
    W = weights(N, K, rng_for(cid, T_W, si)) if with_W else None
    P = orthogonal(K, rng_for(cid, T_P, si)) if with_P else None
    dm, du = default_band(K)
    st = SiteTensors(site, X, W, P, dm, du)
    if site.tac:
        gg = g if g is not None else (cfg.tac_g or default_tac_block(K))
        st.tac_M, st.tac_d = tac_params(K, gg, rng_for(cid, T_TAC, si), identity=tac_identity)
        st.g = gg
    return st


def small_case(seed: int, M: int, K: int, N: int, *, n_out: int = 2, g: int = 0,
               state: Optional[np.ndarray] = None):
    """A free-form small case (for tests): X, state, W, P and optional TAC params."""
    rng = rng_for(1000 + seed, 0)
    if state is None:
        state = (rng.random(M) < 0.5).astype(np.uint8)
    m_idx, u_idx = outlier_channels(K, n_out, rng)
    X = activations(M, K, state, m_idx, u_idx, rng)
    W = weights(N, K, rng)
    P = orthogonal(K, rng)
    out = dict(X=X, state=state, W=W, P=P)
    if g:
        out["tac_M"], out["tac_d"] = tac_params(K, g, rng)
        out["g"] = g
    return out


__all__ = [n for n in dir() if not n.startswith("_")]
