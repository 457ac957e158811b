"""Seeded synthetic inputs for the Video Delta Attention forward pass.

This module only draws random numbers and rounds them to the storage type.
It holds none of the operator's arithmetic, so both the fp64 oracle and the
HIP path can consume exactly the same values from it.

Workloads (all independent head problems are folded into one leading axis,
``H_total = B * H``; each tensor is laid out frame-major ``[H_total][F][N][d]``):

* q, k ~ N(0, 1), then L2-normalised per token (the linear branch's feature
  map normalises queries and keys; Section 2.3 of the paper).
* v ~ N(0, 1).
* beta = sigmoid(sigma * z), z ~ N(0, 1), one write strength per token
  (Section 3.1 defines beta_{t,u} >= 0 per token).
* gate = sigmoid(z), one per head problem.
* Optional correlated writes: a fraction of the tokens in each frame copy
  another token's raw key plus 1e-3 * N(0, 1) noise before normalisation
  (spatially correlated patches, the case Eq. A.3 discusses), and a fraction
  of the write strengths are exactly zero.

Every head problem draws from its own counter-based stream
``numpy.random.default_rng([seed, head])`` (PCG64 seeded by a sequence), so
any subset of heads can be regenerated without drawing the rest; the gates
come from ``default_rng([seed, H_total])``.  Draw order inside a head: q, k,
v (float32 normals), beta logits, then the optional zero mask and duplicate
picks.  q, k, v are rounded to the storage type with round-to-nearest-even
(bf16) or kept as float32.

For the full operator: channel decays alpha uniform in [0.6, 1], a text
state S_T with N(0, 1) / 2 entries and output gates sigmoid(N(0, 1)) per
token and channel, each from its own salted stream.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Workload:
    """Shape, storage type and value distribution of one synthetic workload."""

    name: str
    B: int
    H: int
    F: int
    N: int
    d_k: int
    d_v: int
    dtype: str  # "f32" or "bf16" storage for q, k, v, out
    seed: int
    beta_sigma: float = 1.0
    beta_zero_frac: float = 0.0
    dup_frac: float = 0.0
    grid: tuple | None = None  # latent grid (rows, cols) of the N tokens, when it has one
    description: str = field(default="", compare=False)

    @property
    def heads(self) -> int:
        """Number of independent head problems (batch folded into heads)."""
        return self.B * self.H

    @property
    def tokens(self) -> int:
        """Video tokens per call, B * F * N (heads share tokens)."""
        return self.B * self.F * self.N

    @property
    def frame_heads(self) -> int:
        return self.B * self.H * self.F


# The five workloads the operator is measured and checked on.  The 768p
# long clip is one GPU's head shard: 48x80 latent grid, 36 interior frames.
WORKLOADS = {
    "tiny_f32": Workload("tiny_f32", 1, 2, 4, 64, 64, 64, "f32", 0, grid=(8, 8),
                         description="8x8 grid, 4 frames, fp32 storage"),
    "small_bf16": Workload("small_bf16", 1, 8, 16, 1024, 128, 128, "bf16", 1, grid=(32, 32),
                           description="32x32 grid, 16 frames"),
    "480p_bf16": Workload("480p_bf16", 1, 24, 21, 1560, 128, 128, "bf16", 2, grid=(30, 52),
                          description="30x52 latent grid, 21 frames"),
    "768p_bf16": Workload("768p_bf16", 1, 16, 36, 3840, 128, 128, "bf16", 3, grid=(48, 80),
                          description="48x80 latent grid, 36 frames, 16-head shard"),
    "ragged_bf16": Workload("ragged_bf16", 2, 12, 64, 2025, 64, 128, "bf16", 7, grid=(45, 45),
                            beta_sigma=2.0, beta_zero_frac=0.25, dup_frac=0.10,
                            description="45x45 grid, 64 frames, zero and near-duplicate writes"),
}


# The paper's own shard: 56 heads over 8 GPUs (7 per GPU), a 48x84 latent
# grid and 102 latent frames, 100 of them interior; d = 128 (the head width
# is not stated).  Timed and checked with the full operator's options.
PAPER_SHARD = Workload("paper_shard_bf16", 1, 7, 100, 4032, 128, 128, "bf16", 11, grid=(48, 84),
                       description="48x84 latent grid, 100 interior frames, 7-head shard")


def custom(name: str, B: int, H: int, F: int, N: int, d_k: int, d_v: int,
           dtype: str = "bf16", seed: int = 0, **kw) -> Workload:
    """A workload with arbitrary shape (property sweeps, edge cases)."""
    return Workload(name, B, H, F, N, d_k, d_v, dtype, seed, **kw)


# ----------------------------------------------------------------------------
# bf16 storage helpers (bit manipulation only)
# ----------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 with round-to-nearest-even; return the
    16-bit patterns as uint16.  Inputs are finite."""
    u = np.array(x, dtype=np.float32, copy=True).view(np.uint32)
    bias = u >> np.uint32(16)
    bias &= np.uint32(1)
    bias += np.uint32(0x7FFF)
    u += bias
    u >>= np.uint32(16)
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Expand bf16 bit patterns (uint16) to the float32 values they encode."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


def _sigmoid(z: np.ndarray) -> np.ndarray:
    return 1.0 / (1.0 + np.exp(-z))


def _l2_normalise(x32: np.ndarray) -> np.ndarray:
    """Per-token L2 normalisation in float32 (the stored values are what both
    the oracle and the GPU consume, so this precision is immaterial)."""
    x32 /= np.sqrt(np.einsum("...i,...i->...", x32, x32))[..., None]
    return x32


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    """Cast to the storage type: float32 array, or uint16 bf16 patterns."""
    x32 = x.astype(np.float32, copy=False)
    if dtype == "f32":
        return x32
    if dtype == "bf16":
        return f32_to_bf16_bits(x32)
    raise ValueError(f"unknown storage dtype {dtype!r}")


def head_inputs(w: Workload, hb: int) -> dict:
    """Inputs of head problem ``hb`` in storage form.

    Returns q [F,N,d_k], k [F,N,d_k], v [F,N,d_v] (float32, or uint16 bf16
    patterns) and beta [F,N] float32.
    """
    if not 0 <= hb < w.heads:
        raise IndexError(hb)
    rng = np.random.default_rng([w.seed, hb])
    F, N = w.F, w.N
    q = rng.standard_normal((F, N, w.d_k), dtype=np.float32)
    k = rng.standard_normal((F, N, w.d_k), dtype=np.float32)
    v = rng.standard_normal((F, N, w.d_v), dtype=np.float32)
    z = rng.standard_normal((F, N))
    beta = _sigmoid(w.beta_sigma * z)
    if w.beta_zero_frac > 0:
        beta[rng.random((F, N)) < w.beta_zero_frac] = 0.0
    if w.dup_frac > 0 and N > 1:
        n_dup = int(round(w.dup_frac * N))
        n_dup = min(n_dup, N - 1)
        for t in range(F):
            perm = rng.permutation(N)
            dst, pool = perm[:n_dup], perm[n_dup:]
            src = pool[rng.integers(0, pool.size, n_dup)]
            noise = rng.standard_normal((n_dup, w.d_k), dtype=np.float32)
            k[t, dst] = k[t, src] + np.float32(1e-3) * noise
    return {
        "q": _store(_l2_normalise(q), w.dtype),
        "k": _store(_l2_normalise(k), w.dtype),
        "v": _store(v, w.dtype),
        "beta": beta.astype(np.float32),
    }


def gates(w: Workload) -> np.ndarray:
    """Per-head output gates [H_total], float32 in (0, 1)."""
    rng = np.random.default_rng([w.seed, w.heads])
    return _sigmoid(rng.standard_normal(w.heads)).astype(np.float32)


def make_inputs(w: Workload, heads=None) -> dict:
    """Stack the inputs of the given heads (default: all).

    q, k, v are ``[len(heads)][F][N][d]`` in storage form, beta is
    ``[len(heads)][F][N]`` float32, gate is ``[len(heads)]`` float32.
    """
    hs = range(w.heads) if heads is None else list(heads)
    st = np.float32 if w.dtype == "f32" else np.uint16
    n = len(hs)
    out = {
        "q": np.empty((n, w.F, w.N, w.d_k), st),
        "k": np.empty((n, w.F, w.N, w.d_k), st),
        "v": np.empty((n, w.F, w.N, w.d_v), st),
        "beta": np.empty((n, w.F, w.N), np.float32),
    }
    def fill(i_hb):
        i, hb = i_hb
        hi = head_inputs(w, hb)
        for key in out:
            out[key][i] = hi[key]

    workers = min(n, max(1, min(16, os.cpu_count() or 1)))
    if workers > 1:
        with ThreadPoolExecutor(max_workers=workers) as ex:
            list(ex.map(fill, enumerate(hs)))
    else:
        for item in enumerate(hs):
            fill(item)
    out["gate"] = gates(w)[list(hs)]
    return out


def make_decay(w: Workload, low: float = 0.6, salt: int = 101) -> np.ndarray:
    """Channel decays alpha [H_total][F][d_k] float32, uniform in [low, 1]
    (Proposition 1's range, 0 <= alpha <= 1), from default_rng([seed, salt])."""
    rng = np.random.default_rng([w.seed, salt])
    a = low + (1.0 - low) * rng.random((w.heads, w.F, w.d_k))
    return a.astype(np.float32)


def make_text_state(w: Workload, scale: float = 0.5, salt: int = 102) -> np.ndarray:
    """A text state S_T [H_total][d_v][d_k] float32, scale * N(0, 1), from
    default_rng([seed, salt])."""
    rng = np.random.default_rng([w.seed, salt])
    return (scale * rng.standard_normal((w.heads, w.d_v, w.d_k))).astype(np.float32)


def make_token_gates(w: Workload, salt: int = 103) -> np.ndarray:
    """Content-dependent output gates G^L [H_total][F][N][d_v] = sigmoid(z),
    z ~ N(0, 1), one per token and value channel, in the workload's storage
    type (float32, or bf16 bit patterns), from default_rng([seed, salt])."""
    rng = np.random.default_rng([w.seed, salt])
    z = rng.standard_normal((w.heads, w.F, w.N, w.d_v), dtype=np.float32)
    return _store(_sigmoid(z).astype(np.float32), w.dtype)


def as_float64(x: np.ndarray, dtype: str) -> np.ndarray:
    """The exact values held by a storage array, in float64."""
    if dtype == "bf16":
        return bf16_bits_to_f32(x).astype(np.float64)
    return np.asarray(x, dtype=np.float64)


def make_prep_inputs(B: int, F: int, grid, H: int, d_k: int, d_v: int, seed: int = 0) -> dict:
    """Synthetic inputs of the linear branch's feature map (VDA-Prep):
    token-major projections q, k [B, F, gh*gw, H*d_k], v [B, F, gh*gw,
    H*d_v] ~ N(0, 1), rounded to bf16 (returned as the bf16 bit patterns,
    uint16); depthwise filters, fp32: spatial [H*d, 25] ~ N(0, 1/25) and
    temporal [H*d, 5] ~ N(0, 1/5) for K and for V (so a filtered value has
    about unit variance), from ``default_rng([seed, 1000 + b])`` per clip and
    ``default_rng([seed, 999])`` for the filters."""
    gh, gw = grid
    N = gh * gw
    out = {n: np.empty((B, F, N, H * d), np.uint16)
           for n, d in (("q", d_k), ("k", d_k), ("v", d_v))}
    for b in range(B):
        rng = np.random.default_rng([seed, 1000 + b])
        for n, d in (("q", d_k), ("k", d_k), ("v", d_v)):
            out[n][b] = f32_to_bf16_bits(rng.standard_normal((F, N, H * d), dtype=np.float32))
    rng = np.random.default_rng([seed, 999])
    for n, d in (("k", d_k), ("v", d_v)):
        out[f"w{n}_spatial"] = (rng.standard_normal((H * d, 25)) / 5.0).astype(np.float32)
        out[f"w{n}_temporal"] = (rng.standard_normal((H * d, 5)) / np.sqrt(5.0)).astype(np.float32)
    return out
