"""Helpers shared by the GPU parity tests: host <-> device transfer of the
seeded inputs, the error metric, and oracle evaluation at sampled positions."""
from __future__ import annotations

import numpy as np

import oracle.vda_oracle as O
from paper_2609_20744_amd import inputs as I

# Rel. max-norm tolerances of the parity bar: fp32 storage path, bf16 storage path.
TOL_F32 = 1e-4
TOL_BF16 = 2e-2


def tol_for(w) -> float:
    return TOL_F32 if w.dtype == "f32" else TOL_BF16


def to_device(x: np.ndarray, dtype: str):
    import torch
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def from_device(t) -> np.ndarray:
    """Device tensor -> float64 numpy array of the exact stored values."""
    import torch
    if t.dtype == torch.bfloat16:
        return I.bf16_bits_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
    return t.double().cpu().numpy()


def device_inputs(w, x: dict) -> dict:
    return {"q": to_device(x["q"], w.dtype), "k": to_device(x["k"], w.dtype),
            "v": to_device(x["v"], w.dtype), "beta": to_device(x["beta"], "f32"),
            "gate": to_device(x["gate"], "f32")}


def oracle_inputs(w, x: dict) -> dict:
    return {"q": I.as_float64(x["q"], w.dtype), "k": I.as_float64(x["k"], w.dtype),
            "v": I.as_float64(x["v"], w.dtype), "beta": x["beta"].astype(np.float64),
            "gate": x["gate"].astype(np.float64)}


def rel_max_err(y: np.ndarray, ref: np.ndarray) -> float:
    """||y - ref||_inf / ||ref||_inf (0 when both are zero)."""
    den = float(np.max(np.abs(ref))) if ref.size else 0.0
    num = float(np.max(np.abs(y - ref))) if ref.size else 0.0
    if den == 0.0:
        return num
    return num / den


def fold_partials(P, count: int, tail_frames: int, splits: int):
    """Sum each frame's token-range partials of a [partials, ...] tensor
    (the statistics stage's output under the split plan (tail_frames,
    splits)) into [count, ...]: partial s of split frame i is entry
    count + (s - 1) * tail_frames + (i - (count - tail_frames))."""
    out = P[:count].clone()
    if splits > 1:
        first = count - tail_frames
        for s in range(1, splits):
            out[first:] += P[count + (s - 1) * tail_frames:count + s * tail_frames]
    return out


class ErrorAccumulator:
    """The rel. max-norm error ||y - ref||_inf / ||ref||_inf of a whole
    output tensor [H][F][N][d_v] fed in head groups, with the max-abs error
    and the (head, frame, token) where it occurs."""

    def __init__(self):
        self.num = 0.0
        self.den = 0.0
        self.worst = None

    def add(self, y: np.ndarray, ref: np.ndarray, h0: int):
        d = np.abs(y - ref)
        if d.size:
            i = np.unravel_index(int(np.argmax(d)), d.shape)
            if self.worst is None or d[i] > self.num:
                self.num = float(d[i])
                self.worst = (h0 + int(i[0]), int(i[1]), int(i[2]))
            self.den = max(self.den, float(np.max(np.abs(ref))))

    def rel_max_err(self) -> float:
        return self.num / self.den if self.den > 0 else self.num

    def report(self) -> str:
        return (f"rel max-norm error {self.rel_max_err():.3e}, max abs error {self.num:.3e} "
                f"(|ref|_inf {self.den:.3e}), worst (head, frame, token) {self.worst}")


#: (case, report) of the whole-output parity checks, printed at the end of
#: the session so the margins appear in the test log.
ERROR_RECORDS: list[tuple[str, str]] = []


def record_error(case: str, acc: ErrorAccumulator):
    ERROR_RECORDS.append((case, acc.report()))


def sample_positions(w, rng, per_frame: int):
    """Token indices per frame: the first, the last, the last full 16-token
    group boundary and random ones."""
    N = w.N
    base = {0, N - 1, max(0, (N // 16) * 16 - 1), min(N - 1, (N // 16) * 16)}
    extra = rng.choice(N, size=min(N, per_frame), replace=False)
    toks = sorted(base | set(int(t) for t in extra))
    return toks


def oracle_sampled(w, xo: dict, h_local: int, toks) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Oracle outputs of head ``h_local`` (index into xo) at every frame x toks."""
    F = w.F
    frames = np.repeat(np.arange(F), len(toks))
    tk = np.tile(np.asarray(toks), F)
    y = O.head_forward_sampled(xo["q"][h_local], xo["k"][h_local], xo["v"][h_local],
                               xo["beta"][h_local], float(xo["gate"][h_local]), frames, tk)
    return y, frames, tk


def operand_tile_index(dk: int):
    """(k, n) of every bf16 position of one plane of the split-bf16 operand
    tile layout (include/vda.h): plane position i holds element [k[i]][n[i]]."""
    NB, KB = dk // 16, dk // 32
    nb, ks, lane, e = np.meshgrid(np.arange(NB), np.arange(KB), np.arange(64), np.arange(8),
                                  indexing="ij")
    k = 32 * ks + 4 * (lane // 16) + np.where(e < 4, e, 12 + e)
    n = 16 * nb + lane % 16
    return k.ravel(), n.ravel()


def to_operand_tiles(X: np.ndarray):
    """fp32 matrices [..., d_k, d_k] -> torch bfloat16 [..., 2, d_k*d_k] in
    the tile layout: plane 0 = bf16(x), plane 1 = bf16(x - hi) (torch's
    round-to-nearest-even casts, on the CPU)."""
    import torch
    dk = X.shape[-1]
    k, n = operand_tile_index(dk)
    vals = torch.from_numpy(np.ascontiguousarray(X[..., k, n], dtype=np.float32))
    hi = vals.to(torch.bfloat16)
    lo = (vals - hi.float()).to(torch.bfloat16)
    return torch.stack([hi, lo], dim=-2).contiguous()


def from_operand_tiles(T, dk: int) -> np.ndarray:
    """Tile layout [..., 2, d_k*d_k] (torch bfloat16, any device) -> float64
    matrices hi + lo [..., d_k, d_k]."""
    import torch
    t = T.cpu().to(torch.float64).numpy()
    vals = t[..., 0, :] + t[..., 1, :]
    k, n = operand_tile_index(dk)
    X = np.zeros(t.shape[:-2] + (dk, dk))
    X[..., k, n] = vals
    return X
