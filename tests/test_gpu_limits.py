"""GPU parity at the largest sizes the library accepts.  Byte offsets within
one frame of one head (N * d * 4) and within one head's per-frame matrices
(F * d * d * 4) are 32-bit, so the limits are N <= (2^31 - 1) / (4 d) tokens
per frame and F <= (2^31 - 1) / (4 d^2) frames per head; each case below
sits exactly at one of them, at d = 128.  The oracle evaluates sampled
outputs (the states still come from every frame and every token)."""
import numpy as np
import pytest

from paper_2609_20744_amd import inputs as I
from vda_testutil import (device_inputs, from_device, oracle_inputs, oracle_sampled, rel_max_err,
                          tol_for)

pytestmark = pytest.mark.gpu

LIMIT = 2**31 - 1


@pytest.fixture(scope="module")
def V():
    import torch
    assert torch.cuda.is_available(), "the gpu tests need an MI355X"
    from paper_2609_20744_amd import vda
    return vda


def _log(msg):
    print(msg, flush=True)


def _check(V, w, toks, frames=None):
    import torch
    _log(f"  inputs {w.name}: H={w.heads} F={w.F} N={w.N} d={w.d_k} {w.dtype}")
    x = I.make_inputs(w)
    d = device_inputs(w, x)
    y = V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"])
    torch.cuda.synchronize()
    _log("  forward done; oracle")
    xo = oracle_inputs(w, x)
    ref, fr, tk = oracle_sampled(w, xo, 0, toks)
    if frames is not None:  # keep the listed frames only
        keep = np.isin(fr, frames)
        ref, fr, tk = ref[keep], fr[keep], tk[keep]
    got = from_device(y[0][torch.as_tensor(fr, device=y.device), torch.as_tensor(tk, device=y.device)])
    err = rel_max_err(got, ref)
    _log(f"  rel max-norm error {err:.3e} over {len(fr)} outputs")
    assert err <= tol_for(w), err


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_max_frames_per_head(V, dtype):
    """F = 32767 frames of one d = 128 head: its per-frame matrices (A, Inv, B,
    both states) span 2^31 - 64 KiB bytes each."""
    d = 128
    F = LIMIT // (4 * d * d)
    assert F * 4 * d * d <= LIMIT < (F + 1) * 4 * d * d
    _log(f"max frames per head: F={F} dtype={dtype}")
    w = I.custom("max_frames", 1, 1, F, 16, d, d, dtype, seed=61)
    rng = np.random.default_rng(61)
    frames = np.unique(np.concatenate([[0, 1, F // 2, F - 2, F - 1], rng.integers(0, F, 40)]))
    _check(V, w, toks=[0, 7, 15], frames=frames)


def test_max_tokens_per_frame(V):
    """N = 4194303 tokens per frame (one frame of q, k, v or out at d = 128
    spans 2^31 - 512 bytes in fp32), two frames of one head, bf16 storage."""
    d = 128
    N = LIMIT // (4 * d)
    assert N * 4 * d <= LIMIT < (N + 1) * 4 * d
    _log(f"max tokens per frame: N={N}")
    w = I.custom("max_tokens", 1, 1, 2, N, d, d, "bf16", seed=62)
    rng = np.random.default_rng(62)
    toks = sorted({0, 1, 15, 16, N // 2, N - 17, N - 16, N - 1} |
                  set(int(t) for t in rng.integers(0, N, 40)))
    _check(V, w, toks=toks)
