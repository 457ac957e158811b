"""GPU parity of vda_text_state: the prompt state S_T (Sec. 2.2, Eq. 1b)
formed as one leading frame from the zero state, against the oracle's
text_state, and the forward pass started from it.  The prompt tokens are
drawn like one frame of the workloads (unit keys, N(0, 1) values,
sigmoid write strengths), at prompt lengths from one token to past the
statistics kernel's split point."""
import numpy as np
import pytest

import oracle.vda_oracle as O
from paper_2609_20744_amd import inputs as I
from vda_testutil import from_device, rel_max_err, to_device, TOL_BF16, TOL_F32

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def V():
    import torch
    assert torch.cuda.is_available(), "the gpu tests need an MI355X"
    from paper_2609_20744_amd import vda
    return vda


def _prompt(H, L, dk, dv, dtype, seed):
    """One frame of L tokens per head, as [H][L][d] device tensors and the
    oracle's float64 copies."""
    w = I.custom("prompt", 1, H, 1, L, dk, dv, dtype, seed=seed)
    x = I.make_inputs(w)
    k, v, beta = x["k"][:, 0], x["v"][:, 0], x["beta"][:, 0]
    dev = (to_device(k, dtype), to_device(v, dtype), to_device(beta, "f32"))
    ref = (I.as_float64(k, dtype), I.as_float64(v, dtype), beta.astype(np.float64))
    return dev, ref


CASES = [  # H, L, d_k, d_v
    (3, 1, 128, 128),
    (4, 77, 128, 128),
    (16, 226, 128, 128),
    (2, 1000, 128, 128),   # long enough for the statistics split
    (5, 130, 64, 32),
    (2, 65, 32, 64),
    (3, 40, 16, 16),       # zero-padded narrow heads
    (2, 50, 16, 64),
]


@pytest.mark.parametrize("rule", ["joint", "frozen"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("H,L,dk,dv", CASES, ids=[f"H{c[0]}_L{c[1]}_{c[2]}x{c[3]}" for c in CASES])
def test_text_state_matches_oracle(V, H, L, dk, dv, dtype, rule):
    import torch
    print(f"text state H={H} L={L} d={dk}x{dv} {dtype} {rule}", flush=True)
    (k, v, beta), (k64, v64, b64) = _prompt(H, L, dk, dv, dtype, seed=300 + L)
    S = V.text_state(k, v, beta, rule=rule)
    torch.cuda.synchronize()
    ref = O.text_state(k64, v64, b64, rule)
    err = rel_max_err(from_device(S), ref)
    # The fp32 product and inverse; bf16 storage also rounds beta * k.
    assert err <= (TOL_F32 if dtype == "f32" else TOL_BF16), err


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_forward_from_prompt_state(V, dtype):
    """The whole prompt path: S_T from the prompt tokens, then the full
    operator started from S_T / 2, against the oracle end to end."""
    import torch
    H, F, N, L, d = 2, 5, 96, 120, 64
    print(f"forward from prompt state {dtype}", flush=True)
    (k, v, beta), (k64, v64, b64) = _prompt(H, L, d, d, dtype, seed=331)
    S = V.text_state(k, v, beta)
    w = I.custom("clip", 1, H, F, N, d, d, dtype, seed=332)
    x = I.make_inputs(w)
    dq, dk_, dv_ = (to_device(x[n], dtype) for n in ("q", "k", "v"))
    y = V.forward(dq, dk_, dv_, to_device(x["beta"], "f32"), to_device(x["gate"], "f32"),
                  text_state=S, window=(2, 1, 1))
    torch.cuda.synchronize()
    S_T = O.text_state(k64, v64, b64)
    ref = O.vda_forward_ex(I.as_float64(x["q"], dtype), I.as_float64(x["k"], dtype),
                           I.as_float64(x["v"], dtype), x["beta"].astype(np.float64),
                           x["gate"].astype(np.float64), S_T=S_T, chunk=2, radius=1, offset=1)
    err = rel_max_err(from_device(y), ref)
    assert err <= (TOL_F32 if dtype == "f32" else TOL_BF16), err


def test_text_state_argument_errors(V):
    import torch
    (k, v, beta), _ = _prompt(2, 10, 32, 32, "f32", seed=340)
    with pytest.raises(ValueError):
        V.text_state(k, v, beta, rule="other")
    with pytest.raises(ValueError):
        V.text_state(k, v[:, :9].contiguous(), beta)
    out = torch.empty(2, 32, 32, device=k.device)
    V.text_state(k, v, beta, out=out)
    torch.cuda.synchronize()
    assert torch.isfinite(out).all()
