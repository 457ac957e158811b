"""GPU parity of the full operator (vda_forward_ex): channel decay, local
window with the decay bridge, text state, and the frozen-state rule, against
the fp64 oracle's *_ex functions, through the C ABI.  Same bar as the core:
rel. max-norm error <= 1e-4 (fp32 storage), <= 2e-2 (bf16 storage)."""
import numpy as np
import pytest

import oracle.vda_oracle as O
from paper_2609_20744_amd import inputs as I
from vda_testutil import (device_inputs, from_device, oracle_inputs, rel_max_err, to_device,
                          tol_for)

pytestmark = pytest.mark.gpu

PAPER_WINDOW = (5, 1, 1)   # chunks of five frames, radius one, one leading anchor


@pytest.fixture(scope="module")
def V():
    import torch
    assert torch.cuda.is_available(), "the gpu tests need an MI355X"
    from paper_2609_20744_amd import vda
    return vda


def _log(msg):
    print(msg, flush=True)


def _run(V, w, x, alpha=None, S_T=None, window=None, rule="joint"):
    import torch
    d = device_inputs(w, x)
    a_dev = None if alpha is None else to_device(alpha, "f32")
    t_dev = None if S_T is None else to_device(S_T, "f32")
    y = V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"], alpha=a_dev, text_state=t_dev,
                  window=window, rule=rule)
    torch.cuda.synchronize()
    return from_device(y)


def _oracle(w, x, alpha=None, S_T=None, window=None, rule="joint"):
    xo = oracle_inputs(w, x)
    chunk, radius, offset = window or (1, 0, 0)
    return O.vda_forward_ex(xo["q"], xo["k"], xo["v"], xo["beta"], xo["gate"],
                            None if alpha is None else alpha.astype(np.float64),
                            None if S_T is None else S_T.astype(np.float64),
                            chunk, radius, offset, rule)


CASES = [
    # name, (alpha, text state, window, rule)
    ("decay", (True, False, None, "joint")),
    ("text_state", (False, True, None, "joint")),
    ("window", (False, False, PAPER_WINDOW, "joint")),
    ("all", (True, True, PAPER_WINDOW, "joint")),
    ("frozen", (False, False, None, "frozen")),
    ("frozen_all", (True, True, PAPER_WINDOW, "frozen")),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("name,case", CASES, ids=[c[0] for c in CASES])
def test_full_operator(V, dtype, name, case):
    has_a, has_t, window, rule = case
    _log(f"full operator {name} dtype={dtype}")
    w = I.custom("ex", 1, 2, 12, 150, 64, 64, dtype, seed=41)
    x = I.make_inputs(w)
    alpha = I.make_decay(w) if has_a else None
    S_T = I.make_text_state(w) if has_t else None
    got = _run(V, w, x, alpha, S_T, window, rule)
    exp = _oracle(w, x, alpha, S_T, window, rule)
    err = rel_max_err(got, exp)
    _log(f"  rel err {err:.2e}")
    assert err <= tol_for(w), err


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", [(32, 128), (128, 32), (128, 128), (16, 64), (64, 16)])
def test_full_operator_dims(V, dtype, dk, dv):
    _log(f"full operator dims dtype={dtype} dk={dk} dv={dv}")
    w = I.custom("ex_dims", 1, 2, 9, 100, dk, dv, dtype, seed=dk + 7 * dv)
    x = I.make_inputs(w)
    alpha, S_T = I.make_decay(w), I.make_text_state(w)
    for rule in ("joint", "frozen"):
        got = _run(V, w, x, alpha, S_T, (3, 1, 0), rule)
        exp = _oracle(w, x, alpha, S_T, (3, 1, 0), rule)
        err = rel_max_err(got, exp)
        assert err <= tol_for(w), (rule, err)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_defaults_equal_core(V, dtype):
    """vda_forward_ex with default options is vda_forward, bit for bit."""
    import torch
    w = I.custom("ex_core", 1, 3, 5, 200, 64, 128, dtype, seed=43)
    d = device_inputs(w, I.make_inputs(w))
    y = V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"])
    ye = V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"], window=(1, 0, 0))
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16 if dtype == "bf16" else torch.int32),
                       ye.view(torch.int16 if dtype == "bf16" else torch.int32))


def test_whole_clip_window_reads_text_state(V):
    """A window covering the whole clip: each frame reads only the decayed
    text state (Eq. A.4, both sides at their initial states)."""
    w = I.custom("ex_clip", 1, 2, 6, 80, 64, 64, "f32", seed=44)
    x = I.make_inputs(w)
    alpha, S_T = I.make_decay(w), I.make_text_state(w)
    got = _run(V, w, x, alpha, S_T, (6, 0, 0))
    exp = _oracle(w, x, alpha, S_T, (6, 0, 0))
    assert rel_max_err(got, exp) <= tol_for(w)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ragged_and_single_frame(V, dtype):
    for F, N in ((1, 70), (2, 17), (7, 333)):
        _log(f"full operator ragged F={F} N={N} dtype={dtype}")
        w = I.custom("ex_ragged", 1, 2, F, N, 64, 128, dtype, seed=F * 1000 + N)
        x = I.make_inputs(w)
        alpha, S_T = I.make_decay(w), I.make_text_state(w)
        for rule in ("joint", "frozen"):
            got = _run(V, w, x, alpha, S_T, PAPER_WINDOW, rule)
            exp = _oracle(w, x, alpha, S_T, PAPER_WINDOW, rule)
            assert rel_max_err(got, exp) <= tol_for(w), (F, N, rule)


def test_full_size_sampled(V):
    """A 768p-shaped head pair (36 frames x 3840 tokens, d = 128) with every
    option, at sampled positions: the states come from all frames."""
    w = I.custom("ex_768p", 1, 2, 36, 3840, 128, 128, "bf16", seed=45)
    x = I.make_inputs(w)
    alpha, S_T = I.make_decay(w), I.make_text_state(w)
    got = _run(V, w, x, alpha, S_T, PAPER_WINDOW)
    xo = oracle_inputs(w, x)
    windows = O.local_windows(w.F, *PAPER_WINDOW)
    rng = np.random.default_rng(7)
    for h in range(w.heads):
        As, Bs = O.head_statistics(xo["k"][h], xo["v"][h], xo["beta"][h])
        St = O.gathered_states_ex(As, Bs, S_T[h].astype(np.float64),
                                  alpha[h].astype(np.float64), windows)
        frames = rng.integers(0, w.F, 64)
        toks = rng.integers(0, w.N, 64)
        o = np.einsum("sjc,sc->sj", St[frames], xo["q"][h][frames, toks])
        exp = O.rmsnorm_gate(o, float(xo["gate"][h]))
        err = rel_max_err(got[h][frames, toks], exp)
        assert err <= tol_for(w), (h, err)
