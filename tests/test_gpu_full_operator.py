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


def _run(V, w, x, alpha=None, S_T=None, window=None, rule="joint", G=None):
    import torch
    d = device_inputs(w, x)
    a_dev = None if alpha is None else to_device(alpha, "f32")
    t_dev = None if S_T is None else to_device(S_T, "f32")
    g_dev = None if G is None else to_device(G, w.dtype)
    y = V.forward(d["q"], d["k"], d["v"], d["beta"], None if G is not None else d["gate"],
                  alpha=a_dev, text_state=t_dev, window=window, rule=rule, gate_tokens=g_dev)
    torch.cuda.synchronize()
    return from_device(y)


def _oracle(w, x, alpha=None, S_T=None, window=None, rule="joint", G=None):
    xo = oracle_inputs(w, x)
    chunk, radius, offset = window or (1, 0, 0)
    return O.vda_forward_ex(xo["q"], xo["k"], xo["v"], xo["beta"], xo["gate"],
                            None if alpha is None else alpha.astype(np.float64),
                            None if S_T is None else S_T.astype(np.float64),
                            chunk, radius, offset, rule,
                            gate_tokens=None if G is None else I.as_float64(G, w.dtype))


CASES = [
    # name, (alpha, text state, window, rule, output gate per token)
    ("decay", (True, False, None, "joint", False)),
    ("text_state", (False, True, None, "joint", False)),
    ("window", (False, False, PAPER_WINDOW, "joint", False)),
    ("all", (True, True, PAPER_WINDOW, "joint", False)),
    ("frozen", (False, False, None, "frozen", False)),
    ("frozen_all", (True, True, PAPER_WINDOW, "frozen", False)),
    ("token_gate", (False, False, None, "joint", True)),
    ("all_token_gate", (True, True, PAPER_WINDOW, "joint", True)),
    ("frozen_all_token_gate", (True, True, PAPER_WINDOW, "frozen", True)),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("name,case", CASES, ids=[c[0] for c in CASES])
def test_full_operator(V, dtype, name, case):
    has_a, has_t, window, rule, has_g = case
    _log(f"full operator {name} dtype={dtype}")
    w = I.custom("ex", 1, 2, 12, 150, 64, 64, dtype, seed=41)
    x = I.make_inputs(w)
    alpha = I.make_decay(w) if has_a else None
    S_T = I.make_text_state(w) if has_t else None
    G = I.make_token_gates(w) if has_g else None
    got = _run(V, w, x, alpha, S_T, window, rule, G)
    exp = _oracle(w, x, alpha, S_T, window, rule, G)
    err = rel_max_err(got, exp)
    _log(f"  rel err {err:.2e}")
    assert err <= tol_for(w), err


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", [(32, 128), (128, 32), (128, 128), (16, 64), (64, 16)])
def test_full_operator_dims(V, dtype, dk, dv):
    _log(f"full operator dims dtype={dtype} dk={dk} dv={dv}")
    w = I.custom("ex_dims", 1, 2, 9, 100, dk, dv, dtype, seed=dk + 7 * dv)
    x = I.make_inputs(w)
    alpha, S_T, G = I.make_decay(w), I.make_text_state(w), I.make_token_gates(w)
    for rule in ("joint", "frozen"):
        for gt in (None, G):
            got = _run(V, w, x, alpha, S_T, (3, 1, 0), rule, gt)
            exp = _oracle(w, x, alpha, S_T, (3, 1, 0), rule, gt)
            err = rel_max_err(got, exp)
            assert err <= tol_for(w), (rule, gt is not None, err)


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


@pytest.mark.parametrize("rule", ["joint", "frozen"])
def test_split_frames(V, rule):
    """Frames whose statistics are split into token ranges (12 frames, a
    partial round, 2048 tokens each), with decay, text state and the paper's
    window: the joint rule's inverse and the frozen rule's map tiles both sum
    the partials, and both fold B's."""
    import torch
    _log(f"full operator split frames rule={rule}")
    w = I.custom("ex_split", 1, 2, 6, 2048, 128, 128, "bf16", seed=46)
    tail, splits = V.default_split_plan(w.F, w.N, w.heads, w.d_k, w.d_v, False)
    assert splits > 1 and tail > 0, (tail, splits)
    x = I.make_inputs(w)
    alpha, S_T = I.make_decay(w), I.make_text_state(w)
    got = _run(V, w, x, alpha, S_T, PAPER_WINDOW, rule)
    exp = _oracle(w, x, alpha, S_T, PAPER_WINDOW, rule)
    err = rel_max_err(got, exp)
    _log(f"  rel err {err:.2e} (plan {tail} x {splits})")
    assert err <= tol_for(w), err


@pytest.mark.parametrize("rule", ["joint", "frozen"])
def test_full_size_sampled(V, rule):
    """A 768p-shaped head pair (36 frames x 3840 tokens, d = 128) with every
    option, at sampled positions: the states come from all frames."""
    _log(f"full operator 768p-shaped sampled rule={rule}")
    w = I.custom("ex_768p", 1, 2, 36, 3840, 128, 128, "bf16", seed=45)
    x = I.make_inputs(w)
    alpha, S_T = I.make_decay(w), I.make_text_state(w)
    got = _run(V, w, x, alpha, S_T, PAPER_WINDOW, rule)
    xo = oracle_inputs(w, x)
    windows = O.local_windows(w.F, *PAPER_WINDOW)
    rng = np.random.default_rng(7)
    for h in range(w.heads):
        As, Bs = O.head_statistics(xo["k"][h], xo["v"][h], xo["beta"][h])
        St = O.gathered_states_ex(As, Bs, S_T[h].astype(np.float64),
                                  alpha[h].astype(np.float64), windows, rule=rule,
                                  U=w.N if rule == "frozen" else None)
        frames = rng.integers(0, w.F, 64)
        toks = rng.integers(0, w.N, 64)
        o = np.einsum("sjc,sc->sj", St[frames], xo["q"][h][frames, toks])
        exp = O.rmsnorm_gate(o, float(xo["gate"][h]))
        err = rel_max_err(got[h][frames, toks], exp)
        assert err <= tol_for(w), (h, err)


@pytest.mark.parametrize("dk,dv", [(32, 64), (64, 128), (128, 32), (128, 128)])
def test_chunked_scan_stage(V, dk, dv):
    """Chunk-wise scans (Section 4) fed with the oracle's Inv_t (as split-bf16
    operand tiles) and B_t: the state entering every chunk, forward at its
    first frame and reverse at its last, equals the oracle's chunk-sequence
    scan, with and without decay and text state; other frames stay
    untouched."""
    import torch
    from vda_testutil import to_operand_tiles
    H, F = 3, 13
    _log(f"chunked scan dk={dk} dv={dv}")
    w = I.custom("chunked", 1, H, F, 40, dk, dv, "f32", seed=dk + dv)
    x = I.make_inputs(w)
    xo = oracle_inputs(w, x)
    alpha, S_T = I.make_decay(w), I.make_text_state(w)
    As = np.empty((H, F, dk, dk))
    Bs = np.empty((H, F, dv, dk))
    for h in range(H):
        As[h], Bs[h] = O.head_statistics(xo["k"][h], xo["v"][h], xo["beta"][h])
    Inv = np.linalg.inv(np.eye(dk) + As)
    T = to_operand_tiles(Inv).cuda()
    Bd = to_device(Bs.astype(np.float32), "f32")
    for chunk, offset in ((5, 1), (3, 0), (4, 3), (13, 0), (2, 1)):
        for decay, text in ((False, False), (True, True)):
            a_dev = to_device(alpha, "f32") if decay else None
            t_dev = to_device(S_T, "f32") if text else None
            Sf, Sr = V.state_scan_chunked(T, Bd, chunk, offset, alpha=a_dev, text_state=t_dev)
            torch.cuda.synchronize()
            Sf, Sr = Sf.double().cpu().numpy(), Sr.double().cpu().numpy()
            ranges = O.chunk_ranges(F, chunk, offset)
            firsts = {lo for lo, _ in ranges}
            lasts = {hi for _, hi in ranges}
            for h in range(H):
                S0 = 0.5 * S_T[h].astype(np.float64) if text else np.zeros((dv, dk))
                Pb, Rb = O.chunk_boundary_states(As[h], Bs[h], S0, chunk, offset,
                                                 alpha[h].astype(np.float64) if decay else None)
                for c, (lo, hi) in enumerate(ranges):
                    ef = rel_max_err(Sf[h, lo], Pb[c]) if np.any(Pb[c]) else np.max(np.abs(Sf[h, lo]))
                    er = rel_max_err(Sr[h, hi], Rb[c]) if np.any(Rb[c]) else np.max(np.abs(Sr[h, hi]))
                    assert ef < 1e-4 and er < 1e-4, (chunk, offset, decay, text, h, c, ef, er)
                for t in range(F):
                    if t not in firsts:
                        assert not np.any(Sf[h, t])
                    if t not in lasts:
                        assert not np.any(Sr[h, t])


def test_chunked_scan_many_workgroups(V):
    """Enough chunk chains that several workgroups run per compute unit and
    in more than one round: bitwise repeatable, and equal to the oracle's
    chunk-sequence scan at every boundary."""
    import torch
    from vda_testutil import to_operand_tiles
    H, F, dk, dv = 24, 36, 64, 128
    _log(f"chunked scan many workgroups H={H} F={F}")
    rng = np.random.default_rng(5)
    G = rng.standard_normal((H, F, dk, dk)) / np.sqrt(dk)
    A = G @ np.swapaxes(G, -1, -2)
    Inv = np.linalg.inv(np.eye(dk) + A)
    Bm = rng.standard_normal((H, F, dv, dk))
    alpha = rng.uniform(0.6, 1.0, (H, F, dk))
    T = to_operand_tiles(Inv).cuda()
    Bd, ad = to_device(Bm.astype(np.float32), "f32"), to_device(alpha.astype(np.float32), "f32")
    S1 = V.state_scan_chunked(T, Bd, 5, 1, alpha=ad)
    S2 = V.state_scan_chunked(T, Bd, 5, 1, alpha=ad)
    torch.cuda.synchronize()
    assert torch.equal(S1[0], S2[0]) and torch.equal(S1[1], S2[1])
    Sf, Sr = S1[0].double().cpu().numpy(), S1[1].double().cpu().numpy()
    a32 = alpha.astype(np.float32).astype(np.float64)
    B32 = Bm.astype(np.float32).astype(np.float64)
    for h in (0, H - 1):
        # the oracle's chunk maps from Inv_t directly: A with (I + A)^-1 = Inv
        A_h = np.linalg.inv(Inv[h]) - np.eye(dk)
        Pb, Rb = O.chunk_boundary_states(A_h, B32[h], np.zeros((dv, dk)), 5, 1, a32[h])
        for c, (lo, hi) in enumerate(O.chunk_ranges(F, 5, 1)):
            if c > 0:
                assert rel_max_err(Sf[h, lo], Pb[c]) < 1e-4, (h, c)
            if c < len(Pb) - 1:
                assert rel_max_err(Sr[h, hi], Rb[c]) < 1e-4, (h, c)


@pytest.mark.parametrize("H,dk,dv", [(7, 128, 128), (3, 64, 32)])
def test_full_operator_paper_shard(V, H, dk, dv):
    """The paper's own shard shape (a few heads per GPU, 100 interior frames,
    chunks of five after one anchor, decay and text state), where the
    forward takes the chunk-wise scans: whole output against the oracle.
    The token count is kept small (and ragged) so the oracle stays fast."""
    _log(f"full operator paper shard H={H} dk={dk} dv={dv}")
    w = I.custom("ex_shard", 1, H, 100, 37, dk, dv, "bf16", seed=46 + dk)
    x = I.make_inputs(w)
    alpha, S_T = I.make_decay(w), I.make_text_state(w)
    got = _run(V, w, x, alpha, S_T, PAPER_WINDOW)
    exp = _oracle(w, x, alpha, S_T, PAPER_WINDOW)
    err = rel_max_err(got, exp)
    _log(f"  rel err {err:.2e}")
    assert err <= tol_for(w), err


@pytest.mark.parametrize("rule", ["joint", "frozen"])
def test_full_operator_paper_shard_full_size(V, rule):
    """The paper's own shard at full size: 7 heads x 100 interior frames x
    4032 tokens (48 x 84 grid), d = 128, with decay, a text state and the
    paper's window, in the launch configuration bench.py times (the joint
    rule takes the chunk-wise scans here).  The oracle's states come from
    every frame of every head; outputs are compared at the first and last
    token of every frame and at 256 random (frame, token) positions per
    head."""
    import torch
    w = I.PAPER_SHARD
    _log(f"full operator paper shard full size rule={rule}: H={w.heads} F={w.F} N={w.N}")
    x = I.make_inputs(w)
    alpha, S_T = I.make_decay(w), I.make_text_state(w)
    d = device_inputs(w, x)
    y = V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"], alpha=to_device(alpha, "f32"),
                  text_state=to_device(S_T, "f32"), window=PAPER_WINDOW, rule=rule)
    torch.cuda.synchronize()
    del d
    windows = O.local_windows(w.F, *PAPER_WINDOW)
    rng = np.random.default_rng(11)
    worst = 0.0
    for h in range(w.heads):
        xo = oracle_inputs(w, I.make_inputs(w, heads=[h]))
        As, Bs = O.head_statistics(xo["k"][0], xo["v"][0], xo["beta"][0])
        St = O.gathered_states_ex(As, Bs, S_T[h].astype(np.float64),
                                  alpha[h].astype(np.float64), windows, rule=rule,
                                  U=w.N if rule == "frozen" else None)
        frames = np.concatenate([np.repeat(np.arange(w.F), 2), rng.integers(0, w.F, 256)])
        toks = np.concatenate([np.tile([0, w.N - 1], w.F), rng.integers(0, w.N, 256)])
        o = np.einsum("sjc,sc->sj", St[frames], xo["q"][0][frames, toks])
        exp = O.rmsnorm_gate(o, float(xo["gate"][0]))
        got = from_device(y[h][torch.from_numpy(frames).cuda(), torch.from_numpy(toks).cuda()])
        err = rel_max_err(got, exp)
        worst = max(worst, err)
        assert err <= tol_for(w), (h, err)
    _log(f"  rel max-norm error over the sampled outputs {worst:.3e}")


def _token_major(y, clips, heads):
    """Frame-major per head [clips*heads, F, N, d_v] rearranged to the
    token-major [clips, F, N, heads*d_v] (a layout change only)."""
    _, F, N, dv = y.shape
    return y.reshape(clips, heads, F, N, dv).permute(0, 2, 3, 1, 4).reshape(clips, F, N, heads * dv)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", [(64, 64), (128, 128), (32, 16), (16, 64)])
def test_token_major_output(V, dtype, dk, dv):
    """The epilogue's final layout conversion (vda_options.out_heads): for
    every divisor of the six head problems, with and without the options,
    the token-major output is the frame-major one rearranged, bit for bit
    (the same kernels write it, only to other addresses); once also against
    the oracle's output rearranged."""
    import torch
    _log(f"token-major output dtype={dtype} dk={dk} dv={dv}")
    w = I.custom("ex_tm", 2, 3, 7, 150, dk, dv, dtype, seed=dk + 3 * dv)
    x = I.make_inputs(w)
    d = device_inputs(w, x)
    alpha, S_T, G = I.make_decay(w), I.make_text_state(w), I.make_token_gates(w)
    variants = [
        dict(),
        dict(alpha=to_device(alpha, "f32"), text_state=to_device(S_T, "f32"), window=PAPER_WINDOW),
        dict(gate_tokens=to_device(G, w.dtype), window=(3, 1, 0)),
    ]
    bits = torch.int16 if dtype == "bf16" else torch.int32
    H = w.heads
    for opts in variants:
        gate = None if "gate_tokens" in opts else d["gate"]
        ref = V.forward(d["q"], d["k"], d["v"], d["beta"], gate, **opts)
        for oh in (1, 2, 3, 6):
            y = V.forward(d["q"], d["k"], d["v"], d["beta"], gate, out_heads=oh, **opts)
            torch.cuda.synchronize()
            assert tuple(y.shape) == (H // oh, w.F, w.N, oh * dv)
            assert torch.equal(y.view(bits), _token_major(ref, H // oh, oh).contiguous().view(bits)), \
                (sorted(opts), oh)
    y = V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"], out_heads=3,
                  alpha=to_device(alpha, "f32"), text_state=to_device(S_T, "f32"),
                  window=PAPER_WINDOW)
    torch.cuda.synchronize()
    exp = _oracle(w, x, alpha, S_T, PAPER_WINDOW)
    exp_tm = exp.reshape(2, 3, w.F, w.N, dv).transpose(0, 2, 3, 1, 4).reshape(2, w.F, w.N, 3 * dv)
    err = rel_max_err(from_device(y), exp_tm)
    _log(f"  against the oracle: rel err {err:.2e}")
    assert err <= tol_for(w), err


def _raw_queries(w, seed):
    """Raw query projections per head [H, F, N, d_k] in storage form: normal
    directions with per-token scales spread over e^-3 .. e^3, and a few
    all-zero tokens (whose L2 map is zero, and so is their output)."""
    rng = np.random.default_rng([seed, 77])
    q = rng.standard_normal((w.heads, w.F, w.N, w.d_k))
    q *= np.exp(rng.uniform(-3.0, 3.0, (w.heads, w.F, w.N, 1)))
    q[:, 0, :3] = 0.0
    q[:, -1, -2:] = 0.0
    q32 = q.astype(np.float32)
    return I.f32_to_bf16_bits(q32) if w.dtype == "bf16" else q32


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", [(64, 64), (128, 128), (32, 16), (128, 64)])
def test_raw_query(V, dtype, dk, dv):
    """vda_options.q_heads: the raw token-major query with the L2 map folded
    into the readout's RMSNorm, against the oracle's forward on the
    L2-normalised query (Sec. 2.3), with and without the options, for
    several query and output clip sizes."""
    import torch
    _log(f"raw query dtype={dtype} dk={dk} dv={dv}")
    w = I.custom("ex_rq", 2, 3, 7, 150, dk, dv, dtype, seed=5 * dk + dv)
    x = I.make_inputs(w)
    d = device_inputs(w, x)
    qraw = _raw_queries(w, w.seed)
    alpha, S_T, G = I.make_decay(w), I.make_text_state(w), I.make_token_gates(w)
    H = w.heads
    variants = [
        ("core", {}, {}),
        ("all", dict(alpha=to_device(alpha, "f32"), text_state=to_device(S_T, "f32"),
                     window=(3, 0, 1)), dict(alpha=alpha, S_T=S_T, window=(3, 0, 1))),
        ("token_gate", dict(gate_tokens=to_device(G, w.dtype), window=(3, 1, 0)),
         dict(G=G, window=(3, 1, 0))),
    ]
    xo = oracle_inputs(w, x)
    q_l2 = O.l2_normalise(I.as_float64(qraw, w.dtype))
    for name, opts, oopts in variants:
        exp = O.vda_forward_ex(q_l2, xo["k"], xo["v"], xo["beta"], xo["gate"],
                               None if "alpha" not in oopts else alpha.astype(np.float64),
                               None if "S_T" not in oopts else S_T.astype(np.float64),
                               *(oopts.get("window") or (1, 0, 0)), "joint",
                               gate_tokens=None if "G" not in oopts else
                               I.as_float64(G, w.dtype))
        # zero queries read out zero
        assert np.all(exp[:, 0, :3] == 0.0)
        gate = None if "gate_tokens" in opts else d["gate"]
        for qh, oh in ((1, None), (3, None), (3, 3), (6, 2)):
            qdev = to_device(_token_major_np(qraw, H // qh, qh), w.dtype)
            y = V.forward(qdev, d["k"], d["v"], d["beta"], gate, q_heads=qh, out_heads=oh, **opts)
            torch.cuda.synchronize()
            got = from_device(y)
            ref = exp if oh is None else _token_major_np(exp, H // oh, oh)
            err = rel_max_err(got, ref)
            _log(f"  {name} q_heads={qh} out_heads={oh}: rel err {err:.2e}")
            assert err <= tol_for(w), (name, qh, oh, err)
            if oh is None:
                assert np.all(got[:, 0, :3] == 0.0) and np.all(got[:, -1, -2:] == 0.0)


def _token_major_np(y, clips, heads):
    """numpy version of _token_major."""
    _, F, N, d = y.shape
    return np.ascontiguousarray(
        y.reshape(clips, heads, F, N, d).transpose(0, 2, 3, 1, 4).reshape(clips, F, N, heads * d))
