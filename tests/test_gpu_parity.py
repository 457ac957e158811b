"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Stage tests feed oracle-computed inputs into one kernel and compare with the
oracle's result for that step; whole-operator tests run vda_forward on the
seeded workloads and compare element by element (small sizes) or at sampled
positions (full sizes, in the launch configuration the benchmark times).
The bar: rel. max-norm error <= 1e-4 (fp32 storage) and <= 2e-2 (bf16
storage, fp32 state).
"""
import numpy as np
import pytest

import oracle.vda_oracle as O
from paper_2609_20744_amd import inputs as I
from vda_testutil import (TOL_BF16, TOL_F32, ErrorAccumulator, device_inputs, fold_partials,
                          from_device, from_operand_tiles, oracle_inputs, oracle_sampled,
                          record_error, rel_max_err, sample_positions, to_device,
                          to_operand_tiles, tol_for)

pytestmark = pytest.mark.gpu

DIMS = [(32, 32), (32, 64), (32, 128), (64, 32), (64, 64), (64, 128), (128, 32), (128, 64),
        (128, 128)]


@pytest.fixture(scope="module")
def V():
    import torch
    assert torch.cuda.is_available(), "the gpu tests need an MI355X"
    from paper_2609_20744_amd import vda
    return vda


def _log(msg):
    print(msg, flush=True)


def _forward(V, w, x):
    import torch
    d = device_inputs(w, x)
    y = V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"])
    torch.cuda.synchronize()
    return y


# ----------------------------------------------------------------------------
# Stage parity (oracle-fed)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", DIMS)
def test_stats_stage(V, dtype, dk, dv):
    import torch
    w = I.custom("stats", 1, 2, 3, 200, dk, dv, dtype, seed=11)
    x = I.make_inputs(w)
    xo = oracle_inputs(w, x)
    d = device_inputs(w, x)
    # (tail_frames, splits): no split, every frame in 3 ranges, the last two
    # frames in 3 ranges
    for tail, splits in ((0, 1), (6, 3), (2, 3)):
        _log(f"stats dtype={dtype} dk={dk} dv={dv} tail={tail} splits={splits}")
        A_part, B_part = V.frame_stats(d["k"], d["v"], d["beta"], splits=splits, tail_frames=tail)
        torch.cuda.synchronize()
        assert A_part.shape[0] == 6 + tail * (splits - 1)
        A = fold_partials(A_part.double(), 6, tail, splits).view(2, 3, dk, dk).cpu().numpy()
        B = fold_partials(B_part.double(), 6, tail, splits).view(2, 3, dv, dk).cpu().numpy()
        for h in range(2):
            As, Bs = O.head_statistics(xo["k"][h], xo["v"][h], xo["beta"][h])
            tol = 1e-5 if dtype == "f32" else 1e-2
            assert rel_max_err(A[h], As) < tol
            assert rel_max_err(B[h], Bs) < tol
            if dtype == "bf16":  # off-diagonal 16 x 16 blocks: upper ones mirrored
                for t in range(3):
                    for i in range(dk // 16):
                        for j in range(i + 1, dk // 16):
                            blk = A[h, t, 16 * i:16 * i + 16, 16 * j:16 * j + 16]
                            assert np.array_equal(A[h, t, 16 * j:16 * j + 16, 16 * i:16 * i + 16],
                                                  blk.T)


@pytest.mark.parametrize("dk", [32, 64, 128])
def test_inverse_stage(V, dk):
    import torch
    rng = np.random.default_rng(dk)
    count, U = 6, 3 * dk
    K = rng.standard_normal((count, U, dk))
    K /= np.linalg.norm(K, axis=-1, keepdims=True)
    beta = rng.random((count, U))
    beta[0] = 0.0                        # A = 0: inverse is the identity
    beta[1] *= 10.0                      # stronger writes, larger condition number
    A = np.stack([O.frame_statistics(K[i], K[i][:, :1], beta[i])[0] for i in range(count)])
    expect = np.stack([O.frame_transition(A[i], np.zeros((1, dk)))[0] for i in range(count)])
    # (tail_frames, splits): no split, every frame in 2 ranges, the last
    # three frames in 3 ranges.  Partial s >= 1 of split frame i is matrix
    # i + s * tail.
    for tail, splits in ((0, 1), (count, 2), (3, 3)):
        _log(f"inverse dk={dk} tail={tail} splits={splits}")
        split = np.arange(count) >= count - tail if splits > 1 else np.zeros(count, bool)
        nparts = count + tail * (splits - 1) if splits > 1 else count
        parts = np.empty((nparts, dk, dk), np.float32)
        Bp = np.empty((nparts, 32, dk), np.float32)
        Bsum = np.empty((count, 32, dk), np.float32)
        for i in range(count):
            n = splits if split[i] else 1
            idx = [i] + [i + s * tail for s in range(1, n)]
            for s, m in enumerate(idx):
                parts[m] = A[i] / n
                Bp[m] = float(s + 1)
            Bsum[i] = float(sum(range(1, n + 1)))
        A_dev = to_device(parts, "f32")
        B_dev = to_device(Bp, "f32")
        Inv = V.frame_inverse(A_dev, B_dev, count=count, tail_frames=tail, splits=splits)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(B_dev[:count].cpu().numpy(), Bsum)
        got = Inv.double().cpu().numpy()
        np.testing.assert_array_equal(got[0], np.eye(dk))
        for i in range(count):
            cond = np.linalg.cond(np.eye(dk) + A[i])
            assert rel_max_err(got[i], expect[i]) < 2e-6 * cond, (i, cond)
        # The same inverse as split-bf16 operand tiles: element [k][n] of the
        # tiles is the computed inverse, whose fp32 form is stored transposed
        # (the two agree up to the inverse's rounding asymmetry), split into
        # bf16 hi + lo exactly as torch's RNE casts do on the CPU.
        A_dev = to_device(parts, "f32")
        B_dev = to_device(Bp, "f32")
        T = V.frame_inverse(A_dev, B_dev, count=count, tail_frames=tail, splits=splits,
                            tiles=True)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(B_dev[:count].cpu().numpy(), Bsum)
        T_exp = to_operand_tiles(np.swapaxes(Inv.cpu().numpy(), -1, -2))
        assert torch.equal(T.cpu().view(torch.int16), T_exp.view(torch.int16))
        gt = from_operand_tiles(T, dk)
        for i in range(count):
            cond = np.linalg.cond(np.eye(dk) + A[i])
            assert rel_max_err(gt[i], expect[i]) < 2e-6 * cond + 2e-5, (i, cond)
    # in place onto the partial buffer
    A_dev = to_device(A[None].astype(np.float32), "f32")
    V.frame_inverse(A_dev, Inv=A_dev[0])
    torch.cuda.synchronize()
    assert rel_max_err(A_dev[0].double().cpu().numpy()[3], expect[3]) < 1e-4


@pytest.mark.parametrize("dk,dv", DIMS)
def test_scan_stage(V, dk, dv):
    import torch
    _log(f"scan dk={dk} dv={dv}")
    w = I.custom("scan", 1, 3, 7, 40, dk, dv, "f32", seed=21)
    x = I.make_inputs(w)
    xo = oracle_inputs(w, x)
    Inv = np.empty((3, 7, dk, dk))
    Bm = np.empty((3, 7, dv, dk))
    P_exp = np.empty((3, 7, dv, dk))
    R_exp = np.empty((3, 7, dv, dk))
    for h in range(3):
        As, Bs = O.head_statistics(xo["k"][h], xo["v"][h], xo["beta"][h])
        for t in range(7):
            Inv[h, t] = np.linalg.inv(np.eye(dk) + As[t])
        Bm[h] = Bs
        P = O.forward_states(As, Bs)
        R = O.reverse_states(As, Bs)
        for t in range(1, 8):
            P_exp[h, t - 1] = P[t - 1]
            R_exp[h, t - 1] = R[t + 1]
    # fp32 products: fp32 rounding only; split-bf16 products: ~16-bit operands
    for exact, tol in ((True, 1e-5), (False, 1e-4)):
        Sf, Sr = V.state_scan(to_device(Inv.astype(np.float32), "f32"),
                              to_device(Bm.astype(np.float32), "f32"), exact_f32=exact)
        torch.cuda.synchronize()
        ef = rel_max_err(Sf.double().cpu().numpy(), P_exp)
        er = rel_max_err(Sr.double().cpu().numpy(), R_exp)
        _log(f"  exact_f32={exact}: fwd {ef:.2e} rev {er:.2e}")
        assert ef < tol and er < tol
        assert np.all(Sf[:, 0].cpu().numpy() == 0) and np.all(Sr[:, -1].cpu().numpy() == 0)
    # The scan vda_forward runs with bf16 storage: Inv_t as split-bf16 tiles.
    Sf, Sr = V.state_scan_tiles(to_operand_tiles(Inv).cuda(), to_device(Bm.astype(np.float32), "f32"))
    torch.cuda.synchronize()
    ef = rel_max_err(Sf.double().cpu().numpy(), P_exp)
    er = rel_max_err(Sr.double().cpu().numpy(), R_exp)
    _log(f"  tiles: fwd {ef:.2e} rev {er:.2e}")
    assert ef < 1e-4 and er < 1e-4
    assert np.all(Sf[:, 0].cpu().numpy() == 0) and np.all(Sr[:, -1].cpu().numpy() == 0)


@pytest.mark.parametrize("dk,dv", [(64, 128), (128, 128)])
def test_scan_many_workgroups_per_cu(V, dk, dv):
    """Enough chains that several scan workgroups share a compute unit, where
    waves drift apart and a missing wait before a barrier shows up as wrong,
    run-to-run varying states.  Checked against the fp64 recurrence on the
    same (fp32) Inv_t and B_t, and for bitwise repeatability."""
    import torch
    H, F = 40, 16
    _log(f"scan many workgroups dk={dk} dv={dv} H={H} F={F}")
    rng = np.random.default_rng(dk + dv)
    G = rng.standard_normal((H, F, dk, dk)) / np.sqrt(dk)
    Inv = np.linalg.inv(np.eye(dk) + G @ np.swapaxes(G, -1, -2))
    Inv = (0.5 * (Inv + np.swapaxes(Inv, -1, -2))).astype(np.float32)
    Bm = rng.standard_normal((H, F, dv, dk)).astype(np.float32)
    I64, B64 = Inv.astype(np.float64), Bm.astype(np.float64)
    P_exp = np.zeros((H, F, dv, dk))
    R_exp = np.zeros((H, F, dv, dk))
    for t in range(1, F):
        P_exp[:, t] = (P_exp[:, t - 1] + B64[:, t - 1]) @ I64[:, t - 1]
    for t in range(F - 2, -1, -1):
        R_exp[:, t] = (R_exp[:, t + 1] + B64[:, t + 1]) @ I64[:, t + 1]
    Id, Bd = to_device(Inv, "f32"), to_device(Bm, "f32")
    Td = to_operand_tiles(Inv).cuda()
    for kind, tol in (("exact_f32", 1e-5), ("split", 1e-4), ("tiles", 1e-4)):
        if kind == "tiles":
            Sf, Sr = V.state_scan_tiles(Td, Bd)
            Sf2, Sr2 = V.state_scan_tiles(Td, Bd)
        else:
            Sf, Sr = V.state_scan(Id, Bd, exact_f32=kind == "exact_f32")
            Sf2, Sr2 = V.state_scan(Id, Bd, exact_f32=kind == "exact_f32")
        torch.cuda.synchronize()
        assert torch.equal(Sf, Sf2) and torch.equal(Sr, Sr2)
        ef = rel_max_err(Sf.double().cpu().numpy(), P_exp)
        er = rel_max_err(Sr.double().cpu().numpy(), R_exp)
        _log(f"  {kind}: fwd {ef:.2e} rev {er:.2e}")
        assert ef < tol and er < tol


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", DIMS)
def test_readout_stage(V, dtype, dk, dv):
    import torch
    _log(f"readout dtype={dtype} dk={dk} dv={dv}")
    w = I.custom("readout", 1, 2, 3, 77, dk, dv, dtype, seed=31)
    x = I.make_inputs(w)
    xo = oracle_inputs(w, x)
    rng = np.random.default_rng(5)
    Sf = rng.standard_normal((2, 3, dv, dk)) * 0.3
    Sr = rng.standard_normal((2, 3, dv, dk)) * 0.3
    y = V.readout(to_device(x["q"], dtype), to_device(Sf.astype(np.float32), "f32"),
                  to_device(Sr.astype(np.float32), "f32"), to_device(x["gate"], "f32"))
    torch.cuda.synchronize()
    got = from_device(y)
    Sf32 = Sf.astype(np.float32).astype(np.float64)
    Sr32 = Sr.astype(np.float32).astype(np.float64)
    exp = np.empty_like(got)
    for h in range(2):
        for t in range(3):
            o = O.readout(Sf32[h, t] + Sr32[h, t], xo["q"][h, t])
            exp[h, t] = O.rmsnorm_gate(o, xo["gate"][h])
    tol = 1e-5 if dtype == "f32" else 1e-2
    assert rel_max_err(got, exp) < tol


# ----------------------------------------------------------------------------
# Whole operator on the five workloads
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["tiny_f32", "small_bf16"])
def test_forward_full_oracle(V, name):
    w = I.WORKLOADS[name]
    _log(f"forward {name} (every output against the oracle)")
    x = I.make_inputs(w)
    got = from_device(_forward(V, w, x))
    xo = oracle_inputs(w, x)
    exp = O.vda_forward(xo["q"], xo["k"], xo["v"], xo["beta"], xo["gate"])
    acc = ErrorAccumulator()
    acc.add(got, exp, 0)
    _log(f"  {acc.report()}")
    record_error(f"{name} every output", acc)
    assert acc.rel_max_err() <= tol_for(w)


@pytest.mark.parametrize("name", ["480p_bf16", "768p_bf16", "ragged_bf16"])
def test_forward_full_size_every_output(V, name):
    """Full-size workloads in the benchmark's launch configuration (one call
    over all heads); every output element is compared with the oracle's,
    which runs over groups of heads to bound host memory."""
    w = I.WORKLOADS[name]
    _log(f"forward {name} (every output against the oracle)")
    x = I.make_inputs(w)
    y = _forward(V, w, x)
    del x
    acc = ErrorAccumulator()
    group = 4
    for h0 in range(0, w.heads, group):
        heads = list(range(h0, min(w.heads, h0 + group)))
        xo = oracle_inputs(w, I.make_inputs(w, heads=heads))
        ref = O.vda_forward(xo["q"], xo["k"], xo["v"], xo["beta"], xo["gate"])
        acc.add(from_device(y[h0:h0 + len(heads)]), ref, h0)
    rep = acc.report()
    _log(f"  {rep}")
    record_error(f"{name} every output", acc)
    assert acc.rel_max_err() <= TOL_BF16, rep


# ----------------------------------------------------------------------------
# Edge cases
# ----------------------------------------------------------------------------

def _check_small(V, w, x=None):
    x = I.make_inputs(w) if x is None else x
    got = from_device(_forward(V, w, x))
    xo = oracle_inputs(w, x)
    exp = O.vda_forward(xo["q"], xo["k"], xo["v"], xo["beta"], xo["gate"])
    err = rel_max_err(got, exp)
    assert err <= tol_for(w), err
    return got, exp


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", DIMS)
def test_head_dims(V, dtype, dk, dv):
    _log(f"dims dtype={dtype} dk={dk} dv={dv}")
    _check_small(V, I.custom("dims", 2, 1, 5, 150, dk, dv, dtype, seed=dk + dv))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", [(16, 16), (16, 32), (16, 64), (16, 128), (32, 16), (64, 16),
                                   (128, 16)])
def test_narrow_head_dims(V, dtype, dk, dv):
    # 16-channel heads run zero-padded to 32 channels inside vda_forward
    _log(f"narrow dims dtype={dtype} dk={dk} dv={dv}")
    _check_small(V, I.custom("narrow", 2, 1, 5, 150, dk, dv, dtype, seed=dk * 3 + dv))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_narrow_head_dims_ragged(V, dtype):
    _log(f"narrow ragged dtype={dtype}")
    for N in (1, 17, 333):
        _check_small(V, I.custom("narrow_ragged", 1, 3, 4, N, 16, 16, dtype, seed=N))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("N", [1, 2, 15, 16, 17, 63, 64, 65, 129, 300])
def test_ragged_tokens(V, dtype, N):
    _log(f"ragged N={N} dtype={dtype}")
    _check_small(V, I.custom("ragged", 1, 2, 4, N, 64, 128, dtype, seed=N))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_single_frame_is_zero(V, dtype):
    w = I.custom("f1", 1, 3, 1, 100, 64, 64, dtype, seed=3)
    got, _ = _check_small(V, w)
    assert np.all(got == 0.0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_zero_writes(V, dtype):
    w = I.custom("zero", 1, 2, 5, 70, 64, 64, dtype, seed=4)
    x = I.make_inputs(w)
    x["beta"][:] = 0.0
    got, _ = _check_small(V, w, x)
    assert np.all(got == 0.0)
    x = I.make_inputs(w)
    x["beta"][:, [0, 1, 3, 4]] = 0.0     # only frame 3 (index 2) writes
    got, _ = _check_small(V, w, x)
    assert np.all(got[:, 2] == 0.0)
    assert np.all(np.abs(got[:, [0, 1, 3, 4]]).max(axis=-1) > 0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_duplicate_and_strong_writes(V, dtype):
    w = I.custom("dup", 1, 2, 6, 90, 64, 64, dtype, seed=9, dup_frac=0.3, beta_sigma=3.0,
                 beta_zero_frac=0.2)
    x = I.make_inputs(w)
    x["k"][:, :, 10:20] = x["k"][:, :, 5:6]   # exact duplicates
    x["beta"][:, :, 10:20] = 1.0
    _check_small(V, w, x)


def test_deterministic_and_guarded(V):
    import torch
    w = I.custom("det", 1, 4, 6, 333, 128, 128, "bf16", seed=12)
    x = I.make_inputs(w)
    d = device_inputs(w, x)
    pad = 4096
    buf = torch.full((2 * pad + w.heads * w.F * w.N * w.d_v,), -7, dtype=torch.int16, device="cuda")
    out = buf[pad:pad + w.heads * w.F * w.N * w.d_v].view(torch.bfloat16).view(w.heads, w.F, w.N, w.d_v)
    V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"], out=out)
    y1 = V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"])
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), y1.view(torch.int16))
    assert torch.all(buf[:pad] == -7) and torch.all(buf[-pad:] == -7)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        y2 = V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"])
    s.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


def _staged_forward(V, d, exact_f32):
    """The forward pass through the stage entry points, with the library's
    default split plan of the statistics step.  Returns the output and the
    plan's split count."""
    H, F, N, d_k = d["k"].shape
    d_v = d["v"].shape[-1]
    tail, splits = V.default_split_plan(F, N, H, d_k, d_v, exact_f32)
    A_part, B_part = V.frame_stats(d["k"], d["v"], d["beta"], splits=splits, tail_frames=tail)
    count = H * F
    # With bf16 storage the inverse goes to the scan as split-bf16 tiles.
    Inv = V.frame_inverse(A_part, B_part, count=count, tail_frames=tail, splits=splits,
                          Inv=A_part[:count], tiles=not exact_f32)
    if exact_f32:
        Sf, Sr = V.state_scan(Inv.view(H, F, d_k, d_k), B_part[:count].view(H, F, d_v, d_k),
                              exact_f32=True)
    else:
        Sf, Sr = V.state_scan_tiles(Inv.view(H, F, d_k * d_k), B_part[:count].view(H, F, d_v, d_k))
    return V.readout(d["q"], Sf, Sr, d["gate"]), splits


def test_stages_compose_to_forward(V):
    """vda_forward equals its stages run one after another."""
    import torch
    w = I.custom("compose", 1, 3, 5, 700, 128, 128, "bf16", seed=13)
    d = device_inputs(w, I.make_inputs(w))
    y = V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"])
    y2, splits = _staged_forward(V, d, exact_f32=False)
    assert splits > 1                   # exercises the split reduction
    # the same for fp32 storage
    wf = I.custom("compose32", 1, 2, 4, 100, 64, 64, "f32", seed=14)
    df = device_inputs(wf, I.make_inputs(wf))
    yf = V.forward(df["q"], df["k"], df["v"], df["beta"], df["gate"])
    yf2, _ = _staged_forward(V, df, exact_f32=True)
    # one head: no grouping
    w1 = I.custom("compose1", 1, 1, 3, 300, 64, 128, "bf16", seed=15)
    d1 = device_inputs(w1, I.make_inputs(w1))
    y1 = V.forward(d1["q"], d1["k"], d1["v"], d1["beta"], d1["gate"])
    y12, _ = _staged_forward(V, d1, exact_f32=False)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y2.view(torch.int16))
    assert torch.equal(yf, yf2)
    assert torch.equal(y1.view(torch.int16), y12.view(torch.int16))


def test_forward_on_many_streams(V):
    """Calls issued on several streams at once (sharing the library's
    workspace pool) each equal the single-stream result."""
    import torch
    w = I.custom("streams", 1, 4, 6, 500, 64, 128, "bf16", seed=17)
    d = device_inputs(w, I.make_inputs(w))
    ref = V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"])
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in range(3)]
    outs = []
    for s in streams:
        with torch.cuda.stream(s):
            outs.append(V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"]))
    torch.cuda.synchronize()
    for o in outs:
        assert torch.equal(o.view(torch.int16), ref.view(torch.int16))


def test_invalid_arguments_raise(V):
    import torch
    w = I.custom("bad", 1, 2, 3, 64, 64, 64, "bf16", seed=1)
    d = device_inputs(w, I.make_inputs(w))
    with pytest.raises(ValueError):
        V.forward(d["q"], d["k"], d["v"], d["beta"][..., :10].contiguous(), d["gate"])
    q48 = torch.zeros((2, 3, 64, 48), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError, match="UNSUPPORTED"):
        V.forward(q48, q48, d["v"], d["beta"], d["gate"])
    flat = torch.zeros(2 * 3 * 64 * 64 + 1, dtype=torch.bfloat16, device="cuda")
    q_mis = flat[1:].view(2, 3, 64, 64)
    with pytest.raises(ValueError, match="ALIGN"):
        V.forward(q_mis, d["k"], d["v"], d["beta"], d["gate"])
    with pytest.raises(ValueError, match="OVERLAP"):
        V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"], out=d["v"])
