"""vda_forward_noalloc (the allocation-free forward, workspace in the
library's fixed device scratch array) against vda_forward, through the C
ABI on the current torch stream: two calls in a row, the second smaller; a
call whose workspace exceeds the array (heads in groups) also against the
oracle; 16-channel heads; and the error for a head that cannot fit."""
import ctypes

import numpy as np
import pytest

import oracle.vda_oracle as O
from paper_2609_20744_amd import inputs as I
from vda_testutil import (TOL_BF16, device_inputs, from_device, oracle_inputs,
                          rel_max_err)

pytestmark = pytest.mark.gpu

SCRATCH = 256 << 20


def _noalloc(V, d, F, N, H, dk, dv, out):
    import torch
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return V.lib.vda_forward_noalloc(d["q"].data_ptr(), d["k"].data_ptr(), d["v"].data_ptr(),
                                     d["beta"].data_ptr(), d["gate"].data_ptr(), F, N, H, dk, dv,
                                     out.data_ptr(), stream)


def _case(V, w):
    import torch
    print(f"noalloc {w.name}: H={w.heads} F={w.F} N={w.N} d_k={w.d_k} d_v={w.d_v}", flush=True)
    x = I.make_inputs(w)
    d = device_inputs(w, x)
    ref = V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"])
    out = torch.full_like(ref, float("nan"))
    st = _noalloc(V, d, w.F, w.N, w.heads, w.d_k, w.d_v, out)
    assert st == 0, V.status_string(st)
    torch.cuda.synchronize()
    return x, from_device(out), from_device(ref)


def test_noalloc_matches_forward_two_calls():
    from paper_2609_20744_amd import vda as V
    # First call: every head in one group (same plan and kernels as
    # vda_forward, so the same bits); second call smaller, on the array the
    # first call left behind.
    for w in (I.custom("na_big", 1, 8, 12, 1000, 128, 128, "bf16", seed=41),
              I.custom("na_small", 1, 2, 5, 150, 64, 32, "bf16", seed=42)):
        _, got, ref = _case(V, w)
        assert np.isfinite(got).all()
        assert rel_max_err(got, ref) <= TOL_BF16
        np.testing.assert_array_equal(got, ref)


def test_noalloc_head_groups_and_narrow_heads():
    from paper_2609_20744_amd import vda as V
    # 40 heads x 36 frames at d = 128: about 360 MiB of workspace, so the
    # heads run in groups; checked against vda_forward and the oracle.
    w = I.custom("na_groups", 1, 40, 36, 128, 128, 128, "bf16", seed=43)
    x, got, ref = _case(V, w)
    assert rel_max_err(got, ref) <= TOL_BF16
    xo = oracle_inputs(w, x)
    exp = O.vda_forward(xo["q"], xo["k"], xo["v"], xo["beta"], xo["gate"])
    err = rel_max_err(got, exp)
    print(f"  rel max-norm error against the oracle {err:.3e}", flush=True)
    assert err <= TOL_BF16
    # 16-channel heads (padded copies in the scratch array)
    w = I.custom("na_narrow", 1, 3, 4, 77, 16, 16, "bf16", seed=44)
    _, got, ref = _case(V, w)
    np.testing.assert_array_equal(got, ref)


def test_noalloc_rejects_a_head_larger_than_the_array():
    import torch
    from paper_2609_20744_amd import vda as V
    # One head of 1100 frames at d = 128 needs 1100 * 256 KiB > 256 MiB.
    w = I.custom("na_over", 1, 1, 1100, 1, 128, 128, "bf16", seed=45)
    print("noalloc over the array: H=1 F=1100 N=1", flush=True)
    d = device_inputs(w, I.make_inputs(w))
    out = torch.zeros((1, 1100, 1, 128), dtype=torch.bfloat16, device="cuda")
    st = _noalloc(V, d, 1100, 1, 1, 128, 128, out)
    assert V.STATUS_NAMES[st] == "VDA_ERR_SCRATCH"
    torch.cuda.synchronize()
    assert not out.any()
    with pytest.raises(ValueError):
        V.forward_noalloc(d["q"], d["k"], d["v"], d["beta"], d["gate"], out=out)
