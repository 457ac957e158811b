"""The library's workspace cache on the GPU: vda_release_workspace empties
it, and a forward pass after the release allocates again and gives the same
result bit for bit."""
import numpy as np
import pytest

from paper_2609_20744_amd import inputs as I
from vda_testutil import device_inputs, from_device

pytestmark = pytest.mark.gpu


def test_release_workspace_then_forward_again():
    import torch
    from paper_2609_20744_amd import vda as V
    w = I.custom("ws", 1, 3, 6, 500, 128, 64, "bf16", seed=5)
    print("workspace release: H=3 F=6 N=500 d_k=128 d_v=64 bf16", flush=True)
    d = device_inputs(w, I.make_inputs(w))
    y0 = V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"])
    torch.cuda.synchronize()
    assert V.workspace_bytes() > 0
    freed = V.release_workspace()
    assert freed > 0
    assert V.workspace_bytes() == 0
    assert V.release_workspace() == 0
    y1 = V.forward(d["q"], d["k"], d["v"], d["beta"], d["gate"])
    torch.cuda.synchronize()
    assert V.workspace_bytes() > 0
    np.testing.assert_array_equal(from_device(y1), from_device(y0))
    # the explicit device index of the current device is the same cache
    dev = torch.cuda.current_device()
    assert V.workspace_bytes(dev) == V.workspace_bytes()
    with pytest.raises(ValueError):
        V.release_workspace(torch.cuda.device_count())
