"""Checks of the seeded input generator (CPU)."""
import numpy as np
import torch

from paper_2609_20744_amd import inputs as I


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.005859375, 3.0e38, 1e-40],
                                 dtype=np.float32)])
    bits = I.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(bits, ref)
    back = I.bf16_bits_to_f32(bits)
    np.testing.assert_array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_deterministic_and_per_head():
    w = I.custom("t", 2, 3, 3, 17, 32, 64, "bf16", seed=5, beta_zero_frac=0.25, dup_frac=0.1,
                 beta_sigma=2.0)
    a = I.make_inputs(w)
    b = I.make_inputs(w)
    for key in a:
        np.testing.assert_array_equal(a[key], b[key])
    sub = I.make_inputs(w, heads=[4, 1])
    for key in ["q", "k", "v", "beta"]:
        np.testing.assert_array_equal(sub[key][0], a[key][4])
        np.testing.assert_array_equal(sub[key][1], a[key][1])
    np.testing.assert_array_equal(sub["gate"], a["gate"][[4, 1]])


def test_distributions():
    w = I.WORKLOADS["ragged_bf16"]
    h = I.head_inputs(w, 3)
    k = I.as_float64(h["k"], "bf16")
    q = I.as_float64(h["q"], "bf16")
    assert h["k"].shape == (64, 2025, 64) and h["v"].shape == (64, 2025, 128)
    np.testing.assert_allclose(np.linalg.norm(k, axis=-1), 1.0, atol=1e-2)
    np.testing.assert_allclose(np.linalg.norm(q, axis=-1), 1.0, atol=1e-2)
    beta = h["beta"]
    assert beta.min() >= 0 and beta.max() < 1
    frac0 = np.mean(beta == 0)
    assert 0.23 < frac0 < 0.27
    # near-duplicate keys: about 10% of each frame's tokens have a neighbour at cosine > 0.999
    kk = k[0]
    cos = kk @ kk.T
    np.fill_diagonal(cos, 0)
    dup = np.mean(cos.max(axis=1) > 0.999)
    assert 0.1 <= dup <= 0.25
    g = I.gates(w)
    assert g.shape == (24,) and np.all((g > 0) & (g < 1))


def test_f32_storage():
    w = I.WORKLOADS["tiny_f32"]
    x = I.make_inputs(w)
    assert x["q"].dtype == np.float32 and x["q"].shape == (2, 4, 64, 64)
    assert x["v"].dtype == np.float32
    np.testing.assert_allclose(np.linalg.norm(x["q"].astype(np.float64), axis=-1), 1.0, atol=1e-6)
