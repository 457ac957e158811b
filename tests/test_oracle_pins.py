"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each ``pin_*`` function checks the oracle against something other than its own
code: a hand-derived worked example, a closed form printed in the paper, an
invariant the paper proves, a library routine, or brute force on tiny inputs.
``test_mutants_are_caught`` plants plausible mistakes in the oracle (on the CPU)
and checks that at least one pin fails for each.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle.vda_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


def _unit_rows(x):
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def _random_frame(rng, U=7, d_k=5, d_v=4):
    K = _unit_rows(rng.standard_normal((U, d_k)))
    V = rng.standard_normal((U, d_v))
    beta = 1.0 / (1.0 + np.exp(-rng.standard_normal(U)))
    return K, V, beta


def _random_clip(rng, F=5, N=6, d_k=4, d_v=3):
    q = _unit_rows(rng.standard_normal((F, N, d_k)))
    k = _unit_rows(rng.standard_normal((F, N, d_k)))
    v = rng.standard_normal((F, N, d_v))
    beta = 1.0 / (1.0 + np.exp(-rng.standard_normal((F, N))))
    return q, k, v, beta


def _frac(a):
    return np.vectorize(lambda s: float(Fraction(s)))(np.array(a, dtype=object)).astype(np.float64)


# ----------------------------------------------------------------------------
# Pins
# ----------------------------------------------------------------------------

def _golden_clip():
    """The hand-derived clip of tests/golden as float64 arrays, with its gate
    and the expected outputs y = gate * o / sqrt(ms) (eps = 0)."""
    with open(os.path.join(GOLDEN, "hand_example_dk2_dv2_F3.json")) as f:
        g = json.load(f)
    k = np.stack([_frac(fr["k"]) for fr in g["frames"]])
    v = np.stack([_frac(fr["v"]) for fr in g["frames"]])
    q = np.stack([_frac(fr["q"]) for fr in g["frames"]])
    beta = np.stack([_frac(fr["beta"]) for fr in g["frames"]])
    gate = float(Fraction(g["gate"]))
    y = gate * _frac(g["o"]) / np.sqrt(_frac(g["ms"]))[..., None]
    return g, q, k, v, beta, gate, y


def pin_golden_hand_example():
    """Hand-derived exact example (tests/golden): Eq. 3b, 5, A.1, A.4, 1a, 1c."""
    g, q, k, v, beta, gate, y_expect = _golden_clip()
    As, Bs = O.head_statistics(k, v, beta)
    np.testing.assert_allclose(np.eye(2)[None] + As, _frac(g["A"]), rtol=0, atol=1e-14)
    np.testing.assert_allclose(Bs, _frac(g["B"]), rtol=0, atol=1e-14)
    P = O.forward_states(As, Bs)
    np.testing.assert_allclose(P, _frac(g["P"]), rtol=0, atol=1e-14)
    R = O.reverse_states(As, Bs)
    np.testing.assert_allclose(R[1:], _frac(g["R"]), rtol=0, atol=1e-14)
    St = O.gathered_states(As, Bs)
    np.testing.assert_allclose(St, _frac(g["S_tilde"]), rtol=0, atol=1e-14)
    o_expect = _frac(g["o"])
    ms = _frac(g["ms"])
    for t in range(3):
        o = O.readout(St[t], q[t])
        np.testing.assert_allclose(o, o_expect[t], rtol=0, atol=1e-14)
        y = O.rmsnorm_gate(o, gate, eps=0.0)
        np.testing.assert_allclose(y, gate * o_expect[t] / np.sqrt(ms[t])[:, None],
                                   rtol=1e-14, atol=1e-14)
    y_all = O.head_forward(q, k, v, beta, gate, eps=0.0)
    np.testing.assert_allclose(y_all, y_expect, rtol=1e-14)


def pin_golden_at_head_one_of_two():
    """Eq. 1c and Algorithm 1 act per head: each head problem reads only its
    own inputs and its own gate.  The hand-derived clip sits at head 1 of a
    two-head call whose head 0 is a random clip with a different gate, decay,
    text state and token gate; head 1 must give the hand-derived outputs and
    head 0 its own single-head result, for both multi-head wrappers."""
    _, q1, k1, v1, b1, g1, y1 = _golden_clip()
    rng = _rng(61)
    q0, k0, v0, b0 = _random_clip(rng, F=3, N=2, d_k=2, d_v=2)
    g0 = 0.3
    q, k, v, beta = (np.stack(z) for z in ((q0, q1), (k0, k1), (v0, v1), (b0, b1)))
    gate = np.array([g0, g1])
    y = O.vda_forward(q, k, v, beta, gate, eps=0.0)
    np.testing.assert_allclose(y[1], y1, rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(y[0], O.head_forward(q0, k0, v0, b0, g0, eps=0.0),
                               rtol=1e-14, atol=1e-14)
    # Extended wrapper: head 1 keeps alpha = 1 and no text state (the
    # golden clip's own setting); head 0 has its own decay and text state.
    alpha = np.stack([_random_alpha(rng, 3, 2), np.ones((3, 2))])
    S_T = np.stack([rng.standard_normal((2, 2)), np.zeros((2, 2))])
    ye = O.vda_forward_ex(q, k, v, beta, gate, alpha=alpha, S_T=S_T, eps=0.0)
    np.testing.assert_allclose(ye[1], y1, rtol=1e-14, atol=1e-14)
    ref0 = O.head_forward_ex(q0, k0, v0, b0, g0, alpha[0], S_T[0], O.local_windows(3), "joint", 0.0)
    np.testing.assert_allclose(ye[0], ref0, rtol=1e-13, atol=1e-14)
    # Token gates: head 1's is its head gate everywhere, head 0's is random.
    G = np.stack([rng.uniform(0.05, 1.0, (3, 2, 2)), np.full((3, 2, 2), g1)])
    yg = O.vda_forward_ex(q, k, v, beta, None, alpha=alpha, S_T=S_T, eps=0.0, gate_tokens=G)
    np.testing.assert_allclose(yg[1], y1, rtol=1e-14, atol=1e-14)
    ref0 = O.head_forward_ex(q0, k0, v0, b0, 1.0, alpha[0], S_T[0], O.local_windows(3), "joint",
                             0.0, G[0])
    np.testing.assert_allclose(yg[0], ref0, rtol=1e-13, atol=1e-14)


def pin_stats_outer_product_sum():
    """Eq. 3b, left forms: A = sum_u beta k k^T, B = sum_u beta v k^T (token loop)."""
    rng = _rng(1)
    K, V, beta = _random_frame(rng, U=9, d_k=5, d_v=3)
    A_loop = np.zeros((5, 5))
    B_loop = np.zeros((3, 5))
    for u in range(9):
        for i in range(5):
            for j in range(5):
                A_loop[i, j] += beta[u] * K[u, i] * K[u, j]
        for i in range(3):
            for j in range(5):
                B_loop[i, j] += beta[u] * V[u, i] * K[u, j]
    A, B = O.frame_statistics(K, V, beta)
    np.testing.assert_allclose(A, A_loop, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(B, B_loop, rtol=1e-13, atol=1e-14)


def pin_solve_matches_dense_inverse():
    """Eq. 5 against an explicit dense inverse (library routine)."""
    rng = _rng(2)
    for d_k, d_v, U in [(4, 3, 6), (8, 8, 20), (16, 8, 40)]:
        K, V, beta = _random_frame(rng, U, d_k, d_v)
        S_bar = rng.standard_normal((d_v, d_k))
        A, B = O.frame_statistics(K, V, beta)
        S = O.joint_frame_update(S_bar, A, B)
        S_ref = (S_bar + B) @ np.linalg.inv(np.eye(d_k) + A)
        np.testing.assert_allclose(S, S_ref, rtol=1e-12, atol=1e-13)


def pin_solve_matches_token_space():
    """The key-space solve equals the U x U token-space solve of the same
    first-order condition (the N x N correction solve)."""
    rng = _rng(3)
    for d_k, d_v, U in [(4, 3, 2), (4, 3, 9), (6, 5, 30)]:
        K, V, beta = _random_frame(rng, U, d_k, d_v)
        S_bar = rng.standard_normal((d_v, d_k))
        A, B = O.frame_statistics(K, V, beta)
        S = O.joint_frame_update(S_bar, A, B)
        S_tok = O.joint_frame_update_token_space(S_bar, K, V, beta)
        np.testing.assert_allclose(S, S_tok, rtol=1e-12, atol=1e-13)


def pin_solve_kronecker_bruteforce():
    """Brute force: vec(S C) = (C^T kron I) vec(S) (row-major vec), solved densely."""
    rng = _rng(4)
    d_k, d_v, U = 4, 3, 5
    K, V, beta = _random_frame(rng, U, d_k, d_v)
    S_bar = rng.standard_normal((d_v, d_k))
    C = np.eye(d_k)
    for u in range(U):
        C = C + beta[u] * np.outer(K[u], K[u])
    rhs = S_bar.copy()
    for u in range(U):
        rhs = rhs + beta[u] * np.outer(V[u], K[u])
    # row-major vec: vec(S C)[i*d_k + j] = sum_m S[i,m] C[m,j]
    big = np.kron(np.eye(d_v), C.T)
    S_bf = np.linalg.solve(big, rhs.reshape(-1)).reshape(d_v, d_k)
    A, B = O.frame_statistics(K, V, beta)
    np.testing.assert_allclose(O.joint_frame_update(S_bar, A, B), S_bf, rtol=1e-12, atol=1e-13)


def _eq4(S, S_bar, K, V, beta):
    """Eq. 4 written out token by token."""
    val = 0.5 * float(np.sum((S - S_bar) ** 2))
    for u in range(K.shape[0]):
        r = S @ K[u] - V[u]
        val += 0.5 * beta[u] * float(r @ r)
    return val


def pin_solve_minimises_eq4():
    """Eq. 4: the update is a stationary point (central differences) and a
    strict minimum against random perturbations."""
    rng = _rng(5)
    d_k, d_v, U = 4, 3, 6
    K, V, beta = _random_frame(rng, U, d_k, d_v)
    S_bar = rng.standard_normal((d_v, d_k))
    A, B = O.frame_statistics(K, V, beta)
    S = O.joint_frame_update(S_bar, A, B)
    h = 1e-5
    grad = np.zeros_like(S)
    for i in range(d_v):
        for j in range(d_k):
            E = np.zeros_like(S)
            E[i, j] = h
            grad[i, j] = (_eq4(S + E, S_bar, K, V, beta) - _eq4(S - E, S_bar, K, V, beta)) / (2 * h)
    assert np.max(np.abs(grad)) < 1e-8, grad
    f0 = _eq4(S, S_bar, K, V, beta)
    for _ in range(20):
        D = rng.standard_normal(S.shape) * 1e-3
        assert _eq4(S + D, S_bar, K, V, beta) > f0


def pin_prop1_spectral_norm():
    """Proposition 1 / Eq. A.2: ||Diag(alpha)(I + A)^-1||_2 <= 1 for beta >= 0,
    alpha in [0, 1]; and ||(I+A)^-1||_2 = 1 / (1 + lambda_min(A))."""
    rng = _rng(6)
    for U in [1, 3, 50, 400]:
        K, V, beta = _random_frame(rng, U, 8, 4)
        A, Bm = O.frame_statistics(K, V, beta)
        Cinv = np.linalg.inv(np.eye(8) + A)
        lam_min = np.linalg.eigvalsh(A)[0]
        np.testing.assert_allclose(np.linalg.norm(Cinv, 2), 1.0 / (1.0 + lam_min), rtol=1e-10)
        assert np.linalg.norm(Cinv, 2) <= 1.0 + 1e-12
        alpha = rng.random(8)
        M, _ = O.frame_transition(A, Bm, alpha)
        assert np.linalg.svd(M, compute_uv=False)[0] <= 1.0 + 1e-12


def pin_beta_zero_keeps_state():
    """beta = 0: the frame writes nothing (S_t = S_bar), and zero-strength
    tokens can be deleted without changing the state (Eq. 3b sums)."""
    rng = _rng(7)
    K, V, beta = _random_frame(rng, 6, 5, 3)
    S_bar = rng.standard_normal((3, 5))
    A, B = O.frame_statistics(K, V, np.zeros(6))
    np.testing.assert_array_equal(O.joint_frame_update(S_bar, A, B), S_bar)
    beta2 = beta.copy()
    beta2[[1, 4]] = 0.0
    A2, B2 = O.frame_statistics(K, V, beta2)
    keep = [0, 2, 3, 5]
    A3, B3 = O.frame_statistics(K[keep], V[keep], beta2[keep])
    np.testing.assert_allclose(O.joint_frame_update(S_bar, A2, B2),
                               O.joint_frame_update(S_bar, A3, B3), rtol=1e-13, atol=1e-14)


def pin_repeated_key_eqA3():
    """Eq. A.3: U copies of one unit key with common beta give
    S_t k = s / (1 + U beta) + U beta / (1 + U beta) * vbar, s = S_bar k."""
    rng = _rng(8)
    d_k, d_v = 6, 4
    for U, b in [(1, 0.3), (5, 0.7), (64, 0.5)]:
        k = _unit_rows(rng.standard_normal(d_k))
        K = np.tile(k, (U, 1))
        V = rng.standard_normal((U, d_v))
        S_bar = rng.standard_normal((d_v, d_k))
        A, B = O.frame_statistics(K, V, np.full(U, b))
        S = O.joint_frame_update(S_bar, A, B)
        s = S_bar @ k
        vbar = V.mean(axis=0)
        expect = s / (1 + U * b) + U * b / (1 + U * b) * vbar
        np.testing.assert_allclose(S @ k, expect, rtol=1e-12, atol=1e-13)
        # directions orthogonal to k are untouched
        x = rng.standard_normal(d_k)
        x -= (x @ k) * k
        np.testing.assert_allclose(S @ x, S_bar @ x, rtol=1e-12, atol=1e-13)


def pin_orthonormal_keys_weight():
    """Appendix A.2: orthogonal keys each receive weight beta / (1 + beta):
    S_t k_u = s_u + beta_u / (1 + beta_u) (v_u - s_u)."""
    rng = _rng(9)
    d_k, d_v, U = 8, 3, 5
    Qm, _ = np.linalg.qr(rng.standard_normal((d_k, d_k)))
    K = Qm[:U]
    V = rng.standard_normal((U, d_v))
    beta = rng.random(U) * 2
    S_bar = rng.standard_normal((d_v, d_k))
    A, B = O.frame_statistics(K, V, beta)
    S = O.joint_frame_update(S_bar, A, B)
    for u in range(U):
        s = S_bar @ K[u]
        np.testing.assert_allclose(S @ K[u], s + beta[u] / (1 + beta[u]) * (V[u] - s),
                                   rtol=1e-12, atol=1e-13)


def pin_token_permutation_invariance():
    """The frame update imposes no patch order: permuting a frame's tokens
    (k, v, beta together) leaves the state unchanged."""
    rng = _rng(10)
    K, V, beta = _random_frame(rng, 11, 6, 4)
    S_bar = rng.standard_normal((4, 6))
    perm = rng.permutation(11)
    A, B = O.frame_statistics(K, V, beta)
    Ap, Bp = O.frame_statistics(K[perm], V[perm], beta[perm])
    np.testing.assert_allclose(O.joint_frame_update(S_bar, A, B),
                               O.joint_frame_update(S_bar, Ap, Bp), rtol=1e-12, atol=1e-13)


def pin_n1_reduces_to_token_delta_rule():
    """One token per frame: the forward scan equals the token-wise delta rule
    of Eq. 2 (alpha = 1) with write strength beta' = beta / (1 + beta ||k||^2)
    (Sherman-Morrison), and differs from it with the same beta."""
    rng = _rng(11)
    F, d_k, d_v = 9, 5, 4
    k = rng.standard_normal((F, 1, d_k))          # not unit: exercises ||k||^2
    v = rng.standard_normal((F, 1, d_v))
    beta = rng.random((F, 1)) * 1.5
    As, Bs = O.head_statistics(k, v, beta)
    P = O.forward_states(As, Bs)
    kn2 = np.sum(k[:, 0] ** 2, axis=1)
    beta_p = beta[:, 0] / (1 + beta[:, 0] * kn2)
    S_tok = O.token_delta_rule(np.zeros((d_v, d_k)), k[:, 0], v[:, 0], beta_p)
    np.testing.assert_allclose(P[F], S_tok, rtol=1e-12, atol=1e-13)
    S_same = O.token_delta_rule(np.zeros((d_v, d_k)), k[:, 0], v[:, 0], beta[:, 0])
    assert np.max(np.abs(P[F] - S_same)) > 1e-3
    # a non-zero entering state as well
    S0 = rng.standard_normal((d_v, d_k))
    P2 = O.forward_states(As, Bs, S0)
    np.testing.assert_allclose(P2[F], O.token_delta_rule(S0, k[:, 0], v[:, 0], beta_p),
                               rtol=1e-12, atol=1e-13)


def pin_reverse_is_forward_on_reversed_frames():
    """Algorithm 1 step 5: the reverse scan is the forward scan run on the
    time-reversed frames, reversed back; and it matches an explicit
    descending loop of Eq. A.1."""
    rng = _rng(12)
    q, k, v, beta = _random_clip(rng, F=6)
    As, Bs = O.head_statistics(k, v, beta)
    R = O.reverse_states(As, Bs)
    Pr = O.forward_states(As[::-1], Bs[::-1])
    F = 6
    for j in range(1, F + 2):
        np.testing.assert_allclose(R[j], Pr[F + 1 - j], rtol=1e-13, atol=1e-14)
    S = np.zeros_like(Bs[0])
    for t in range(F, 0, -1):
        M, J = O.frame_transition(As[t - 1], Bs[t - 1])
        S = S @ M + J
        np.testing.assert_allclose(R[t], S, rtol=1e-12, atol=1e-13)


def pin_perturbation_contracts():
    """Eq. A.2: changing the entering state by dS changes the frame's result
    by at most ||dS||_F."""
    rng = _rng(13)
    for U in [1, 4, 100]:
        K, V, beta = _random_frame(rng, U, 6, 5)
        A, B = O.frame_statistics(K, V, beta)
        for _ in range(10):
            S1 = rng.standard_normal((5, 6))
            dS = rng.standard_normal((5, 6))
            d_out = O.joint_frame_update(S1 + dS, A, B) - O.joint_frame_update(S1, A, B)
            assert np.linalg.norm(d_out) <= np.linalg.norm(dS) * (1 + 1e-12)


def pin_affine_composition():
    """Eq. A.1: frames a..b compose into one affine map S -> S M + J with
    M = M_a ... M_b, J = (...(J_a M_{a+1} + J_{a+1}) M_{a+2} ...) + J_b."""
    rng = _rng(14)
    q, k, v, beta = _random_clip(rng, F=7)
    As, Bs = O.head_statistics(k, v, beta)
    S0 = rng.standard_normal(Bs[0].shape)
    P = O.forward_states(As, Bs, S0)
    M_tot = np.eye(As.shape[1])
    J_tot = np.zeros_like(Bs[0])
    for t in range(2, 6):          # frames 3..6 in paper numbering
        M, J = O.frame_transition(As[t], Bs[t])
        M_tot = M_tot @ M
        J_tot = J_tot @ M + J
    np.testing.assert_allclose(P[2] @ M_tot + J_tot, P[6], rtol=1e-12, atol=1e-13)


def pin_whole_operator_orthonormal_keys():
    """Whole operator, before the epilogue: with every key of the clip
    mutually orthonormal, each frame write stays in its own key directions, so
    o_{t,u} = sum_{j != t} sum_w beta/(1+beta) (k_{j,w} . q_{t,u}) v_{j,w}."""
    rng = _rng(15)
    F, N, d_k, d_v = 4, 3, 16, 5
    Qm, _ = np.linalg.qr(rng.standard_normal((d_k, d_k)))
    k = Qm[: F * N].reshape(F, N, d_k)
    v = rng.standard_normal((F, N, d_v))
    beta = rng.random((F, N)) * 3
    q = _unit_rows(rng.standard_normal((F, N, d_k)))
    As, Bs = O.head_statistics(k, v, beta)
    St = O.gathered_states(As, Bs)
    for t in range(F):
        for u in range(N):
            expect = np.zeros(d_v)
            for j in range(F):
                if j == t:
                    continue
                for w in range(N):
                    expect += beta[j, w] / (1 + beta[j, w]) * (k[j, w] @ q[t, u]) * v[j, w]
            np.testing.assert_allclose(O.readout(St[t], q[t])[u], expect, rtol=1e-12, atol=1e-13)


def pin_single_frame_and_lone_writer():
    """Eq. A.4 edge cases: a one-frame clip reads no distant video (y = 0);
    when only frame j writes, frame j reads nothing and every other frame
    reads exactly frame j's single-frame state B_j (I + A_j)^-1."""
    rng = _rng(16)
    q, k, v, beta = _random_clip(rng, F=1)
    y = O.head_forward(q, k, v, beta, 0.7)
    assert np.all(y == 0.0)
    q, k, v, beta = _random_clip(rng, F=5)
    beta[[0, 1, 3, 4]] = 0.0
    As, Bs = O.head_statistics(k, v, beta)
    St = O.gathered_states(As, Bs)
    lone = Bs[2] @ np.linalg.inv(np.eye(As.shape[1]) + As[2])
    assert np.all(St[2] == 0.0)
    for t in [0, 1, 3, 4]:
        np.testing.assert_allclose(St[t], lone, rtol=1e-12, atol=1e-13)


def pin_rmsnorm_library_and_invariances():
    """Eq. 1c: matches torch's RMSNorm (library routine) times the gate; y is
    invariant to v -> c v (c > 0; o is linear in v from a zero state) up to
    eps, and linear in the gate."""
    import torch
    rng = _rng(17)
    o = rng.standard_normal((10, 7))
    y = O.rmsnorm_gate(o, 0.3, eps=1e-6)
    ref = 0.3 * torch.nn.functional.rms_norm(torch.from_numpy(o), (7,), eps=1e-6).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-14)
    q, k, v, beta = _random_clip(rng, F=4)
    y1 = O.head_forward(q, k, v, beta, 0.5, eps=0.0)
    y2 = O.head_forward(q, k, 3.0 * v, beta, 0.5, eps=0.0)
    np.testing.assert_allclose(y1, y2, rtol=1e-11, atol=1e-12)
    y3 = O.head_forward(q, k, v, beta, 0.25, eps=0.0)
    np.testing.assert_allclose(y3, 0.5 * y1, rtol=1e-13, atol=1e-15)
    # per-token mean square of the normalised output is gate^2 (eps = 0)
    np.testing.assert_allclose(np.mean(y1 ** 2, axis=-1), 0.25, rtol=1e-12)


def pin_sampled_matches_full():
    """The sampled readout used at full sizes equals the full operator."""
    rng = _rng(18)
    q, k, v, beta = _random_clip(rng, F=5, N=9, d_k=6, d_v=4)
    y = O.head_forward(q, k, v, beta, 0.8)
    frames = [0, 2, 4, 4, 1]
    toks = [3, 8, 0, 5, 1]
    ys = O.head_forward_sampled(q, k, v, beta, 0.8, frames, toks)
    np.testing.assert_allclose(ys, y[frames, toks], rtol=1e-13, atol=1e-14)


# ----------------------------------------------------------------------------
# Pins of the full gather (decay, window, text state) and the frozen rule
# ----------------------------------------------------------------------------

def _random_alpha(rng, F, d_k, low=0.6):
    return low + (1.0 - low) * rng.random((F, d_k))


def pin_ex_reduces_to_core():
    """alpha = 1, own-frame window, no text state, joint rule: the extended
    operator is the core operator (itself pinned above)."""
    rng = _rng(31)
    q, k, v, beta = _random_clip(rng, F=6, N=7, d_k=5, d_v=4)
    y = O.head_forward(q, k, v, beta, 0.7)
    ye = O.head_forward_ex(q, k, v, beta, 0.7)
    np.testing.assert_allclose(ye, y, rtol=1e-13, atol=1e-14)
    yw = O.head_forward_ex(q, k, v, beta, 0.7, alpha=np.ones((6, 5)),
                           windows=O.local_windows(6, 1, 0, 0))
    np.testing.assert_allclose(yw, y, rtol=1e-13, atol=1e-14)


def pin_decay_single_token_is_token_rule():
    """With one token per frame the decayed joint update is the token-wise
    delta rule of Eq. 2 with decay alpha and write strength
    beta' = beta / (1 + beta |k|^2) (Sherman-Morrison), brute force per token."""
    rng = _rng(32)
    F, d_k, d_v = 6, 4, 3
    keys = _unit_rows(rng.standard_normal((F, d_k))) * 1.3
    vals = rng.standard_normal((F, d_v))
    betas = rng.random(F)
    alphas = _random_alpha(rng, F, d_k)
    S0 = rng.standard_normal((d_v, d_k))
    As = np.stack([betas[t] * np.outer(keys[t], keys[t]) for t in range(F)])
    Bs = np.stack([betas[t] * np.outer(vals[t], keys[t]) for t in range(F)])
    P = O.forward_states_ex(As, Bs, S0, alphas)
    bprime = betas / (1.0 + betas * np.sum(keys * keys, axis=1))
    for j in range(1, F + 1):
        ref = O.token_delta_rule(S0, keys[:j], vals[:j], bprime[:j], alphas[:j])
        np.testing.assert_allclose(P[j], ref, rtol=1e-11, atol=1e-12)


def pin_bridge_is_scan_without_writes():
    """Appendix A.3: the bridge decays the gathered state over the skipped
    local frames without their writes.  So each side of S~_t equals a scan
    that reaches frame t with the window's frames given zero writes (beta = 0
    there: A = B = 0, each such frame only decays)."""
    rng = _rng(33)
    F, N, d_k, d_v = 11, 5, 4, 3
    q, k, v, beta = _random_clip(rng, F=F, N=N, d_k=d_k, d_v=d_v)
    alphas = _random_alpha(rng, F, d_k)
    S_T = rng.standard_normal((d_v, d_k))
    As, Bs = O.head_statistics(k, v, beta)
    windows = O.local_windows(F, 3, 1, 1)
    St = O.gathered_states_ex(As, Bs, S_T, alphas, windows)
    for t in range(1, F + 1):
        lo, hi = windows[t - 1]
        Af, Bf = As.copy(), Bs.copy()
        Af[lo - 1:], Bf[lo - 1:] = 0.0, 0.0           # no writes from frame l_t on
        fwd = O.scan_states_ex(Af[:t], Bf[:t], 0.5 * S_T, alphas[:t])[t]
        Ar, Br = As.copy(), Bs.copy()
        Ar[:hi], Br[:hi] = 0.0, 0.0                   # no writes up to frame h_t
        rev = O.scan_states_ex(Ar[t - 1:][::-1], Br[t - 1:][::-1], 0.5 * S_T,
                               alphas[t - 1:][::-1])[F - t + 1]
        np.testing.assert_allclose(St[t - 1], fwd + rev, rtol=1e-12, atol=1e-13)


def pin_text_state_counted_once():
    """Eq. 1b: with no writes (beta = 0) and alpha = 1 every frame reads
    (S_T/2 + S_T/2) q = S_T q, for any window; with decay the two halves are
    S_T/2 decayed over frames 1..t and over t..F (closed form)."""
    rng = _rng(34)
    F, N, d_k, d_v = 7, 3, 4, 5
    q, k, v, _ = _random_clip(rng, F=F, N=N, d_k=d_k, d_v=d_v)
    beta = np.zeros((F, N))
    S_T = rng.standard_normal((d_v, d_k))
    As, Bs = O.head_statistics(k, v, beta)
    for windows in (None, O.local_windows(F, 2, 1, 0)):
        St = O.gathered_states_ex(As, Bs, S_T, None, windows)
        np.testing.assert_allclose(St, np.broadcast_to(S_T, St.shape), rtol=1e-14, atol=1e-14)
    alphas = _random_alpha(rng, F, d_k)
    St = O.gathered_states_ex(As, Bs, S_T, alphas, O.local_windows(F, 2, 1, 1))
    for t in range(1, F + 1):
        ref = 0.5 * S_T * np.prod(alphas[:t], axis=0)[None, :] \
            + 0.5 * S_T * np.prod(alphas[t - 1:], axis=0)[None, :]
        np.testing.assert_allclose(St[t - 1], ref, rtol=1e-13, atol=1e-14)


def pin_text_state_closed_forms():
    """S_T from the prompt as one frame from zero.  One token: the joint
    solve is Sherman-Morrison's beta/(1 + beta ||k||^2) v k^T and the frozen
    rule (U = 1) is beta v k^T.  Orthonormal keys: each token's weight is
    beta/(1 + beta) (the joint solve decouples), and the frozen rule divides
    by sqrt(L)."""
    rng = _rng(53)
    dk, dv = 5, 4
    k = rng.normal(size=(2, 1, dk))
    v = rng.normal(size=(2, 1, dv))
    beta = rng.uniform(0.1, 1.5, size=(2, 1))
    for h in range(2):
        b, kk, vv = beta[h, 0], k[h, 0], v[h, 0]
        np.testing.assert_allclose(O.text_state(k, v, beta)[h],
                                   b / (1 + b * kk @ kk) * np.outer(vv, kk), rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(O.text_state(k, v, beta, "frozen")[h], b * np.outer(vv, kk),
                                   rtol=1e-12, atol=1e-14)
    L = 3
    Q, _ = np.linalg.qr(rng.normal(size=(dk, dk)))
    k = Q[:L][None]                                   # orthonormal rows
    v = rng.normal(size=(1, L, dv))
    beta = rng.uniform(0.1, 1.5, size=(1, L))
    w = beta[0] / (1 + beta[0])
    np.testing.assert_allclose(O.text_state(k, v, beta)[0],
                               sum(w[u] * np.outer(v[0, u], k[0, u]) for u in range(L)),
                               rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(O.text_state(k, v, beta, "frozen")[0],
                               sum(beta[0, u] * np.outer(v[0, u], k[0, u]) for u in range(L)) / np.sqrt(L),
                               rtol=1e-12, atol=1e-14)


def pin_text_state_minimises_eq4():
    """The joint rule's S_T is the minimiser of Eq. 4 with S_bar = 0 over the
    prompt tokens: no direction lowers the objective (central differences
    vanish and second differences are positive)."""
    rng = _rng(54)
    L, dk, dv = 9, 4, 3
    k = _unit_rows(rng.normal(size=(1, L, dk)))
    v = rng.normal(size=(1, L, dv))
    beta = rng.uniform(0, 1, size=(1, L))
    S = O.text_state(k, v, beta)[0]
    f = lambda X: _eq4(X, np.zeros_like(S), k[0], v[0], beta[0])
    for _ in range(5):
        E = rng.normal(size=S.shape)
        eps = 1e-4
        assert abs(f(S + eps * E) - f(S - eps * E)) / (2 * eps) < 1e-7
        assert f(S + eps * E) > f(S) and f(S - eps * E) > f(S)


def pin_frozen_rule_is_scaled_token_sum():
    """Eq. 3a with every key scaled by 1/sqrt(U) (SANA-WM's scaling, Section
    3.2): Sbar + sum_u beta_u (v_u - Sbar k'_u) k'_u^T with k' = k / sqrt(U),
    summed token by token, is the frozen rule of Eq. 3c with A/U, B/sqrt(U)."""
    rng = _rng(35)
    K, V, beta = _random_frame(rng, U=9, d_k=5, d_v=4)
    S_prev = rng.standard_normal((4, 5))
    alpha = _random_alpha(rng, 1, 5)[0]
    S_bar = S_prev * alpha[None, :]
    Ks = K / np.sqrt(K.shape[0])
    S = S_bar.copy()
    for u in range(K.shape[0]):
        S = S + beta[u] * np.outer(V[u] - S_bar @ Ks[u], Ks[u])
    A, B = O.frame_statistics(K, V, beta)
    got = O.decayed_frame_update(S_prev, A, B, alpha, rule="frozen", U=K.shape[0])
    np.testing.assert_allclose(got, S, rtol=1e-12, atol=1e-13)


def pin_frozen_rule_non_expansive_with_scaling():
    """Appendix A.2: with unit keys and write strengths in [0, 1], the scaled
    additive factor I - A/U has eigenvalues in [0, 1], so the frozen rule's
    inherited-state transition does not expand (checked on differences of
    entering states), while the unscaled factor I - A can (aligned keys)."""
    rng = _rng(36)
    U, d_k, d_v = 12, 4, 3
    base = _unit_rows(rng.standard_normal(d_k))
    K = _unit_rows(base[None, :] + 0.05 * rng.standard_normal((U, d_k)))
    V = rng.standard_normal((U, d_v))
    beta = 0.5 + 0.5 * rng.random(U)
    A, B = O.frame_statistics(K, V, beta)
    ev = np.linalg.eigvalsh(np.eye(d_k) - A / U)
    assert ev.min() >= -1e-12 and ev.max() <= 1 + 1e-12
    assert np.linalg.eigvalsh(np.eye(d_k) - A).min() < -1.0   # unscaled: expands
    for _ in range(5):
        S1, S2 = rng.standard_normal((2, d_v, d_k))
        d1 = O.decayed_frame_update(S1, A, B, rule="frozen", U=U)
        d2 = O.decayed_frame_update(S2, A, B, rule="frozen", U=U)
        assert np.linalg.norm(d1 - d2) <= np.linalg.norm(S1 - S2) * (1 + 1e-12)


def pin_token_gate_reduces_to_head_gate():
    """Eq. 1c with a content-dependent gate G^L: a gate that is constant over
    tokens and channels is the per-head gate, and a gate of ones leaves
    RMSNorm(o) itself."""
    rng = _rng(51)
    H, F, N, dk, dv = 2, 4, 6, 3, 5
    q, k, v, beta = (np.stack(z) for z in zip(*[_random_clip(rng, F, N, dk, dv) for _ in range(H)]))
    gate = np.array([0.3, 0.8])
    base = O.vda_forward_ex(q, k, v, beta, gate, chunk=2, radius=1)
    full = np.broadcast_to(gate[:, None, None, None], (H, F, N, dv)).copy()
    np.testing.assert_allclose(O.vda_forward_ex(q, k, v, beta, None, chunk=2, radius=1,
                                                gate_tokens=full), base, rtol=1e-13, atol=0)
    ones = O.vda_forward_ex(q, k, v, beta, None, chunk=2, radius=1, gate_tokens=np.ones((H, F, N, dv)))
    np.testing.assert_allclose(ones * gate[:, None, None, None], base, rtol=1e-13, atol=0)


def pin_token_gate_applies_after_norm():
    """The gate multiplies the normalised readout channel by channel: scaling
    one channel of one token's gate by c scales exactly that output by c, and
    the result equals torch's rms_norm of the readout times the gate (not the
    norm of the gated readout)."""
    import torch
    rng = _rng(52)
    F, N, dk, dv = 3, 5, 4, 6
    q, k, v, beta = _random_clip(rng, F, N, dk, dv)
    G = rng.uniform(0.05, 1.0, (F, N, dv))
    y = O.head_forward_ex(q, k, v, beta, 1.0, gate_tokens=G)
    G2 = G.copy()
    G2[1, 2, 3] *= 7.0
    y2 = O.head_forward_ex(q, k, v, beta, 1.0, gate_tokens=G2)
    np.testing.assert_allclose(y2[1, 2, 3], 7.0 * y[1, 2, 3], rtol=1e-13)
    mask = np.ones_like(y, dtype=bool)
    mask[1, 2, 3] = False
    np.testing.assert_array_equal(y2[mask], y[mask])
    As, Bs = O.head_statistics(k, v, beta)
    St = O.gathered_states_ex(As, Bs)
    o = np.einsum("tjc,tuc->tuj", St, q)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(o), (dv,), eps=O.RMS_EPS).numpy() * G
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-14)


def pin_local_windows_paper_layout():
    """Section 2.1: chunks of five latent frames, each query chunk sees itself
    and one chunk on each side, a 15-frame window away from the sequence
    ends; every window holds its own frame and all frames of its chunk share
    it; windows are clipped to the interior frames (Appendix A.3)."""
    F = 40
    w = O.local_windows(F, chunk=5, radius=1, offset=1)
    for t in range(1, F + 1):
        lo, hi = w[t - 1]
        assert 1 <= lo <= t <= hi <= F
        first = max(1, 5 * (t // 5))       # first interior frame of t's chunk
        assert w[t - 1] == w[first - 1]
        if lo > 1 and hi < F:
            assert hi - lo + 1 == 15
    # a brute-force membership check: frame r is in t's window iff their
    # chunks differ by at most the radius
    for t in range(1, F + 1):
        lo, hi = w[t - 1]
        inside = [r for r in range(1, F + 1) if abs(r // 5 - t // 5) <= 1]
        assert (lo, hi) == (min(inside), max(inside))
    assert O.local_windows(4, 1, 0, 0) == [(1, 1), (2, 2), (3, 3), (4, 4)]


def pin_chunk_ranges_tile_the_window_grid():
    """Section 2.1 / Section 4: the chunks of the window grid, clipped to the
    clip, cover every frame once, in order, and two frames share a chunk
    exactly when they share a radius-0 window.  Hand-derived layout: 12
    frames in chunks of 5 after one leading anchor are frames 0-3, 4-8 and
    9-11 (array numbering)."""
    assert O.chunk_ranges(12, 5, 1) == [(0, 3), (4, 8), (9, 11)]
    assert O.chunk_ranges(10, 5, 0) == [(0, 4), (5, 9)]
    assert O.chunk_ranges(3, 5, 4) == [(0, 0), (1, 2)]
    assert O.chunk_ranges(4, 1, 0) == [(0, 0), (1, 1), (2, 2), (3, 3)]
    for F, chunk, offset in ((1, 3, 0), (7, 3, 2), (36, 5, 1), (40, 5, 0), (13, 4, 3)):
        ranges = O.chunk_ranges(F, chunk, offset)
        frames = [t for lo, hi in ranges for t in range(lo, hi + 1)]
        assert frames == list(range(F))
        assert all(hi - lo + 1 <= chunk for lo, hi in ranges)
        own = O.local_windows(F, chunk, 0, offset)      # paper numbering
        for lo, hi in ranges:
            for t in range(lo, hi + 1):
                assert own[t] == (lo + 1, hi + 1)


def pin_chunk_scan_matches_frame_scan():
    """Section 4, chunk-wise scans: composing each chunk into S_out = S_in M
    + J (Eq. A.1) and scanning the chunk sequence gives, at every chunk
    boundary and in both directions, the states of the frame-by-frame scans
    (with decay and a text state)."""
    rng = _rng(31)
    q, k, v, beta = _random_clip(rng, F=11, N=5, d_k=4, d_v=3)
    As, Bs = O.head_statistics(k, v, beta)
    alphas = _random_alpha(rng, 11, 4)
    S0 = 0.5 * rng.standard_normal((3, 4))
    P = O.forward_states_ex(As, Bs, S0, alphas)
    R = O.reverse_states_ex(As, Bs, S0, alphas)
    for chunk, offset in ((5, 1), (3, 0), (4, 2), (11, 0), (1, 0)):
        Pb, Rb = O.chunk_boundary_states(As, Bs, S0, chunk, offset, alphas)
        for c, (lo, hi) in enumerate(O.chunk_ranges(11, chunk, offset)):
            np.testing.assert_allclose(Pb[c], P[lo], rtol=1e-11, atol=1e-12)
            np.testing.assert_allclose(Rb[c], R[hi + 2], rtol=1e-11, atol=1e-12)


def _prep_case(rng, F=4, gh=5, gw=6, H=2, d=3):
    C = H * d
    x = {n: rng.standard_normal((F, gh * gw, C)) for n in ("q", "k", "v")}
    w = {n: rng.standard_normal(shape) for n, shape in
         (("ks", (C, 5, 5)), ("kt", (C, 5)), ("vs", (C, 5, 5)), ("vt", (C, 5)))}
    return x, w, (gh, gw), H


def pin_prep_conv_matches_library():
    """Section 2.3: the depthwise 5 x 5 spatial and five-tap temporal filters
    equal torch's grouped 3-D cross-correlation with the separable kernel
    w_t[c, dt] w_s[c, dy, dx] and zero padding 2 (a textbook reduction)."""
    import torch
    rng = _rng(41)
    F, gh, gw, C = 6, 5, 7, 3
    x = rng.standard_normal((F, gh, gw, C))
    ws, wt = rng.standard_normal((C, 5, 5)), rng.standard_normal((C, 5))
    got = O.depthwise_conv3(x, ws, wt)
    kern = torch.from_numpy(wt[:, :, None, None] * ws[:, None, :, :])[:, None]   # [C,1,5,5,5]
    xt = torch.from_numpy(np.ascontiguousarray(x.transpose(3, 0, 1, 2)))[None]   # [1,C,F,gh,gw]
    ref = torch.nn.functional.conv3d(xt, kern, padding=2, groups=C)[0].numpy().transpose(1, 2, 3, 0)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def pin_prep_conv_hand_cases():
    """Hand-derived cases: centred unit taps pass the input through; a spatial
    tap at offset (0, +1) reads the right-hand neighbour (zero past the last
    column); a temporal tap at offset -1 reads the previous frame (zero before
    the first)."""
    rng = _rng(42)
    F, gh, gw, C = 3, 2, 3, 2
    x = rng.standard_normal((F, gh, gw, C))
    ws = np.zeros((C, 5, 5))
    wt = np.zeros((C, 5))
    ws[:, 2, 2] = 1.0
    wt[:, 2] = 1.0
    np.testing.assert_array_equal(O.depthwise_conv3(x, ws, wt), x)
    ws2 = np.zeros((C, 5, 5))
    ws2[:, 2, 3] = 1.0
    exp = np.zeros_like(x)
    exp[:, :, :-1] = x[:, :, 1:]
    np.testing.assert_array_equal(O.depthwise_conv3(x, ws2, wt), exp)
    wt2 = np.zeros((C, 5))
    wt2[:, 1] = 1.0
    exp = np.zeros_like(x)
    exp[1:] = x[:-1]
    np.testing.assert_array_equal(O.depthwise_conv3(x, ws, wt2), exp)


def pin_prep_feature_map():
    """Section 2.3: K and V are convolved then passed through SiLU (torch's
    silu), Q and K are L2-normalised per token and head (unit norm when the
    norm dwarfs eps; torch's normalize), V is not normalised, and the layout
    is [head][frame][token][channel] with head h taking channels h*d..h*d+d-1."""
    import torch
    rng = _rng(43)
    x, w, grid, H = _prep_case(rng, d=8)
    q, k, v = O.vda_prep(x["q"], x["k"], x["v"], grid, H, w["ks"], w["kt"], w["vs"], w["vt"])
    F, N, C = x["q"].shape
    d = C // H
    conv = lambda t, ws, wt: O.depthwise_conv3(t.reshape(F, grid[0], grid[1], C), ws, wt).reshape(F, N, C)
    silu = lambda t: torch.nn.functional.silu(torch.from_numpy(t)).numpy()
    norm = lambda t: torch.nn.functional.normalize(torch.from_numpy(t), dim=-1).numpy()
    kc, vc = silu(conv(x["k"], w["ks"], w["kt"])), silu(conv(x["v"], w["vs"], w["vt"]))
    for h in range(H):
        sl = slice(h * d, (h + 1) * d)
        # eps inside the square root moves the result by ~eps / (2 |x|^2)
        np.testing.assert_allclose(q[h], norm(x["q"][:, :, sl]), rtol=2e-5, atol=1e-9)
        np.testing.assert_allclose(k[h], norm(kc[:, :, sl]), rtol=2e-5, atol=1e-9)
        np.testing.assert_allclose(v[h], vc[:, :, sl], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(np.linalg.norm(q, axis=-1), 1.0, atol=2e-5)


def pin_prep_filters_commute():
    """The spatial and temporal filters are linear and act on different axes,
    so applying the temporal filter first (as a pass with a unit spatial
    tap) and the spatial one second gives the same result."""
    rng = _rng(44)
    F, gh, gw, C = 5, 4, 6, 2
    x = rng.standard_normal((F, gh, gw, C))
    ws, wt = rng.standard_normal((C, 5, 5)), rng.standard_normal((C, 5))
    unit_s = np.zeros((C, 5, 5))
    unit_s[:, 2, 2] = 1.0
    unit_t = np.zeros((C, 5))
    unit_t[:, 2] = 1.0
    two_pass = O.depthwise_conv3(O.depthwise_conv3(x, unit_s, wt), ws, unit_t)
    np.testing.assert_allclose(O.depthwise_conv3(x, ws, wt), two_pass, rtol=1e-12, atol=1e-12)


def pin_query_l2_folds_into_rmsnorm():
    """Section 2.3 with Eq. 1c: the readout is linear in the query and RMSNorm
    is scale-invariant up to its epsilon, so with the raw query q and
    n = |q|^2 + eps_l2, RMSNorm(S (q / sqrt(n))) = S q / sqrt(mean((S q)^2) +
    eps_rms n) times the gate: the form in which a readout of the raw query
    applies the L2 map.  Checked on scales from 1e-3 to 1e3 and a zero query
    (whose output is zero either way)."""
    rng = _rng(45)
    S = rng.standard_normal((6, 5))
    q = rng.standard_normal((9, 5)) * np.exp(rng.uniform(-7.0, 7.0, (9, 1)))
    q[4] = 0.0
    eps_rms = O.RMS_EPS
    y = O.rmsnorm_gate(O.readout(S, O.l2_normalise(q)), 0.7, eps=eps_rms)
    o = q @ S.T
    n = np.sum(q * q, axis=-1, keepdims=True) + O.L2_EPS
    folded = 0.7 * o / np.sqrt(np.mean(o * o, axis=-1, keepdims=True) + eps_rms * n)
    np.testing.assert_allclose(y, folded, rtol=1e-12, atol=1e-15)
    assert np.all(y[4] == 0.0)


PINS = [f for name, f in sorted(globals().items()) if name.startswith("pin_")]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin()


# ----------------------------------------------------------------------------
# Planted mistakes: each must be caught by at least one pin
# ----------------------------------------------------------------------------

def _mut_stats_no_beta(K, V, beta):
    return K.T @ K, V.T @ K


def _mut_stats_beta_squared(K, V, beta):
    KD = K * (beta ** 2)[:, None]
    return K.T @ KD, V.T @ KD


def _mut_update_no_identity(S_bar, A, B):
    return (S_bar + B) @ np.linalg.pinv(A)


def _mut_update_frozen_state(S_bar, A, B):
    return S_bar @ (np.eye(A.shape[0]) - A) + B


def _mut_update_drop_inherited(S_bar, A, B):
    return B @ np.linalg.inv(np.eye(A.shape[0]) + A)


def _mut_update_wrong_sign(S_bar, A, B):
    return (S_bar - B) @ np.linalg.inv(np.eye(A.shape[0]) + A)


def _mut_gather_inclusive(As, Bs):
    F = As.shape[0]
    P = O.forward_states(As, Bs)
    R = O.reverse_states(As, Bs)
    return np.stack([P[t] + R[t] for t in range(1, F + 1)])


def _mut_gather_forward_only(As, Bs):
    F = As.shape[0]
    P = O.forward_states(As, Bs)
    return np.stack([P[t - 1] for t in range(1, F + 1)])


def _mut_gather_swapped(As, Bs):
    F = As.shape[0]
    P = O.forward_states(As, Bs)
    R = O.reverse_states(As, Bs)
    zero = np.zeros_like(P[0])
    return np.stack([(R[t - 1] if t >= 2 else zero) + (P[t + 1] if t + 1 <= F else zero)
                     for t in range(1, F + 1)])


def _mut_reverse_not_reversed(As, Bs, S0=None):
    F, d_v, d_k = Bs.shape
    fwd = O.scan_states(As, Bs, np.zeros((d_v, d_k)) if S0 is None else S0)
    R = np.zeros((F + 2, d_v, d_k))
    for j in range(1, F + 2):
        R[j] = fwd[F + 1 - j]
    return R


def _mut_readout_transposed(S_tilde, q):
    return q @ S_tilde


def _mut_rms_sum_not_mean(o, gate, eps=O.RMS_EPS):
    return gate * o / np.sqrt(np.sum(o * o, axis=-1, keepdims=True) + eps)


def _mut_rms_gate_inside(o, gate, eps=O.RMS_EPS):
    og = gate * o
    return og / np.sqrt(np.mean(og * og, axis=-1, keepdims=True) + eps)


def _mut_decay_after_update(S_prev, A, B, alpha=None, rule="joint", U=None):
    if rule == "joint":
        S = O.joint_frame_update(S_prev, A, B)
    else:
        S = O.frozen_state_update(S_prev, A, B, U)
    return S if alpha is None else S * np.asarray(alpha)[None, :]


def _mut_frozen_unscaled(S_prev, A, B, alpha=None, rule="joint", U=None):
    S_bar = S_prev if alpha is None else S_prev * np.asarray(alpha)[None, :]
    if rule == "joint":
        return O.joint_frame_update(S_bar, A, B)
    return O.frozen_state_update(S_bar, A, B, None)


def _mut_bridge_skips_own_decay(As, Bs, S_T=None, alphas=None, windows=None, rule="joint", U=None):
    F, d_v, d_k = Bs.shape
    S0 = np.zeros((d_v, d_k)) if S_T is None else 0.5 * np.asarray(S_T)
    P = O.forward_states_ex(As, Bs, S0, alphas, rule, U)
    R = O.reverse_states_ex(As, Bs, S0, alphas, rule, U)
    windows = windows or [(t, t) for t in range(1, F + 1)]
    out = np.empty((F, d_v, d_k))
    for t in range(1, F + 1):
        lo, hi = windows[t - 1]
        df = np.ones(d_k) if alphas is None else np.prod(alphas[lo - 1:t - 1], axis=0)
        dr = np.ones(d_k) if alphas is None else np.prod(alphas[t - 1:hi], axis=0)
        out[t - 1] = P[lo - 1] * df[None, :] + R[hi + 1] * dr[None, :]
    return out


def _mut_text_state_not_halved(As, Bs, S_T=None, alphas=None, windows=None, rule="joint", U=None):
    S2 = None if S_T is None else 2.0 * np.asarray(S_T)
    return _ORIG_GATHER_EX(As, Bs, S2, alphas, windows, rule, U)


def _mut_windows_ignore_offset(F, chunk=1, radius=0, offset=0):
    return _ORIG_WINDOWS(F, chunk, radius, 0)


def _mut_chunk_map_wrong_order(As, Bs, frames, alphas=None):
    d_k, d_v = As.shape[1], Bs.shape[1]
    M, J = np.eye(d_k), np.zeros((d_v, d_k))
    for t in frames:
        Mt, Jt = O.frame_transition(As[t], Bs[t], None if alphas is None else alphas[t])
        M = Mt @ M
        J = J @ Mt + Jt
    return M, J


def _mut_chunk_ranges_unclipped(F, chunk, offset=0):
    return [(lo, min(F - 1, lo + chunk - 1)) for lo, _ in _ORIG_CHUNK_RANGES(F, chunk, offset)]


def _mut_conv_wraps(x, w_spatial, w_temporal):
    F, gh, gw, C = x.shape
    s = np.zeros_like(x)
    for dy in range(5):
        for dx in range(5):
            s += w_spatial[:, dy, dx] * np.roll(x, (2 - dy, 2 - dx), axis=(1, 2))
    out = np.zeros_like(x)
    for dt in range(5):
        out += w_temporal[:, dt] * np.roll(s, 2 - dt, axis=0)
    return out


def _mut_conv_flipped(x, w_spatial, w_temporal):
    return _ORIG_CONV(x, w_spatial[:, ::-1, ::-1], w_temporal[:, ::-1])


def _mut_l2_over_tokens(x, eps=O.L2_EPS):
    return x / np.sqrt(np.sum(x * x, axis=-2, keepdims=True) + eps)


def _mut_silu_is_sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


_ORIG_CONV = O.depthwise_conv3
_ORIG_GATHER_EX = O.gathered_states_ex
_ORIG_WINDOWS = O.local_windows
_ORIG_CHUNK_RANGES = O.chunk_ranges

_ORIG_HEAD_FORWARD_EX = O.head_forward_ex


def _mut_token_gate_before_norm(q, k, v, beta, gate, alpha=None, S_T=None, windows=None,
                                rule="joint", eps=O.RMS_EPS, gate_tokens=None):
    if gate_tokens is None:
        return _ORIG_HEAD_FORWARD_EX(q, k, v, beta, gate, alpha, S_T, windows, rule, eps)
    As, Bs = O.head_statistics(k, v, beta)
    St = O.gathered_states_ex(As, Bs, S_T, alpha, windows, rule, U=k.shape[1])
    y = np.empty(q.shape[:2] + (v.shape[2],))
    for t in range(q.shape[0]):
        y[t] = O.rmsnorm_gate(gate_tokens[t] * O.readout(St[t], q[t]), 1.0, eps)
    return y


_ORIG_TEXT_STATE = O.text_state


def _mut_text_state_halved(k, v, beta, rule="joint"):
    return 0.5 * _ORIG_TEXT_STATE(k, v, beta, rule)


def _mut_text_state_frame_u(k, v, beta, rule="joint"):
    if rule != "frozen":
        return _ORIG_TEXT_STATE(k, v, beta, rule)
    return np.stack([O.frame_statistics(k[h], v[h], beta[h])[1] for h in range(k.shape[0])])


_ORIG_FORWARD = O.vda_forward
_ORIG_FORWARD_EX = O.vda_forward_ex


def _mut_forward_gate0(q, k, v, beta, gate, eps=O.RMS_EPS):
    return np.stack([O.head_forward(q[h], k[h], v[h], beta[h], float(gate[0]), eps)
                     for h in range(q.shape[0])])


def _mut_forward_heads_reversed(q, k, v, beta, gate, eps=O.RMS_EPS):
    return _ORIG_FORWARD(q, k, v, beta, gate, eps)[::-1]


def _mut_forward_ex_alpha0(q, k, v, beta, gate, alpha=None, S_T=None, chunk=1, radius=0,
                           offset=0, rule="joint", eps=O.RMS_EPS, gate_tokens=None):
    a = None if alpha is None else np.broadcast_to(alpha[:1], alpha.shape)
    return _ORIG_FORWARD_EX(q, k, v, beta, gate, a, S_T, chunk, radius, offset, rule, eps,
                            gate_tokens)


def _mut_forward_ex_text_state0(q, k, v, beta, gate, alpha=None, S_T=None, chunk=1, radius=0,
                                offset=0, rule="joint", eps=O.RMS_EPS, gate_tokens=None):
    s = None if S_T is None else np.broadcast_to(S_T[:1], S_T.shape)
    return _ORIG_FORWARD_EX(q, k, v, beta, gate, alpha, s, chunk, radius, offset, rule, eps,
                            gate_tokens)


def _mut_forward_ex_token_gate0(q, k, v, beta, gate, alpha=None, S_T=None, chunk=1, radius=0,
                                offset=0, rule="joint", eps=O.RMS_EPS, gate_tokens=None):
    G = None if gate_tokens is None else np.broadcast_to(gate_tokens[:1], gate_tokens.shape)
    return _ORIG_FORWARD_EX(q, k, v, beta, gate, alpha, S_T, chunk, radius, offset, rule, eps, G)


def _mut_forward_ex_heads_reversed(*args, **kw):
    return _ORIG_FORWARD_EX(*args, **kw)[::-1]


MUTANTS = [
    ("vda_forward", _mut_forward_gate0),
    ("vda_forward", _mut_forward_heads_reversed),
    ("vda_forward_ex", _mut_forward_ex_alpha0),
    ("vda_forward_ex", _mut_forward_ex_text_state0),
    ("vda_forward_ex", _mut_forward_ex_token_gate0),
    ("vda_forward_ex", _mut_forward_ex_heads_reversed),
    ("decayed_frame_update", _mut_decay_after_update),
    ("decayed_frame_update", _mut_frozen_unscaled),
    ("gathered_states_ex", _mut_bridge_skips_own_decay),
    ("gathered_states_ex", _mut_text_state_not_halved),
    ("local_windows", _mut_windows_ignore_offset),
    ("head_forward_ex", _mut_token_gate_before_norm),
    ("text_state", _mut_text_state_halved),
    ("text_state", _mut_text_state_frame_u),
    ("chunk_map", _mut_chunk_map_wrong_order),
    ("depthwise_conv3", _mut_conv_wraps),
    ("depthwise_conv3", _mut_conv_flipped),
    ("l2_normalise", _mut_l2_over_tokens),
    ("silu", _mut_silu_is_sigmoid),
    ("chunk_ranges", _mut_chunk_ranges_unclipped),
    ("frame_statistics", _mut_stats_no_beta),
    ("frame_statistics", _mut_stats_beta_squared),
    ("joint_frame_update", _mut_update_no_identity),
    ("joint_frame_update", _mut_update_frozen_state),
    ("joint_frame_update", _mut_update_drop_inherited),
    ("joint_frame_update", _mut_update_wrong_sign),
    ("gathered_states", _mut_gather_inclusive),
    ("gathered_states", _mut_gather_forward_only),
    ("gathered_states", _mut_gather_swapped),
    ("reverse_states", _mut_reverse_not_reversed),
    ("readout", _mut_readout_transposed),
    ("rmsnorm_gate", _mut_rms_sum_not_mean),
    ("rmsnorm_gate", _mut_rms_gate_inside),
]


@pytest.mark.parametrize("target,mutant", MUTANTS, ids=[m.__name__ for _, m in MUTANTS])
def test_mutants_are_caught(monkeypatch, target, mutant):
    monkeypatch.setattr(O, target, mutant)
    caught = []
    for pin in PINS:
        try:
            with np.errstate(all="ignore"):
                pin()
        except Exception:
            caught.append(pin.__name__)
    assert caught, f"no pin detects the planted mistake {mutant.__name__}"
