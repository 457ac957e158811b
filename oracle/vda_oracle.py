"""Plain fp64 CPU oracle for the Video Delta Attention (VDA) forward pass.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports or calls this
module; only the test-suite, the smoke check and the benchmark's CPU-baseline
leg may.  It shares no code, constants or helpers with the HIP library.

It computes the operator straight from its definition in the paper
(arXiv 2609.20744, "Video DeltaNet"), in float64, one head problem at a time,
with no blocking, fusion or reordering beyond what the equations state:

* Frame statistics, Eq. 3b (Section 3.1):
      A_t = K_t^T Diag(beta_t) K_t,   B_t = V_t^T Diag(beta_t) K_t.
* Joint frame update, Eq. 4 -> Eq. 5 (Section 3.2): the unique minimiser
      S_t = (Sbar_t + B_t)(I + A_t)^{-1},
  evaluated with a Cholesky solve of the SPD key-space matrix I + A_t.
* With no decay input, Sbar_t = S_{t-1} (alpha = 1), so each frame is the
  affine map S_t = S_{t-1} M_t + J_t of Eq. A.1 (Appendix A.1), scanned in
  both temporal directions (Algorithm 1, step 5) from a zero initial state
  (Eq. 1b with no text state).
* Boundary gather, Eq. A.4 (Appendix A.3), with the local window reduced to
  the query's own frame and alpha = 1: frame t reads P_{t-1} + R_{t+1}, the
  forward state through the previous frame plus the reverse state through
  the next one (the two regions are disjoint, Section 2.2, Eq. 1a).
* Readout o_{t,u} = S~_t q_{t,u}, then the branch epilogue of Eq. 1c:
      y = g * RMSNorm(o),  RMSNorm(o) = o / sqrt(mean_j o_j^2 + eps),
  over the d_v channels of one token of one head, no learnable weight.

The chunk-wise scans (chunk_map, chunk_boundary_states) compose each chunk
of the window grid into one affine map of Eq. A.1 and scan the chunk
sequence (Section 4); they give the states at chunk boundaries, which equal
the frame-by-frame scans' states there.

The feature map before the operator (vda_prep: depthwise 5 x 5 spatial and
five-tap temporal convolution of K and V, SiLU, L2 normalisation of Q and K,
frame-major layout per head) is the VDA-Prep step of Section 4.

The full gather (the *_ex functions at the end) adds what the core leaves
at its special values: the channel-wise decay alpha_t (S_bar_t =
S_{t-1} Diag(alpha_t), Eq. 3a/5 and A.1), the text state S_T starting both
scans at S_T / 2 (Eq. 1b; text_state forms S_T from the prompt), the local
window [l_t, h_t] with the decay bridge of Eq. A.4, the content-dependent output gate G^L of Eq. 1c (one value per
token and channel, applied after RMSNorm, in place of the per-head gate),
and, as a selectable rule, the frozen-state additive update of Eq. 3c with
the 1/sqrt(U) key scaling the paper compares against (Section 3.2, Appendix
A.2).

Index convention: the paper numbers frames 1..F; arrays here use 0..F-1, so
array frame i is the paper's frame t = i + 1.

Every function here is pinned by the CPU tests against values the paper's
equations fix independently of this code (closed forms, invariants, a
hand-derived worked example, library routines and brute force).
"""
from __future__ import annotations

import numpy as np
import scipy.linalg

#: RMSNorm epsilon.  The paper does not state it; 1e-6 is the reading used.
RMS_EPS = 1e-6


# ----------------------------------------------------------------------------
# One frame
# ----------------------------------------------------------------------------

def frame_statistics(K: np.ndarray, V: np.ndarray, beta: np.ndarray):
    """Eq. 3b: A = K^T Diag(beta) K (d_k x d_k), B = V^T Diag(beta) K (d_v x d_k).

    K [U, d_k], V [U, d_v], beta [U] (all float64).
    """
    KD = K * beta[:, None]          # Diag(beta) K
    A = K.T @ KD
    B = V.T @ KD
    return A, B


def joint_frame_update(S_bar: np.ndarray, A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """Eq. 5: the S solving S (I + A) = S_bar + B.

    I + A is symmetric positive definite (A is a beta-weighted Gram matrix,
    beta >= 0; Appendix A.1), so the right solve X C = Y is done as
    C X^T = Y^T with a Cholesky factorisation.
    """
    C = np.eye(A.shape[0]) + A
    Y = S_bar + B
    factor = scipy.linalg.cho_factor(C, lower=True)
    return scipy.linalg.cho_solve(factor, Y.T).T


def frame_transition(A: np.ndarray, B: np.ndarray, alpha: np.ndarray | None = None):
    """Eq. A.1: M = Diag(alpha) (I + A)^{-1}, J = B (I + A)^{-1}.

    Used by the composition and contraction checks; the scan itself uses
    joint_frame_update, which is the same map.
    """
    Cinv = np.linalg.inv(np.eye(A.shape[0]) + A)
    M = Cinv if alpha is None else np.diag(alpha) @ Cinv
    return M, B @ Cinv


# ----------------------------------------------------------------------------
# One head problem: scans, gather, readout, epilogue
# ----------------------------------------------------------------------------

def head_statistics(k: np.ndarray, v: np.ndarray, beta: np.ndarray):
    """Eq. 3b for every frame of one head.  k [F,N,d_k], v [F,N,d_v], beta [F,N]."""
    F = k.shape[0]
    As = np.empty((F, k.shape[2], k.shape[2]))
    Bs = np.empty((F, v.shape[2], k.shape[2]))
    for t in range(F):
        As[t], Bs[t] = frame_statistics(k[t], v[t], beta[t])
    return As, Bs


def scan_states(As: np.ndarray, Bs: np.ndarray, S0: np.ndarray) -> np.ndarray:
    """Apply the frame map of Eq. 5 (alpha = 1) to frames 0..F-1 in order.

    Returns [F+1, d_v, d_k]: element j is the state after the first j frames
    (element 0 is the initial state S0).
    """
    F = As.shape[0]
    out = np.empty((F + 1,) + S0.shape)
    out[0] = S0
    for t in range(F):
        out[t + 1] = joint_frame_update(out[t], As[t], Bs[t])
    return out


def forward_states(As, Bs, S0=None):
    """Forward scan (Algorithm 1, step 5).  P[j] = state through frames 1..j
    (paper numbering), P[0] the virtual initial state."""
    d_v, d_k = Bs.shape[1], Bs.shape[2]
    S0 = np.zeros((d_v, d_k)) if S0 is None else S0
    return scan_states(As, Bs, S0)


def reverse_states(As, Bs, S0=None):
    """Reverse scan (Algorithm 1, step 5), the same frame map applied from the
    last frame down.  Returns R of length F+2 in paper numbering:
    R[j] = state through frames F..j for j = 1..F, R[F+1] = initial state,
    R[0] unused (zero)."""
    F, d_v, d_k = Bs.shape
    S0 = np.zeros((d_v, d_k)) if S0 is None else S0
    rev = scan_states(As[::-1], Bs[::-1], S0)      # rev[m] = through last m frames
    R = np.zeros((F + 2, d_v, d_k))
    for j in range(1, F + 2):
        R[j] = rev[F + 1 - j]
    return R


def gathered_states(As, Bs) -> np.ndarray:
    """Eq. A.4 with window [t, t] and alpha = 1, no text state: the state read
    by array frame i (paper frame t = i + 1) is P_{t-1} + R_{t+1}.
    Returns [F, d_v, d_k]."""
    F = As.shape[0]
    P = forward_states(As, Bs)
    R = reverse_states(As, Bs)
    return np.stack([P[t - 1] + R[t + 1] for t in range(1, F + 1)])


def readout(S_tilde: np.ndarray, q: np.ndarray) -> np.ndarray:
    """Eq. A.4 last line / Eq. 1a: o_{t,u} = S~_t q_{t,u}.  q [U, d_k] -> [U, d_v]."""
    return q @ S_tilde.T


def rmsnorm_gate(o: np.ndarray, gate, eps: float = RMS_EPS) -> np.ndarray:
    """Eq. 1c, linear branch: G * RMSNorm(o), the RMS over the last (d_v)
    axis; G is one value per head, or an array of o's shape (the
    content-dependent output gate, elementwise)."""
    ms = np.mean(o * o, axis=-1, keepdims=True)
    return gate * o / np.sqrt(ms + eps)


def head_forward(q, k, v, beta, gate: float, eps: float = RMS_EPS) -> np.ndarray:
    """Whole operator for one head problem.  q,k [F,N,d_k], v [F,N,d_v],
    beta [F,N] (float64, beta >= 0) -> y [F,N,d_v]."""
    if np.any(beta < 0):
        raise ValueError("write strengths must be non-negative")
    As, Bs = head_statistics(k, v, beta)
    St = gathered_states(As, Bs)
    y = np.empty(q.shape[:2] + (v.shape[2],))
    for t in range(q.shape[0]):
        y[t] = rmsnorm_gate(readout(St[t], q[t]), gate, eps)
    return y


def vda_forward(q, k, v, beta, gate, eps: float = RMS_EPS) -> np.ndarray:
    """All head problems: q,k [H,F,N,d_k], v [H,F,N,d_v], beta [H,F,N],
    gate [H] (float64) -> y [H,F,N,d_v]."""
    return np.stack([head_forward(q[h], k[h], v[h], beta[h], float(gate[h]), eps)
                     for h in range(q.shape[0])])


def head_forward_sampled(q, k, v, beta, gate: float, frames, tokens,
                         eps: float = RMS_EPS) -> np.ndarray:
    """Outputs of one head at the listed (frame, token) positions only.

    The states still come from every frame of the head (the scans need all of
    them); only the readout is restricted.  Returns [len(frames), d_v].
    """
    As, Bs = head_statistics(k, v, beta)
    St = gathered_states(As, Bs)
    frames = np.asarray(frames)
    tokens = np.asarray(tokens)
    o = np.einsum("sjc,sc->sj", St[frames], q[frames, tokens])
    return rmsnorm_gate(o, gate, eps)


# ----------------------------------------------------------------------------
# Other forms of the same rule, and neighbouring rules, for the checks
# ----------------------------------------------------------------------------

def joint_frame_update_token_space(S_bar, K, V, beta) -> np.ndarray:
    """The same minimiser reached through a U x U solve in token space.

    The first-order condition of Eq. 4 reads S = S_bar + W^T K with
    W = Diag(beta)(V - K S^T) (Appendix A.2's rearranged form); substituting
    S gives (I_U + Diag(beta) K K^T) W = Diag(beta)(V - K S_bar^T).
    """
    U = K.shape[0]
    D = np.diag(beta)
    W = np.linalg.solve(np.eye(U) + D @ K @ K.T, D @ (V - K @ S_bar.T))
    return S_bar + W.T @ K


def token_delta_rule(S0, keys, values, betas, alphas=None) -> np.ndarray:
    """Eq. 2, one token per step: Sbar = S Diag(alpha); S = Sbar + beta (v - Sbar k) k^T.
    keys [T,d_k], values [T,d_v], betas [T]; returns the final state."""
    S = np.array(S0, dtype=np.float64)
    for i in range(keys.shape[0]):
        if alphas is not None:
            S = S @ np.diag(alphas[i])
        kk, vv = keys[i], values[i]
        S = S + betas[i] * np.outer(vv - S @ kk, kk)
    return S


def frozen_state_update(S_bar, A, B, U: int | None = None) -> np.ndarray:
    """Eq. 3c: S = S_bar (I - A) + B; with U given, the 1/sqrt(U) key scaling
    of Appendix A.2 (A -> A/U, B -> B/sqrt(U))."""
    if U is not None:
        A, B = A / U, B / np.sqrt(U)
    return S_bar @ (np.eye(A.shape[0]) - A) + B


# ----------------------------------------------------------------------------
# The full gather: decay, local window, text state; the frozen-state rule
# ----------------------------------------------------------------------------
#
# Section 2.2 (Eq. 1a, 1b), Section 3.1 (Eq. 3c), Appendix A.1 (Eq. A.1),
# Appendix A.3 (Eq. A.4) and Algorithm 1, steps 3-7.  The core functions
# above are the special case alpha = 1, window = own frame, S_T = 0 and the
# joint rule.

RULES = ("joint", "frozen")


def decayed_frame_update(S_prev, A, B, alpha=None, rule="joint", U=None):
    """One frame of either rule from the entering state S_prev.

    The decayed state is Sbar = S_prev Diag(alpha) (alpha per key channel,
    None = 1).  'joint': Eq. 5, S = (Sbar + B)(I + A)^{-1} (so S = S_prev M + J
    with M = Diag(alpha)(I + A)^{-1}, J = B (I + A)^{-1}, Eq. A.1).  'frozen':
    Eq. 3c with the 1/sqrt(U) key scaling, S = Sbar (I - A/U) + B/sqrt(U).
    """
    S_bar = S_prev if alpha is None else S_prev * np.asarray(alpha)[None, :]
    if rule == "joint":
        return joint_frame_update(S_bar, A, B)
    if rule == "frozen":
        return frozen_state_update(S_bar, A, B, U)
    raise ValueError(f"unknown rule {rule!r}")


def scan_states_ex(As, Bs, S0, alphas=None, rule="joint", U=None):
    """decayed_frame_update over frames 0..F-1 in order from S0.
    Returns [F+1, d_v, d_k]; element j is the state after the first j frames."""
    F = As.shape[0]
    out = np.empty((F + 1,) + S0.shape)
    out[0] = S0
    for t in range(F):
        a = None if alphas is None else alphas[t]
        out[t + 1] = decayed_frame_update(out[t], As[t], Bs[t], a, rule, U)
    return out


def forward_states_ex(As, Bs, S0, alphas=None, rule="joint", U=None):
    """P[j] = state through frames 1..j (paper numbering), P[0] = S0."""
    return scan_states_ex(As, Bs, S0, alphas, rule, U)


def reverse_states_ex(As, Bs, S0, alphas=None, rule="joint", U=None):
    """R[j] = state through frames F..j (paper numbering) for j = 1..F,
    R[F+1] = S0; R[0] unused (zero).  Each frame applies its own decay."""
    F = Bs.shape[0]
    a_rev = None if alphas is None else alphas[::-1]
    rev = scan_states_ex(As[::-1], Bs[::-1], S0, a_rev, rule, U)
    R = np.zeros((F + 2,) + S0.shape)
    for j in range(1, F + 2):
        R[j] = rev[F + 1 - j]
    return R


def local_windows(F: int, chunk: int = 1, radius: int = 0, offset: int = 0):
    """Local Softmax window [l_t, h_t] of every interior frame t = 1..F.

    Frames are grouped into chunks of `chunk` consecutive frames, counted
    from `offset` positions before interior frame 1 (for example the leading
    anchor frame); a query frame's window is its own chunk and `radius`
    chunks on each side (Section 2.1: chunks of five latent frames, radius
    one), clipped to the interior frames (Appendix A.3).  Returns a list of
    (l_t, h_t) in paper numbering.
    """
    out = []
    for t in range(1, F + 1):
        c = (t - 1 + offset) // chunk
        lo = (c - radius) * chunk - offset + 1
        hi = (c + radius + 1) * chunk - offset
        out.append((max(1, lo), min(F, hi)))
    return out


def gathered_states_ex(As, Bs, S_T=None, alphas=None, windows=None, rule="joint", U=None):
    """Eq. A.4: S~_t = P_{l_t-1} Diag(prod_{r=l_t..t} alpha_r)
                     + R_{h_t+1} Diag(prod_{r=t..h_t} alpha_r),
    with both scans started from S_T / 2 (Eq. 1b).  windows: list of
    (l_t, h_t) (default: the own frame).  Returns [F, d_v, d_k] (array frame
    i is paper frame i + 1)."""
    F, d_v, d_k = Bs.shape
    S0 = np.zeros((d_v, d_k)) if S_T is None else 0.5 * np.asarray(S_T)
    P = forward_states_ex(As, Bs, S0, alphas, rule, U)
    R = reverse_states_ex(As, Bs, S0, alphas, rule, U)
    if windows is None:
        windows = [(t, t) for t in range(1, F + 1)]
    out = np.empty((F, d_v, d_k))
    for t in range(1, F + 1):
        lo, hi = windows[t - 1]
        df = np.ones(d_k)
        dr = np.ones(d_k)
        if alphas is not None:
            for r in range(lo, t + 1):
                df = df * alphas[r - 1]
            for r in range(t, hi + 1):
                dr = dr * alphas[r - 1]
        out[t - 1] = P[lo - 1] * df[None, :] + R[hi + 1] * dr[None, :]
    return out


def head_forward_ex(q, k, v, beta, gate: float, alpha=None, S_T=None, windows=None,
                    rule="joint", eps: float = RMS_EPS, gate_tokens=None) -> np.ndarray:
    """The full linear branch for one head problem (Algorithm 1, steps 3-7):
    q, k [F,N,d_k], v [F,N,d_v], beta [F,N], alpha [F,d_k] or None, S_T
    [d_v,d_k] or None, windows as in gathered_states_ex -> y [F,N,d_v].
    gate_tokens [F,N,d_v], when given, is the output gate G^L of Eq. 1c per
    token and channel, and replaces the per-head gate."""
    if np.any(beta < 0):
        raise ValueError("write strengths must be non-negative")
    As, Bs = head_statistics(k, v, beta)
    St = gathered_states_ex(As, Bs, S_T, alpha, windows, rule, U=k.shape[1])
    y = np.empty(q.shape[:2] + (v.shape[2],))
    for t in range(q.shape[0]):
        g = gate if gate_tokens is None else gate_tokens[t]
        y[t] = rmsnorm_gate(readout(St[t], q[t]), g, eps)
    return y


def vda_forward_ex(q, k, v, beta, gate, alpha=None, S_T=None, chunk=1, radius=0, offset=0,
                   rule="joint", eps: float = RMS_EPS, gate_tokens=None) -> np.ndarray:
    """All head problems: alpha [H,F,d_k] or None, S_T [H,d_v,d_k] or None,
    gate_tokens [H,F,N,d_v] or None (then gate [H] applies), one window
    layout for every head."""
    H, F = q.shape[0], q.shape[1]
    windows = local_windows(F, chunk, radius, offset)
    return np.stack([
        head_forward_ex(q[h], k[h], v[h], beta[h],
                        1.0 if gate is None else float(gate[h]),
                        None if alpha is None else alpha[h],
                        None if S_T is None else S_T[h], windows, rule, eps,
                        None if gate_tokens is None else gate_tokens[h])
        for h in range(H)])


def text_state(k, v, beta, rule="joint") -> np.ndarray:
    """S_T per head: the prompt summarised into one state, taken as a leading
    virtual frame updated from the zero state (Sec. 2.2, Eq. 1b; Sec. 4).
    k [H,L,d_k], v [H,L,d_v], beta [H,L] over the L prompt tokens; returns
    [H,d_v,d_k].  The frame's statistics are Eq. 3b over its tokens; from
    S_prev = 0 the joint rule gives S_T = B_T (I + A_T)^{-1} (Eq. 5) and the
    frozen rule B_T / sqrt(L) (Eq. 3c, U = L, the prompt's own token count)."""
    H, L, d_k = k.shape
    out = np.empty((H, v.shape[-1], d_k))
    for h in range(H):
        A, B = frame_statistics(k[h], v[h], beta[h])
        out[h] = decayed_frame_update(np.zeros_like(B), A, B, rule=rule, U=L)
    return out


# ----------------------------------------------------------------------------
# Chunk-wise scans (Section 4): each chunk of frames composed into one affine
# map (Eq. A.1), then the chunk sequence scanned in both directions
# ----------------------------------------------------------------------------

def chunk_ranges(F: int, chunk: int, offset: int = 0):
    """The chunks of the local-window grid (Section 2.1, as in local_windows):
    `chunk` consecutive frames counted from `offset` positions before array
    frame 0, clipped to the clip.  Returns (first, last) array frame indices
    (inclusive) of every non-empty chunk, in frame order."""
    out = []
    c = 0
    while c * chunk - offset <= F - 1:
        lo = max(0, c * chunk - offset)
        hi = min(F - 1, (c + 1) * chunk - offset - 1)
        if hi >= lo:
            out.append((lo, hi))
        c += 1
    return out


def chunk_map(As, Bs, frames, alphas=None):
    """Eq. A.1 composed over array frames `frames`, applied in the order
    given (the scan order): the map S_in -> S_out of the joint rule is
    S_out = S_in M + J with, frame by frame, M <- M M_t and J <- J M_t + J_t
    (M_t = Diag(alpha_t)(I + A_t)^{-1}, J_t = B_t (I + A_t)^{-1})."""
    d_k, d_v = As.shape[1], Bs.shape[1]
    M = np.eye(d_k)
    J = np.zeros((d_v, d_k))
    for t in frames:
        Mt, Jt = frame_transition(As[t], Bs[t], None if alphas is None else alphas[t])
        M = M @ Mt
        J = J @ Mt + Jt
    return M, J


def chunk_boundary_states(As, Bs, S0, chunk: int, offset: int = 0, alphas=None):
    """Both scans over the chunk sequence (joint rule), from S0 each.
    Returns (Pb, Rb), one entry per chunk of chunk_ranges: Pb[c] is the
    forward state entering chunk c (after every earlier frame), Rb[c] the
    reverse state entering it from the right (after every later frame)."""
    ranges = chunk_ranges(Bs.shape[0], chunk, offset)
    Pb, Rb = [], [None] * len(ranges)
    P = np.array(S0, dtype=np.float64)
    for lo, hi in ranges:
        Pb.append(P)
        M, J = chunk_map(As, Bs, range(lo, hi + 1), alphas)
        P = P @ M + J
    R = np.array(S0, dtype=np.float64)
    for c in range(len(ranges) - 1, -1, -1):
        lo, hi = ranges[c]
        Rb[c] = R
        M, J = chunk_map(As, Bs, range(hi, lo - 1, -1), alphas)
        R = R @ M + J
    return Pb, Rb


# ----------------------------------------------------------------------------
# VDA-Prep (Section 2.3 and Section 4): the linear branch's feature map
# ----------------------------------------------------------------------------

#: Epsilon of the L2 normalisation of Q and K (not stated in the paper).
L2_EPS = 1e-6


def depthwise_conv3(x: np.ndarray, w_spatial: np.ndarray, w_temporal: np.ndarray) -> np.ndarray:
    """The separable short convolution of K and V: a depthwise 5 x 5 spatial
    filter and a depthwise five-tap temporal filter (Section 2.3), centred,
    as cross-correlations with zero padding at the clip and frame borders.

    x [F, gh, gw, C] (C channels, one filter per channel); w_spatial
    [C, 5, 5] indexed [c, dy, dx] for offsets dy - 2, dx - 2; w_temporal
    [C, 5] for frame offsets dt - 2.  Both filters are linear in x, so the
    order of the two passes does not matter; here spatial, then temporal."""
    F, gh, gw, C = x.shape
    r = w_spatial.shape[1] // 2
    rt = w_temporal.shape[1] // 2
    xp = np.zeros((F, gh + 2 * r, gw + 2 * r, C))
    xp[:, r:r + gh, r:r + gw] = x
    s = np.zeros((F, gh, gw, C))
    for dy in range(2 * r + 1):
        for dx in range(2 * r + 1):
            s += w_spatial[:, dy, dx] * xp[:, dy:dy + gh, dx:dx + gw]
    sp = np.zeros((F + 2 * rt, gh, gw, C))
    sp[rt:rt + F] = s
    out = np.zeros_like(s)
    for dt in range(2 * rt + 1):
        out += w_temporal[:, dt] * sp[dt:dt + F]
    return out


def silu(x: np.ndarray) -> np.ndarray:
    """SiLU(x) = x * sigmoid(x)."""
    return x / (1.0 + np.exp(-x))


def l2_normalise(x: np.ndarray, eps: float = L2_EPS) -> np.ndarray:
    """x / sqrt(sum x^2 + eps) over the last axis (one token of one head)."""
    return x / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps)


def vda_prep(q, k, v, grid, H: int, wk_spatial, wk_temporal, wv_spatial, wv_temporal,
             eps: float = L2_EPS):
    """The linear branch's feature map (Section 2.3; VDA-Prep of Section 4)
    for one clip: K and V pass through their separable short convolution and
    SiLU, Q and K are L2-normalised per token and head, and everything is
    laid out frame-major per head.

    q, k, v [F, N, H*d] (token-major projections, N = gh * gw tokens per
    frame in row-major grid order, H heads of d channels each); grid =
    (gh, gw); w*_spatial [H*d, 5, 5], w*_temporal [H*d, 5].
    Returns (q, k, v) each [H, F, N, d]."""
    F, N, Cq = q.shape
    gh, gw = grid
    assert gh * gw == N

    def heads(x):
        d = x.shape[-1] // H
        return np.ascontiguousarray(x.reshape(F, N, H, d).transpose(2, 0, 1, 3))

    kc = silu(depthwise_conv3(k.reshape(F, gh, gw, -1), wk_spatial, wk_temporal)).reshape(F, N, -1)
    vc = silu(depthwise_conv3(v.reshape(F, gh, gw, -1), wv_spatial, wv_temporal)).reshape(F, N, -1)
    return l2_normalise(heads(q), eps), l2_normalise(heads(kc), eps), heads(vc)
