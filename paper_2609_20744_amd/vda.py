"""Thin Python binding of libvda.so (the C ABI in include/vda.h).

Argument marshalling only: every step of the operator runs in the HIP
kernels of libvda.so.  PyTorch supplies device memory and the stream.
Importing this module raises ImportError if the library is not built.

Tensor layout (batch and heads folded into one leading axis, or kept as any
number of leading axes, which are flattened):
    q, k  [..., F, N, d_k]   v, out [..., F, N, d_v]
    beta  [..., F, N] fp32   gate   [...] fp32
q, k, v, out are torch.bfloat16 (vda_forward) or torch.float32
(vda_forward_f32), contiguous, on one GPU.
"""
from __future__ import annotations

import ctypes
import math
import os
import re

# torch is imported before libvda.so is loaded: torch bundles its own HIP
# runtime (soname libamdhip64.so.7), and loading it first makes libvda.so's
# dependency resolve to that same runtime, so torch's streams and memory are
# valid in the library's calls.  Loading libvda.so first would bring in a
# second runtime instance whose streams are unrelated to torch's.
import torch  # noqa: F401  (load order matters, see above)

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libvda.so")
HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "vda.h")

VDA_OK = 0
STATUS_NAMES = {0: "VDA_OK", 1: "VDA_ERR_NULL", 2: "VDA_ERR_SIZE", 3: "VDA_ERR_UNSUPPORTED",
                4: "VDA_ERR_ALIGN", 5: "VDA_ERR_OVERLAP", 6: "VDA_ERR_HIP", 7: "VDA_ERR_NOMEM",
                8: "VDA_ERR_SCRATCH"}

_P = ctypes.c_void_p
_I = ctypes.c_int

class VdaOptions(ctypes.Structure):
    """struct vda_options (include/vda.h)."""
    _fields_ = [("rule", ctypes.c_int), ("alpha", ctypes.c_void_p),
                ("text_state", ctypes.c_void_p), ("window_chunk", ctypes.c_int),
                ("window_radius", ctypes.c_int), ("window_offset", ctypes.c_int),
                ("gate_tokens", ctypes.c_void_p), ("out_heads", ctypes.c_int),
                ("q_heads", ctypes.c_int)]


RULES = {"joint": 0, "frozen": 1}

_SIGNATURES = {
    "vda_status_string": (ctypes.c_char_p, [_I]),
    "vda_forward": (_I, [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _P, _P]),
    "vda_forward_f32": (_I, [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _P, _P]),
    "vda_forward_noalloc": (_I, [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _P, _P]),
    "vda_forward_ex": (_I, [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _P, _P, _P]),
    "vda_forward_ex_f32": (_I, [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _P, _P, _P]),
    "vda_text_state": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _I, _P, _P]),
    "vda_default_split_plan": (_I, [_I, _I, _I, _I, _I, _I, _P, _P]),
    "vda_frame_stats": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _P, _P, _P]),
    "vda_frame_inverse": (_I, [_P, _P, _I, _I, _I, _I, _I, _P, _P]),
    "vda_frame_inverse_tiles": (_I, [_P, _P, _I, _I, _I, _I, _I, _P, _P]),
    "vda_state_scan": (_I, [_P, _P, _I, _I, _I, _I, _I, _P, _P, _P]),
    "vda_state_scan_tiles": (_I, [_P, _P, _I, _I, _I, _I, _P, _P, _P]),
    "vda_state_scan_chunked": (_I, [_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _P, _P, _P, _P]),
    "vda_state_scan_chunked_workspace": (ctypes.c_size_t, [_I, _I, _I, _I, _I, _I]),
    "vda_prep": (_I, [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _P, _P, _P, _P]),
    "vda_readout": (_I, [_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _P, _P]),
    "vda_release_workspace": (_I, [_I, _P]),
    "vda_workspace_bytes": (_I, [_I, _P]),
}


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run `python -m paper_2609_20744_amd.build` "
            "(the VDA operator has no fallback path)")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()


class VDAError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)}")


def status_string(status: int) -> str:
    return lib.vda_status_string(int(status)).decode()


def header_functions() -> list[str]:
    """Names of the entry points declared in include/vda.h."""
    with open(HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(vda_\w+)\s*\(", text, flags=re.M)))


def _check(status: int, where: str) -> None:
    if status != VDA_OK:
        if status == 1:
            raise ValueError(f"{where}: {status_string(status)}")
        if status in (2, 3, 4, 5, 8):
            raise ValueError(f"{where}: {status_string(status)}")
        raise VDAError(status, where)


# ----------------------------------------------------------------------------
# torch-facing wrappers
# ----------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _stream_ptr(device, stream=None) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return int(s.cuda_stream)


def _require(t, name, dtype, device):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _shape(q, k, v, beta, gate=None, q_heads=0):
    if k.dim() < 3:
        raise ValueError("k must be [..., F, N, d_k]")
    lead = tuple(k.shape[:-3])
    F, N, d_k = k.shape[-3:]
    d_v = v.shape[-1]
    H = math.prod(lead) if lead else 1
    if q_heads:
        if H % q_heads:
            raise ValueError(f"q_heads {q_heads} must divide the {H} head problems")
        qshape = (H // q_heads, F, N, q_heads * d_k)
        if tuple(q.shape) != qshape:
            raise ValueError(f"raw q shape {tuple(q.shape)} must be {qshape}")
    elif tuple(k.shape) != tuple(q.shape):
        raise ValueError(f"k shape {tuple(k.shape)} != q shape {tuple(q.shape)}")
    if tuple(v.shape) != lead + (F, N, d_v):
        raise ValueError(f"v shape {tuple(v.shape)} does not match k")
    if tuple(beta.shape) != lead + (F, N):
        raise ValueError(f"beta shape {tuple(beta.shape)} must be {lead + (F, N)}")
    if gate is not None and gate.numel() != H:
        raise ValueError(f"gate must have {H} elements (one per head problem)")
    return lead, F, N, H, d_k, d_v


def forward(q, k, v, beta, gate, out=None, stream=None, alpha=None, text_state=None,
            window=None, rule="joint", gate_tokens=None, out_heads=None, q_heads=None):
    """VDA forward (vda_forward for bf16 tensors, vda_forward_f32 for fp32).

    With any of the full-operator options it calls vda_forward_ex(_f32):
    alpha [..., F, d_k] fp32 channel decays, text_state [..., d_v, d_k] fp32
    S_T, window = (chunk, radius, offset) of the local window, rule 'joint'
    (Eq. 5) or 'frozen' (Eq. 3c with 1/sqrt(U) key scaling), and
    gate_tokens [..., F, N, d_v] (q's dtype), the output gate G^L of Eq. 1c
    per token and channel, which replaces the per-head gate (gate may then
    be None).  out_heads (> 0) selects the token-major output
    [H / out_heads, F, N, out_heads * d_v] of clips of out_heads heads, H the
    number of head problems (the product of the leading dimensions).
    q_heads (> 0) passes the raw token-major query [H / q_heads, F, N,
    q_heads * d_k] (as vda_prep's input) and leaves its L2 map to the
    readout; k, v and the other arguments keep their per-head layouts."""
    torch = _torch()
    dt = q.dtype
    if dt not in (torch.bfloat16, torch.float32):
        raise ValueError(f"q dtype {dt} must be bfloat16 or float32")
    dev = q.device
    if dev.type != "cuda":
        raise ValueError("VDA runs on the GPU only; tensors must be on a cuda device")
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        _require(t, n, dt, dev)
    _require(beta, "beta", torch.float32, dev)
    if gate is not None or gate_tokens is None:
        _require(gate, "gate", torch.float32, dev)
    qh = int(q_heads or 0)
    if qh < 0:
        raise ValueError(f"q_heads {q_heads} must be positive")
    lead, F, N, H, d_k, d_v = _shape(q, k, v, beta, gate, qh)
    oh = int(out_heads or 0)
    if oh < 0 or (oh and H % oh):
        raise ValueError(f"out_heads {out_heads} must divide the {H} head problems")
    oshape = (H // oh, F, N, oh * d_v) if oh else lead + (F, N, d_v)
    if out is None:
        out = torch.empty(oshape, dtype=dt, device=dev)
    else:
        _require(out, "out", dt, dev)
        if tuple(out.shape) != oshape:
            raise ValueError(f"out shape {tuple(out.shape)} must be {oshape}")
    if alpha is None and text_state is None and window is None and rule == "joint" and \
            gate_tokens is None and not oh and not qh:
        fn = lib.vda_forward if dt == torch.bfloat16 else lib.vda_forward_f32
        with torch.cuda.device(dev):
            st = fn(q.data_ptr(), k.data_ptr(), v.data_ptr(), beta.data_ptr(), gate.data_ptr(),
                    F, N, H, d_k, d_v, out.data_ptr(), _stream_ptr(dev, stream))
        _check(st, fn.__name__)
        return out
    if rule not in RULES:
        raise ValueError(f"rule must be one of {sorted(RULES)}")
    if alpha is not None:
        _require(alpha, "alpha", torch.float32, dev)
        if tuple(alpha.shape) != lead + (F, d_k):
            raise ValueError(f"alpha shape {tuple(alpha.shape)} must be {lead + (F, d_k)}")
    if text_state is not None:
        _require(text_state, "text_state", torch.float32, dev)
        if tuple(text_state.shape) != lead + (d_v, d_k):
            raise ValueError(f"text_state shape {tuple(text_state.shape)} must be "
                             f"{lead + (d_v, d_k)}")
    if gate_tokens is not None:
        _require(gate_tokens, "gate_tokens", dt, dev)
        if tuple(gate_tokens.shape) != lead + (F, N, d_v):
            raise ValueError(f"gate_tokens shape {tuple(gate_tokens.shape)} must be "
                             f"{lead + (F, N, d_v)}")
    chunk, radius, offset = (1, 0, 0) if window is None else (int(x) for x in window)
    opts = VdaOptions(RULES[rule], alpha.data_ptr() if alpha is not None else None,
                      text_state.data_ptr() if text_state is not None else None,
                      chunk, radius, offset,
                      gate_tokens.data_ptr() if gate_tokens is not None else None, oh, qh)
    fn = lib.vda_forward_ex if dt == torch.bfloat16 else lib.vda_forward_ex_f32
    with torch.cuda.device(dev):
        st = fn(q.data_ptr(), k.data_ptr(), v.data_ptr(), beta.data_ptr(),
                gate.data_ptr() if gate is not None else None,
                F, N, H, d_k, d_v, ctypes.byref(opts), out.data_ptr(), _stream_ptr(dev, stream))
    _check(st, fn.__name__)
    return out


def text_state(k, v, beta, rule="joint", out=None, stream=None):
    """The prompt state S_T (vda_text_state): k [..., L, d_k], v [..., L, d_v]
    (bfloat16 or float32), beta [..., L] float32; returns [..., d_v, d_k]
    float32, the text_state argument of forward."""
    torch = _torch()
    dt = k.dtype
    if dt not in (torch.bfloat16, torch.float32):
        raise ValueError(f"k dtype {dt} must be bfloat16 or float32")
    dev = k.device
    if dev.type != "cuda":
        raise ValueError("VDA runs on the GPU only; tensors must be on a cuda device")
    _require(k, "k", dt, dev)
    _require(v, "v", dt, dev)
    _require(beta, "beta", torch.float32, dev)
    if rule not in RULES:
        raise ValueError(f"rule must be one of {sorted(RULES)}")
    if k.dim() < 2:
        raise ValueError("k must be [..., L, d_k]")
    lead = tuple(k.shape[:-2])
    L, d_k = k.shape[-2:]
    d_v = v.shape[-1]
    H = math.prod(lead) if lead else 1
    if tuple(v.shape) != lead + (L, d_v):
        raise ValueError(f"v shape {tuple(v.shape)} does not match k")
    if tuple(beta.shape) != lead + (L,):
        raise ValueError(f"beta shape {tuple(beta.shape)} must be {lead + (L,)}")
    if out is None:
        out = torch.empty(lead + (d_v, d_k), dtype=torch.float32, device=dev)
    else:
        _require(out, "out", torch.float32, dev)
        if tuple(out.shape) != lead + (d_v, d_k):
            raise ValueError(f"out shape {tuple(out.shape)} must be {lead + (d_v, d_k)}")
    with torch.cuda.device(dev):
        st = lib.vda_text_state(k.data_ptr(), v.data_ptr(), beta.data_ptr(), L, H, d_k, d_v,
                                RULES[rule], int(dt == torch.float32), out.data_ptr(),
                                _stream_ptr(dev, stream))
    _check(st, "vda_text_state")
    return out


def forward_noalloc(q, k, v, beta, gate, out=None, stream=None):
    """vda_forward_noalloc: vda_forward (bf16 tensors) with the library's
    fixed device scratch array as workspace; the library allocates nothing
    (out is allocated here by torch when not given)."""
    torch = _torch()
    dev = q.device
    if q.dtype != torch.bfloat16:
        raise ValueError("vda_forward_noalloc takes bfloat16 q, k, v")
    if dev.type != "cuda":
        raise ValueError("VDA runs on the GPU only; tensors must be on a cuda device")
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        _require(t, n, torch.bfloat16, dev)
    _require(beta, "beta", torch.float32, dev)
    _require(gate, "gate", torch.float32, dev)
    lead, F, N, H, d_k, d_v = _shape(q, k, v, beta, gate)
    if out is None:
        out = torch.empty(lead + (F, N, d_v), dtype=q.dtype, device=dev)
    else:
        _require(out, "out", q.dtype, dev)
        if tuple(out.shape) != lead + (F, N, d_v):
            raise ValueError(f"out shape {tuple(out.shape)} must be {lead + (F, N, d_v)}")
    with torch.cuda.device(dev):
        st = lib.vda_forward_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), beta.data_ptr(),
                                     gate.data_ptr(), F, N, H, d_k, d_v, out.data_ptr(),
                                     _stream_ptr(dev, stream))
    _check(st, "vda_forward_noalloc")
    return out


def release_workspace(device: int = -1) -> int:
    """Free the library's cached workspace buffers on `device` (-1: the
    current one) that no call is using (vda_release_workspace); waits for
    their last work on the host.  Returns the bytes freed."""
    n = ctypes.c_size_t(0)
    _check(lib.vda_release_workspace(int(device), ctypes.byref(n)), "vda_release_workspace")
    return n.value


def workspace_bytes(device: int = -1) -> int:
    """Bytes of workspace the library holds cached on `device` (-1: the
    current one) (vda_workspace_bytes)."""
    n = ctypes.c_size_t(0)
    _check(lib.vda_workspace_bytes(int(device), ctypes.byref(n)), "vda_workspace_bytes")
    return n.value


def default_split_plan(F: int, N: int, H: int, d_k: int, d_v: int,
                       is_f32: bool = False) -> tuple[int, int]:
    """(tail_frames, splits) of the statistics step that vda_forward uses on
    the current device (vda_default_split_plan)."""
    t, s = ctypes.c_int(0), ctypes.c_int(0)
    st = lib.vda_default_split_plan(F, N, H, d_k, d_v, int(bool(is_f32)), ctypes.byref(t),
                                    ctypes.byref(s))
    _check(st, "vda_default_split_plan")
    return t.value, s.value


def partial_count(count: int, tail_frames: int, splits: int) -> int:
    """Number of partial matrices of a split plan over `count` frames."""
    return count + tail_frames * (splits - 1) if splits > 1 else count


def frame_stats(k, v, beta, splits=None, tail_frames=None, A_part=None, B_part=None,
                stream=None):
    """Step a1 (vda_frame_stats): partial A [P, d_k, d_k] and B [P, d_v, d_k],
    fp32, under the split plan (tail_frames, splits); the first H*F partials
    are the frames in [H, F] order.  Defaults: the library's plan; with only
    `splits` given, every frame is split."""
    torch = _torch()
    dev, dt = k.device, k.dtype
    for t, n in ((k, "k"), (v, "v")):
        _require(t, n, dt, dev)
    _require(beta, "beta", torch.float32, dev)
    lead, F, N, H, d_k, d_v = _shape(k, k, v, beta)
    if splits is None:
        with torch.cuda.device(dev):
            tail_frames, splits = default_split_plan(F, N, H, d_k, d_v, dt == torch.float32)
    elif tail_frames is None:
        tail_frames = H * F
    splits, tail_frames = int(splits), int(tail_frames)
    P = partial_count(H * F, tail_frames, splits)
    if A_part is None:
        A_part = torch.empty((P, d_k, d_k), dtype=torch.float32, device=dev)
    if B_part is None:
        B_part = torch.empty((P, d_v, d_k), dtype=torch.float32, device=dev)
    with torch.cuda.device(dev):
        st = lib.vda_frame_stats(k.data_ptr(), v.data_ptr(), beta.data_ptr(), F, N, H, d_k, d_v,
                                 tail_frames, splits, int(dt == torch.float32), A_part.data_ptr(),
                                 B_part.data_ptr(), _stream_ptr(dev, stream))
    _check(st, "vda_frame_stats")
    return A_part, B_part


def frame_inverse(A_part, B_part=None, count=None, tail_frames=0, splits=1, Inv=None,
                  stream=None, tiles=False):
    """Step a2 (vda_frame_inverse): Inv [count, d_k, d_k] = (I + sum of each
    frame's A partials)^-1, fp32, under the split plan that made the partials
    (A_part [P, d_k, d_k]; count defaults to P when splits == 1).  With
    splits > 1 each frame's B partials ([P, d_v, d_k]) are folded in place into
    B_part[frame].  tiles=True (vda_frame_inverse_tiles) writes each inverse
    as split-bf16 operand tiles instead: Inv is then [count, 2, d_k * d_k]
    bfloat16 (hi plane, lo plane; the layout of include/vda.h), or any
    buffer of the same size in bytes."""
    torch = _torch()
    d_k = A_part.shape[-1]
    if count is None:
        if splits > 1:
            raise ValueError("count is required with a split plan")
        count = math.prod(A_part.shape[:-2])
    d_v = B_part.shape[-2] if B_part is not None else d_k
    if splits > 1 and B_part is None:
        raise ValueError("B_part is required when there is more than one split")
    if Inv is None:
        Inv = (torch.empty((count, 2, d_k * d_k), dtype=torch.bfloat16, device=A_part.device)
               if tiles else
               torch.empty((count, d_k, d_k), dtype=torch.float32, device=A_part.device))
    fn = lib.vda_frame_inverse_tiles if tiles else lib.vda_frame_inverse
    with torch.cuda.device(A_part.device):
        st = fn(A_part.data_ptr(), B_part.data_ptr() if B_part is not None else None,
                int(tail_frames), int(splits), int(count), d_k, d_v, Inv.data_ptr(),
                _stream_ptr(A_part.device, stream))
    _check(st, fn.__name__)
    return Inv


def state_scan(Inv, B, S_fwd=None, S_rev=None, exact_f32=False, stream=None):
    """Steps a3/a4 (vda_state_scan).  Inv [H, F, d_k, d_k], B [H, F, d_v, d_k]
    (the reduced statistic, e.g. B_part[0] after frame_inverse).
    exact_f32 selects fp32 matrix products (the fp32 storage path); otherwise
    split-bf16 products with fp32 accumulation (the bf16 storage path)."""
    torch = _torch()
    H, F, d_v, d_k = B.shape
    dev = B.device
    if S_fwd is None:
        S_fwd = torch.empty((H, F, d_v, d_k), dtype=torch.float32, device=dev)
    if S_rev is None:
        S_rev = torch.empty((H, F, d_v, d_k), dtype=torch.float32, device=dev)
    with torch.cuda.device(dev):
        st = lib.vda_state_scan(Inv.data_ptr(), B.data_ptr(), F, H, d_k, d_v,
                                int(bool(exact_f32)), S_fwd.data_ptr(), S_rev.data_ptr(),
                                _stream_ptr(dev, stream))
    _check(st, "vda_state_scan")
    return S_fwd, S_rev


def state_scan_tiles(Inv_tiles, B, S_fwd=None, S_rev=None, stream=None):
    """Steps a3/a4 from split-bf16 operand tiles (vda_state_scan_tiles), the
    kernel vda_forward runs with bf16 storage.  Inv_tiles: [H, F, ...] with
    d_k * d_k * 4 bytes per frame (as written by frame_inverse(tiles=True));
    B [H, F, d_v, d_k] fp32."""
    torch = _torch()
    H, F, d_v, d_k = B.shape
    dev = B.device
    if Inv_tiles.numel() * Inv_tiles.element_size() != H * F * d_k * d_k * 4:
        raise ValueError("Inv_tiles must hold d_k * d_k * 4 bytes per frame")
    if S_fwd is None:
        S_fwd = torch.empty((H, F, d_v, d_k), dtype=torch.float32, device=dev)
    if S_rev is None:
        S_rev = torch.empty((H, F, d_v, d_k), dtype=torch.float32, device=dev)
    with torch.cuda.device(dev):
        st = lib.vda_state_scan_tiles(Inv_tiles.data_ptr(), B.data_ptr(), F, H, d_k, d_v,
                                      S_fwd.data_ptr(), S_rev.data_ptr(), _stream_ptr(dev, stream))
    _check(st, "vda_state_scan_tiles")
    return S_fwd, S_rev


def state_scan_chunked(Inv_tiles, B, chunk, offset=0, alpha=None, text_state=None, S_fwd=None,
                       S_rev=None, work=None, stream=None):
    """Chunk-wise scans for a chunked window (vda_state_scan_chunked): the
    states entering every chunk of the window grid, forward at the chunk's
    first frame of S_fwd, reverse at its last frame of S_rev (other frames
    untouched; new outputs are zero-filled).  Inv_tiles as for
    state_scan_tiles, B [H, F, d_v, d_k] fp32, alpha [H, F, d_k] and
    text_state [H, d_v, d_k] fp32 or None; work: a device buffer of
    chunked_workspace(...) bytes (allocated if None)."""
    torch = _torch()
    H, F, d_v, d_k = B.shape
    dev = B.device
    if Inv_tiles.numel() * Inv_tiles.element_size() != H * F * d_k * d_k * 4:
        raise ValueError("Inv_tiles must hold d_k * d_k * 4 bytes per frame")
    for t, n in ((alpha, "alpha"), (text_state, "text_state")):
        if t is not None:
            _require(t, n, torch.float32, dev)
    if S_fwd is None:
        S_fwd = torch.zeros((H, F, d_v, d_k), dtype=torch.float32, device=dev)
    if S_rev is None:
        S_rev = torch.zeros((H, F, d_v, d_k), dtype=torch.float32, device=dev)
    if work is None:
        nbytes = chunked_workspace(F, H, d_k, d_v, chunk, offset)
        work = torch.empty((max(nbytes, 16),), dtype=torch.uint8, device=dev)
    with torch.cuda.device(dev):
        st = lib.vda_state_scan_chunked(
            Inv_tiles.data_ptr(), B.data_ptr(), alpha.data_ptr() if alpha is not None else None,
            text_state.data_ptr() if text_state is not None else None, F, H, d_k, d_v, int(chunk),
            int(offset), work.data_ptr(), S_fwd.data_ptr(), S_rev.data_ptr(),
            _stream_ptr(dev, stream))
    _check(st, "vda_state_scan_chunked")
    return S_fwd, S_rev


def chunked_workspace(F: int, H: int, d_k: int, d_v: int, chunk: int, offset: int = 0) -> int:
    """Bytes of the work buffer of state_scan_chunked."""
    return int(lib.vda_state_scan_chunked_workspace(F, H, d_k, d_v, int(chunk), int(offset)))


def prep(q, k, v, grid, wk_spatial, wk_temporal, wv_spatial, wv_temporal, H, outs=None,
         stream=None):
    """VDA-Prep (vda_prep): q, k [B, F, N, H*d_k], v [B, F, N, H*d_v] bf16
    projections with N = grid[0] * grid[1]; filters fp32 wk_spatial
    [H*d_k, 25] (or [H*d_k, 5, 5]), wk_temporal [H*d_k, 5], likewise for v.
    Returns (q', k', v') [B*H, F, N, d] bf16 (or fills `outs`).  With q None
    the query map is skipped (forward with q_heads = H applies it to the raw
    query) and q' is None."""
    torch = _torch()
    dev = k.device
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        if t is not None or n != "q":
            _require(t, n, torch.bfloat16, dev)
    for t, n in ((wk_spatial, "wk_spatial"), (wk_temporal, "wk_temporal"),
                 (wv_spatial, "wv_spatial"), (wv_temporal, "wv_temporal")):
        _require(t, n, torch.float32, dev)
    B, F, N, Ck = k.shape
    Cv = v.shape[-1]
    gh, gw = grid
    if gh * gw != N or (q is not None and q.shape != k.shape) or v.shape[:3] != k.shape[:3]:
        raise ValueError("q, k, v must be [B, F, grid_h*grid_w, H*d]")
    if Ck % H or Cv % H:
        raise ValueError("channels must split into H heads")
    d_k, d_v = Ck // H, Cv // H
    if outs is None:
        outs = (torch.empty((B * H, F, N, d_k), dtype=torch.bfloat16, device=dev)
                if q is not None else None,
                torch.empty((B * H, F, N, d_k), dtype=torch.bfloat16, device=dev),
                torch.empty((B * H, F, N, d_v), dtype=torch.bfloat16, device=dev))
    elif (outs[0] is None) != (q is None):
        raise ValueError("q and its output must both be given or both be None")
    with torch.cuda.device(dev):
        st = lib.vda_prep(q.data_ptr() if q is not None else None, k.data_ptr(), v.data_ptr(),
                          wk_spatial.data_ptr(), wk_temporal.data_ptr(), wv_spatial.data_ptr(),
                          wv_temporal.data_ptr(), B, F, gh, gw, H, d_k, d_v,
                          outs[0].data_ptr() if outs[0] is not None else None,
                          outs[1].data_ptr(), outs[2].data_ptr(), _stream_ptr(dev, stream))
    _check(st, "vda_prep")
    return outs


def readout(q, S_fwd, S_rev, gate, d_v=None, out=None, stream=None):
    """Steps a5-a7 (vda_readout).  q [H, F, N, d_k], S_* [H, F, d_v, d_k], gate [H]."""
    torch = _torch()
    H, F, N, d_k = q.shape
    d_v = S_fwd.shape[-2] if d_v is None else d_v
    dev = q.device
    if out is None:
        out = torch.empty((H, F, N, d_v), dtype=q.dtype, device=dev)
    with torch.cuda.device(dev):
        st = lib.vda_readout(q.data_ptr(), S_fwd.data_ptr(), S_rev.data_ptr(), gate.data_ptr(),
                             F, N, H, d_k, d_v, int(q.dtype == torch.float32), out.data_ptr(),
                             _stream_ptr(dev, stream))
    _check(st, "vda_readout")
    return out
