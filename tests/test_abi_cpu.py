"""Host-side checks of the C ABI (no GPU): the library loads, exports every
entry point that include/vda.h declares, and rejects invalid arguments
before anything is enqueued (these calls never reach the HIP runtime)."""
import ctypes

import pytest

vda = pytest.importorskip("paper_2609_20744_amd.vda", reason="libvda.so not built")

P = 0x10000  # a 64 KiB-aligned fake device address; validation never dereferences it


def test_exports_every_declared_symbol():
    names = vda.header_functions()
    assert set(names) >= {"vda_forward", "vda_forward_f32", "vda_status_string", "vda_frame_stats",
                          "vda_frame_inverse", "vda_state_scan", "vda_readout",
                          "vda_default_split_plan", "vda_forward_ex", "vda_forward_ex_f32"}
    for n in names:
        assert hasattr(vda.lib, n), n
    assert set(names) == set(vda._SIGNATURES)


def test_status_strings():
    for code, name in vda.STATUS_NAMES.items():
        assert vda.status_string(code).startswith(name)
    assert "unknown" in vda.status_string(99)


def _fwd(**kw):
    a = dict(q=P, k=P * 2, v=P * 3, beta=P * 4, gate=P * 5, F=4, N=64, H=2, d_k=64, d_v=64,
             out=P * 16, stream=None)
    a.update(kw)
    return vda.lib.vda_forward(a["q"], a["k"], a["v"], a["beta"], a["gate"], a["F"], a["N"],
                               a["H"], a["d_k"], a["d_v"], a["out"], a["stream"])


def test_forward_validation():
    # distinct far-apart fake buffers: out = 16 * 64 KiB, inputs below it
    big = 1 << 32
    ok = dict(q=big, k=2 * big, v=3 * big, beta=4 * big, gate=5 * big, out=6 * big)
    assert _fwd(q=None, **{k: v for k, v in ok.items() if k != "q"}) == 1
    assert _fwd(**{**ok, "out": None}) == 1
    assert _fwd(**ok, F=0) == 2
    assert _fwd(**ok, N=0) == 2
    assert _fwd(**ok, H=-1) == 2
    assert _fwd(**ok, d_k=48) == 3
    assert _fwd(**ok, d_v=256) == 3
    assert _fwd(**ok, d_k=8) == 3
    assert _fwd(**ok, d_v=24) == 3
    # 16-channel heads pass the forward's shape check (padded to 32 inside);
    # the output-overlap check still runs on the true sizes
    assert _fwd(**{**ok, "out": 3 * big + 64}, d_k=16, d_v=16) == 5
    assert _fwd(**{**ok, "q": big + 8}) == 4
    assert _fwd(**{**ok, "beta": 4 * big + 2}) == 4
    # out overlapping v
    assert _fwd(**{**ok, "out": 3 * big + 64}) == 5
    # out overlapping beta
    assert _fwd(**{**ok, "out": 4 * big - 16}) == 5
    # H * F too large for the launch grid
    assert _fwd(**ok, H=1 << 20, F=1 << 10) == 2


def test_stage_validation():
    big = 1 << 32
    L = vda.lib
    st = L.vda_frame_stats
    # (k, v, beta, F, N, H, d_k, d_v, tail_frames, splits, is_f32, A_part, B_part, stream)
    assert st(None, big, 2 * big, 4, 64, 2, 64, 64, 0, 1, 0, 3 * big, 4 * big, None) == 1
    assert st(big, 2 * big, 3 * big, 4, 64, 2, 64, 64, 0, 0, 0, 4 * big, 5 * big, None) == 2
    # two ranges of a 64-token frame, a split plan without frames, too many frames
    assert st(big, 2 * big, 3 * big, 4, 64, 2, 64, 64, 8, 2, 0, 4 * big, 5 * big, None) == 2
    assert st(big, 2 * big, 3 * big, 4, 256, 2, 64, 64, 0, 2, 0, 4 * big, 5 * big, None) == 2
    assert st(big, 2 * big, 3 * big, 4, 256, 2, 64, 64, 9, 2, 0, 4 * big, 5 * big, None) == 2
    assert st(big, 2 * big, 3 * big, 4, 64, 2, 64, 64, 0, 1, 0, 4 * big + 4, 5 * big, None) == 4
    assert st(big, 2 * big, 3 * big, 4, 64, 2, 64, 64, 0, 1, 0, big, 5 * big, None) == 5
    # B partials of a tail plan (8 + 3 * 2 matrices) running into A's range
    mat = 64 * 64 * 4
    assert st(big, 2 * big, 3 * big, 4, 256, 2, 64, 64, 3, 3, 0, 4 * big,
              4 * big + 13 * mat, None) == 5
    inv = L.vda_frame_inverse
    # (A_part, B_part, tail_frames, splits, count, d_k, d_v, Inv, stream)
    assert inv(None, None, 0, 1, 8, 64, 64, big, None) == 1
    assert inv(big, None, 8, 2, 8, 64, 64, 2 * big, None) == 1
    assert inv(big, None, 0, 1, 8, 96, 64, 2 * big, None) == 3
    assert inv(big, None, 0, 0, 8, 64, 64, 2 * big, None) == 2
    assert inv(big, 3 * big, 9, 2, 8, 64, 64, 2 * big, None) == 2
    # in place onto the first partials is allowed (would launch), onto the extra ones is not
    assert inv(big, 3 * big, 8, 2, 8, 64, 64, big + 8 * mat, None) == 5
    assert inv(big, 3 * big, 2, 3, 8, 64, 64, big + 4 * mat, None) == 5
    # B partials may not overlap the A partials or Inv
    assert inv(big, big + 4096, 8, 2, 8, 64, 64, 2 * big, None) == 5
    assert L.vda_default_split_plan(4, 64, 2, 64, 64, 0, None, None) == 1
    assert L.vda_state_scan(big, 2 * big, 4, 2, 64, 64, 0, 3 * big, 3 * big, None) == 5
    assert L.vda_state_scan(big, 2 * big, 4, 2, 64, 48, 0, 3 * big, 4 * big, None) == 3
    assert L.vda_readout(big, 2 * big, 3 * big, 4 * big, 4, 64, 2, 64, 64, 0, big, None) == 5
    assert L.vda_readout(big, 2 * big, 3 * big, None, 4, 64, 2, 64, 64, 0, 5 * big, None) == 1
    # the stage entry points take only the kernels' own widths (no 16)
    assert L.vda_frame_stats(big, 2 * big, 3 * big, 4, 64, 2, 16, 64, 0, 1, 0, 4 * big, 5 * big,
                             None) == 3
    assert L.vda_frame_inverse(big, None, 0, 1, 8, 16, 64, 2 * big, None) == 3
    assert L.vda_state_scan(big, 2 * big, 4, 2, 64, 16, 0, 3 * big, 4 * big, None) == 3
    assert L.vda_readout(big, 2 * big, 3 * big, 4 * big, 4, 64, 2, 64, 16, 0, 5 * big, None) == 3
    # tiled inverse and scan: the same checks as their fp32-layout forms
    it = L.vda_frame_inverse_tiles
    assert it(None, None, 0, 1, 8, 64, 64, big, None) == 1
    assert it(big, None, 0, 1, 8, 96, 64, 2 * big, None) == 3
    assert it(big, 3 * big, 8, 2, 8, 64, 64, big + 8 * mat, None) == 5
    sct = L.vda_state_scan_tiles
    assert sct(None, 2 * big, 4, 2, 64, 64, 3 * big, 4 * big, None) == 1
    assert sct(big, 2 * big, 4, 2, 64, 64, 3 * big, 3 * big, None) == 5
    assert sct(big, 2 * big, 4, 2, 64, 48, 3 * big, 4 * big, None) == 3
    assert sct(big + 4, 2 * big, 4, 2, 64, 64, 3 * big, 4 * big, None) == 4
    # the frames of one head must stay within 32-bit byte offsets
    assert sct(big, 2 * big, 40000, 1, 128, 128, 3 * big, 4 * big, None) == 2
    # chunked scan: (Inv_tiles, B, alpha, text_state, F, H, d_k, d_v, chunk, offset, work,
    #                S_fwd, S_rev, stream)
    ch = L.vda_state_scan_chunked
    assert ch(big, 2 * big, None, None, 12, 2, 64, 64, 5, 1, None, 3 * big, 4 * big, None) == 1
    assert ch(big, 2 * big, None, None, 12, 2, 64, 64, 0, 0, 5 * big, 3 * big, 4 * big, None) == 2
    assert ch(big, 2 * big, None, None, 12, 2, 64, 64, 5, 5, 5 * big, 3 * big, 4 * big, None) == 2
    assert ch(big, 2 * big, None, None, 12, 2, 64, 64, 5, -1, 5 * big, 3 * big, 4 * big, None) == 2
    assert ch(big, 2 * big, big + 8, None, 12, 2, 64, 64, 5, 1, 5 * big, 3 * big, 4 * big,
              None) == 4
    assert ch(big, 2 * big, None, None, 12, 2, 64, 64, 5, 1, 5 * big + 8, 3 * big, 4 * big,
              None) == 4
    assert ch(big, 2 * big, None, 6 * big + 4, 12, 2, 64, 64, 5, 1, 5 * big, 3 * big, 4 * big,
              None) == 4
    assert ch(big, 2 * big, None, None, 12, 2, 64, 64, 5, 1, 3 * big, 3 * big, 4 * big, None) == 5
    assert ch(big, 2 * big, None, None, 12, 2, 64, 48, 5, 1, 5 * big, 3 * big, 4 * big, None) == 3
    pr = L.vda_prep
    # (q, k, v, wks, wkt, wvs, wvt, B, F, gh, gw, H, d_k, d_v, q_out, k_out, v_out, stream)
    w = [9 * big, 9 * big + 4096, 9 * big + 8192, 9 * big + 12288]
    outs = [4 * big, 5 * big, 6 * big]
    assert pr(None, 2 * big, 3 * big, *w, 1, 4, 6, 8, 2, 128, 128, *outs, None) == 1
    # q and q_out NULL together skip the query map (the size check is then
    # the first to fail); either alone is a NULL error
    assert pr(big, 2 * big, 3 * big, *w, 1, 4, 6, 8, 2, 128, 128, None, 5 * big, 6 * big,
              None) == 1
    assert pr(None, 2 * big, 3 * big, *w, 1, 0, 6, 8, 2, 128, 128, None, 5 * big, 6 * big,
              None) == 2
    assert pr(None, 2 * big, 3 * big, *w, 1, 4, 6, 8, 2, 128, 128, None, 5 * big + 8, 6 * big,
              None) == 4
    assert pr(big, 2 * big, 3 * big, *w, 1, 0, 6, 8, 2, 128, 128, *outs, None) == 2
    assert pr(big, 2 * big, 3 * big, *w, 1, 4, 6, 8, 2, 96, 128, *outs, None) == 3
    assert pr(big, 2 * big, 3 * big, *w, 1, 4, 6, 8, 2, 128, 32, *outs, None) == 3
    assert pr(big + 8, 2 * big, 3 * big, *w, 1, 4, 6, 8, 2, 128, 128, *outs, None) == 4
    assert pr(big, 2 * big, 3 * big, *w, 1, 4, 6, 8, 2, 128, 128, big, 5 * big, 6 * big,
              None) == 5
    assert pr(big, 2 * big, 3 * big, *w, 1, 4, 6, 8, 2, 128, 128, 4 * big, 4 * big, 6 * big,
              None) == 5
    # one clip's projections beyond 32-bit byte offsets
    assert pr(big, 2 * big, 3 * big, *w, 1, 4096, 64, 64, 2, 128, 128, *outs, None) == 2
    ws = L.vda_state_scan_chunked_workspace
    # 3 chunks (frames 0-3, 4-8, 9-11) x 2 directions x 2 heads x (M tiles + J)
    assert ws(12, 2, 64, 32, 5, 1) == 3 * 2 * 2 * (64 * 64 * 4 + 32 * 64 * 4)
    assert ws(12, 2, 64, 32, 5, 5) == 0 and ws(12, 2, 64, 48, 5, 1) == 0


def test_single_hip_runtime_loaded():
    """The binding and torch must share one HIP runtime instance, or torch's
    streams would be unknown to the library."""
    import os
    maps = open(f"/proc/{os.getpid()}/maps").read()
    libs = {l.split()[-1] for l in maps.splitlines() if "libamdhip64" in l}
    assert len(libs) == 1, libs


def test_forward_ex_validation():
    import ctypes
    big = 1 << 32
    L = vda.lib

    def ex(opts, out=6 * big, d_k=64, d_v=64):
        return L.vda_forward_ex(big, 2 * big, 3 * big, 4 * big, 5 * big, 4, 64, 2, d_k, d_v,
                                None if opts is None else ctypes.byref(opts), out, None)

    def opts(rule=0, alpha=None, ts=None, chunk=1, radius=0, offset=0):
        return vda.VdaOptions(rule, alpha, ts, chunk, radius, offset)

    assert ex(opts(rule=2)) == 3                        # unknown rule
    assert ex(opts(chunk=0)) == 2
    assert ex(opts(radius=-1)) == 2
    assert ex(opts(chunk=5, offset=5)) == 2             # offset must be < chunk
    assert ex(opts(alpha=7 * big + 8)) == 4             # alpha 16-byte aligned
    assert ex(opts(ts=7 * big + 2)) == 4
    # the text state is read with 16-byte loads (also when 16-channel heads
    # pad it): 4- and 8-byte offsets are rejected, 16-byte ones accepted
    assert ex(opts(ts=7 * big + 4)) == 4
    assert ex(opts(ts=7 * big + 8), d_k=16, d_v=16) == 4
    assert ex(opts(ts=7 * big + 16), d_k=16, d_v=16) != 4
    # out overlapping alpha or the text state
    assert ex(opts(alpha=7 * big), out=7 * big + 64) == 5
    assert ex(opts(ts=8 * big), out=8 * big - 64) == 5
    assert ex(opts(), d_k=48) == 3
    assert L.vda_forward_ex(None, 2 * big, 3 * big, 4 * big, 5 * big, 4, 64, 2, 64, 64, None,
                            6 * big, None) == 1
    # output gates per token: 16-byte aligned, not overlapping out, and the
    # per-head gate may then be NULL (but not both)
    assert ex(vda.VdaOptions(0, None, None, 1, 0, 0, 9 * big + 8)) == 4
    assert ex(vda.VdaOptions(0, None, None, 1, 0, 0, 9 * big), out=9 * big + 64) == 5
    assert L.vda_forward_ex(big, 2 * big, 3 * big, 4 * big, None, 4, 64, 2, 64, 64,
                            ctypes.byref(opts()), 6 * big, None) == 1
    assert L.vda_forward_ex(big, 2 * big, 3 * big, 4 * big, None, 4, 64, 2, 64, 64, None,
                            6 * big, None) == 1
    # token-major output: out_heads >= 0, dividing H, one frame's rows within
    # 32-bit byte offsets
    assert ex(vda.VdaOptions(0, None, None, 1, 0, 0, None, -1)) == 2
    assert ex(vda.VdaOptions(0, None, None, 1, 0, 0, None, 3)) == 2
    assert L.vda_forward_ex(big, 2 * big, 3 * big, 4 * big, 5 * big, 1, 1 << 21, 4, 128, 128,
                            ctypes.byref(vda.VdaOptions(0, None, None, 1, 0, 0, None, 4)),
                            8 * big, None) == 2
    # raw token-major query: q_heads >= 0, dividing H, a kernel key width
    # (no padded 16-channel key), one frame's rows within 32-bit offsets
    assert ex(vda.VdaOptions(0, None, None, 1, 0, 0, None, 0, -1)) == 2
    assert ex(vda.VdaOptions(0, None, None, 1, 0, 0, None, 0, 3)) == 2
    assert ex(vda.VdaOptions(0, None, None, 1, 0, 0, None, 0, 2), d_k=16) == 3
    assert L.vda_forward_ex(big, 2 * big, 3 * big, 4 * big, 5 * big, 1, 1 << 21, 4, 128, 128,
                            ctypes.byref(vda.VdaOptions(0, None, None, 1, 0, 0, None, 0, 4)),
                            8 * big, None) == 2
    assert L.vda_forward_ex_f32(big, 2 * big, 3 * big, 4 * big, 5 * big, 1, 1 << 20, 4, 128, 128,
                                ctypes.byref(vda.VdaOptions(0, None, None, 1, 0, 0, None, 0, 4)),
                                8 * big, None) == 2


def test_text_state_validation():
    """vda_text_state rejects bad arguments before touching the device."""
    big = 1 << 32
    ts = vda.lib.vda_text_state
    # (k, v, beta, L, H, d_k, d_v, rule, is_f32, S_T, stream)
    assert ts(None, 2 * big, 3 * big, 77, 4, 128, 128, 0, 0, 4 * big, None) == 1
    assert ts(big, 2 * big, 3 * big, 77, 4, 128, 128, 0, 0, None, None) == 1
    assert ts(big, 2 * big, 3 * big, 0, 4, 128, 128, 0, 0, 4 * big, None) == 2
    assert ts(big, 2 * big, 3 * big, 77, 0, 128, 128, 0, 0, 4 * big, None) == 2
    assert ts(big, 2 * big, 3 * big, 77, 4, 48, 128, 0, 0, 4 * big, None) == 3
    assert ts(big, 2 * big, 3 * big, 77, 4, 128, 128, 2, 0, 4 * big, None) == 3
    assert ts(big + 8, 2 * big, 3 * big, 77, 4, 128, 128, 0, 0, 4 * big, None) == 4
    assert ts(big, 2 * big, 3 * big, 77, 4, 128, 128, 0, 0, 4 * big + 4, None) == 4
    # S_T [4][128][128] fp32 over the tail of v, or over beta
    assert ts(big, 2 * big, 3 * big, 77, 4, 128, 128, 0, 1, 2 * big + 4096, None) == 5
    assert ts(big, 2 * big, 3 * big, 77, 4, 128, 128, 1, 0, 3 * big - 4096, None) == 5
    # one prompt frame of d = 128 stays within 32-bit byte offsets
    assert ts(big, 2 * big, 3 * big, 1 << 22, 1, 128, 128, 0, 0, 4 * big, None) == 2


def test_workspace_entry_points_validation():
    """vda_release_workspace / vda_workspace_bytes reject device indices below
    -1 or beyond the library's device table before any runtime call, and a
    NULL result pointer; *bytes_freed is cleared first."""
    n = ctypes.c_size_t(123)
    assert vda.lib.vda_release_workspace(-2, ctypes.byref(n)) == 2
    assert n.value == 0
    assert vda.lib.vda_release_workspace(64, None) == 2
    assert vda.lib.vda_workspace_bytes(0, None) == 1
    n = ctypes.c_size_t(123)
    assert vda.lib.vda_workspace_bytes(-7, ctypes.byref(n)) == 2
    assert n.value == 0
