#!/usr/bin/env python3
"""Throughput of the VDA forward pass on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload 768p_bf16] [--no-cpu-baseline]

A step is one whole forward pass (frame statistics, inverse, both scans,
readout + RMSNorm + gate) over the workload's synthetic inputs, which are
resident in HBM before timing starts.  The first timed region runs K steps of
the library's forward entry point (the value reported).  A second timed
region runs the same kernel launches (same head ranges and splits) through
the stage entry points with HIP events around each launch on the launch
stream, so each kernel's average launch duration is measured live (for the
roofline).  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "VDA fwd tokens/s and TFLOP/s (% bf16 MFMA peak) on one MI355X, 768p-shaped"
PEAK_BF16_TFLOPS = 2500.0   # dense bf16 MFMA, MI355X
PEAK_HBM_GBS = 8000.0       # HBM3E, MI355X
PEAK_F32_TFLOPS = 157.3     # dense fp32 MFMA, MI355X


def flops_alg(w) -> float:
    """FLOPs of the method per call: A_t (2 N d_k^2), B_t and the readout
    (4 N d_k d_v), the SPD inverse (d_k^3) and two scan products (4 d_v d_k^2)
    per frame and head."""
    dk, dv, N = w.d_k, w.d_v, w.N
    return w.frame_heads * (2 * N * dk * dk + 4 * N * dk * dv + dk ** 3 + 4 * dv * dk * dk)


def bytes_alg(w) -> float:
    """Bytes the operator must move: q, k, v, out (storage type), fp32 beta and gate."""
    e = 4 if w.dtype == "f32" else 2
    return w.heads * w.F * w.N * (e * (2 * w.d_k + w.d_v) + e * w.d_v + 4) + 4 * w.heads


def head_groups(H: int):
    """Head ranges of the forward pass's launches: one launch of each kernel
    over all heads, as the library schedules them."""
    return [(0, H)]


def kernel_bytes(w, heads=None):
    """Algorithmic bytes per launch of each kernel over `heads` heads (default:
    all): what it must read and write once (its inputs and its outputs),
    without split partials."""
    e = 4 if w.dtype == "f32" else 2
    heads = w.heads if heads is None else heads
    fh, N, dk, dv = heads * w.F, w.N, w.d_k, w.d_v
    return {
        "frame_stats": fh * (N * (e * (dk + dv) + 4) + 4 * (dk * dk + dv * dk)),
        "frame_inverse": fh * 8 * dk * dk,
        "state_scan": fh * 2 * (4 * dk * dk + 4 * dv * dk + 4 * dv * dk),
        "readout": fh * (N * e * (dk + dv) + 8 * dv * dk) + 4 * heads,
    }


def prep_kernel_bytes(w):
    """Algorithmic HBM bytes per launch of the VDA-Prep kernels: each reads
    its bf16 projection once and writes the bf16 features once.  The K and V
    convolutions are two launches of one kernel, so theirs is the mean."""
    tok_heads = w.B * w.F * w.N * w.H
    return {"prep_conv": tok_heads * 2 * 2 * (w.d_k + w.d_v) // 2,
            "prep_qnorm": tok_heads * 2 * 2 * w.d_k}


# Kernel of each stage, and the sources whose change makes counters taken
# on it stale.
KERNEL_OF = {"frame_stats": "stats_bf16_kernel", "frame_inverse": "inverse_kernel",
             "state_scan": "scan_tiled_kernel", "readout": "readout_bf16_kernel",
             "prep_conv": "prep_conv_kernel", "prep_qnorm": "prep_qnorm_kernel"}
def instance_of(w):
    """The template instance of each stage's kernel that one pass of the
    workload runs (bf16 storage); the summary reads its counters, not those
    of other instances of the same kernel (the chunk-wise and frozen-rule
    scans share the scan kernel's name).  The prep convolution keeps its bare
    name: its K and V launches are two instances, averaged."""
    dk, dv = w.d_k, w.d_v
    return {"frame_stats": f"stats_bf16_kernel<{dk},{dv}>",
            "frame_inverse": f"inverse_kernel<{dk},true>",
            "state_scan": f"scan_tiled_kernel<{dk},false,false>",
            "readout": f"readout_bf16_kernel<{dk},{dv},false,false>",
            "prep_qnorm": f"prep_qnorm_kernel<{dk}>"}


SOURCE_OF = {"frame_stats": ("vda_stats.hip",),
             "frame_inverse": ("vda_inverse.hip", "vda_inverse_body.h"),
             "state_scan": ("vda_scan_tiled.hip",), "readout": ("vda_readout.hip",),
             "prep_conv": ("vda_prep.hip",), "prep_qnorm": ("vda_prep.hip",)}


def _code_only(text: str) -> str:
    """C++ source without comments and with whitespace collapsed, so that an
    edit of the comments alone does not mark measured counters stale."""
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def source_hash(stage: str) -> str:
    """SHA-256 over the code (comments and layout aside) of the kernel's
    source files and the shared device header."""
    import hashlib
    h = hashlib.sha256()
    for f in SOURCE_OF[stage] + ("vda_common.h",):
        with open(os.path.join(ROOT, "paper_2609_20744_amd", "csrc", f)) as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()


def traffic_file(workload: str) -> str:
    return os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.json")


def measured_traffic(workload: str, stage: str):
    """HBM bytes per launch of `stage` from the committed counter summary, or
    None when there is none or the kernel's source has changed since."""
    path = traffic_file(workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        summ = json.load(f)
    k = summ.get("kernels", {}).get(stage)
    if not k or k.get("source_sha256") != source_hash(stage):
        return None
    return k["hbm_bytes_per_launch"]


def pmc_summary(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, copy_gib, workload):
    """Turn four rocprofv3 --pmc runs (FETCH_SIZE and WRITE_SIZE of the bench,
    and of the --calibrate-copy run) into HBM bytes per launch per kernel.
    Each counter (KiB per dispatch) is scaled by the factor that makes it
    match the bytes a plain copy of known size reads or writes."""
    import csv
    import re

    def load(d):
        """Average bytes per dispatch, by kernel: the library's kernels both
        by function name and by template instance ("name<args>", no
        spaces), the calibration copy (torch's neg) as "copy"."""
        out = {}
        with open(os.path.join(d, "run_counter_collection.csv")) as f:
            for r in csv.DictReader(f):
                full = r["Kernel_Name"]
                names = []
                if "neg_kernel" in full:
                    names = ["copy"]
                else:
                    m = re.search(r"::(\w+)(<[^()]*>)?\(", full)
                    if m:
                        names = [m.group(1)]
                        if m.group(2):
                            names.append(m.group(1) + m.group(2).replace(" ", ""))
                    else:
                        names = [full]
                for name in names:
                    out.setdefault(name, []).append(float(r["Counter_Value"]) * 1024.0)
        return {n: sum(v) / len(v) for n, v in out.items()}

    copy_bytes = copy_gib * (1 << 30)
    f_fetch = copy_bytes / load(copy_fetch_dir)["copy"]
    f_write = copy_bytes / load(copy_write_dir)["copy"]
    fetch, write = load(fetch_dir), load(write_dir)
    w = __import__("paper_2609_20744_amd.inputs", fromlist=["WORKLOADS"]).WORKLOADS[workload]
    kb = {**kernel_bytes(w), **prep_kernel_bytes(w)}
    kernels = {}
    inst = instance_of(w)
    for stage, kname in KERNEL_OF.items():
        kname = inst.get(stage, kname)
        if kname not in fetch or kname not in write:
            continue
        rd, wr = fetch[kname] * f_fetch, write[kname] * f_write
        kernels[stage] = {"kernel": kname, "fetch_size_bytes_raw": fetch[kname],
                          "write_size_bytes_raw": write[kname], "hbm_read_bytes": rd,
                          "hbm_write_bytes": wr, "hbm_bytes_per_launch": rd + wr,
                          "algorithmic_bytes_per_launch": kb[stage],
                          "traffic_over_algorithmic": (rd + wr) / kb[stage],
                          "source_sha256": source_hash(stage)}
    return {"workload": workload, "copy_gib": copy_gib, "fetch_factor": f_fetch,
            "write_factor": f_write, "kernels": kernels}


def _time_calls(torch, fn, K, warm=3):
    """Average ms of K back-to-back calls of fn on the current stream."""
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(K):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / K


def prep_bench(vda, torch, w, K):
    """Time vda_prep on the workload's shape (B clips, F frames, H heads,
    latent grid, d_k / d_v channels) from seeded synthetic projections.  Its
    algorithmic bytes are the three bf16 inputs and outputs (filters are
    negligible).  Also timed: vda_prep of K and V only, and the two ways from
    the projections to the token-major attention output -- vda_prep of all
    three then vda_forward_ex (out_heads = H), and vda_prep of K and V then
    vda_forward_ex on the raw query (q_heads = out_heads = H), whose readout
    applies the query's L2 map."""
    import numpy as np
    from paper_2609_20744_amd import inputs as I
    if w.dtype != "bf16" or w.grid is None or w.d_k not in (64, 128) or w.d_v not in (64, 128):
        return None
    x = I.make_prep_inputs(w.B, w.F, w.grid, w.H, w.d_k, w.d_v, seed=w.seed)
    bf = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    f32 = lambda a: torch.from_numpy(a).cuda()
    qp = bf(x["q"])
    rest = (bf(x["k"]), bf(x["v"]), w.grid, f32(x["wk_spatial"]), f32(x["wk_temporal"]),
            f32(x["wv_spatial"]), f32(x["wv_temporal"]), w.H)
    outs = vda.prep(qp, *rest)
    ms = _time_calls(torch, lambda: vda.prep(qp, *rest, outs=outs), K)
    kv_outs = (None,) + tuple(outs[1:])
    ms_kv = _time_calls(torch, lambda: vda.prep(None, *rest, outs=kv_outs), K)
    tok = w.B * w.F * w.N
    nbytes = 2 * tok * w.H * 2 * (2 * w.d_k + w.d_v)
    print(f"[bench] vda_prep: {ms:.4f} ms; K and V only: {ms_kv:.4f} ms", file=sys.stderr,
          flush=True)
    # the pipelines, with the workload's beta and per-head gate shapes
    g = torch.Generator(device="cuda").manual_seed(w.seed)
    HB = w.B * w.H
    beta = torch.sigmoid(torch.randn((HB, w.F, w.N), generator=g, device="cuda"))
    gate = torch.sigmoid(torch.randn((HB,), generator=g, device="cuda"))
    y = torch.empty((w.B, w.F, w.N, w.H * w.d_v), dtype=torch.bfloat16, device="cuda")

    def two_step():
        vda.prep(qp, *rest, outs=outs)
        vda.forward(outs[0], outs[1], outs[2], beta, gate, out=y, out_heads=w.H)

    def raw_query():
        vda.prep(None, *rest, outs=kv_outs)
        vda.forward(qp, outs[1], outs[2], beta, gate, out=y, out_heads=w.H, q_heads=w.H)

    ms_two = _time_calls(torch, two_step, K)
    ms_raw = _time_calls(torch, raw_query, K)
    print(f"[bench] prep + forward: {ms_two:.4f} ms; K/V prep + raw-query forward: "
          f"{ms_raw:.4f} ms", file=sys.stderr, flush=True)
    return {"ms": ms, "tokens_per_s": tok / (ms / 1e3), "hbm_gbs_alg": nbytes / (ms / 1e3) / 1e9,
            "frac_hbm_peak": nbytes / (ms / 1e3) / 1e9 / PEAK_HBM_GBS, "bytes_alg": nbytes,
            "kv_only_ms": ms_kv,
            "pipeline_token_major": {"prep_then_forward_ms": ms_two,
                                     "kv_prep_then_raw_query_forward_ms": ms_raw}}


def scan_paths(vda, torch, H, F, dk, dv, chunk, offset, K):
    """Time the frame-by-frame and the chunk-wise scans of one shape on
    synthetic inverses (I + G G^T / d_k)^{-1}, written as operand tiles by the
    library's inverse, and random B."""
    g = torch.Generator(device="cuda").manual_seed(11)
    G = torch.randn((H * F, dk, dk), device="cuda", generator=g) / dk ** 0.5
    A = torch.bmm(G, G.transpose(1, 2).contiguous())
    T = vda.frame_inverse(A, tiles=True).view(H, F, -1)
    B = torch.randn((H, F, dv, dk), device="cuda", generator=g)
    Sf = torch.zeros((H, F, dv, dk), device="cuda")
    Sr = torch.zeros_like(Sf)
    work = torch.empty((vda.chunked_workspace(F, H, dk, dv, chunk, offset),), dtype=torch.uint8,
                       device="cuda")
    runs = {"frame_scan_ms": lambda: vda.state_scan_tiles(T, B, Sf, Sr),
            "chunk_scan_ms": lambda: vda.state_scan_chunked(T, B, chunk, offset, S_fwd=Sf,
                                                            S_rev=Sr, work=work)}
    out = {"heads": H, "frames": F, "d_k": dk, "d_v": dv, "chunk": chunk, "offset": offset}
    for name, fn in runs.items():
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(K):
            fn()
        e1.record()
        torch.cuda.synchronize()
        out[name] = e0.elapsed_time(e1) / K
    print(f"[bench] scans H={H} F={F}: frame by frame {out['frame_scan_ms']:.4f} ms, "
          f"chunk-wise {out['chunk_scan_ms']:.4f} ms", file=sys.stderr, flush=True)
    return out


def cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo), else what platform reports."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.lower().startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def blas_info() -> dict:
    """The BLAS library NumPy calls (threadpoolctl), with its default thread count."""
    try:
        from threadpoolctl import threadpool_info
        for p in threadpool_info():
            if p.get("user_api") == "blas":
                return {"library": p.get("internal_api"), "version": p.get("version"),
                        "threads": p.get("num_threads"),
                        "file": os.path.basename(p.get("filepath", ""))}
    except Exception:
        pass
    return {"library": "unknown", "threads": int(os.environ.get("OMP_NUM_THREADS", "1"))}


def time_oracle(w, threads, budget_s: float) -> dict:
    """The fp64 oracle on whole heads of the workload, with BLAS limited to
    `threads` (None: the library's default), until about budget_s seconds."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle.vda_oracle as O
    from paper_2609_20744_amd import inputs as I
    spent, heads = 0.0, 0
    with threadpool_limits(limits=threads, user_api="blas"):
        used = blas_info()["threads"]
        for hb in range(w.heads):
            x = I.make_inputs(w, heads=[hb])
            f = {k: I.as_float64(x[k], w.dtype)[0] for k in ("q", "k", "v")}
            b = x["beta"][0].astype(np.float64)
            g = float(x["gate"][0])
            t0 = time.perf_counter()
            O.head_forward(f["q"], f["k"], f["v"], b, g)
            spent += time.perf_counter() - t0
            heads += 1
            if spent >= budget_s:
                break
    s_per_head = spent / heads
    return {"threads": used, "heads_timed": heads, "seconds": spent,
            "seconds_whole_workload": s_per_head * w.heads,
            "tokens_per_s": w.tokens / (s_per_head * w.heads)}


def cpu_baseline(w, budget_s: float = 20.0) -> dict:
    """The fp64 oracle timed on the host on whole heads of the same workload,
    at one BLAS thread and at the library's default (all the cores it is
    given), each for about budget_s / 2 seconds, scaled to the whole job's
    tokens/s.  `value` and `cores` are the all-cores figures."""
    one = time_oracle(w, 1, budget_s / 2)
    allc = time_oracle(w, None, budget_s / 2)
    return {"value": allc["tokens_per_s"], "unit": "tokens/s", "cores": allc["threads"],
            "kind": "oracle",
            "sample": f"{allc['heads_timed']} of {w.heads} heads of the {w.name} workload (all "
                      f"{w.F} frames x {w.N} tokens, fp64 NumPy oracle, {allc['seconds']:.1f} s "
                      f"at {allc['threads']} BLAS threads), scaled to all heads",
            "one_thread": one, "all_cores": allc, "cpu_model": cpu_model(), "blas": blas_info(),
            "nproc": os.cpu_count()}


def input_copies(w) -> int:
    """Input sets the timed loop rotates through, so that a workload whose
    inputs and output fit in the 256 MB last-level cache is still read from
    HBM: about 1 GiB in all, at most 64 sets."""
    return max(1, min(64, math.ceil((1 << 30) / bytes_alg(w))))


def device_sets(torch, w, x, copies):
    """`copies` device copies of (q, k, v, beta, gate, out) for the workload."""
    import numpy as np

    def dev(a, dt):
        if dt == "bf16":
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a)).cuda()

    first = (dev(x["q"], w.dtype), dev(x["k"], w.dtype), dev(x["v"], w.dtype),
             dev(x["beta"], "f32"), dev(x["gate"], "f32"))
    sets = [first] + [tuple(t.clone() for t in first) for _ in range(copies - 1)]
    outs = [torch.empty((w.heads, w.F, w.N, w.d_v), dtype=first[0].dtype, device="cuda")
            for _ in range(copies)]
    return [st + (o,) for st, o in zip(sets, outs)]


def time_forward(vda, torch, sets, K, warmup, settle):
    """Untimed passes for `settle` seconds (the clocks settle under load),
    `warmup` more, then K timed passes of vda_forward bracketed by HIP
    events on the current stream, rotating through the input sets."""
    n = len(sets)

    def fwd(i):
        q, k, v, beta, gate, out = sets[i % n]
        vda.forward(q, k, v, beta, gate, out=out)

    t0 = time.perf_counter()
    i = 0
    while time.perf_counter() - t0 < settle:
        fwd(i)
        i += 1
        torch.cuda.synchronize()
    for j in range(warmup):
        fwd(j)
    torch.cuda.synchronize()
    fev = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    wall0 = time.perf_counter()
    fev[0].record()
    for j in range(K):
        fwd(j)
        fev[j + 1].record()
    host = time.perf_counter() - wall0
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = fev[0].elapsed_time(fev[K]) / K
    step_ms = sorted(fev[j].elapsed_time(fev[j + 1]) for j in range(K))
    pct = lambda p: step_ms[min(K - 1, int(p * (K - 1) + 0.5))]
    return {"ms": ms, "p10_p50_p90": [pct(0.1), pct(0.5), pct(0.9)], "wall_s": wall,
            "input_sets": n, "host_ms_per_call": host / K * 1e3}


def throughput(w, ms) -> dict:
    t = ms / 1e3
    tflops = flops_alg(w) / t / 1e12
    gbs = bytes_alg(w) / t / 1e9
    return {"tokens_per_s": w.tokens / t, "token_heads_per_s": w.tokens * w.H / t,
            "tflops": tflops, "pct_bf16_mfma_peak": 100.0 * tflops / PEAK_BF16_TFLOPS,
            "hbm_gbs_alg": gbs, "pct_hbm_peak": 100.0 * gbs / PEAK_HBM_GBS,
            "hbm_floor_ms": bytes_alg(w) / (PEAK_HBM_GBS * 1e9) * 1e3}


def all_workloads(vda, torch, K, warmup, settle, cpu_budget):
    """One JSON line per workload: vda_forward's time (rotating input sets
    where the working set fits in the last-level cache), its throughput
    against both rooflines, and the oracle's time at one and at all BLAS
    threads."""
    from paper_2609_20744_amd import inputs as I
    for name, w in I.WORKLOADS.items():
        print(f"[bench] {name}: inputs", file=sys.stderr, flush=True)
        x = I.make_inputs(w)
        sets = device_sets(torch, w, x, input_copies(w))
        del x
        r = time_forward(vda, torch, sets, K, warmup, settle)
        per_launch, staged_ms, plans, _ = staged_kernel_times(vda, torch, w, sets[0], K)
        del sets
        torch.cuda.empty_cache()
        line = {"workload": name, "B": w.B, "H": w.H, "F": w.F, "N": w.N, "d_k": w.d_k,
                "d_v": w.d_v, "storage": w.dtype, "ms_per_step": r["ms"],
                "step_ms_p10_p50_p90": r["p10_p50_p90"], "input_sets": r["input_sets"],
                "host_ms_per_call": r["host_ms_per_call"],
                **throughput(w, r["ms"]), "kernel_ms_per_launch": per_launch,
                "staged_ms_per_step": staged_ms, "split_plan": plans}
        print(f"[bench] {name}: {r['ms']:.4f} ms/step; timing the oracle", file=sys.stderr,
              flush=True)
        if cpu_budget > 0:
            one = time_oracle(w, 1, cpu_budget / 2)
            allc = time_oracle(w, None, cpu_budget / 2)
            line["oracle"] = {"one_thread_s": one["seconds_whole_workload"],
                              "all_cores_s": allc["seconds_whole_workload"],
                              "all_cores_threads": allc["threads"],
                              "heads_timed": [one["heads_timed"], allc["heads_timed"]]}
        print(json.dumps(line), flush=True)
    print(json.dumps({"cpu_model": cpu_model(), "blas": blas_info(), "nproc": os.cpu_count()}),
          flush=True)


def paper_shard(vda, torch, K, warmup):
    """The paper's own shard (7 heads, 100 interior frames, 4032 tokens, d =
    128), inputs resident in HBM: vda_forward, and vda_forward_ex with channel
    decay, a text state and the paper's window (chunks of five frames after one
    anchor, radius one) for both rules."""
    from paper_2609_20744_amd import inputs as I
    w = I.PAPER_SHARD
    print(f"[bench] paper shard: inputs", file=sys.stderr, flush=True)
    x = I.make_inputs(w)
    (q, k, v, beta, gate, out), = device_sets(torch, w, x, 1)
    del x
    alpha = torch.from_numpy(I.make_decay(w)).cuda()
    text_state = torch.from_numpy(I.make_text_state(w)).cuda()
    runs = {"forward": lambda: vda.forward(q, k, v, beta, gate, out=out)}
    for rule in ("joint", "frozen"):
        runs[f"{rule}_decay_text_window"] = (
            lambda rule=rule: vda.forward(q, k, v, beta, gate, out=out, alpha=alpha,
                                          text_state=text_state, window=(5, 1, 1), rule=rule))
    res = {"workload": w.name, "H": w.H, "F": w.F, "N": w.N, "d_k": w.d_k, "d_v": w.d_v,
           "window": {"chunk": 5, "radius": 1, "offset": 1}}
    for name, fn in runs.items():
        for _ in range(max(2, warmup)):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(K):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / K
        res[name] = {"ms_per_step": ms, "tokens_per_s": w.tokens / (ms / 1e3)}
        print(f"[bench] paper shard {name}: {ms:.4f} ms/step", file=sys.stderr, flush=True)
    return res


def counter_summary(dirs) -> dict:
    """Per kernel instance, the mean of each counter over its dispatches in
    rocprofv3 --pmc runs (run_counter_collection.csv in each directory), the
    mean dispatch duration, and the matrix-core figures derived from them:
    MFMA FLOPs (512 per MOPS unit) and their rate over the dispatch, as a
    fraction of the dense bf16 or fp32 MFMA peak."""
    import csv
    import re
    per = {}   # (dir, dispatch) -> {"name", "dur", counters}
    for d in dirs:
        with open(os.path.join(d, "run_counter_collection.csv")) as f:
            for r in csv.DictReader(f):
                full = r["Kernel_Name"]
                m = re.search(r"::(\w+)(<[^()]*>)?\(", full)
                if not m:
                    continue
                name = m.group(1) + (m.group(2) or "").replace(" ", "")
                e = per.setdefault((d, r["Dispatch_Id"]), {"name": name, "c": {}})
                e["c"][r["Counter_Name"]] = float(r["Counter_Value"])
                e["dur"] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
    kern = {}
    for e in per.values():
        k = kern.setdefault(e["name"], {"dispatches": 0, "dur": [], "c": {}})
        k["dispatches"] += 1
        k["dur"].append(e["dur"])
        for c, v in e["c"].items():
            k["c"].setdefault(c, []).append(v)
    out = {}
    for name, k in kern.items():
        c = {n: sum(v) / len(v) for n, v in k["c"].items()}
        dur = sum(k["dur"]) / len(k["dur"])
        row = {"dispatches": k["dispatches"], "mean_duration_us": dur * 1e6, "counters": c}
        bf = c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16")
        f32 = c.get("SQ_INSTS_VALU_MFMA_MOPS_F32")
        if bf is not None and dur > 0:
            row["mfma_bf16_tflops"] = bf * 512 / dur / 1e12
            row["frac_bf16_mfma_peak"] = row["mfma_bf16_tflops"] / PEAK_BF16_TFLOPS
        if f32 is not None and dur > 0:
            row["mfma_f32_tflops"] = f32 * 512 / dur / 1e12
            row["frac_f32_mfma_peak"] = row["mfma_f32_tflops"] / PEAK_F32_TFLOPS
        out[name] = row
    return out


def staged_kernel_times(vda, torch, w, inputs, K):
    """The pass's kernel launches (same head ranges and splits as
    vda_forward) through the stage entry points on one stream, with HIP
    events around every launch: mean duration per launch of each kernel (ms),
    the mean staged pass (ms) and the split plans."""
    q, k, v, beta, gate, out = inputs
    H, F, N, dk, dv = w.heads, w.F, w.N, w.d_k, w.d_v
    names = ["frame_stats", "frame_inverse", "state_scan", "readout"]
    groups = head_groups(H)
    bufs = []
    for h0, h1 in groups:
        Hg = h1 - h0
        plan = vda.default_split_plan(F, N, Hg, dk, dv, w.dtype == "f32")
        P = vda.partial_count(Hg * F, *plan)
        A_part = torch.empty((P, dk, dk), dtype=torch.float32, device="cuda")
        B_part = torch.empty((P, dv, dk), dtype=torch.float32, device="cuda")
        S_fwd = torch.empty((Hg, F, dv, dk), dtype=torch.float32, device="cuda")
        S_rev = torch.empty((Hg, F, dv, dk), dtype=torch.float32, device="cuda")
        bufs.append((slice(h0, h1), plan, A_part, B_part, S_fwd, S_rev))

    def staged(evs=None):
        j = 0
        for sl, (tail, sp), A_part, B_part, S_fwd, S_rev in bufs:
            c = S_fwd.shape[0] * F
            Inv = A_part[:c]
            launches = (
                lambda: vda.frame_stats(k[sl], v[sl], beta[sl], splits=sp, tail_frames=tail,
                                        A_part=A_part, B_part=B_part),
                lambda: vda.frame_inverse(A_part, B_part, count=c, tail_frames=tail, splits=sp,
                                          Inv=Inv, tiles=(w.dtype != "f32")),
                (lambda: vda.state_scan(Inv.view(-1, F, dk, dk), B_part[:c].view(-1, F, dv, dk),
                                        S_fwd, S_rev, exact_f32=True)) if w.dtype == "f32" else
                (lambda: vda.state_scan_tiles(Inv.view(-1, F, dk * dk),
                                              B_part[:c].view(-1, F, dv, dk), S_fwd, S_rev)),
                lambda: vda.readout(q[sl], S_fwd, S_rev, gate[sl], out=out[sl]),
            )
            for fn in launches:
                fn()
                if evs is not None:
                    evs[j + 1].record()
                j += 1

    for _ in range(2):
        staged()
    torch.cuda.synchronize()
    nl = 4 * len(groups)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nl + 1)] for _ in range(K)]
    for i in range(K):
        evs[i][0].record()
        staged(evs[i])
    torch.cuda.synchronize()
    launch_ms = {n: [] for n in names}
    for i in range(K):
        for j in range(nl):
            launch_ms[names[j % 4]].append(evs[i][j].elapsed_time(evs[i][j + 1]))
    per_launch = {n: sum(v_) / len(v_) for n, v_ in launch_ms.items()}
    staged_ms = sum(evs[i][0].elapsed_time(evs[i][nl]) for i in range(K)) / K

    plans = [{"tail_frames": b[1][0], "splits": b[1][1]} for b in bufs]
    return per_launch, staged_ms, plans, len(groups)


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="768p_bf16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--settle", type=float, default=0.3,
                    help="seconds of untimed forward passes before the warm-up steps")
    ap.add_argument("--calibrate-copy", type=float, default=0.0, metavar="GIB",
                    help="instead of the operator, run a plain elementwise copy (torch.neg) "
                         "reading and writing GIB GiB, to calibrate HBM byte counters")
    ap.add_argument("--pmc-summary", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR",
                                                       "COPY_WRITE_DIR"),
                    help="summarise rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE runs of this "
                         "benchmark and of --calibrate-copy into HBM bytes per launch (no GPU)")
    ap.add_argument("--copy-gib", type=float, default=1.0,
                    help="size given to --calibrate-copy in the counter runs")
    ap.add_argument("--counter-summary", nargs="+", metavar="DIR",
                    help="summarise rocprofv3 --pmc runs (matrix-core counters) per kernel "
                         "instance (no GPU)")
    ap.add_argument("--all-workloads", action="store_true",
                    help="instead of the headline line, one line per workload: vda_forward's "
                         "time and throughput, and the oracle at one and at all BLAS threads")
    ap.add_argument("--no-extras", action="store_true",
                    help="time only the headline and the per-kernel launches")
    ap.add_argument("--prep-only", action="store_true",
                    help="instead of the headline line, time only VDA-Prep and the two ways from "
                         "the projections to the token-major output on the workload's shape")
    args = ap.parse_args()
    if args.pmc_summary:
        print(json.dumps(pmc_summary(*args.pmc_summary, args.copy_gib, args.workload), indent=1))
        return 0
    if args.counter_summary:
        print(json.dumps(counter_summary(args.counter_summary), indent=1))
        return 0
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (the operator is one GPU's head shard); "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2609_20744_amd import inputs as I
    from paper_2609_20744_amd import vda

    torch.cuda.set_device(0)
    if args.calibrate_copy > 0:
        n = int(args.calibrate_copy * (1 << 30)) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(args.warmup):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            torch.neg(src, out=dst)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        print(json.dumps({"calibration": "torch.neg fp32 copy", "bytes_read": 4 * n,
                          "bytes_written": 4 * n, "ms": ms,
                          "gbs_read_plus_write": 8 * n / ms / 1e6}), flush=True)
        return 0
    if args.all_workloads:
        all_workloads(vda, torch, args.steps, args.warmup, args.settle, args.cpu_budget)
        return 0
    w = I.WORKLOADS[args.workload]
    if args.prep_only:
        print(json.dumps({"workload": w.name, "prep": prep_bench(vda, torch, w, args.steps)}),
              flush=True)
        return 0
    print(f"[bench] generating {w.name} inputs", file=sys.stderr, flush=True)
    x = I.make_inputs(w)
    sets = device_sets(torch, w, x, input_copies(w))
    del x
    q, k, v, beta, gate, out = sets[0]
    H, F, N, dk, dv = w.heads, w.F, w.N, w.d_k, w.d_v
    K = args.steps

    # 1. The headline: the library's forward entry point.  The GPU's clocks
    #    take a few tens of milliseconds of load to settle (the first 20
    #    passes were measured 7% slower), so untimed passes run for
    #    args.settle seconds before the W warm-up steps.  Workloads whose
    #    working set fits in the last-level cache rotate through input sets.
    print(f"[bench] settle {args.settle} s, warmup {args.warmup}", file=sys.stderr, flush=True)
    head = time_forward(vda, torch, sets, K, args.warmup, args.settle)
    ms, wall = head["ms"], head["wall_s"]
    print(f"[bench] timed {K} forward steps: {ms:.4f} ms/step", file=sys.stderr, flush=True)

    # 2. Per-kernel durations: the same launches (same head ranges and splits)
    #    through the stage entry points on one stream, HIP events around every
    #    launch.
    names = ["frame_stats", "frame_inverse", "state_scan", "readout"]
    per_launch, staged_ms, plans, n_groups = staged_kernel_times(vda, torch, w, sets[0], K)
    groups = head_groups(H)

    t = ms / 1e3
    tp = throughput(w, ms)
    # Per-launch algorithmic bytes (mean over the launches timed).
    kb = {n: sum(kernel_bytes(w, h1 - h0)[n] for h0, h1 in groups) / len(groups) for n in names}
    dominant = max(("frame_stats", "readout"), key=lambda n: per_launch[n])
    ach = kb[dominant] / (per_launch[dominant] / 1e3) / 1e9
    result = {
        "metric": METRIC,
        "value": w.tokens / t,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic (seeded; L2-normalised q,k; sigmoid write strengths and gates)",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "F": F, "N": N, "d_k": dk, "d_v": dv,
                   "storage": w.dtype, "state": "fp32", "head_groups": len(groups),
                   "split_plan": plans},
        "tflops": tp["tflops"],
        "pct_bf16_mfma_peak": tp["pct_bf16_mfma_peak"],
        "hbm_gbs_alg": tp["hbm_gbs_alg"],
        "pct_hbm_peak": tp["pct_hbm_peak"],
        "hbm_floor_ms": tp["hbm_floor_ms"],
        "token_heads_per_s": tp["token_heads_per_s"],
        "step_ms_p10_p50_p90": head["p10_p50_p90"],
        "input_sets": head["input_sets"],
        "kernel_ms_per_launch": per_launch,
        "kernel_launches_per_step": len(groups),
        "staged_ms_per_step": staged_ms,
        "wall_s_timed_region": wall,
        "roofline": {"bound": "hbm", "kernel": dominant, "achieved": ach, "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": ach / PEAK_HBM_GBS,
                     "traffic": measured_traffic(w.name, dominant)},
    }
    # 3. The full operator (vda_forward_ex) on the same workload, with every
    #    option: channel decay, text state, the paper's local window (chunks
    #    of five frames, radius one, one leading anchor), for both rules, and
    #    the joint rule with the output gate per token and channel (which
    #    adds one read of an output-sized tensor).  Reported beside the
    #    headline, not as it.
    if args.no_extras:
        if not args.no_cpu_baseline:
            print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
            result["cpu_baseline"] = cpu_baseline(w, args.cpu_budget)
        print(json.dumps(result), flush=True)
        return 0

    def dev(a, dt):
        if dt == "bf16":
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a)).cuda()

    alpha = dev(I.make_decay(w), "f32")
    text_state = dev(I.make_text_state(w), "f32")
    gtok = dev(I.make_token_gates(w), w.dtype) if w.dtype == "bf16" else None
    full = {}
    for rule, tg in (("joint", False), ("frozen", False), ("joint", True)):
        if tg and gtok is None:
            continue
        def fwd_ex():
            vda.forward(q, k, v, beta, None if tg else gate, out=out, alpha=alpha,
                        text_state=text_state, window=(5, 1, 1), rule=rule,
                        gate_tokens=gtok if tg else None)
        for _ in range(max(2, args.warmup)):
            fwd_ex()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(K):
            fwd_ex()
        e1.record()
        torch.cuda.synchronize()
        ms_ex = e0.elapsed_time(e1) / K
        name = f"{rule}_decay_text_window" + ("_token_gate" if tg else "")
        full[name] = {"ms_per_step": ms_ex, "tokens_per_s": w.tokens / (ms_ex / 1e3)}
        print(f"[bench] vda_forward_ex ({name}): {ms_ex:.4f} ms/step", file=sys.stderr,
              flush=True)
    # The core operator with the epilogue's token-major output
    # ([clips][F][N][heads * d_v], vda_options.out_heads), the layout the
    # model's output projection reads.
    out_tm = torch.empty((w.B, F, N, w.H * dv), dtype=out.dtype, device=out.device)
    def fwd_tm():
        vda.forward(q, k, v, beta, gate, out=out_tm, out_heads=w.H)
    for _ in range(max(2, args.warmup)):
        fwd_tm()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(K):
        fwd_tm()
    e1.record()
    torch.cuda.synchronize()
    ms_tm = e0.elapsed_time(e1) / K
    full["token_major_output"] = {"ms_per_step": ms_tm, "tokens_per_s": w.tokens / (ms_tm / 1e3)}
    print(f"[bench] vda_forward_ex (token-major output): {ms_tm:.4f} ms/step", file=sys.stderr,
          flush=True)
    # ... and reading the raw token-major query (vda_options.q_heads), whose
    # L2 map the readout applies; the timing reads q's buffer in that layout.
    q_tm = q.view(w.B, F, N, w.H * dk)
    ms_rq = _time_calls(torch, lambda: vda.forward(q_tm, k, v, beta, gate, out=out_tm,
                                                   out_heads=w.H, q_heads=w.H),
                        K, max(2, args.warmup))
    full["raw_query_token_major"] = {"ms_per_step": ms_rq, "tokens_per_s": w.tokens / (ms_rq / 1e3)}
    print(f"[bench] vda_forward_ex (raw token-major query and output): {ms_rq:.4f} ms/step",
          file=sys.stderr, flush=True)
    del out_tm
    # The prompt state itself (vda_text_state): a 512-token prompt per head of
    # the workload, one frame from zero, joint rule.
    pw = I.custom("prompt", 1, w.heads, 1, 512, w.d_k, w.d_v, w.dtype, seed=w.seed + 77)
    px = I.make_inputs(pw)
    pk, pv = dev(px["k"][:, 0], w.dtype), dev(px["v"][:, 0], w.dtype)
    pb = dev(px["beta"][:, 0], "f32")
    s_out = vda.text_state(pk, pv, pb)
    for _ in range(max(2, args.warmup)):
        vda.text_state(pk, pv, pb, out=s_out)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(K):
        vda.text_state(pk, pv, pb, out=s_out)
    e1.record()
    torch.cuda.synchronize()
    full["text_state_prompt512"] = {"ms_per_call": e0.elapsed_time(e1) / K, "prompt_tokens": 512,
                                    "heads": w.heads}
    print(f"[bench] vda_text_state (512 prompt tokens): {e0.elapsed_time(e1) / K:.4f} ms/call",
          file=sys.stderr, flush=True)
    result["full_operator"] = full
    # 4. VDA-Prep (the feature map before the operator) on this workload's
    #    shape: token-major bf16 projections -> frame-major features.
    result["prep"] = prep_bench(vda, torch, w, K)
    # 5. The two scan paths of a chunked window, alone: frame by frame
    #    (vda_state_scan_tiles) and chunk-wise (vda_state_scan_chunked, chunks
    #    of five after one anchor), on this workload's heads and frames and on
    #    the paper's own shard (7 heads per GPU, 100 interior frames).
    #    The same at narrower heads (d = 64 and 32), which the path choice
    #    also covers.
    result["scan_paths"] = [scan_paths(vda, torch, Hs, Fs, d, d, 5, 1, K)
                            for d in (dk, 64, 32) for Hs, Fs in ((H, F), (7, 100))]
    # 6. The paper's own shard at full size (7 heads x 100 frames x 4032
    #    tokens): the core pass and the full operator.
    del sets, q, k, v, beta, gate, out, alpha, text_state, gtok
    torch.cuda.empty_cache()
    result["paper_shard"] = paper_shard(vda, torch, K, args.warmup)
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_budget)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
