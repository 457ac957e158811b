"""Host-side checks of bench.py: the one-GPU guard and the counter summary
that feeds roofline.traffic (no GPU needed)."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_kernel_bytes_formula_at_768p():
    from paper_2609_20744_amd.inputs import WORKLOADS
    kb = bench.kernel_bytes(WORKLOADS["768p_bf16"])
    fh, N, d = 16 * 36, 3840, 128
    # K, V in bf16 plus fp32 beta per token; A and B out in fp32.
    assert kb["frame_stats"] == fh * (N * (2 * 2 * d + 4) + 4 * 2 * d * d)
    # q in, out out (bf16); both fp32 states in; one fp32 gate per head.
    assert kb["readout"] == fh * (N * 2 * 2 * d + 2 * 4 * d * d) + 4 * 16


def _write_counters(dirpath, rows):
    os.makedirs(dirpath, exist_ok=True)
    with open(os.path.join(dirpath, "run_counter_collection.csv"), "w") as f:
        f.write('"Kernel_Name","Counter_Value"\n')
        for name, kib in rows:
            f.write(f'"{name}",{kib}\n')


def test_pmc_summary_scales_by_copy_factor(tmp_path):
    neg = "void at::native::vectorized_elementwise_kernel<4, at::native::neg_kernel_cuda(x)>(int)"
    fill = "void at::native::vectorized_elementwise_kernel<4, at::native::FillFunctor<float> >(int)"
    stats = "void vda::(anonymous namespace)::stats_bf16_kernel<128, 128>(unsigned short const*)"
    gib_kib = 1 << 20
    _write_counters(tmp_path / "cf", [(fill, 10.0), (neg, gib_kib / 2), (neg, gib_kib / 2)])
    _write_counters(tmp_path / "cw", [(fill, gib_kib), (neg, gib_kib)])
    _write_counters(tmp_path / "f", [(stats, 1000.0), (stats, 3000.0)])
    _write_counters(tmp_path / "w", [(stats, 500.0)])
    s = bench.pmc_summary(str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "cf"),
                          str(tmp_path / "cw"), 1.0, "768p_bf16")
    assert s["fetch_factor"] == pytest.approx(2.0)
    assert s["write_factor"] == pytest.approx(1.0)
    k = s["kernels"]["frame_stats"]
    assert k["hbm_read_bytes"] == pytest.approx(2000.0 * 1024 * 2.0)
    assert k["hbm_write_bytes"] == pytest.approx(500.0 * 1024)
    assert set(s["kernels"]) == {"frame_stats"}


def test_traffic_is_null_once_the_kernel_changed(tmp_path, monkeypatch):
    summ = {"kernels": {"frame_stats": {"source_sha256": bench.source_hash("frame_stats"),
                                        "hbm_bytes_per_launch": 123.0},
                        "readout": {"source_sha256": "0" * 64, "hbm_bytes_per_launch": 456.0}}}
    path = tmp_path / "t.json"
    path.write_text(json.dumps(summ))
    monkeypatch.setattr(bench, "traffic_file", lambda w: str(path))
    assert bench.measured_traffic("768p_bf16", "frame_stats") == 123.0
    assert bench.measured_traffic("768p_bf16", "readout") is None
    assert bench.measured_traffic("768p_bf16", "state_scan") is None


def test_committed_traffic_summary_is_well_formed():
    path = bench.traffic_file("768p_bf16")
    if not os.path.exists(path):
        pytest.skip("no counter summary committed")
    s = json.load(open(path))
    assert s["write_factor"] > 0 and s["fetch_factor"] > 0
    for stage, k in s["kernels"].items():
        assert stage in bench.KERNEL_OF
        assert k["hbm_bytes_per_launch"] == pytest.approx(k["hbm_read_bytes"] + k["hbm_write_bytes"])


def test_source_hash_ignores_comments_and_layout():
    """Counters stay attached to a kernel whose comments alone change."""
    a = "int f(int x) {  // doubles\n  return 2 * x;  /* twice */\n}\n"
    b = "// a new header comment\nint f(int x) {\n\n  return 2 * x;\n}\n"
    c = "int f(int x) { return 3 * x; }"
    assert bench._code_only(a) == bench._code_only(b)
    assert bench._code_only(a) != bench._code_only(c)


def test_counter_summary_derives_mfma_rates(tmp_path):
    """Matrix-core counters per kernel instance: mean over dispatches, 512
    FLOPs per MOPS unit, rate over the dispatch's own duration."""
    d = tmp_path / "pmc"
    os.makedirs(d)
    inv = "void vda::(anonymous namespace)::inverse_kernel<128, true>(float const*, int)"
    rows = []
    # two dispatches of 10 us each: 1e6 and 3e6 F32 MOPS units
    for disp, mops in ((1, 1e6), (2, 3e6)):
        for cname, val in (("SQ_INSTS_VALU_MFMA_MOPS_F32", mops), ("MfmaUtil", 10.0 * disp)):
            rows.append(f'{disp},"{inv}","{cname}",{val},1000,11000')
    (d / "run_counter_collection.csv").write_text(
        '"Dispatch_Id","Kernel_Name","Counter_Name","Counter_Value","Start_Timestamp",'
        '"End_Timestamp"\n' + "\n".join(rows) + "\n")
    s = bench.counter_summary([str(d)])
    k = s["inverse_kernel<128,true>"]
    assert k["dispatches"] == 2
    assert k["mean_duration_us"] == pytest.approx(10.0)
    assert k["counters"]["MfmaUtil"] == pytest.approx(15.0)
    assert k["mfma_f32_tflops"] == pytest.approx(2e6 * 512 / 1e-5 / 1e12)
    assert k["frac_f32_mfma_peak"] == pytest.approx(k["mfma_f32_tflops"] / 157.3)
