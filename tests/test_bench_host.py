"""Host-side pieces of bench.py (CPU): the one-GPU guard, the algorithmic
byte counts behind roofline.achieved, the counter-summary lookup behind
roofline.traffic and the shape of the cpu_baseline record."""
import os
import subprocess
import sys

import bench
from paper_2607_10611_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_bytes_per_param_counts_each_array_once():
    assert bench.bytes_per_param("bf16", "fp32") == 2 + 4 + 12 + 2 + 12
    assert bench.bytes_per_param("bf16", "bf16") == 2 + 4 + 6 + 2 + 6
    assert bench.bytes_per_param("e4m3", "fp32") == 30
    assert bench.bytes_per_param("nvfp4", "fp32") == 29


def test_algorithmic_bytes_of_the_7b_settings():
    sizes = [s.numel for s in W.specs("c5")]
    n = sum(sizes)
    plain = [("bf16", False, False)] * len(sizes)
    assert bench.algorithmic_bytes(sizes, plain, "fp32") == 32 * n == 215629299712
    lin = [s for s, p in zip(sizes, W.low_precision_master_plan("c5", "e4m3")) if p[1]]
    nl, nt = sum(lin), len(lin)
    rest = n - nl
    fp8 = bench.algorithmic_bytes(sizes, W.low_precision_master_plan("c5", "e4m3"), "fp32")
    assert fp8 == nl * (30 + 2) + rest * 32 + nl // 128 * 4
    mx = bench.algorithmic_bytes(sizes, W.low_precision_master_plan("c5", "mxfp4"), "fp32")
    assert mx == nl * (29 + 2) + rest * 32 + nl // 32 * 2
    nv = bench.algorithmic_bytes(sizes, W.low_precision_master_plan("c5", "nvfp4"), "fp32")
    assert nv == nl * (29 + 2) + rest * 32 + nl // 16 * 2 + 4 * nt
    cs = bench.algorithmic_bytes(sizes, W.low_precision_master_plan("c5", "nvfp4_current"),
                                 "fp32")
    assert cs == nl * (29 + 2) + rest * 32 + nl // 16 * 2 + 8 * nt
    plan = W.low_precision_master_plan("c5", "nvfp4_current")
    assert bench.scratch_bytes(sizes, plan) == 8 * nl + 12 * nt


def test_traffic_is_reported_only_for_the_profiled_kernel_source(monkeypatch, tmp_path):
    summary = tmp_path / "pmc.md"
    summary.write_text(f"kernel_code_sha256: {bench.kernel_sha()}\n"
                       "traffic_bytes_per_launch: 2.5e+11\n")
    monkeypatch.setattr(bench, "PMC_SUMMARY", str(summary))
    assert bench.traffic_from_profile() == 2.5e11
    summary.write_text("kernel_code_sha256: " + "0" * 64 + "\ntraffic_bytes_per_launch: 2.5e+11\n")
    assert bench.traffic_from_profile() is None
    monkeypatch.setattr(bench, "PMC_SUMMARY", str(tmp_path / "missing.md"))
    assert bench.traffic_from_profile() is None


def test_kernel_hash_ignores_comments_and_blank_lines(monkeypatch, tmp_path):
    a, b = tmp_path / "a.hip", tmp_path / "b.hip"
    a.write_text("int f() {\n  return 1;  // one\n}\n")
    b.write_text("/* note */\nint f() {\n\n  return 1;\n}\n")
    monkeypatch.setattr(bench, "KERNEL_SRC", str(a))
    ha = bench.kernel_sha()
    monkeypatch.setattr(bench, "KERNEL_SRC", str(b))
    assert bench.kernel_sha() == ha
    b.write_text("int f() {\n  return 2;\n}\n")
    assert bench.kernel_sha() != ha


def test_cpu_baseline_record():
    rec = bench.cpu_baseline("c5", 1 << 12, 2, "fp32", threads=2, seconds=0.0)
    assert rec["kind"] == "oracle" and rec["unit"] == "Gparam/s" and rec["cores"] == 2
    assert rec["value"] > 0 and "2 steps" in rec["sample"]
    assert "logical CPUs" in rec["host"]
