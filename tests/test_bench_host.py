"""Host-side logic of the benchmark and the trainer's schedule (no GPU)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_1806_00512_amd.inputs import WORKLOADS  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_roofline_entry_bounds():
    # an MFMA-bound launch: 1 TFLOP in 10 ms = 100 TFLOP/s against the fp32 peak
    e = bench.roofline_entry("k", {"flops": 1e12, "bytes": 1e6}, 0.01, "f32", None)
    assert e["bound"] == "mfma" and e["achieved"] == pytest.approx(100.0)
    assert e["frac"] == pytest.approx(100.0 / bench.PEAK["f32_tflops"], rel=1e-3)
    # an HBM-bound launch: 8 GB in 2 ms = 4000 GB/s
    e = bench.roofline_entry("k", {"flops": 0.0, "bytes": 8e9}, 0.002, "f32", 9e9)
    assert e["bound"] == "hbm" and e["achieved"] == pytest.approx(4000.0)
    assert e["frac"] == pytest.approx(0.5) and e["traffic"] == 9e9


def test_kernel_work_counts():
    wl = WORKLOADS["lstm4_enc_h2048_b128_t50_f32"]
    I, H, B, T = 2048, 2048, 128, 50
    Kp = 4 * H // 2
    w = bench.kernel_work(wl, 1, Kp, 4)
    assert w["data_grad_gemm"]["flops"] == 2 * T * (I + H) * B * Kp
    assert w["weight_grad_gemm"]["flops"] == 2 * T * Kp * (I + H) * B
    # dW is written once per layer call (fp32)
    assert w["weight_grad_gemm"]["bytes"] >= 4 * H * (I + H) * 4
    # the kept rows and index move from the gate kernels to the dh product
    # when the selection runs inside it; the total stays the same
    ws = bench.kernel_work(wl, 1, Kp, 4, select_in_product=True)
    compact = T * (Kp * B * 4 + Kp // 4 * 4)
    assert w["gates_select_compact"]["bytes"] - ws["gates_select_compact"]["bytes"] == compact
    assert ws["data_grad_gemm"]["bytes"] - w["data_grad_gemm"]["bytes"] == compact
    assert ws["data_grad_gemm"]["flops"] == w["data_grad_gemm"]["flops"]


def test_traffic_needs_matching_sources(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    os.makedirs(tmp_path / "profiles")
    f = tmp_path / "profiles" / "traffic_wgrad_kernel_w.txt"
    f.write_text("sources_sha256_16: 0000\nhbm_bytes_per_launch: 123\n")
    monkeypatch.setattr(bench, "sources_digest", lambda: "0000")
    assert bench.traffic_on_file("weight_grad_gemm", "w") == 123.0
    monkeypatch.setattr(bench, "sources_digest", lambda: "ffff")
    assert bench.traffic_on_file("weight_grad_gemm", "w") is None


def test_dense_after_sparse_schedule():
    from paper_1806_00512_amd.train import dense_after_sparse
    assert dense_after_sparse(8) == [True] * 6 + [False] * 2
    assert dense_after_sparse(10, 0.9) == [True] * 9 + [False]
    assert dense_after_sparse(3, 0.0) == [False] * 3
    with pytest.raises(ValueError):
        dense_after_sparse(4, 1.5)


def test_sweep_entries_and_integer_removals():
    # the H = 1024 workload's sweep removes a whole number of slices per region
    wl = WORKLOADS["lstm2_h1024_b64_t35_f32"]
    assert wl.sweep == (0.0, 0.25, 0.5, 0.75)
    for s in wl.sweep:
        assert abs(s * wl.R - round(s * wl.R)) < 1e-9
    assert "lstm2_h1024_b64_t35_f32" in bench.ALSO_WORKLOADS
    e = bench.sweep_entries({"dn_ms": 2.0, "sweep": [(0.0, 2.0), (0.5, 1.6), (0.75, 1.25)]})
    assert [p["sparsity"] for p in e] == [0.0, 0.5, 0.75]
    assert [p["speedup_vs_dense"] for p in e] == [1.0, 1.25, 1.6]


def test_rocprof_duration_needs_matching_sources(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    os.makedirs(tmp_path / "profiles")
    f = tmp_path / "profiles" / "kernels_w.txt"
    f.write_text("# summary\nsources_sha256_16: 0000\nrocprof_avg_us_data_grad_gemm: 40.0\n")
    monkeypatch.setattr(bench, "sources_digest", lambda: "0000")
    assert bench.rocprof_on_file("data_grad_gemm", "w") == 40.0
    assert bench.rocprof_on_file("weight_grad_gemm", "w") is None
    monkeypatch.setattr(bench, "sources_digest", lambda: "ffff")
    assert bench.rocprof_on_file("data_grad_gemm", "w") is None
    # both fractions: from the live event time and from the profiler's time
    e = bench.roofline_entry("k", {"flops": 1e12, "bytes": 1e6}, 0.01, "f32", None, 8000.0)
    assert e["frac"] == pytest.approx(100.0 / bench.PEAK["f32_tflops"], rel=1e-3)
    assert e["frac_rocprof"] == pytest.approx(125.0 / bench.PEAK["f32_tflops"], rel=1e-3)


def test_every_workload_is_measured():
    """The default workload plus every other one under "also"."""
    assert bench.DEFAULT_WORKLOAD in WORKLOADS
    assert set(bench.ALSO_WORKLOADS) | {bench.DEFAULT_WORKLOAD} == set(WORKLOADS)
