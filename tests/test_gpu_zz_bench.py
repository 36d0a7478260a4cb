"""The benchmark's JSON line on a short run: every field the report needs,
with consistent roofline and CPU-baseline entries (the small workload, so the
run takes seconds)."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_json_line():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "lstm1_h128_b16_t20_f32",
           "--steps", "3", "--warmup", "1", "--no-also", "--no-fine", "--no-train", "--no-bidir"]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
              "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
              "roofline", "cpu_baseline"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["dtype"] == "f32" and d["config"]["workload"] == "lstm1_h128_b16_t20_f32"
    assert d["value"] > 0 and d["ms_per_step"] > 0
    rl = d["roofline"]
    assert rl["bound"] in ("hbm", "mfma", "alu") and rl["unit"] in ("GB/s", "TFLOP/s")
    assert rl["frac"] == pytest.approx(rl["achieved"] / rl["peak"], rel=1e-2, abs=1e-4)
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb["value"] > 0 and cb["sample"]
    one = cb["single_core"]
    assert one["cores"] == 1 and one["value"] > 0 and one["sample"]
    assert set(d["roofline_all"]) == {"gates_select_compact", "data_grad_gemm",
                                      "weight_grad_gemm"}
