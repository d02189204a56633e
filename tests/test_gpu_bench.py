"""bench.py end to end on the smallest model-shaped stack: one JSON line with the fields the
measurement contract names (metric, value, roofline with traffic, cpu_baseline of the oracle,
library reference timings), all finite and in range."""
import json
import math
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_json_line():
    p = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--config", "opt-1.3b",
                        "--steps", "1", "--warmup", "0", "--cpu-budget", "1"],
                       capture_output=True, text=True, timeout=110, cwd=ROOT)
    assert p.returncode == 0, p.stderr[-2000:]
    lines = [l for l in p.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, p.stdout[-2000:]
    d = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
              "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 1 and d["warmup"] == 0
    assert d["unit"] == "TFLOP/s" and d["dtype"] == "bf16" and d["data"] == "synthetic"
    assert d["higher_is_better"] is True and d["vs_baseline"] is None
    assert "workload" in d["config"] and "model" not in d["config"]
    assert 0 < d["value"] < 2516.6 and math.isfinite(d["ms_per_step"])
    rf = d["roofline"]
    assert rf["bound"] == "mfma" and rf["unit"] == "TFLOP/s" and rf["peak"] == 2516.6
    assert 0 < rf["achieved"] < rf["peak"] and abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-3
    assert "traffic" in rf  # null: the committed counters are for the OPT-13B workload
    up = d["update"]
    assert up["bound"] == "hbm" and 0 < up["achieved"] < up["peak"] == 8000.0
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb["value"] > 0 and cb["sample"]
    pk = d["practical_peaks"]
    assert pk["gemm_torch_matmul"]["tflops"] > 0 and pk["copy_2gib_gbs"] > 0 and pk["inplace_rmw_2gib_gbs"] > 0
