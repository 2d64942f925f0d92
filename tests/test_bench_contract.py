"""The benchmark's one-line JSON contract (a short run) and its refusal of
more than one GPU."""
from __future__ import annotations

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout.strip() == ""


@pytest.mark.gpu
def test_bench_line_has_the_contract_fields():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "3",
                        "--warmup", "2", "--prewarm-ms", "20", "--no-gemm", "--cpu-seconds",
                        "0.5"],
                       capture_output=True, text=True, timeout=600, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, lines
    rec = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline"):
        assert key in rec, key
    assert rec["n_gpus"] == 1 and rec["steps"] == 3 and rec["warmup"] == 2
    assert rec["value"] > 0 and rec["unit"] == "TFLOP/s" and rec["higher_is_better"] is True
    assert rec["config"]["workload"] == "prefill_b1_h32_s8192_d128"
    assert rec["prewarm_ms"] >= 20
    roof = rec["roofline"]
    for key in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert key in roof, key
    assert roof["bound"] == "mfma" and roof["unit"] == "TFLOP/s"
    assert abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-9
    cpu = rec["cpu_baseline"]
    for key in ("value", "unit", "cores", "kind", "sample"):
        assert key in cpu, key
    assert cpu["kind"] == "oracle" and cpu["cores"] >= 1 and cpu["value"] > 0
    legs = rec["legs"]
    assert set(legs) == {"prefill_b1_h32_s8192_d128", "prefill_b4_h16_s2048_d128_causal",
                         "decode_b16_h32_s8192_d128", "decode_b1_h32_s131072_d128"}
    assert legs["prefill_b1_h32_s8192_d128"]["value"] == rec["value"]
    for name, leg in legs.items():
        assert leg["roofline"]["bound"] == ("hbm" if name.startswith("decode") else "mfma")
        assert leg["value"] > 0 and leg["ms_per_call"] > 0
