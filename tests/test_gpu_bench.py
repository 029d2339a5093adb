"""The benchmark's JSON line on the GPU: a short `bench.py` run (headline layer
only, no CPU baseline) prints exactly one line with the keys, units and ranges
the reporting contract fixes: one GPU, the requested step counts, effective
TFLOP/s over the step time, and the fused kernel's roofline entry with its
fraction of the fp32 matrix peak."""

import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_line_keeps_the_contract():
    print("\n[gpu] bench.py --steps 3 --warmup 1 --no-layers --no-cpu", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "3", "--warmup", "1",
                        "--no-layers", "--no-cpu"], capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, r.stdout
    d = json.loads(lines[0])
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["unit"] == "TFLOP/s" and d["higher_is_better"] is True and d["scaling"] == "weak"
    assert d["dtype"] == "f32" and d["data"] == "synthetic" and d["vs_baseline"] is None
    assert d["config"]["workload"] == "N32_C64_K64_224x224/F(4x4,3x3)"
    # value: direct-convolution flops of the layer over the mean step time
    flops = 2 * 32 * 64 * 64 * 224 * 224 * 9
    assert d["ms_per_step"] > 0
    assert abs(d["value"] - flops / (d["ms_per_step"] * 1e-3) / 1e12) <= 1e-6 * d["value"]
    rf = d["roofline"]
    assert rf["bound"] == "mfma" and rf["unit"] == "TFLOP/s" and rf["peak"] == 157.3
    assert 0.0 < rf["frac"] < 1.0 and abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-9
    assert rf["kernel"].startswith("fused_ws_kernel<M=4")
    # the kernel's own time is part of the step (kernel transform + fused kernel)
    assert 0 < rf["kernel_ms"] <= d["ms_per_step"] * 1.05
    assert rf["traffic"] is None or rf["traffic"] > 0
    assert d["cpu_baseline"] is None and d["layers"] is None
