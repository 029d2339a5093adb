"""Host-side checks of bench.py (no GPU): it refuses more than one GPU with a
message before touching a device, its measured-traffic lookup only accepts
entries taken on the current kernel source, and every workload of the table
exists."""

import json
import os
import subprocess
import sys

import bench
from paper_1912_02165_amd import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_entries_match_the_kernel_source():
    with open(bench.TRAFFIC_FILE) as f:
        data = json.load(f)
    entries = data if isinstance(data, list) else data.get("entries", [])
    assert entries, "no measured traffic entries"
    h = bench.kernel_source_hash()
    headline = workloads.LAYER_BY_ID[2].tag(4)
    got = bench.measured_traffic("fused", headline)
    if any(e.get("source_hash") == h and e.get("workload") == headline for e in entries):
        # calibrated bytes per launch: at least the algorithmic x + y of the layer
        layer = workloads.LAYER_BY_ID[2]
        assert got is not None and got >= 2 * 4 * layer.N * layer.C * layer.H * layer.W
    else:
        assert got is None
    assert bench.measured_traffic("fused", "no such workload") is None
