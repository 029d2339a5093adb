"""Host-side checks of bench.py (no GPU): it refuses more than one GPU with a
message before touching a device, its measured-traffic lookup only accepts
entries taken on the current kernel source, and its per-call timing takes
exactly the requested calls for the timed steps and a longer window only where
asked."""

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


class _FakeTimer:
    """Stands in for a window of n back-to-back calls of `ms_each` milliseconds."""

    def __init__(self, ms_each):
        self.ms_each = ms_each
        self.windows = []

    def __call__(self, n):
        self.windows.append(n)
        return n * self.ms_each


def test_timed_steps_are_exactly_the_requested_calls():
    for ms_each in (0.008, 0.37):
        t = _FakeTimer(ms_each)
        assert abs(bench.per_call_ms(t, 100, exact=True) - ms_each) < 1e-12
        assert t.windows == [100]


def test_short_windows_are_lengthened_to_the_minimum_time():
    t = _FakeTimer(0.008)  # 20 calls of 8 us: 0.16 ms, below MIN_TIMED_MS
    assert abs(bench.per_call_ms(t, 20) - 0.008) < 1e-12
    assert t.windows[0] == 20 and len(t.windows) == 2
    assert t.windows[1] * 0.008 >= bench.MIN_TIMED_MS
    assert t.windows[1] <= bench.MAX_TIMED_CALLS
    long = _FakeTimer(0.37)  # 20 calls of 370 us already cover the minimum
    bench.per_call_ms(long, 20)
    assert long.windows == [20]
    tiny = _FakeTimer(1e-7)  # never more than MAX_TIMED_CALLS
    bench.per_call_ms(tiny, 20)
    assert tiny.windows[1] == bench.MAX_TIMED_CALLS
