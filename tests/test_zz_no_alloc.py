"""wino_conv_run_noalloc (the entry point that allocates nothing) through the C ABI,
against wino_conv_run with a plan of the same default blocking: the same kernels,
so the same bits, and within tolerance of the oracle; two calls in a row on one
GPU share the scratch array, the second with a smaller input; layers whose scratch
exceeds the array are refused."""

import re

import numpy as np
import pytest
import torch

import paper_1912_02165_amd as wc
from paper_1912_02165_amd import workloads
from oracle.direct import direct_conv
from parity import assert_close

pytestmark = pytest.mark.gpu


def _plan_run(x, w, m):
    N, C, H, W = x.shape
    K = w.shape[0]
    y = torch.full((N, K, H, W), float("nan"), device="cuda")
    with wc.Plan(N, C, K, H, W, m) as p:
        p.run(x, w, y)
        p.status()
    return y


def _noalloc_run(x, w, m, status):
    N, C, H, W = x.shape
    K = w.shape[0]
    y = torch.full((N, K, H, W), float("nan"), device="cuda")
    wc.wino_conv_run_noalloc(N, C, K, H, W, m, x, w, y, status)
    return y


# pairs of calls in a row: (first shape, second, smaller, shape, m, whether the
# first has split items); a first call with split items keeps partial outputs and
# counters in the scratch; the full-size 28x28 layer (N=64, C=K=128) uses 2.4 MB
# of transformed kernels, the C=K=256 one 9.4 MB
PAIRS = [
    ((1, 256, 256, 28, 28), (1, 20, 24, 17, 19), 4, True),
    ((1, 64, 64, 56, 56), (1, 9, 17, 13, 11), 2, False),
    ((2, 256, 64, 14, 14), (1, 5, 17, 13, 11), 6, True),
    ((2, 250, 40, 14, 15), (1, 20, 24, 17, 19), 5, True),
    ((64, 128, 128, 28, 28), (3, 64, 64, 20, 20), 4, False),
]


def _split_items(shape, m):
    with wc.Plan(*shape, m) as p:
        found = re.search(r"split items (\d+) x", p.describe())
    return int(found.group(1)) if found else 0


@pytest.mark.parametrize("pair", PAIRS, ids=lambda p: "m%d-%s" % (p[2], "x".join(map(str, p[0]))))
def test_noalloc_matches_run_twice(pair):
    first, second, m, split = pair
    assert (_split_items(first, m) > 0) == split
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    for i, shape in enumerate((first, second)):
        N, C, K, H, W = shape
        x, w = workloads.random_inputs(N, C, K, H, W, seed=500 + 7 * i + sum(shape) + m)
        xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
        print(f"\n[gpu] noalloc call {i + 1} m={m} shape={shape}", flush=True)
        y_na = _noalloc_run(xd, wd, m, status)
        torch.cuda.synchronize()
        y_plan = _plan_run(xd, wd, m)
        assert torch.equal(y_na, y_plan), f"call {i + 1}: differs from wino_conv_run"
        assert_close(y_na.cpu().numpy(), direct_conv(x, w), m, f"noalloc call {i + 1} F({m}) {shape}")
    assert int(status.item()) == 0, "a bounded wait gave up"


def test_noalloc_repeated_calls_bitwise():
    """Calls repeated on the shared scratch (its counters cleared by each call's
    kernel transform) give identical bits."""
    N, C, K, H, W = 1, 64, 64, 56, 56
    x, w = workloads.random_inputs(N, C, K, H, W, seed=77)
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    ys = [_noalloc_run(xd, wd, 2, None) for _ in range(3)]
    torch.cuda.synchronize()
    assert torch.equal(ys[0], ys[1]) and torch.equal(ys[0], ys[2])


def test_noalloc_refuses_too_large():
    """C = K = 512 at F(6x6,3x3) needs 67 MB of transformed kernels: refused (before
    any HIP call); at F(4x4,3x3), 38 MB: refused too; y untouched."""
    N, C, K, H, W = 64, 512, 512, 14, 14
    x = torch.zeros((N, C, H, W), device="cuda")
    w = torch.zeros((K, C, 3, 3), device="cuda")
    y = torch.full((N, K, H, W), 3.0, device="cuda")
    for m in (6, 4):
        with pytest.raises(wc.WinoError, match="scratch") as e:
            wc.wino_conv_run_noalloc(N, C, K, H, W, m, x, w, y)
        assert e.value.status == wc.wino.WINO_EUNSUPPORTED
    torch.cuda.synchronize()
    assert bool((y == 3.0).all())


def test_noalloc_rejects_bad_arguments():
    N, C, K, H, W = 1, 4, 8, 8, 8
    x = torch.zeros((N, C, H, W), device="cuda")
    w = torch.zeros((K, C, 3, 3), device="cuda")
    y = torch.zeros((N, K, H, W), device="cuda")
    with pytest.raises(wc.WinoError, match="only F"):
        wc.wino_conv_run_noalloc(N, C, K, H, W, 3, x, w, y)
    with pytest.raises(wc.WinoError, match="overlaps"):
        wc.wino_conv_run_noalloc(N, C, C, H, W, 4, x, torch.zeros((C, C, 3, 3), device="cuda"), x)
    host = np.zeros(N * K * H * W, np.float32)
    with pytest.raises(wc.WinoError, match="device"):
        wc.wino_conv_run_noalloc(N, C, K, H, W, 4, x, w, host.ctypes.data)
