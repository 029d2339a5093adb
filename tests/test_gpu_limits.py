"""Parity at the largest sizes the library accepts: the kernels address x and y
with 32-bit byte offsets, and a plan takes each of them only below 2^31 bytes.
An output y (and, separately, an input x) of 99 % of that limit is run and
checked against the oracle on three output planes: the first, one in the
middle and the last, whose stores sit at the largest offsets of y; the layers
read the whole of x for each of them.  The planes are computed once per shape
and shared by the tile sizes and algorithms (Winograd F(2)-F(7) and the FFT
tiles)."""

import numpy as np
import pytest
import torch

import paper_1912_02165_amd as wc
from oracle.direct import direct_conv_planes
from parity import assert_close

pytestmark = pytest.mark.gpu

Y_LIMIT = (1, 16, 128, 2040, 2040)   # y: 128 * 2040^2 * 4 = 2,130,739,200 bytes
X_LIMIT = (1, 128, 16, 2040, 2040)   # x: the same bytes on the input side
CASES = [(Y_LIMIT, 2, "fused"), (Y_LIMIT, 4, "fused"), (Y_LIMIT, 5, "fused"), (Y_LIMIT, 6, "fused"),
         (Y_LIMIT, 4, "three_stage"), (Y_LIMIT, 7, "three_stage"),
         (Y_LIMIT, 14, "fft"),
         (X_LIMIT, 4, "fused"), (X_LIMIT, 6, "fused"), (X_LIMIT, 4, "three_stage"), (X_LIMIT, 14, "fft")]

_cache = {}


def _inputs_and_planes(shape):
    if shape not in _cache:
        _cache.clear()
        N, C, K, H, W = shape
        rng = np.random.default_rng(7001 + C)
        x = rng.random((N, C, H, W), dtype=np.float32) * 2.0 - 1.0
        w = (rng.standard_normal((K, C, 3, 3), dtype=np.float32) * np.float32(np.sqrt(2.0 / (9 * C))))
        planes = [(0, 0), (0, K // 2), (N - 1, K - 1)]
        _cache[shape] = (x, w, planes, direct_conv_planes(x, w, planes))
    return _cache[shape]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{'x'.join(map(str, c[0]))}-m{c[1]}-{c[2]}")
def test_largest_accepted_sizes(case):
    shape, m, algo = case
    N, C, K, H, W = shape
    assert 4 * N * max(C, K) * H * W < 2**31 and 4 * N * max(C, K) * H * W > 0.99 * 2**31
    print(f"\n[gpu] limit {case}", flush=True)
    x, w, planes, ref = _inputs_and_planes(shape)
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y = torch.full((N, K, H, W), float("nan"), dtype=torch.float32, device="cuda")
    with wc.Plan(N, C, K, H, W, m, algo) as p:
        p.run(xd, wd, y)
        p.status()
    got = np.stack([y[n, k].cpu().numpy() for n, k in planes])
    del y, xd, wd
    torch.cuda.empty_cache()
    assert_close(got, ref, m, f"{case} planes {planes}")
