"""Seeded random shapes for every algorithm and tile size against the fp64
direct oracle: sizes drawn so that channel counts, image sides and batch sizes
fall on and off the blockings (4 input channels, 16 output channels, 16 or 32
tiles per work item, tile edges m), including one-pixel and one-channel
extremes.  The shapes are fixed by the seed, so a failure names its case."""

import numpy as np
import pytest
import torch

import paper_1912_02165_amd as wc
from paper_1912_02165_amd import workloads
from oracle.direct import direct_conv
from parity import assert_close

pytestmark = pytest.mark.gpu


def run_gpu(x, w, m, algo):
    N, C, H, W = x.shape
    K = w.shape[0]
    y = torch.full((N, K, H, W), float("nan"), dtype=torch.float32, device="cuda")
    with wc.Plan(N, C, K, H, W, m, algo) as p:
        p.run(torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda(), y)
        torch.cuda.synchronize()
    return y


def _shapes(seed, count):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        N = int(rng.integers(1, 4))
        C = int(rng.choice([1, 3, 4, 5, 16, 17, 31, 64, 70]))
        K = int(rng.choice([1, 2, 15, 16, 17, 33, 64, 65]))
        H = int(rng.integers(1, 41))
        W = int(rng.integers(1, 41))
        out.append((N, C, K, H, W))
    return out


CASES = ([(s, m, "fused") for m in (2, 4, 5, 6) for s in _shapes(100 + m, 6)]
         + [(s, m, "three_stage") for m in (2, 4, 6, 7) for s in _shapes(200 + m, 3)]
         + [(s, 14, "fft") for s in _shapes(314, 6)])


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[2]}-m{c[1]}-{'x'.join(map(str, c[0]))}")
def test_random_shapes(case):
    (N, C, K, H, W), m, algo = case
    x, w = workloads.random_inputs(N, C, K, H, W, seed=N * 7 + C * 11 + K * 13 + H * 17 + W * 19 + m)
    print(f"\n[gpu] random {algo} m={m} shape={(N, C, K, H, W)}", flush=True)
    y = run_gpu(x, w, m, algo).cpu().numpy()
    assert_close(y, direct_conv(x, w), m, f"{algo} F({m}) {(N, C, K, H, W)}")
