"""A seeded sweep of 300 small random problems over every algorithm, tile size
and built fused blocking, some with channel splitting, against the fp64 direct
oracle: channel counts around and across the 4-channel steps, 16-channel stages
and the 8-stage split pieces (up to 300), output channels around the 16-channel
blocks, image sides 1-60, batches 1-5.  A second call on the same plan must
reproduce the first bit for bit, and the status word must stay clear.  The cases
are fixed by the seed, so a failure names its case."""

import numpy as np
import pytest
import torch

import paper_1912_02165_amd as wc
from paper_1912_02165_amd import workloads
from oracle.direct import direct_conv
from parity import assert_close

pytestmark = pytest.mark.gpu

# the blockings the fused kernel is built for, as in include/wino_conv.h
BLOCKINGS = {2: [(32, 64), (16, 64), (32, 32), (16, 32), (16, 16)], 4: [(16, 64), (16, 32)],
             5: [(16, 32), (16, 16)], 6: [(16, 32), (16, 16)]}


def _cases(seed=2024, count=300):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(count):
        m = int(rng.choice([2, 4, 5, 6, 7, 14]))
        algo = "fft" if m == 14 else ("three_stage" if m == 7 else str(rng.choice(["fused", "fused", "three_stage"])))
        N = int(rng.integers(1, 6))
        C = int(rng.choice([1, 2, 3, 4, 7, 8, 15, 16, 17, 33, 48, 63, 64, 96, 128, 129, 250, 256, 300]))
        K = int(rng.choice([1, 2, 5, 16, 17, 31, 32, 48, 64, 65, 100, 128, 160, 256, 300]))
        H, W = int(rng.integers(1, 61)), int(rng.integers(1, 61))
        while N * C * K * H * W * 18 > 4e8 and (H > 1 or W > 1):
            H, W = max(1, H // 2), max(1, W // 2)
        tuning = None
        if algo == "fused":
            r = rng.random()
            if r < 0.4:
                R, kit = BLOCKINGS[m][int(rng.integers(0, len(BLOCKINGS[m])))]
                tuning = {"tiles_per_wg": R, "k_per_wg": kit}
            elif r < 0.55 and C >= 32:
                tuning = {"channel_splits": int(rng.integers(2, 5))}
        out.append((i, (N, C, K, H, W), m, algo, tuning))
    return out


def _id(c):
    i, s, m, algo, t = c
    extra = "" if t is None else "-" + "-".join(f"{k[0]}{v}" for k, v in t.items())
    return f"{i}-{algo}-m{m}-{'x'.join(map(str, s))}{extra}"


def test_blockings_table_matches_the_library():
    built = {}
    for m, R, kit in wc.wino_fused_blockings():
        built.setdefault(m, []).append((R, kit))
    assert {m: sorted(v) for m, v in built.items()} == {m: sorted(v) for m, v in BLOCKINGS.items()}


@pytest.mark.parametrize("case", _cases(), ids=_id)
def test_sweep(case):
    i, (N, C, K, H, W), m, algo, tuning = case
    print(f"\n[gpu] sweep {_id(case)}", flush=True)
    x, w = workloads.random_inputs(N, C, K, H, W, seed=5000 + i)
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y1 = torch.full((N, K, H, W), float("nan"), device="cuda")
    y2 = torch.full_like(y1, float("nan"))
    with wc.Plan(N, C, K, H, W, m, algo, tuning) as p:
        p.run(xd, wd, y1)
        p.status()
        p.run(xd, wd, y2)
        p.status()
    assert torch.equal(y1, y2), "a second call differs"
    assert_close(y1.cpu().numpy(), direct_conv(x, w), m, _id(case))
