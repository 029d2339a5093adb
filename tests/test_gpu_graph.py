"""A call captured in a HIP graph (torch.cuda.CUDAGraph) replays correctly: the
run path allocates nothing and issues no memset, and the split path's arrival
counters are left at zero by every call.  Each replay, with eager work and
synchronisations between replays, must equal the eager result bit for bit."""

import re

import pytest
import torch

import paper_1912_02165_amd as wc
from paper_1912_02165_amd import workloads

pytestmark = pytest.mark.gpu

CASES = [
    # (N, C, K, H, W, m, algo); the C=256 28x28 layer splits its last round of
    # items into channel pieces (partial outputs, arrival counters)
    ((1, 256, 256, 28, 28), 4, "fused"),
    ((1, 64, 64, 56, 56), 4, "fused"),
    ((1, 64, 64, 56, 56), 2, "fused"),
    ((2, 37, 45, 29, 35), 6, "fused"),
    ((2, 37, 45, 29, 35), 4, "three_stage"),
    ((2, 37, 45, 29, 35), 14, "fft"),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{'x'.join(map(str, c[0]))}-m{c[1]}-{c[2]}")
def test_graph_replay_matches_eager(case):
    (N, C, K, H, W), m, algo = case
    x, w = workloads.random_inputs(N, C, K, H, W, seed=31 + m)
    print(f"\n[gpu] graph replay {case}", flush=True)
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    with wc.Plan(N, C, K, H, W, m, algo) as p:
        if C == 256:
            assert re.search(r"split items [1-9]", p.describe()), p.describe()
        ref = torch.empty((N, K, H, W), device="cuda")
        p.run(xd, wd, ref)
        torch.cuda.synchronize()
        y = torch.full((N, K, H, W), float("nan"), device="cuda")
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):            # one eager call on the capture stream first
            p.run(xd, wd, y, s.cuda_stream)
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            p.run(xd, wd, y, s.cuda_stream)
        for i in range(3):
            y.fill_(float("nan"))
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(y, ref), f"replay {i} differs from the eager result"
            p.run(xd, wd, ref)                # eager work between replays
            torch.cuda.synchronize()
        del g
