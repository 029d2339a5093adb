"""GPU parity of the FFT-tile algorithm (16 x 16 tiles, 14 x 14 outputs) against
the fp64 oracles: the direct convolution for y, the oracle's kernel spectra for
the transformed kernels the plan holds.  Inputs are the seeded synthetic layers
and random small shapes; shapes cover one-pixel images, ragged edge tiles, input
channels that leave a partial step of 4, output channels that leave a partial
block of 16, and tile counts that leave a partial group of 16."""

import numpy as np
import pytest
import torch

import paper_1912_02165_amd as wc
from paper_1912_02165_amd import workloads
from oracle.direct import direct_conv, direct_conv_planes
from oracle.fft_conv import kernel_spectrum
from parity import assert_close

pytestmark = pytest.mark.gpu

M = 14
SMALL = [(1, 1, 1, 1, 1), (1, 2, 3, 2, 5), (1, 3, 5, 7, 9), (2, 4, 16, 14, 14), (1, 5, 17, 15, 30),
         (3, 8, 20, 17, 23), (2, 37, 45, 29, 35), (1, 64, 64, 20, 20), (4, 12, 40, 6, 6),
         (1, 130, 18, 9, 10), (5, 9, 33, 28, 15)]


def run_fft(x, w):
    N, C, H, W = x.shape
    K = w.shape[0]
    y = torch.full((N, K, H, W), float("nan"), dtype=torch.float32, device="cuda")
    with wc.Plan(N, C, K, H, W, M, "fft") as p:
        p.run(torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda(), y)
        torch.cuda.synchronize()
    return y


@pytest.mark.parametrize("shape", SMALL, ids=lambda s: "x".join(map(str, s)))
def test_fft_small_shapes(shape):
    N, C, K, H, W = shape
    x, w = workloads.random_inputs(N, C, K, H, W, seed=sum(shape) + 14)
    print(f"\n[gpu] fft shape={shape}", flush=True)
    y = run_fft(x, w).cpu().numpy()
    rel, mx = assert_close(y, direct_conv(x, w), M, f"FFT {shape}")
    print(f"rel_l2={rel:.3e} max={mx:.3e}")


def test_fft_kernel_spectra():
    """The plan's transformed kernels are the oracle's spectra of the zero-padded
    kernels, as {Re, Im, -Im, 0} in matrix-core operand order, zero for padding
    channels."""
    N, C, K, H, W = 1, 6, 20, 16, 16
    x, w = workloads.random_inputs(N, C, K, H, W, seed=21)
    print("\n[gpu] fft kernel spectra", flush=True)
    with wc.Plan(N, C, K, H, W, M, "fft") as p:
        p.set_weights(torch.from_numpy(w).cuda())
        torch.cuda.synchronize()
        dims = wc.wino_conv_intermediate_dims(p.handle, wc.WINO_BUF_WEIGHTS)
        Cs, Kb = (C + 3) // 4, (K + 15) // 16
        assert tuple(dims) == (Cs, Kb, 144, 256)
        got = p.intermediate(wc.WINO_BUF_WEIGHTS).reshape(Cs, Kb, 144, 4, 16, 4)  # lane = c4 * 16 + k16
    ref = kernel_spectrum(w, 16).reshape(K, C, 144)                               # f = p * 9 + q
    full = np.zeros((Cs * 4, Kb * 16, 144), dtype=np.complex128)
    full[:C, :K] = ref.transpose(1, 0, 2)
    want = full.reshape(Cs, 4, Kb, 16, 144).transpose(0, 2, 4, 1, 3)              # [cs][kb][f][c4][k16]
    scale = np.abs(ref).max()
    assert np.abs(got[..., 0] - want.real).max() <= 1e-5 * scale
    assert np.abs(got[..., 1] - want.imag).max() <= 1e-5 * scale
    assert np.array_equal(got[..., 2], -got[..., 1])
    assert not got[..., 3].any()


def sample_planes(N, K, seed, count=8):
    rng = np.random.default_rng(seed)
    planes = {(0, 0), (N - 1, K - 1), (N // 2, K // 3), (min(1, N - 1), K - 1), (N - 1, 0)}
    while len(planes) < count:
        planes.add((int(rng.integers(N)), int(rng.integers(K))))
    return sorted(planes)


@pytest.mark.parametrize("lid", [1, 2, 3, 4, 5])
def test_fft_full_layers_sampled(lid):
    layer = workloads.LAYER_BY_ID[lid]
    x, w = workloads.layer_inputs(layer)
    label = f"{layer.name}/FFT 16x16 tiles"
    print(f"\n[gpu] {label} full size", flush=True)
    y = run_fft(x, w)
    assert bool(torch.isfinite(y).all()), "non-finite output"
    planes = sample_planes(layer.N, layer.K, seed=layer.id * 10 + M)
    n_idx = torch.tensor([p[0] for p in planes], device="cuda")
    k_idx = torch.tensor([p[1] for p in planes], device="cuda")
    got = y[n_idx, k_idx].cpu().numpy()
    rel, mx = assert_close(got, direct_conv_planes(x, w, planes), M, f"{label} planes {planes}")
    print(f"rel_l2={rel:.3e} max={mx:.3e} over {len(planes)} planes")


def test_fft_reproducible_and_pretransformed():
    N, C, K, H, W = 2, 24, 40, 31, 27
    x, w = workloads.random_inputs(N, C, K, H, W, seed=22)
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    ys = [torch.full((N, K, H, W), float("nan"), device="cuda") for _ in range(3)]
    with wc.Plan(N, C, K, H, W, M, "fft") as p:
        p.run(xd, wd, ys[0])
        p.run(xd, wd, ys[1])
        p.set_weights(wd)
        p.run_pretransformed(xd, ys[2])
        torch.cuda.synchronize()
    assert torch.equal(ys[0], ys[1]) and torch.equal(ys[0], ys[2])
    assert_close(ys[0].cpu().numpy(), direct_conv(x, w), M, "fft repeated")
