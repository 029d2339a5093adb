"""Pins for the direct-convolution oracle (oracle/direct_conv.c).

Eq. 1 of the paper read as a 3x3 cross-correlation with zero padding 1.  Pinned
against: a pure-Python brute force on tiny shapes; PyTorch's CPU conv2d in
float64 (a library routine computing the same cross-correlation); an impulse
input, which fixes correlation versus convolution and the pad offset; a
constant input; zero weights; linearity in x and in w.
"""

import numpy as np
import pytest
import torch

from oracle.direct import direct_conv, direct_conv_planes, num_threads


def brute_force(x, w):
    N, C, H, W = x.shape
    K = w.shape[0]
    y = np.zeros((N, K, H, W), dtype=np.float64)
    for n in range(N):
        for k in range(K):
            for h in range(H):
                for v in range(W):
                    acc = 0.0
                    for c in range(C):
                        for r in range(3):
                            for s in range(3):
                                hh, vv = h + r - 1, v + s - 1
                                if 0 <= hh < H and 0 <= vv < W:
                                    acc += float(x[n, c, hh, vv]) * float(w[k, c, r, s])
                    y[n, k, h, v] = acc
    return y


def rand(shape, seed):
    return np.random.default_rng(seed).uniform(-1, 1, size=shape).astype(np.float32)


TINY = [(1, 1, 1, 1, 1), (1, 1, 1, 2, 2), (2, 3, 2, 3, 3), (1, 2, 3, 5, 7),
        (2, 3, 3, 7, 5), (1, 1, 2, 1, 6), (1, 2, 1, 4, 1)]


@pytest.mark.parametrize("N,C,K,H,W", TINY)
def test_brute_force(N, C, K, H, W):
    x = rand((N, C, H, W), 1)
    w = rand((K, C, 3, 3), 2)
    np.testing.assert_allclose(direct_conv(x, w), brute_force(x, w), rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("N,C,K,H,W", [(2, 5, 4, 9, 11), (1, 64, 64, 56, 56), (3, 16, 8, 14, 14)])
def test_torch_conv2d_float64(N, C, K, H, W):
    x = rand((N, C, H, W), 3)
    w = rand((K, C, 3, 3), 4)
    ref = torch.nn.functional.conv2d(torch.from_numpy(x).double(), torch.from_numpy(w).double(),
                                     padding=1).numpy()
    np.testing.assert_allclose(direct_conv(x, w), ref, rtol=1e-12, atol=1e-11)


def test_impulse_fixes_correlation_and_pad():
    H, W = 6, 7
    w = rand((2, 1, 3, 3), 5)
    for h0, v0 in [(0, 0), (2, 3), (5, 6), (0, 6)]:
        x = np.zeros((1, 1, H, W), dtype=np.float32)
        x[0, 0, h0, v0] = 1.0
        y = direct_conv(x, w)
        expect = np.zeros((1, 2, H, W))
        for r in range(3):
            for s in range(3):
                h, v = h0 - r + 1, v0 - s + 1
                if 0 <= h < H and 0 <= v < W:
                    expect[0, :, h, v] = w[:, 0, r, s]
        np.testing.assert_array_equal(y, expect)


def test_constant_input():
    x = np.ones((1, 3, 5, 6), dtype=np.float32)
    w = rand((2, 3, 3, 3), 6)
    y = direct_conv(x, w)
    interior = w.astype(np.float64).sum(axis=(1, 2, 3))
    for k in range(2):
        np.testing.assert_allclose(y[0, k, 1:-1, 1:-1], interior[k], rtol=1e-14)
    # corner: only r, s in {1, 2} see the image
    np.testing.assert_allclose(y[0, :, 0, 0], w[:, :, 1:, 1:].astype(np.float64).sum(axis=(1, 2, 3)),
                               rtol=1e-14)


def test_zero_weights():
    x = rand((2, 3, 5, 5), 7)
    assert not direct_conv(x, np.zeros((4, 3, 3, 3), np.float32)).any()


def test_linearity():
    # Disjoint supports keep a*x1 + b*x2 exact in fp32, so the only difference
    # left is fp64 summation order.
    mask = np.random.default_rng(14).random((2, 4, 8, 9)) < 0.5
    x1 = np.where(mask, rand((2, 4, 8, 9), 8), 0).astype(np.float32)
    x2 = np.where(mask, 0, rand((2, 4, 8, 9), 9)).astype(np.float32)
    wmask = np.random.default_rng(15).random((3, 4, 3, 3)) < 0.5
    w1 = np.where(wmask, rand((3, 4, 3, 3), 10), 0).astype(np.float32)
    w2 = np.where(wmask, 0, rand((3, 4, 3, 3), 11)).astype(np.float32)
    a, b = np.float32(0.5), np.float32(-2.0)
    y = direct_conv(a * x1 + b * x2, w1)
    np.testing.assert_allclose(y, a * direct_conv(x1, w1) + b * direct_conv(x2, w1),
                               rtol=1e-12, atol=1e-12)
    y = direct_conv(x1, a * w1 + b * w2)
    np.testing.assert_allclose(y, a * direct_conv(x1, w1) + b * direct_conv(x1, w2),
                               rtol=1e-12, atol=1e-12)


def test_planes_match_full():
    x = rand((3, 5, 9, 8), 12)
    w = rand((4, 5, 3, 3), 13)
    full = direct_conv(x, w)
    planes = [(0, 0), (2, 3), (1, 2), (2, 0)]
    got = direct_conv_planes(x, w, planes)
    for i, (n, k) in enumerate(planes):
        np.testing.assert_array_equal(got[i], full[n, k])
    with pytest.raises(RuntimeError):
        direct_conv_planes(x, w, [(3, 0)])


def test_threads_reported():
    assert num_threads() >= 1
