"""Pins for the fp64 CPU Winograd (oracle/winograd.py).

It must reproduce the direct convolution (itself pinned to PyTorch and a brute
force) to fp64 rounding for every supported m, including images smaller than
one tile and sizes that leave ragged edge tiles.  Each intermediate is also
checked against its definition on single tiles.
"""

import numpy as np
import pytest

from oracle import toom_cook, winograd
from oracle.direct import direct_conv

SHAPES = [(1, 1, 1, 1, 1), (1, 2, 3, 2, 2), (2, 3, 2, 5, 7), (1, 4, 5, 9, 11),
          (2, 5, 3, 14, 14), (1, 3, 4, 13, 6), (1, 2, 2, 1, 17)]


def rand(shape, seed):
    return np.random.default_rng(seed).uniform(-1, 1, size=shape).astype(np.float32)


@pytest.mark.parametrize("m", toom_cook.SUPPORTED_M)
@pytest.mark.parametrize("N,C,K,H,W", SHAPES)
def test_matches_direct(m, N, C, K, H, W):
    x = rand((N, C, H, W), 20 + H)
    w = rand((K, C, 3, 3), 30 + W)
    y = winograd.winograd_conv(x, w, m)
    ref = direct_conv(x, w)
    scale = max(1.0, np.abs(ref).max())
    assert y.shape == ref.shape
    assert np.abs(y - ref).max() <= 1e-12 * scale * (1 + C)


def test_tile_counts():
    assert winograd.tile_counts(56, 56, 4) == (14, 14)
    assert winograd.tile_counts(112, 112, 6) == (19, 19)
    assert winograd.tile_counts(14, 14, 6) == (3, 3)
    assert winograd.tile_counts(1, 5, 2) == (1, 3)


@pytest.mark.parametrize("m", toom_cook.SUPPORTED_M)
def test_intermediates_on_one_tile(m):
    AT, G, BT = toom_cook.matrices_f64(m)
    T = m + 2
    x = rand((1, 2, 2 * m + 1, 3 * m + 1), 40)
    w = rand((3, 2, 3, 3), 41)
    N, C, H, W = x.shape
    TH, TW = winograd.tile_counts(H, W, m)
    d = winograd.input_tiles(x, m)
    # tile (ty, tx) = (1, 2) of channel 1 reads rows m-1.., columns 2m-1.. with zero fill
    xp = np.pad(x.astype(np.float64), ((0, 0), (0, 0), (1, T), (1, T)))
    np.testing.assert_array_equal(d[0, 1, 1, 2], xp[0, 1, m:m + T, 2 * m:2 * m + T])
    U = winograd.input_transform(x, m)
    t = 1 * TW + 2
    np.testing.assert_allclose(U[:, 1, t].reshape(T, T), BT @ d[0, 1, 1, 2] @ BT.T, rtol=1e-14,
                               atol=1e-14)
    Wt = winograd.weight_transform(w, m)
    np.testing.assert_allclose(Wt[:, 1, 2].reshape(T, T), G @ w[2, 1].astype(np.float64) @ G.T,
                               rtol=1e-14, atol=1e-14)
    Mf = winograd.frequency_gemm(U, Wt)
    np.testing.assert_allclose(Mf[:, 2, t], (Wt[:, :, 2] * U[:, :, t]).sum(axis=1), rtol=1e-13,
                               atol=1e-13)
    y = winograd.output_transform(Mf, m, N, 3, H, W)
    np.testing.assert_allclose(y[0, 2, m:2 * m, 2 * m:3 * m], AT @ Mf[:, 2, t].reshape(T, T) @ AT.T,
                               rtol=1e-13, atol=1e-13)
