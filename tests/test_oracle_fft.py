"""Pins for the fp64 CPU FFT-tile convolution (oracle/fft_conv.py).

The tile spectra are checked against closed forms (impulse, constant tile) and
against numpy's FFT (a library routine); the convolution against the direct
oracle (itself pinned to PyTorch and a brute force) to fp64 rounding, at the
16-point tiles the GPU path uses and at other even tile edges, on images
smaller than one tile and with ragged edge tiles.  A kernel spectrum used
without its complex conjugate computes a convolution with the flipped kernel,
which the random, non-symmetric kernels here tell apart.
"""

import numpy as np
import pytest

from oracle import fft_conv
from oracle.direct import direct_conv

SHAPES = [(1, 1, 1, 1, 1), (1, 2, 3, 2, 2), (2, 3, 2, 15, 15), (1, 4, 5, 14, 14),
          (1, 3, 4, 29, 6), (2, 2, 3, 17, 31), (1, 2, 2, 1, 33)]


def rand(shape, seed):
    return np.random.default_rng(seed).uniform(-1, 1, size=shape).astype(np.float32)


@pytest.mark.parametrize("T", (16, 8, 6))
def test_spectrum_of_impulses_and_constants(T):
    """An impulse at (a, b) has spectrum exp(-2 pi i (p a + q b) / T); a constant
    tile of value v has T^2 v at frequency (0, 0) and zero elsewhere."""
    p = np.arange(T)[:, None]
    q = np.arange(T // 2 + 1)[None, :]
    for a, b in ((0, 0), (1, 3), (T - 1, 2)):
        d = np.zeros((T, T))
        d[a, b] = 1.0
        want = np.exp(-2j * np.pi * (p * a + q * b) / T)
        np.testing.assert_allclose(fft_conv.tile_spectrum(d), want, atol=1e-12)
    D = fft_conv.tile_spectrum(np.full((T, T), 0.75))
    want = np.zeros((T, T // 2 + 1), dtype=complex)
    want[0, 0] = 0.75 * T * T
    np.testing.assert_allclose(D, want, atol=1e-12)


@pytest.mark.parametrize("T", (16, 8))
def test_spectrum_matches_numpy_fft(T):
    d = rand((3, T, T), 5).astype(np.float64)
    np.testing.assert_allclose(fft_conv.tile_spectrum(d), np.fft.rfft2(d), atol=1e-11)
    full = fft_conv.full_from_half(fft_conv.tile_spectrum(d), T)
    np.testing.assert_allclose(full, np.fft.fft2(d), atol=1e-11)


def test_inverse_is_numpy_irfft():
    T = 16
    Z = np.fft.rfft2(rand((2, T, T), 6).astype(np.float64))
    np.testing.assert_allclose(fft_conv.inverse_tile(Z, T), np.fft.irfft2(Z, s=(T, T)), atol=1e-12)


def test_kernel_spectrum_layout():
    """Wp[k, c] is the spectrum of w[k, c] padded with zeros at the high indices."""
    w = rand((2, 3, 3, 3), 7).astype(np.float64)
    T = 16
    padded = np.zeros((2, 3, T, T))
    padded[:, :, :3, :3] = w
    np.testing.assert_allclose(fft_conv.kernel_spectrum(w, T), np.fft.rfft2(padded), atol=1e-12)


@pytest.mark.parametrize("T", (16, 8, 6))
@pytest.mark.parametrize("N,C,K,H,W", SHAPES)
def test_matches_direct(T, N, C, K, H, W):
    x = rand((N, C, H, W), 20 + H)
    w = rand((K, C, 3, 3), 30 + W)
    y = fft_conv.fft_conv(x, w, T)
    ref = direct_conv(x, w)
    scale = max(1.0, np.abs(ref).max())
    assert y.shape == ref.shape
    assert np.abs(y - ref).max() <= 1e-12 * scale * (1 + C)


def test_conjugate_decides_the_orientation():
    """Without the conjugate the kernel acts flipped (a convolution, not the
    correlation of Eq. 1): the result is far from the direct oracle's."""
    x = rand((1, 2, 14, 14), 8)
    w = rand((3, 2, 3, 3), 9)
    T, m = 16, 14
    xp = np.zeros((1, 2, T, T))
    xp[:, :, 1:15, 1:15] = x
    Dh = fft_conv.tile_spectrum(xp)
    Wh = fft_conv.kernel_spectrum(w, T)
    wrong = fft_conv.inverse_tile(np.einsum("ncpq,kcpq->nkpq", Dh, Wh), T)[:, :, :m, :m]
    ref = direct_conv(x, w)
    assert np.abs(wrong - ref).max() > 0.1 * np.abs(ref).max()
