"""fp64 CPU FFT-tile convolution, 3 x 3 kernels, pad 1.  Oracle code (test
infrastructure only: imported by tests/, never by the library).

The paper's transformed convolutions (Sec. 2.1, Sec. 4) take either Winograd or
FFT transforms; for FFT it names tiles of at least 16 (Sec. 4) and notes that the
spectra of real tiles are conjugate symmetric, so about half of each is stored
and multiplied (Sec. 2.1).  This module computes that method plainly:

* Overlap-add tiling (Sec. 2.1): input tiles of edge T overlapping by K - 1 = 2,
  output tiles of edge T - 2.  With pad 1 the tile at (ty, tx) reads input rows
  ty*(T-2) - 1 .. ty*(T-2) + T - 2 (likewise columns), zero outside the image.
* Transform: the 2-D discrete Fourier transform of each T x T tile,
  D[p, q] = sum_{i,j} d[i, j] exp(-2 pi i (p i + q j) / T), written out from its
  definition as a product with the T x T DFT matrix; only q = 0 .. T/2 is kept
  (the rest is the complex conjugate of a kept value).
* Kernels: the 3 x 3 kernel zero-padded to T x T, transformed the same way.
* Per frequency: Z[p, q, k] = sum_c D[p, q, c] conj(Wp[p, q, k, c]) -- the
  convolution theorem for the cross-correlation of Eq. 1, which is circular on
  a T x T tile and agrees with the linear one on the first T - 2 rows and
  columns, the output tile.
* Inverse: z = (1/T^2) sum_{p,q} Z[p, q] exp(+2 pi i (p i + q j) / T) over the
  full spectrum (the dropped half restored by conjugate symmetry); the output
  tile is z[0:T-2, 0:T-2], clipped at the image edge.
"""

import numpy as np


def dft_matrix(T, sign=-1):
    """F[a, b] = exp(sign * 2 pi i a b / T), from the definition."""
    a = np.arange(T)
    return np.exp(sign * 2j * np.pi * np.outer(a, a) / T)


def tile_spectrum(d):
    """Half spectrum of real T x T tiles d[..., T, T]: D[..., p, q], q <= T/2."""
    d = np.asarray(d, dtype=np.float64)
    T = d.shape[-1]
    F = dft_matrix(T)
    full = np.einsum("pi,...ij,qj->...pq", F, d, F)
    return full[..., : T // 2 + 1]


def full_from_half(Dh, T):
    """Restore the full spectrum from the kept half: D[p, q] = conj(D[-p, -q])."""
    Dh = np.asarray(Dh)
    full = np.zeros(Dh.shape[:-1] + (T,), dtype=np.complex128)
    full[..., : T // 2 + 1] = Dh
    p = np.arange(T)
    for q in range(T // 2 + 1, T):
        full[..., :, q] = np.conj(Dh[..., (-p) % T, T - q])
    return full


def inverse_tile(Zh, T):
    """Real T x T tiles from half spectra Zh[..., p, q] (q <= T/2)."""
    full = full_from_half(Zh, T)
    G = dft_matrix(T, sign=+1)
    z = np.einsum("ip,...pq,jq->...ij", G, full, G) / (T * T)
    return z.real


def kernel_spectrum(w, T):
    """Half spectra of the kernels zero-padded to T x T: Wp[k, c, p, q]."""
    w = np.asarray(w, dtype=np.float64)
    K, C, R, S = w.shape
    wp = np.zeros((K, C, T, T), dtype=np.float64)
    wp[:, :, :R, :S] = w
    return tile_spectrum(wp)


def fft_conv(x, w, T=16):
    """y[n, k] = FFT-tile convolution of x (N, C, H, W) with w (K, C, 3, 3), pad 1."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    N, C, H, W = x.shape
    K = w.shape[0]
    m = T - 2
    TH, TW = -(-H // m), -(-W // m)
    xp = np.zeros((N, C, TH * m + 2, TW * m + 2), dtype=np.float64)
    xp[:, :, 1:H + 1, 1:W + 1] = x
    Wh = kernel_spectrum(w, T)                            # (K, C, T, T/2+1)
    y = np.zeros((N, K, TH * m, TW * m), dtype=np.float64)
    for ty in range(TH):
        for tx in range(TW):
            d = xp[:, :, ty * m:ty * m + T, tx * m:tx * m + T]   # (N, C, T, T)
            Dh = tile_spectrum(d)                                 # (N, C, T, T/2+1)
            Zh = np.einsum("ncpq,kcpq->nkpq", Dh, np.conj(Wh))
            z = inverse_tile(Zh, T)                               # (N, K, T, T)
            y[:, :, ty * m:(ty + 1) * m, tx * m:(tx + 1) * m] = z[:, :, :m, :m]
    return y[:, :, :H, :W]
