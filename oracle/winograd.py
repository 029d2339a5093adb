"""fp64 CPU Winograd F(m x m, 3 x 3) convolution, pad 1.  Oracle code.

This is the second, test-only oracle.  It follows the paper's formulation step
by step so that each GPU stage can be compared with its counterpart:

* Eq. 3 (Sec. 2.1): I' = A [ sum_c (G W G^T) (.) (B I B^T) ] A^T, with the
  transform matrices of ``toom_cook`` (``AT``, ``G``, ``BT`` in Lavin-Gray form).
* Overlap-add tiling (Sec. 2.1): input tiles of edge T = m + 2 overlapping by
  K - 1 = 2, output tiles of edge m.  With pad 1 the tile at (ty, tx) reads
  input rows ty*m - 1 .. ty*m + T - 2 and columns tx*m - 1 .. tx*m + T - 2, zero
  outside the image; the number of tiles is N * ceil(H/m) * ceil(W/m) (the
  paper's tile count divides by T, which must be T' = m here).  Output tiles
  that run past H or W are clipped.
* The three steps of Sec. 3: (1) transform every input tile into T^2 values,
  read as T^2 vectors over the C channels; (2) multiply vector f by the C x C'
  kernel matrix of frequency f, obtained ahead of time by transforming the
  kernels; (3) inverse-transform the C' resulting tiles.

Layouts of the intermediates (frequency f = i*T + j for transform-domain row i
and column j; tile t = (n*TH + ty)*TW + tx):
    weight_transform -> Wt[f, c, k]
    input_transform  -> U[f, c, t]
    frequency_gemm   -> Mf[f, k, t] = sum_c Wt[f, c, k] U[f, c, t]
    output_transform -> y[n, k, h, w]
"""

import numpy as np

from .toom_cook import matrices_f64, tile_edge


def tile_counts(H, W, m):
    """Tiles per column and per row: ceil(H/m), ceil(W/m)."""
    return -(-H // m), -(-W // m)


def weight_transform(w, m):
    """Wt[f, c, k] = (G w[k, c] G^T)[f] for every kernel (Sec. 3, step 2's right-hand matrices)."""
    _, G, _ = matrices_f64(m)
    T = tile_edge(m)
    w = np.asarray(w, dtype=np.float64)
    K, C = w.shape[:2]
    wt = np.einsum("iu,kcuv,jv->ijck", G, w, G)        # (T, T, C, K)
    return wt.reshape(T * T, C, K)


def input_tiles(x, m):
    """d[n, c, ty, tx, a, b] = x[n, c, ty*m - 1 + a, tx*m - 1 + b], zero outside the image."""
    x = np.asarray(x, dtype=np.float64)
    N, C, H, W = x.shape
    T = tile_edge(m)
    TH, TW = tile_counts(H, W, m)
    xp = np.zeros((N, C, TH * m + 2, TW * m + 2), dtype=np.float64)
    xp[:, :, 1:H + 1, 1:W + 1] = x
    d = np.empty((N, C, TH, TW, T, T), dtype=np.float64)
    for ty in range(TH):
        for tx in range(TW):
            d[:, :, ty, tx] = xp[:, :, ty * m:ty * m + T, tx * m:tx * m + T]
    return d


def input_transform(x, m):
    """U[f, c, t] = (B^T d B)[f] for the input tile d of tile t, channel c (Sec. 3, step 1)."""
    _, _, BT = matrices_f64(m)
    T = tile_edge(m)
    d = input_tiles(x, m)                                # (N, C, TH, TW, T, T)
    N, C, TH, TW = d.shape[:4]
    u = np.einsum("ia,nchwab,jb->ijcnhw", BT, d, BT)     # (T, T, C, N, TH, TW)
    return u.reshape(T * T, C, N * TH * TW)


def frequency_gemm(U, Wt):
    """Mf[f] = Wt[f]^T U[f]: the T^2 per-frequency products over channels (Sec. 3, step 2)."""
    return np.matmul(np.transpose(Wt, (0, 2, 1)), U)    # (T^2, K, Ntile)


def output_transform(Mf, m, N, K, H, W):
    """y tile = A^T Mf[:, k, t] A, reshaped T x T, clipped to H x W (Sec. 3, step 3)."""
    AT, _, _ = matrices_f64(m)
    T = tile_edge(m)
    TH, TW = tile_counts(H, W, m)
    Mt = Mf.reshape(T, T, K, N, TH, TW)
    yt = np.einsum("ia,abknhw,jb->nkhiwj", AT, Mt, AT)   # (N, K, TH, m, TW, m)
    y = yt.reshape(N, K, TH * m, TW * m)
    return np.ascontiguousarray(y[:, :, :H, :W])


def winograd_conv(x, w, m):
    """Full Winograd F(m x m, 3 x 3) convolution, pad 1, computed in fp64 (Eq. 3 + OLA)."""
    x = np.asarray(x)
    N, C, H, W = x.shape
    K = w.shape[0]
    Wt = weight_transform(w, m)
    U = input_transform(x, m)
    Mf = frequency_gemm(U, Wt)
    return output_transform(Mf, m, N, K, H, W)
