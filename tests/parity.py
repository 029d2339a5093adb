"""Shared helpers of the GPU parity tests: tolerances and error measures.

Tolerances (relative L2 error over the compared outputs, and the largest
element error normalised by the largest reference magnitude):
    F(2x2,3x3): rel_l2 <= 1e-5;  F(4x4,3x3), F(6x6,3x3): rel_l2 <= 1e-4;
    F(5x5,3x3) (not among the stated tolerances; its tile lies between F(4) and
    F(6), so it takes theirs): rel_l2 <= 1e-4;
    F(7x7,3x3) (three-stage only; not among the stated tolerances): its transforms
    on the points +-1, +-2, +-1/2, +-1/4 are less well conditioned, about 4e-5
    relative L2 in fp32 over random tiles, so it takes F(4)-F(6)'s rel_l2 <= 1e-4;
    FFT tiles (16 x 16, m = 14; not among the stated tolerances): rel_l2 <= 1e-5.
    The error of an fp32 radix-2 FFT grows with the number of butterfly levels,
    about eps * log2(n) relative: 8 levels forward and 8 inverse on 16 x 16
    tiles give ~1e-6 (eps = 6e-8), a tenth of the bound, to which the products
    add the usual fp32 sum over 9C terms;
    all: max|y - y_ref| / max|y_ref| <= 1e-3.
The reference is the fp64 oracle; the GPU computes in fp32.
"""

import numpy as np

REL_L2 = {2: 1e-5, 4: 1e-4, 5: 1e-4, 6: 1e-4, 7: 1e-4, 14: 1e-5}
MAX_ERR = 1e-3


def errors(y, ref):
    y = np.asarray(y, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert y.shape == ref.shape, (y.shape, ref.shape)
    diff = y - ref
    nref = np.linalg.norm(ref)
    rel = np.linalg.norm(diff) / nref if nref > 0 else np.linalg.norm(diff)
    mref = np.abs(ref).max() if ref.size else 0.0
    mx = np.abs(diff).max() / mref if mref > 0 else (np.abs(diff).max() if diff.size else 0.0)
    return float(rel), float(mx)


def assert_close(y, ref, m, label=""):
    assert np.isfinite(y).all(), f"{label}: non-finite outputs"
    rel, mx = errors(y, ref)
    assert rel <= REL_L2[m] and mx <= MAX_ERR, (
        f"{label}: rel_l2={rel:.3e} (tol {REL_L2[m]:.0e}), max_err/max|y|={mx:.3e} (tol {MAX_ERR:.0e})")
    return rel, mx
