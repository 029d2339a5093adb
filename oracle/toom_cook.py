"""Exact Winograd / Toom-Cook transform matrices for F(m x m, 3 x 3).  Oracle code.

The paper writes the 2D transformed convolution as (Sec. 2.1, Eq. 3)

    I'_{b,c'} = A [ sum_c (G W_{c,c'} G^T) (.) (B I_{b,c} B^T) ] A^T

with A, B, G "transform matrices" that it does not print (it cites Lavin and
Gray).  Here they are built from first principles, the Toom-Cook way, and
returned as exact ``fractions.Fraction`` matrices.  In this package's naming
(Lavin-Gray form) the paper's A is ``AT`` (m x T), its B is ``BT`` (T x T) and
its G is ``G`` (T x 3), with T = m + 2 the input tile edge and m = T - K + 1 the
output tile edge of the overlap-add tiling (Sec. 2.1).

Construction (a reading: the paper is silent on it).  Pick
T - 1 distinct finite interpolation points p_j and the point at infinity.  The
1D correlation y_i = sum_{u<3} g_u d_{i+u} (i < m) is the transpose of the
polynomial product a(x) g(x) with deg a = m - 1, so with

    Eval_a[j][i] = p_j^i            (the infinity row is [i == m - 1])
    Eval_g[j][u] = p_j^u            (the infinity row is [u == 2])
    L_j(x)       = prod_{l != j} (x - p_l) / prod_{l != j} (p_j - p_l)

the product is c = Interp (Eval_g g (.) Eval_a a) where column j of Interp holds
the ascending coefficients of L_j and the infinity column those of
prod_l (x - p_l).  Transposing gives y = Eval_a^T [ (Eval_g g) (.) (Interp^T d) ].
The divisor of L_j is moved from Interp^T to row j of Eval_g, so

    AT[i][j] = p_j^i,                         AT[i][inf] = [i == m - 1]
    G[j][u]  = p_j^u / prod_{l != j}(p_j - p_l), G[inf][u] = [u == 2]
    BT[j][:] = coefficients of prod_{l != j}(x - p_l), BT[inf][:] = those of prod_l (x - p_l)

Point sets (in frequency order; infinity is always last):
    F(2,3): 0, 1, -1
    F(4,3): 0, 1, -1, 2, -2
    F(5,3): 1, -1, 2, -2, 1/2, -1/2     (the paper's T = 7 tile, Sec. 6; the paper
                                         gives no points: six finite points in +-p
                                         pairs, without 0, so that every point
                                         but infinity has its mirror)
    F(6,3): 0, 1, -1, 2, -2, 1/2, -1/2
    F(7,3): 1, -1, 2, -2, 1/2, -1/2, 1/4, -1/4
                                        (T = 9: eight finite points in +-p pairs,
                                         as for F(5); of the natural next pairs
                                         +-3, +-3/2 and +-1/4, the last keeps the
                                         fp32 error lowest, ~4e-5 relative L2)
"""

from fractions import Fraction

R = 3  # kernel edge: the paper's K for 3x3 kernels

_POINTS = {
    2: (Fraction(0), Fraction(1), Fraction(-1)),
    4: (Fraction(0), Fraction(1), Fraction(-1), Fraction(2), Fraction(-2)),
    5: (Fraction(1), Fraction(-1), Fraction(2), Fraction(-2), Fraction(1, 2), Fraction(-1, 2)),
    6: (Fraction(0), Fraction(1), Fraction(-1), Fraction(2), Fraction(-2),
        Fraction(1, 2), Fraction(-1, 2)),
    7: (Fraction(1), Fraction(-1), Fraction(2), Fraction(-2), Fraction(1, 2), Fraction(-1, 2),
        Fraction(1, 4), Fraction(-1, 4)),
}

SUPPORTED_M = tuple(sorted(_POINTS))


def points(m):
    """Finite interpolation points for F(m, 3), in frequency order."""
    if m not in _POINTS:
        raise ValueError(f"F({m},3) is not supported; m must be one of {SUPPORTED_M}")
    return _POINTS[m]


def tile_edge(m):
    """Input tile edge T = m + K - 1 of the overlap-add tiling (Sec. 2.1)."""
    return m + R - 1


def _poly_from_roots(roots, length):
    """Ascending coefficients of prod (x - r) over ``roots``, zero-padded to ``length``."""
    coef = [Fraction(1)]
    for r in roots:
        nxt = [Fraction(0)] * (len(coef) + 1)
        for i, a in enumerate(coef):
            nxt[i + 1] += a       # a * x
            nxt[i] -= a * r       # a * (-r)
        coef = nxt
    return coef + [Fraction(0)] * (length - len(coef))


def matrices(m):
    """Return (AT, G, BT) for F(m x m, 3 x 3) as lists of lists of Fractions.

    AT is m x T, G is T x 3, BT is T x T (T = m + 2).
    """
    p = points(m)
    T = tile_edge(m)
    assert len(p) == T - 1

    AT = [[pj ** i for pj in p] + [Fraction(1 if i == m - 1 else 0)] for i in range(m)]

    G = []
    for j, pj in enumerate(p):
        denom = Fraction(1)
        for l, pl in enumerate(p):
            if l != j:
                denom *= (pj - pl)
        G.append([pj ** u / denom for u in range(R)])
    G.append([Fraction(1 if u == R - 1 else 0) for u in range(R)])

    BT = []
    for j in range(len(p)):
        BT.append(_poly_from_roots([pl for l, pl in enumerate(p) if l != j], T))
    BT.append(_poly_from_roots(list(p), T))

    return AT, G, BT


def matrices_f64(m):
    """The same matrices as float64 NumPy arrays (for the fp64 oracle)."""
    import numpy as np
    AT, G, BT = matrices(m)
    conv = lambda A: np.array([[float(v) for v in row] for row in A], dtype=np.float64)
    return conv(AT), conv(G), conv(BT)
