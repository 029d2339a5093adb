"""Pins for the exact transform matrices (oracle/toom_cook.py).

What fixes them is mathematics, not the code: a Winograd F(m, 3) algorithm is
correct exactly when A^T[(G g) (.) (B^T d)] equals the valid correlation of d
with g, for every d and g (Eq. 3 in 1D); in 2D the same must hold for
A^T[(G g G^T) (.) (B^T d B)]A.  Both are checked over the rationals on basis
inputs, which covers every input by linearity.  Planted mistakes (a flipped sign,
a dropped entry, a transposed operand) must make the check fail.
"""

import itertools
import random
from fractions import Fraction

import pytest

from oracle import toom_cook

MS = toom_cook.SUPPORTED_M


def correlate_1d(d, g, m):
    return [sum(g[u] * d[i + u] for u in range(3)) for i in range(m)]


def winograd_1d(AT, G, BT, d, g):
    Gg = [sum(G[f][u] * g[u] for u in range(3)) for f in range(len(G))]
    Bd = [sum(BT[f][a] * d[a] for a in range(len(d))) for f in range(len(BT))]
    prod = [Gg[f] * Bd[f] for f in range(len(G))]
    return [sum(AT[i][f] * prod[f] for f in range(len(prod))) for i in range(len(AT))]


def identity_1d_holds(AT, G, BT, m):
    T = m + 2
    for a in range(T):
        for u in range(3):
            d = [Fraction(int(k == a)) for k in range(T)]
            g = [Fraction(int(k == u)) for k in range(3)]
            if winograd_1d(AT, G, BT, d, g) != correlate_1d(d, g, m):
                return False
    return True


def matmul(A, B):
    return [[sum(A[i][k] * B[k][j] for k in range(len(B))) for j in range(len(B[0]))]
            for i in range(len(A))]


def transpose(A):
    return [list(r) for r in zip(*A)]


def winograd_2d(AT, G, BT, d, g):
    Wt = matmul(matmul(G, g), transpose(G))
    U = matmul(matmul(BT, d), transpose(BT))
    Mm = [[Wt[i][j] * U[i][j] for j in range(len(U))] for i in range(len(U))]
    return matmul(matmul(AT, Mm), transpose(AT))


def correlate_2d(d, g, m):
    return [[sum(g[u][v] * d[i + u][j + v] for u in range(3) for v in range(3))
             for j in range(m)] for i in range(m)]


@pytest.mark.parametrize("m", MS)
def test_shapes(m):
    AT, G, BT = toom_cook.matrices(m)
    T = m + 2
    assert toom_cook.tile_edge(m) == T
    assert (len(AT), len(AT[0])) == (m, T)
    assert (len(G), len(G[0])) == (T, 3)
    assert (len(BT), len(BT[0])) == (T, T)


@pytest.mark.parametrize("m", MS)
def test_identity_1d_exact(m):
    AT, G, BT = toom_cook.matrices(m)
    assert identity_1d_holds(AT, G, BT, m)


@pytest.mark.parametrize("m", MS)
def test_identity_2d_exact_on_basis_pairs(m):
    AT, G, BT = toom_cook.matrices(m)
    T = m + 2
    pairs = list(itertools.product(range(T), range(T), range(3), range(3)))
    if m == 6:  # 576 exact 8x8 evaluations is slow in Fractions; sample a fixed third
        pairs = random.Random(6).sample(pairs, 192) + [(0, 0, 0, 0), (T - 1, T - 1, 2, 2)]
    for a, b, u, v in pairs:
        d = [[Fraction(int(i == a and j == b)) for j in range(T)] for i in range(T)]
        g = [[Fraction(int(i == u and j == v)) for j in range(3)] for i in range(3)]
        assert winograd_2d(AT, G, BT, d, g) == correlate_2d(d, g, m), (a, b, u, v)


@pytest.mark.parametrize("m", MS)
def test_identity_on_random_rationals(m):
    rng = random.Random(100 + m)
    AT, G, BT = toom_cook.matrices(m)
    T = m + 2
    d = [[Fraction(rng.randint(-9, 9), rng.randint(1, 5)) for _ in range(T)] for _ in range(T)]
    g = [[Fraction(rng.randint(-9, 9), rng.randint(1, 5)) for _ in range(3)] for _ in range(3)]
    assert winograd_2d(AT, G, BT, d, g) == correlate_2d(d, g, m)


def test_f2_tables_by_hand():
    """F(2,3) worked out by hand from the construction with points 0, 1, -1, inf."""
    AT, G, BT = toom_cook.matrices(2)
    h = Fraction(1, 2)
    assert AT == [[1, 1, 1, 0], [0, 1, -1, 1]]
    assert G == [[-1, 0, 0], [h, h, h], [h, -h, h], [0, 0, 1]]
    assert BT == [[-1, 0, 1, 0], [0, 1, 1, 0], [0, -1, 1, 0], [0, -1, 0, 1]]


def test_points_pair_structure():
    """Points come in +-p pairs (after 0 when 0 is a point: even T), so the B^T rows
    of a pair are the same polynomial at x and -x (coefficient i times (-1)^i, and
    negated once more when 0 is not a point: the row's degree is then odd), and A^T
    columns of a pair differ by (-1)^i (properties the GPU code may use)."""
    for m in MS:
        p = toom_cook.points(m)
        AT, _, BT = toom_cook.matrices(m)
        assert len(p) == m + 1
        j0 = 1 if p[0] == 0 else 0
        assert (j0 == 1) == (m % 2 == 0)
        assert 0 not in p[j0:]
        for j in range(j0, len(p), 2):
            assert p[j + 1] == -p[j]
            for i in range(m):
                assert AT[i][j + 1] == (AT[i][j] if i % 2 == 0 else -AT[i][j])
            sgn = 1 if j0 == 1 else -1
            for i, (a, b) in enumerate(zip(BT[j], BT[j + 1])):
                assert b == sgn * (a if i % 2 == 0 else -a)


def test_unsupported_m():
    with pytest.raises(ValueError):
        toom_cook.matrices(3)


# --- planted mistakes: the identity check must catch each of them ----------

def _mutations(m):
    AT, G, BT = toom_cook.matrices(m)
    out = []
    for name, mat in (("AT", AT), ("G", G), ("BT", BT)):
        nz = [(i, j) for i in range(len(mat)) for j in range(len(mat[0])) if mat[i][j] != 0]
        for i, j in nz[:: max(1, len(nz) // 6)]:
            flipped = [row[:] for row in mat]
            flipped[i][j] = -flipped[i][j]
            out.append((f"{name}[{i}][{j}] sign", name, flipped))
            dropped = [row[:] for row in mat]
            dropped[i][j] = 0
            out.append((f"{name}[{i}][{j}] dropped", name, dropped))
    # a transposed square operand
    out.append(("BT transposed", "BT", transpose(BT)))
    # two frequencies swapped in one matrix only
    sw = [row[:] for row in G]
    sw[1], sw[2] = sw[2], sw[1]
    out.append(("G rows 1,2 swapped", "G", sw))
    return AT, G, BT, out


@pytest.mark.parametrize("m", MS)
def test_planted_mistakes_are_caught(m):
    AT, G, BT, muts = _mutations(m)
    assert muts
    for label, name, mat in muts:
        mats = {"AT": AT, "G": G, "BT": BT}
        mats[name] = mat
        assert not identity_1d_holds(mats["AT"], mats["G"], mats["BT"], m), label
