"""Shared buffer of the L3-fused task (Sec. 4.2, Fig. 1).  Oracle code.

A task holds n = T^2 left-hand matrices (R x C, S_left bytes each) and produces
n result matrices (R x C', S_res bytes each).  Stored separately they need
n * (S_left + S_res).  The paper's shared buffer stores the left-hand matrices
back to back at the end of one buffer and writes result i from the start; result
i may overwrite left-hand matrices 0..i-1 (already consumed) but never the i-th
or later ones, which are still to be read.  Its size is

    n * S_max + S_min,   S_max = max(S_left, S_res), S_min = min(S_left, S_res).

``simulate`` plays the multiplications in order on that layout and reports any
write that would clobber a live left-hand matrix.
"""


def separate_size(n, s_left, s_res):
    """Size when left-hand and result matrices are stored separately."""
    return n * (s_left + s_res)


def shared_size(n, s_left, s_res):
    """Size of the shared buffer: n * S_max + S_min (Sec. 4.2)."""
    return n * max(s_left, s_res) + min(s_left, s_res)


def layout(n, s_left, s_res, size):
    """Offsets (left_i, result_i) for a buffer of ``size``: left-hand matrices packed
    at the end of the buffer, results packed from the start."""
    left = [size - (n - i) * s_left for i in range(n)]
    res = [i * s_res for i in range(n)]
    return left, res


def simulate(n, s_left, s_res, size):
    """Run the n multiplications on the layout; return the list of violations.

    Multiplication i reads left-hand matrix i and writes result i.  A violation
    is a write of result i that overlaps a left-hand matrix j >= i (still live),
    or any region outside [0, size).
    """
    left, res = layout(n, s_left, s_res, size)
    bad = []
    if n and left[0] < 0:
        bad.append(("left-out-of-buffer", 0))
    for i in range(n):
        r0, r1 = res[i], res[i] + s_res
        if r1 > size:
            bad.append(("result-out-of-buffer", i))
        for j in range(i, n):
            l0, l1 = left[j], left[j] + s_left
            if r0 < l1 and l0 < r1:
                bad.append(("overwrites-live-left", i, j))
    return bad


def minimal_size(n, s_left, s_res):
    """Smallest buffer for which ``simulate`` finds no violation (brute force)."""
    size = 0
    while simulate(n, s_left, s_res, size):
        size += 1
    return size
