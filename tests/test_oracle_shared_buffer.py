"""Pins for the shared buffer of Sec. 4.2 (oracle/shared_buffer.py).

Fixed by the worked examples of Fig. 1 (tests/golden/fig1_shared_buffer.txt) and
by brute force: the size formula n * S_max + S_min must be exactly the smallest
buffer on which playing the multiplications in order never overwrites a live
left-hand matrix.
"""

import os
import random

import pytest

from oracle import shared_buffer as sb

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "fig1_shared_buffer.txt")


def golden_rows():
    rows = []
    for line in open(GOLDEN):
        line = line.strip()
        if line and not line.startswith("#"):
            n, sl, sr, shared, sep, pct = line.split()
            rows.append((int(n), int(sl), int(sr), int(shared), int(sep), float(pct)))
    return rows


def test_golden_file_has_both_examples():
    assert len(golden_rows()) == 2


@pytest.mark.parametrize("row", golden_rows())
def test_fig1_examples(row):
    n, sl, sr, shared, sep, pct = row
    assert sb.shared_size(n, sl, sr) == shared
    assert sb.separate_size(n, sl, sr) == sep
    assert 100.0 * (sep - shared) / sep == pytest.approx(pct, abs=1e-12)
    assert sb.simulate(n, sl, sr, shared) == []
    assert sb.simulate(n, sl, sr, shared - 1) != []
    assert sb.minimal_size(n, sl, sr) == shared


def test_fig1a_final_contents():
    # Equal sizes: after the last multiplication the results fill the first n
    # slots' worth and the last left-hand matrix sits behind them.
    left, res = sb.layout(4, 8, 8, 40)
    assert res == [0, 8, 16, 24]
    assert left == [8, 16, 24, 32]
    assert res[-1] + 8 == left[-1]


def test_formula_is_minimal_brute_force():
    rng = random.Random(0)
    for _ in range(60):
        n = rng.randint(1, 9)
        sl, sr = rng.randint(1, 12), rng.randint(1, 12)
        assert sb.minimal_size(n, sl, sr) == sb.shared_size(n, sl, sr), (n, sl, sr)


def test_result_never_overwrites_current_left():
    # a buffer that only holds the separate left-hand block cannot work
    assert sb.simulate(3, 5, 5, 15) != []
