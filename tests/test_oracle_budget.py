"""Pins of the branching-budget oracle (oracle/budget.py)."""

import math

import numpy as np
import pytest

from oracle import budget as B


def test_even_transfer_closed_form():
    """Sec. 2.2 budget transfer: N^d spread evenly -- floor(total/n) each, the
    first total mod n paths one more."""
    for n, total in ((1, 1), (3, 8), (5, 16), (7, 64), (4, 4), (6, 3)):
        b = B.branch_budget([0.0] * n, total, "even")
        if total >= n:
            assert b == [total // n + (1 if k < total % n else 0) for k in range(n)]
        else:
            assert b == [1] * n


@pytest.mark.parametrize("mode", ["high", "low"])
def test_sum_min_one_and_order(mode):
    rng = np.random.default_rng(3)
    for _ in range(50):
        n = int(rng.integers(1, 12))
        total = int(rng.integers(n, 80))
        s = list(rng.normal(-20, 10, size=n))
        b = B.branch_budget(s, total, mode, 2.0)
        assert sum(b) == total and min(b) >= 1
        # monotone: a higher (high mode) or lower (low mode) score never gets fewer branches
        key = np.array(s) if mode == "high" else -np.array(s)
        for i in range(n):
            for j in range(n):
                if key[i] > key[j]:
                    assert b[i] >= b[j]


def test_two_paths_closed_form():
    """Two paths, scores 0 and -T ln 3 at temperature T: weights 3/4 and 1/4 in
    high mode; 2 + 8 branches -> 1 + 6 and 1 + 2."""
    T = 2.0
    s = [0.0, -T * math.log(3.0)]
    assert B.branch_budget(s, 10, "high", T) == [7, 3]
    assert B.branch_budget(s, 10, "low", T) == [3, 7]


def test_infinite_temperature_is_even():
    s = [-1.0, -50.0, -3.0, -8.0]
    assert B.branch_budget(s, 20, "high", 1e12) == B.branch_budget(s, 20, "even")


def test_largest_remainder_ties_to_lower_index():
    """Equal scores: even split, the extra branches to the first paths."""
    assert B.branch_budget([-5.0] * 3, 8, "high", 2.0) == [3, 3, 2]
