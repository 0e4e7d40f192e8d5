"""Pins of the oracle's top-K selection (Section 3.3.3, Eq. topk)."""
import math

import numpy as np
import pytest

import oracle
from synth import generator


def _bruteforce(scores, k):
    """Pure Python: order by (NaN last, value descending, index ascending)."""
    vals = [float(x) for x in scores]

    def key(i):
        v = vals[i]
        return (1, 0.0, i) if math.isnan(v) else (0, -v, i)

    return sorted(sorted(range(len(vals)), key=key)[:k])


@pytest.mark.parametrize("n,k,levels", [(1, 1, 3), (10, 3, 4), (257, 100, 8), (1000, 999, 5), (64, 0, 2)])
def test_matches_bruteforce_with_duplicates(n, k, levels):
    s = generator.quantised_scores(n + k, n, levels)
    assert list(oracle.select_topk(s, k)) == _bruteforce(s, k)


def test_hand_example():
    s = np.array([0.5, 0.9, 0.5, 0.1, 0.9], dtype=np.float32)
    assert list(oracle.select_topk(s, 3)) == [0, 1, 4]
    assert list(oracle.select_topk(s, 2)) == [1, 4]
    assert list(oracle.select_topk(s, 4)) == [0, 1, 2, 4]


def test_degenerate_k():
    s = np.random.default_rng(0).random(50).astype(np.float32)
    assert oracle.select_topk(s, 0).shape == (0,)
    assert list(oracle.select_topk(s, 50)) == list(range(50))
    assert list(oracle.select_topk(np.full(50, 0.3, np.float32), 7)) == list(range(7))
    with pytest.raises(ValueError):
        oracle.select_topk(s, 51)


def test_signed_zero_nan_and_infinities():
    s = np.array([np.nan, -0.0, 0.0, -np.inf, np.inf, np.nan, -1.0], dtype=np.float32)
    # Order: inf(4), -0.0(1) == 0.0(2) by index, -1(6), -inf(3), nan(0), nan(5).
    assert list(oracle.select_topk(s, 1)) == [4]
    assert list(oracle.select_topk(s, 2)) == [1, 4]
    assert list(oracle.select_topk(s, 3)) == [1, 2, 4]
    assert list(oracle.select_topk(s, 5)) == [1, 2, 3, 4, 6]
    assert list(oracle.select_topk(s, 6)) == [0, 1, 2, 3, 4, 6]
    assert list(oracle.select_topk(s, 6)) == _bruteforce(s, 6)


def test_unique_ascending_and_threshold():
    s = np.random.default_rng(1).standard_normal(4096).astype(np.float32)
    idx = oracle.select_topk(s, 1229)
    assert np.all(np.diff(idx) > 0)
    kth = np.sort(s)[::-1][1228]
    assert np.all(s[idx] >= kth)
    rest = np.setdiff1d(np.arange(4096), idx)
    assert np.all(s[rest] <= kth)
