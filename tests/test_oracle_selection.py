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


# ---------------------------------------------------------------------------
# The paper's tie-break perturbation (Section 3.3) and batched selection.

def _fp32_sums(scores, delta):
    """fp32 sums rounded once: float64 adds of fp32 values of similar size are
    exact, so one rounding to fp32 gives the correctly rounded sum."""
    return [float(np.float32(float(a) + float(b))) for a, b in zip(scores, delta)]


def test_perturbed_hand_example():
    s = np.array([0.5, 0.9, 0.5, 0.1, 0.9], dtype=np.float32)
    d = np.array([0.0, -1e-6, 1e-6, 0.0, 0.0], dtype=np.float32)
    # 0.9 (4) > 0.9 - 1e-6 (1) > 0.5 + 1e-6 (2) > 0.5 (0): the perturbation, not the index, breaks the ties.
    assert list(oracle.select_topk_perturbed(s, d, 3)) == [1, 2, 4]
    assert list(oracle.select_topk(s, 3)) == [0, 1, 4]


def test_perturbed_zero_delta_is_plain_selection():
    s = generator.quantised_scores(3, 500, 6)
    assert list(oracle.select_topk_perturbed(s, np.zeros(500, np.float32), 123)) == list(oracle.select_topk(s, 123))


@pytest.mark.parametrize("n,k,levels", [(300, 100, 4), (1000, 333, 8), (64, 64, 2)])
def test_perturbed_matches_bruteforce(n, k, levels):
    s = generator.quantised_scores(n, n, levels)
    d = generator.tiebreak_noise(n, n)
    assert list(oracle.select_topk_perturbed(s, d, k)) == _bruteforce(_fp32_sums(s, d), k)
    # The perturbation only reorders ties: every kept score is at least every dropped one.
    sel = set(oracle.select_topk_perturbed(s, d, k).tolist())
    kept = [s[i] for i in sel]
    dropped = [s[i] for i in range(n) if i not in sel]
    if kept and dropped:
        assert min(kept) >= max(dropped)


def test_batched_is_per_segment_bruteforce():
    g = np.random.default_rng(5)
    sizes = [7, 1, 300, 64, 1000]
    ks = [3, 1, 0, 64, 250]
    off = np.concatenate([[0], np.cumsum(sizes)])
    s = generator.quantised_scores(9, int(off[-1]), 5)
    got = oracle.select_topk_batched(s, off, ks)
    want = []
    for b in range(len(sizes)):
        want += _bruteforce(s[off[b]:off[b + 1]], ks[b])
    assert got.tolist() == want
    d = generator.tiebreak_noise(9, int(off[-1]))
    got = oracle.select_topk_batched(s, off, ks, delta=d)
    want = []
    for b in range(len(sizes)):
        want += _bruteforce(_fp32_sums(s[off[b]:off[b + 1]], d[off[b]:off[b + 1]]), ks[b])
    assert got.tolist() == want
