"""Pins of the coordinate-bound noise oracle (Section 3.2 re-injection; the
generator's published definition and its known-answer vectors)."""
import json
import math
import os

import numpy as np
import pytest
from scipy import stats

import oracle
from oracle import noise as nz

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.json")


def test_philox_known_answers():
    for v in json.load(open(GOLDEN))["vectors"]:
        ctr = np.array([[int(x, 16) for x in v["ctr"]]], dtype=np.uint64)
        key = [int(x, 16) for x in v["key"]]
        got = nz.philox4x32_10(ctr, key)[0]
        assert [int(x) for x in got] == [int(x, 16) for x in v["out"]]


def test_uniforms_are_open_interval_and_exact():
    w = np.array([0, 255, 256, 0xFFFFFFFF], dtype=np.uint64)
    u = nz.uniform24(w)
    np.testing.assert_array_equal(u, [2.0 ** -25, 2.0 ** -25, 3 * 2.0 ** -25, 1 - 2.0 ** -25])
    assert np.all((u > 0) & (u < 1))


def test_box_muller_hand_values():
    # u0 = u2 = 1/2 + 2^-25 gives r = sqrt(2 ln 2) = 1.17741002...; u1 = 1/4 + 2^-25 puts the
    # angle at pi/2 (cos ~ 0, sin ~ 1); u3 = 2^-25 puts it at 0 (cos ~ 1, sin ~ 0).
    w = np.array([[0x80000000, 0x40000000, 0x80000000, 0]], dtype=np.uint64)
    z = nz.box_muller(w)[0]
    assert abs(z[0]) < 1e-6 and abs(z[3]) < 1e-6
    assert z[1] == pytest.approx(1.1774100225154747, rel=1e-6)
    assert z[2] == pytest.approx(1.1774100225154747, rel=1e-6)
    assert z[3] > 0 and z[0] < 0


def test_noise_is_standard_normal():
    C = 64
    eps = nz.pixel_noise(np.arange(4096), C, seed=7)
    x = eps.reshape(-1)
    n = x.size
    assert abs(x.mean()) < 5 / math.sqrt(n)
    assert abs(x.var() - 1.0) < 5 * math.sqrt(2.0 / n)
    assert abs(stats.kurtosis(x, fisher=False) - 3.0) < 0.05
    assert stats.kstest(x, "norm").pvalue > 1e-3
    # Neighbouring channels and pixels uncorrelated.
    assert abs(np.corrcoef(eps[:, :-1].reshape(-1), eps[:, 1:].reshape(-1))[0, 1]) < 0.01
    assert abs(np.corrcoef(eps[:-1].reshape(-1), eps[1:].reshape(-1))[0, 1]) < 0.01


def test_noise_is_bound_to_the_coordinate():
    C = 16
    pix = np.array([5, 900, 3, 77, 5])
    a = nz.pixel_noise(pix, C, seed=3)
    b = nz.pixel_noise(pix[::-1], C, seed=3)[::-1]
    np.testing.assert_array_equal(a, b)                       # order-free
    np.testing.assert_array_equal(a[0], a[4])                 # same pixel, same noise
    assert not np.allclose(a[0], nz.pixel_noise([5], C, seed=4)[0])   # the seed changes it
    # Channel groups of one pixel come from consecutive counters; words map to channels in order.
    bits = nz.pixel_noise_bits([900], 8, seed=3)[0]
    w1 = nz.philox4x32_10(np.array([[900, 1, 0, 0]], dtype=np.uint64), (3, 0))[0]
    np.testing.assert_array_equal(bits[4:], w1)


def test_block_noise_is_scaled_mean_of_children():
    W_lr, C = 5, 8
    blocks = np.array([0, 7, 24])
    got = nz.block_noise(blocks, W_lr, C, seed=11)
    W_hr = 2 * W_lr
    for i, b in enumerate(blocks):
        r, c = divmod(int(b), W_lr)
        kids = [(2 * r + dr) * W_hr + 2 * c + dc for dr in (0, 1) for dc in (0, 1)]
        np.testing.assert_allclose(got[i], nz.pixel_noise(kids, C, seed=11).mean(axis=0) * 2.0, rtol=1e-14)
    big = nz.block_noise(np.arange(32 * 32), 32, 16, seed=2).reshape(-1)
    assert abs(big.var() - 1.0) < 0.05


def test_halfunit_positions_select_pixel_or_block_noise():
    W_lr, C = 4, 8
    W_hr = 2 * W_lr
    pos = np.array([[0, 2 * 3, 2 * 5],          # pixel (3, 5)
                    [0, 4 * 1 + 1, 4 * 2 + 1],  # block (1, 2)
                    [0, 0, 0]])                 # pixel (0, 0)
    got = nz.halfunit_noise(pos, W_hr, C, seed=9)
    np.testing.assert_array_equal(got[0], nz.pixel_noise([3 * W_hr + 5], C, seed=9)[0])
    np.testing.assert_array_equal(got[1], nz.block_noise([1 * W_lr + 2], W_lr, C, seed=9)[0])
    np.testing.assert_array_equal(got[2], nz.pixel_noise([0], C, seed=9)[0])
    with pytest.raises(ValueError):
        nz.halfunit_noise(np.array([[0, 1, 2]]), W_hr, C, seed=9)


def test_reinject_limits():
    g = np.random.default_rng(0)
    x, e = g.standard_normal((6, 8)), g.standard_normal((6, 8))
    np.testing.assert_array_equal(nz.reinject(x, e, 0.0), x)
    np.testing.assert_array_equal(nz.reinject(x, e, 1.0), e)
    np.testing.assert_allclose(nz.reinject(x, e, 0.25), 0.75 * x + 0.25 * e, rtol=1e-15)
    # Re-injecting into noise-free zeros gives t eps: unit-variance noise scaled to level t.
    z = nz.reinject(np.zeros((4096, 16)), nz.pixel_noise(np.arange(4096), 16, 1), 0.6)
    assert abs(z.std() - 0.6) < 0.01
    assert oracle.reinject is nz.reinject
