"""Pins of the oracle's gather / upsample / scatter (Section 3.2, Stages 2 and 3)."""
import numpy as np
import pytest
import torch

import oracle


def _grid(H, W, D, seed=0):
    return np.random.default_rng(seed).standard_normal((H * W, D))


def test_nearest_equals_repeat():
    g = _grid(5, 7, 3)
    up = oracle.upsample_nearest(g, 5, 7)
    ref = np.repeat(np.repeat(g.reshape(5, 7, 3), 2, axis=0), 2, axis=1).reshape(-1, 3)
    np.testing.assert_array_equal(up, ref)


@pytest.mark.parametrize("H,W", [(4, 4), (3, 5), (1, 6), (7, 2)])
def test_bilinear_equals_torch_interpolate(H, W):
    g = _grid(H, W, 4, seed=H * 10 + W)
    up = oracle.upsample_bilinear(g, H, W)
    t = torch.from_numpy(g.reshape(H, W, 4).transpose(2, 0, 1)[None].copy())
    ref = torch.nn.functional.interpolate(t, scale_factor=2, mode="bilinear", align_corners=False)
    ref = ref[0].numpy().transpose(1, 2, 0).reshape(-1, 4)
    np.testing.assert_allclose(up, ref, atol=1e-14)


def test_bilinear_of_constant_and_linear_ramp():
    H, W = 6, 5
    np.testing.assert_allclose(oracle.upsample_bilinear(np.full((H * W, 2), 1.5), H, W), 1.5)
    # Interior of a row ramp x = c: output at column o is (o + 0.5)/2 - 0.5.
    ramp = np.tile(np.arange(W, dtype=float), H).reshape(-1, 1)
    up = oracle.upsample_bilinear(ramp, H, W).reshape(2 * H, 2 * W)
    for o in range(1, 2 * W - 1):
        assert abs(up[3, o] - ((o + 0.5) / 2 - 0.5)) < 1e-14


def test_gather_keep_all_and_keep_none():
    H, W, D = 4, 3, 5
    N = 4 * H * W
    g = np.random.default_rng(2)
    low, high, pre = g.standard_normal((H * W, D)), g.standard_normal((N, D)), g.standard_normal((6, D))
    idx_all = np.arange(N, dtype=np.int32)
    compact, pos, canvas = oracle.gather_upsample(low, high, pre, idx_all, H, W)
    np.testing.assert_array_equal(canvas, high)
    np.testing.assert_array_equal(compact, np.concatenate([pre, high]))
    compact, pos, canvas = oracle.gather_upsample(low, high, pre, np.zeros(0, np.int32), H, W)
    np.testing.assert_array_equal(canvas, oracle.upsample_nearest(low, H, W))
    np.testing.assert_array_equal(compact, pre)
    assert pos.shape == (0, 3)


def test_gather_mixed_and_positions():
    H, W, D = 3, 4, 2
    g = np.random.default_rng(3)
    low, high = g.standard_normal((H * W, D)), g.standard_normal((4 * H * W, D))
    idx = np.array([0, 9, 17, 47], dtype=np.int32)
    compact, pos, canvas = oracle.gather_upsample(low, high, np.zeros((0, D)), idx, H, W)
    np.testing.assert_array_equal(compact, high[idx])
    # W_hr = 8: 9 -> (1, 1), 17 -> (2, 1), 47 -> (5, 7).
    assert pos.tolist() == [[0, 0, 0], [0, 1, 1], [0, 2, 1], [0, 5, 7]]
    up = oracle.upsample_nearest(low, H, W)
    for p in range(4 * H * W):
        np.testing.assert_array_equal(canvas[p], high[p] if p in idx else up[p])
    # Position 47 = (5, 7) on the high-res grid is low-res cell (2, 3) = 11.
    np.testing.assert_array_equal(up[47], low[11])


def test_scatter_roundtrip():
    g = np.random.default_rng(4)
    high = g.standard_normal((64, 3))
    idx = np.sort(g.permutation(64)[:20]).astype(np.int32)
    compact, _, canvas = oracle.gather_upsample(g.standard_normal((16, 3)), high,
                                                g.standard_normal((5, 3)), idx, 4, 4)
    np.testing.assert_array_equal(oracle.scatter(compact, idx, 5, canvas), canvas)
    out = g.standard_normal(compact.shape)
    c2 = oracle.scatter(out, idx, 5, canvas)
    np.testing.assert_array_equal(c2[idx], out[5:])
    rest = np.setdiff1d(np.arange(64), idx)
    np.testing.assert_array_equal(c2[rest], canvas[rest])
