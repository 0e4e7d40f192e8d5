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


# ---------------------------------------------------------------------------
# The mixed-resolution Stage-2 sequence (Section 3.2): selected low-res tokens
# expanded to 2x2 children, the rest kept at low resolution.

def _hr_index(pos_half, W_lr):
    """High-res raster index of a child from its half-unit position."""
    return (pos_half[:, 1] // 2) * (2 * W_lr) + pos_half[:, 2] // 2


def test_mixed_worked_example():
    # M' = 2x2, parents 1 = (0, 1) and 2 = (1, 0) selected; worked by hand.
    # Children come parent by parent in (dr, dc) raster order at twice their
    # high-res coordinate; kept parents 0 and 3 sit at their block centres
    # (0.5, 0.5) and (2.5, 2.5), i.e. (1, 1) and (5, 5) in half units.
    low = np.arange(8, dtype=float).reshape(4, 2)
    pre = np.full((1, 2), -1.0)
    compact, pos, children = oracle.gather_mixed(low, pre, [1, 2], 2, 2)
    assert pos.tolist() == [[0, 0, 4], [0, 0, 6], [0, 2, 4], [0, 2, 6],
                            [0, 4, 0], [0, 4, 2], [0, 6, 0], [0, 6, 2],
                            [0, 1, 1], [0, 5, 5]]
    assert children.tolist() == [2, 3, 6, 7, 8, 9, 12, 13]
    want = [[-1, -1]] + [[2, 3]] * 4 + [[4, 5]] * 4 + [[0, 1], [6, 7]]
    np.testing.assert_array_equal(compact, want)


@pytest.mark.parametrize("mode,up", [("nearest", oracle.upsample_nearest), ("bilinear", oracle.upsample_bilinear)])
def test_mixed_keep_all_is_the_upsampled_grid(mode, up):
    # rho = 1: every token expanded; placing each row at the pixel its
    # position names rebuilds the 2x upsampled grid, and the children are
    # every high-res index.
    H, W, D = 3, 5, 4
    low = _grid(H, W, D, seed=11)
    compact, pos, children = oracle.gather_mixed(low, None, np.arange(H * W), H, W, mode)
    assert compact.shape == (4 * H * W, D)
    assert (pos % 2 == 0).all()
    q = _hr_index(pos, W)
    assert sorted(q.tolist()) == list(range(4 * H * W))
    grid = np.empty((4 * H * W, D))
    grid[q] = compact
    np.testing.assert_array_equal(grid, up(low, H, W))
    np.testing.assert_array_equal(children, np.arange(4 * H * W))


def test_mixed_keep_none_is_the_lowres_grid():
    H, W, D = 4, 3, 2
    low = _grid(H, W, D, seed=12)
    pre = _grid(1, 3, D, seed=13)
    compact, pos, children = oracle.gather_mixed(low, pre, np.zeros(0, np.int64), H, W)
    np.testing.assert_array_equal(compact, np.concatenate([pre, low]))
    assert children.shape == (0,)
    # A kept token sits at the mean of its four children's positions.
    _, pos_all, _ = oracle.gather_mixed(low, None, np.arange(H * W), H, W)
    centres = pos_all.reshape(H * W, 4, 3).mean(axis=1)
    np.testing.assert_array_equal(pos, centres)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_mixed_partition_and_roundtrip(seed):
    g = np.random.default_rng(seed)
    H, W, D = 5, 6, 3
    Mp = H * W
    k = int(g.integers(1, Mp))
    idx = np.sort(g.permutation(Mp)[:k])
    low = g.standard_normal((Mp, D))
    pre = g.standard_normal((2, D))
    compact, pos, children = oracle.gather_mixed(low, pre, idx, H, W)
    assert compact.shape == (2 + 4 * k + Mp - k, D) and pos.shape == (4 * k + Mp - k, 3)
    # Every low-res cell is covered once: by its four children or by itself.
    cover = np.zeros((2 * H, 2 * W), dtype=int)
    for (_, r2, c2) in pos:
        if r2 % 2 == 0:
            cover[r2 // 2, c2 // 2] += 1
        else:
            cover[(r2 - 1) // 2:(r2 + 3) // 2, (c2 - 1) // 2:(c2 + 3) // 2] += 1
    assert (cover == 1).all()
    assert len({tuple(p) for p in pos}) == len(pos)
    assert (np.diff(children) > 0).all()
    np.testing.assert_array_equal(np.sort(_hr_index(pos[:4 * k], W)), children)
    # Identity blocks: the scatter sends every row back where it came from.
    canvas0 = g.standard_normal((4 * Mp, D))
    state0 = g.standard_normal((Mp, D))
    canvas, state = oracle.scatter_mixed(compact, idx, 2, H, W, canvas0, state0)
    up = oracle.upsample_nearest(low, H, W)
    np.testing.assert_array_equal(canvas[children], up[children])
    rest = np.setdiff1d(np.arange(4 * Mp), children)
    np.testing.assert_array_equal(canvas[rest], canvas0[rest])
    kept = np.setdiff1d(np.arange(Mp), idx)
    np.testing.assert_array_equal(state[kept], low[kept])
    np.testing.assert_array_equal(state[idx], state0[idx])
    # Stage 3: expanding the kept tokens over that canvas gives the upsampled grid.
    _, _, full = oracle.gather_upsample(state, canvas, None, children, H, W)
    np.testing.assert_array_equal(full, up)


def test_half_unit_positions_rotate_halfway():
    # A token between two grid positions is rotated by the mean of their angles.
    pos = np.array([[0, 3, 4], [0, 4, 5], [0, 3.5, 4.5]])
    ang = oracle.rope_angles(pos, 64)
    np.testing.assert_allclose(ang[2], (ang[0] + ang[1]) / 2, rtol=0, atol=1e-12)
