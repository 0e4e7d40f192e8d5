"""Token re-layout around the selective block (paper Section 3.2, Stage 2/3).

Test infrastructure: used only by tests, the smoke check and the CPU baseline.

Readings: the "orthogonal upsampling" of Stage 2 is read as 2x nearest
upsampling (bilinear, half-pixel centres, edge clamp, is a variant); the
unselected tokens are filled by upsampling the low-res latent and do not enter
the block; the compacted sequence is [text; reference; selected tokens in
ascending index order]; selected rows carry their high-res grid position
(0, row, col) for RoPE.
"""
from __future__ import annotations

import numpy as np


def upsample_nearest(lowres, H_lr: int, W_lr: int):
    """2x nearest upsampling of a raster-ordered [H_lr*W_lr, D] grid."""
    x = np.asarray(lowres)
    D = x.shape[1]
    g = x.reshape(H_lr, W_lr, D)
    out = np.empty((2 * H_lr, 2 * W_lr, D), dtype=x.dtype)
    for r in range(2 * H_lr):
        for c in range(2 * W_lr):
            out[r, c] = g[r // 2, c // 2]
    return out.reshape(4 * H_lr * W_lr, D)


def upsample_bilinear(lowres, H_lr: int, W_lr: int):
    """2x bilinear upsampling with half-pixel centres and edge clamping (fp64).

    Output pixel r samples source coordinate (r + 0.5) / 2 - 0.5, clamped to
    the grid; weights are the linear interpolation weights on each axis.
    """
    x = np.asarray(lowres, dtype=np.float64)
    D = x.shape[1]
    g = x.reshape(H_lr, W_lr, D)

    def taps(n_out, n_in):
        res = []
        for o in range(n_out):
            src = max((o + 0.5) / 2.0 - 0.5, 0.0)
            i0 = min(int(np.floor(src)), n_in - 1)
            i1 = min(i0 + 1, n_in - 1)
            w1 = src - i0
            res.append((i0, i1, 1.0 - w1, w1))
        return res

    rt, ct = taps(2 * H_lr, H_lr), taps(2 * W_lr, W_lr)
    out = np.empty((2 * H_lr, 2 * W_lr, D))
    for r, (r0, r1, wr0, wr1) in enumerate(rt):
        row = wr0 * g[r0] + wr1 * g[r1]                      # [W_lr, D]
        for c, (c0, c1, wc0, wc1) in enumerate(ct):
            out[r, c] = wc0 * row[c0] + wc1 * row[c1]
    return out.reshape(4 * H_lr * W_lr, D)


def selected_positions(idx, W_hr: int) -> np.ndarray:
    """(frame, row, col) = (0, idx // W_hr, idx % W_hr) for each selected index."""
    idx = np.asarray(idx, dtype=np.int64)
    pos = np.zeros((idx.shape[0], 3), dtype=np.int32)
    pos[:, 1] = idx // W_hr
    pos[:, 2] = idx % W_hr
    return pos


def gather_upsample(lowres, highres_prev, prefix, idx, H_lr: int, W_lr: int,
                    mode: str = "nearest"):
    """Build the compacted block input and the canvas of unselected tokens.

    Returns (compact [LR + k, D], pos_sel [k, 3], canvas [N, D]):
      compact = [prefix rows; highres_prev[idx]];
      canvas[p] = highres_prev[p] where p is selected, else upsample(lowres)[p].
    """
    highres_prev = np.asarray(highres_prev)
    idx = np.asarray(idx, dtype=np.int64)
    N = highres_prev.shape[0]
    if mode == "nearest":
        up = upsample_nearest(lowres, H_lr, W_lr)
    elif mode == "bilinear":
        up = upsample_bilinear(lowres, H_lr, W_lr)
    else:
        raise ValueError(mode)
    mask = np.zeros(N, dtype=bool)
    mask[idx] = True
    canvas = np.where(mask[:, None], highres_prev, up)
    prefix = np.asarray(prefix).reshape(-1, highres_prev.shape[1])
    compact = np.concatenate([prefix, highres_prev[idx]], axis=0)
    return compact, selected_positions(idx, 2 * W_lr), canvas


def scatter(out, idx, row_offset: int, canvas):
    """Stage-3 re-layout: canvas[idx[j]] = out[row_offset + j] (returns a copy)."""
    canvas = np.array(canvas, copy=True)
    idx = np.asarray(idx, dtype=np.int64)
    canvas[idx] = np.asarray(out)[row_offset:row_offset + idx.shape[0]]
    return canvas
