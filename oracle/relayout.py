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
    prefix = np.zeros((0, highres_prev.shape[1])) if prefix is None else np.asarray(prefix).reshape(-1, highres_prev.shape[1])
    compact = np.concatenate([prefix, highres_prev[idx]], axis=0)
    return compact, selected_positions(idx, 2 * W_lr), canvas


def scatter(out, idx, row_offset: int, canvas):
    """Stage-3 re-layout: canvas[idx[j]] = out[row_offset + j] (returns a copy)."""
    canvas = np.array(canvas, copy=True)
    idx = np.asarray(idx, dtype=np.int64)
    canvas[idx] = np.asarray(out)[row_offset:row_offset + idx.shape[0]]
    return canvas


# ---------------------------------------------------------------------------
# The paper's own Stage 2 (Section 3.2): selection at low-res granularity, the
# selected tokens expanded 2x2, the others kept at low resolution in the same
# sequence.  Readings: a low-res token sits at the centre of its 2x2 block,
# (2r + 1/2, 2c + 1/2) in high-res coordinates, so RoPE rotates it by
# fractional positions; positions are given in half units (twice the
# coordinate) so they stay integers; children of a selected parent come in
# raster order (dr, dc), parents in ascending index order, then the
# unselected parents in ascending order.


def mixed_layout(idx, H_lr: int, W_lr: int):
    """Rows of the mixed sequence after the prefix, as (parent, dr, dc) with
    dr = dc = -1 for a token kept at low resolution; and their positions in
    half units (frame, 2 row, 2 col) [4K + M' - K, 3]."""
    idx = np.asarray(idx, dtype=np.int64)
    Mp = H_lr * W_lr
    sel = np.zeros(Mp, dtype=bool)
    sel[idx] = True
    rows, pos = [], []
    for p in idx:
        r, c = divmod(int(p), W_lr)
        for dr in (0, 1):
            for dc in (0, 1):
                rows.append((int(p), dr, dc))
                pos.append((0, 2 * (2 * r + dr), 2 * (2 * c + dc)))
    for p in np.nonzero(~sel)[0]:
        r, c = divmod(int(p), W_lr)
        rows.append((int(p), -1, -1))
        pos.append((0, 4 * r + 1, 4 * c + 1))
    return rows, np.array(pos, dtype=np.int32).reshape(-1, 3)


def gather_mixed(lowres, prefix, idx, H_lr: int, W_lr: int, mode: str = "nearest"):
    """The mixed-resolution block input of Stage 2.

    Returns (compact [LR + 4K + M' - K, D], pos [4K + M' - K, 3] in half units,
    children [4K], the high-res raster indices of the expanded tokens in
    ascending order).  A child takes the upsampled value of its high-res
    pixel (nearest: its parent's row; bilinear: the variant's interpolation);
    a kept token takes its low-res row.
    """
    lowres = np.asarray(lowres)
    W_hr = 2 * W_lr
    up = upsample_nearest(lowres, H_lr, W_lr) if mode == "nearest" else upsample_bilinear(lowres, H_lr, W_lr)
    rows, pos = mixed_layout(idx, H_lr, W_lr)
    body = []
    children = []
    for p, dr, dc in rows:
        if dr < 0:
            body.append(lowres[p])
        else:
            r, c = divmod(p, W_lr)
            q = (2 * r + dr) * W_hr + 2 * c + dc
            body.append(up[q])
            children.append(q)
    prefix = np.zeros((0, lowres.shape[1])) if prefix is None else np.asarray(prefix).reshape(-1, lowres.shape[1])
    body = np.array(body, dtype=up.dtype).reshape(-1, lowres.shape[1])
    compact = np.concatenate([prefix.astype(up.dtype), body], axis=0)
    return compact, pos, np.sort(np.array(children, dtype=np.int64))


def scatter_mixed(out, idx, row_offset: int, H_lr: int, W_lr: int, canvas_hr, state_lr):
    """After the Stage-2 blocks: each expanded token's row goes to its
    high-res pixel of canvas_hr; each kept token's row goes to its row of the
    low-res state.  Returns (canvas_hr, state_lr) copies."""
    canvas_hr = np.array(canvas_hr, copy=True)
    state_lr = np.array(state_lr, copy=True)
    out = np.asarray(out)
    rows, _ = mixed_layout(idx, H_lr, W_lr)
    W_hr = 2 * W_lr
    for j, (p, dr, dc) in enumerate(rows):
        if dr < 0:
            state_lr[p] = out[row_offset + j]
        else:
            r, c = divmod(p, W_lr)
            canvas_hr[(2 * r + dr) * W_hr + 2 * c + dc] = out[row_offset + j]
    return canvas_hr, state_lr
