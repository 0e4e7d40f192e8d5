"""The joint image-text attention block run on the compacted sequence, fp64.

Test infrastructure: used only by tests, the smoke check and the CPU baseline.

The paper names the block (Section 3.3.1: double-stream blocks computing
joint self-attention over [C; Z], Eq. joint_qk, with the model's
QK-normalisation) but not its internals.  The reading used here is the
FLUX-style MMDiT block:

double-stream, per stream s in {text rows, image rows}, each with its own
weights (PyTorch Linear layout W[out, in], biases present):
    h   = LN(x) * (1 + scale1_s) + shift1_s           (LN: no affine, eps 1e-6)
    q, k, v = split(h W_qkv^T + b_qkv)                 (each [rows, H, d])
    q = RMSNorm_d(q) * g_q ; k = RMSNorm_d(k) * g_k    (eps 1e-6)
    q, k = RoPE(q, pos), RoPE(k, pos)                  (rows in sequence order)
    o   = softmax(q k^T / sqrt(d)) v  over all rows of both streams
    x   = x + gate1_s * (o W_o^T + b_o)
    x   = x + gate2_s * (GELU_tanh((LN(x)(1 + scale2_s) + shift2_s) W_1^T + b_1) W_2^T + b_2)
single-stream, one weight set:
    h = LN(x)(1 + scale) + shift ; [q k v m] = h W_in^T + b_in
    q, k normalised and rotated as above ; o = attention(q, k, v)
    x = x + gate * ([o ; GELU_tanh(m)] W_out^T + b_out)
Modulation rows: double (shift1, scale1, gate1, shift2, scale2, gate2),
single (shift, scale, gate).

RoPE reading: three position axes (frame, row, col) splitting the head dim as
(d/8, 7d/16, 7d/16); within an axis of width n, pair m rotates by angle
pos * theta^(-2m/n) with theta = 10000; pairs are adjacent dims (2m, 2m+1).
"""
from __future__ import annotations

import numpy as np

LN_EPS = 1e-6
RMS_EPS = 1e-6
ROPE_THETA = 10000.0


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def layer_norm(x, eps: float = LN_EPS):
    """Layer norm over the last axis without affine parameters (biased variance)."""
    x = _f64(x)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def rms_norm(x, g, eps: float = RMS_EPS):
    """RMS norm over the last axis, times the gain g (the model's QK-norm)."""
    x = _f64(x)
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps) * _f64(g)


def rope_axes(d: int):
    return (d // 8, 7 * d // 16, 7 * d // 16)


def rope_angles(pos, d: int, theta: float = ROPE_THETA):
    """Rotation angle of each adjacent pair: [S, d/2] for pos [S, 3].

    Positions are real: the grid's are integers, the low-res tokens of the
    mixed-resolution Stage-2 sequence sit at half-integer block centres.
    """
    pos = np.asarray(pos, dtype=np.float64)
    parts = []
    for a, n in enumerate(rope_axes(d)):
        m = np.arange(n // 2, dtype=np.float64)
        omega = theta ** (-2.0 * m / n)
        parts.append(pos[:, a:a + 1] * omega[None, :])
    return np.concatenate(parts, axis=1)


def apply_rope(x, angles):
    """Rotate adjacent pairs (2m, 2m+1) of x [S, H, d] by angles [S, d/2]."""
    x = _f64(x)
    c = np.cos(angles)[:, None, :]
    s = np.sin(angles)[:, None, :]
    x0, x1 = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2] = x0 * c - x1 * s
    out[..., 1::2] = x0 * s + x1 * c
    return out


def attention(q, k, v, row_chunk: int = 1024):
    """Non-causal softmax attention per head.

    q: [Sq, H, d], k, v: [Sk, H, d].  Returns (o [Sq, H, d], lse [H, Sq]) with
    lse the natural-log normaliser of each softmax row.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    Sq, H, d = q.shape
    o = np.empty((Sq, H, v.shape[2]))
    lse = np.empty((H, Sq))
    scale = 1.0 / np.sqrt(d)
    for h in range(H):
        kh, vh = k[:, h, :], v[:, h, :]
        for r0 in range(0, Sq, row_chunk):
            p = (q[r0:r0 + row_chunk, h, :] @ kh.T) * scale
            m = p.max(axis=1, keepdims=True)
            e = np.exp(p - m)
            l = e.sum(axis=1, keepdims=True)
            o[r0:r0 + row_chunk, h, :] = (e @ vh) / l
            lse[h, r0:r0 + row_chunk] = m[:, 0] + np.log(l[:, 0])
    return o, lse


def gelu_tanh(x):
    """GELU, tanh form: x/2 * (1 + tanh(sqrt(2/pi) * (x + 0.044715 x^3)))."""
    x = _f64(x)
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))


def _modulate(x, shift, scale):
    return layer_norm(x) * (1.0 + _f64(scale)) + _f64(shift)


def _rows_in(rows, lo, hi):
    sel = (rows >= lo) & (rows < hi)
    return np.nonzero(sel)[0], rows[sel]


def double_block(x, pos, n_txt: int, w_txt: dict, w_img: dict, H: int, rows=None):
    """Double-stream block on x [S, D] with positions pos [S, 3].

    Rows [0, n_txt) use the text-stream weights, the rest the image-stream
    weights.  ``rows`` (optional) restricts the returned outputs to those
    sequence rows; keys and values always cover the whole sequence.
    Returns (out [len(rows), D], lse [H, len(rows)]).
    """
    x = _f64(x)
    S, D = x.shape
    d = D // H
    rows = np.arange(S) if rows is None else np.asarray(rows, dtype=np.int64)
    ang = rope_angles(pos, d)
    k_all = np.empty((S, H, d))
    v_all = np.empty((S, H, d))
    q_r = np.empty((rows.shape[0], H, d))
    for lo, hi, w in ((0, n_txt, w_txt), (n_txt, S, w_img)):
        if hi <= lo:
            continue
        mod, W, b = _f64(w["mod"]), _f64(w["w_qkv"]), _f64(w["b_qkv"])
        h = _modulate(x[lo:hi], mod[0], mod[1])
        k = h @ W[D:2 * D].T + b[D:2 * D]
        v = h @ W[2 * D:].T + b[2 * D:]
        k_all[lo:hi] = rms_norm(k.reshape(-1, H, d), w["g_k"])
        v_all[lo:hi] = v.reshape(-1, H, d)
        slot, r = _rows_in(rows, lo, hi)
        if r.size:
            hq = _modulate(x[r], mod[0], mod[1])
            q = hq @ W[:D].T + b[:D]
            q_r[slot] = rms_norm(q.reshape(-1, H, d), w["g_q"])
    k_all = apply_rope(k_all, ang)
    q_r = apply_rope(q_r, ang[rows])
    o, lse = attention(q_r, k_all, v_all)
    o = o.reshape(-1, D)
    out = np.empty((rows.shape[0], D))
    for lo, hi, w in ((0, n_txt, w_txt), (n_txt, S, w_img)):
        slot, r = _rows_in(rows, lo, hi)
        if not r.size:
            continue
        mod = _f64(w["mod"])
        y = x[r] + mod[2] * (o[slot] @ _f64(w["w_o"]).T + _f64(w["b_o"]))
        h2 = _modulate(y, mod[3], mod[4])
        m = gelu_tanh(h2 @ _f64(w["w_mlp1"]).T + _f64(w["b_mlp1"]))
        out[slot] = y + mod[5] * (m @ _f64(w["w_mlp2"]).T + _f64(w["b_mlp2"]))
    return out, lse


def block_qk(x, pos, n_txt: int, w_txt: dict | None, w_img: dict | None, H: int, single: dict | None = None):
    """Normalised, rotated queries and keys of a block's first stage.

    These are the q and k whose joint softmax the block's attention takes
    (Section 3.3.1, Eq. joint_qk) and from which Eq. spatial reads the
    image-to-text attention mass: per row, h = LN(x)(1 + scale1) + shift1,
    q = RMSNorm(h W_q^T + b_q) * g_q, k likewise, both rotated at pos.  For a
    double block rows [0, n_txt) use w_txt and the rest w_img; with ``single``
    given, every row uses the single-block weights (W_q, W_k = the first 2D
    rows of W_in).  Returns (q, k), each [S, H, d].
    """
    x = _f64(x)
    S, D = x.shape
    d = D // H
    ang = rope_angles(pos, d)
    q = np.empty((S, H, d))
    k = np.empty((S, H, d))
    parts = ((0, S, single, "w_in", "b_in"),) if single is not None else \
        ((0, n_txt, w_txt, "w_qkv", "b_qkv"), (n_txt, S, w_img, "w_qkv", "b_qkv"))
    for lo, hi, w, wn, bn in parts:
        if hi <= lo:
            continue
        mod, W, b = _f64(w["mod"]), _f64(w[wn]), _f64(w[bn])
        h = _modulate(x[lo:hi], mod[0], mod[1])
        q[lo:hi] = rms_norm((h @ W[:D].T + b[:D]).reshape(-1, H, d), w["g_q"])
        k[lo:hi] = rms_norm((h @ W[D:2 * D].T + b[D:2 * D]).reshape(-1, H, d), w["g_k"])
    return apply_rope(q, ang), apply_rope(k, ang)


def single_block(x, pos, w: dict, H: int, rows=None):
    """Single-stream block on x [S, D]; ``rows`` as in double_block."""
    x = _f64(x)
    S, D = x.shape
    d = D // H
    rows = np.arange(S) if rows is None else np.asarray(rows, dtype=np.int64)
    ang = rope_angles(pos, d)
    mod, W, b = _f64(w["mod"]), _f64(w["w_in"]), _f64(w["b_in"])
    h = _modulate(x, mod[0], mod[1])
    k = rms_norm((h @ W[D:2 * D].T + b[D:2 * D]).reshape(S, H, d), w["g_k"])
    v = (h @ W[2 * D:3 * D].T + b[2 * D:3 * D]).reshape(S, H, d)
    hr = h[rows]
    q = rms_norm((hr @ W[:D].T + b[:D]).reshape(-1, H, d), w["g_q"])
    mlp = gelu_tanh(hr @ W[3 * D:].T + b[3 * D:])
    k = apply_rope(k, ang)
    q = apply_rope(q, ang[rows])
    o, lse = attention(q, k, v)
    cat = np.concatenate([o.reshape(-1, D), mlp], axis=1)
    y = cat @ _f64(w["w_out"]).T + _f64(w["b_out"])
    return x[rows] + mod[2] * y, lse


def block_batched(x, pos, txt_off, img_off, H: int, w_txt: dict | None = None, w_img: dict | None = None,
                  single: dict | None = None):
    """B images through one block, rows packed by stream: the text rows of all
    images first (image b's at txt_off[b]:txt_off[b+1]), then their image rows
    (image b's at T + img_off[b]:img_off[b+1], T = txt_off[-1]).  Each image
    is its own joint sequence [text_b; image_b] (Section 3.3.1 per image):
    its rows attend only to its own rows.  Returns (out [S, D], lse [H, S])
    in the packed row order."""
    x = _f64(x)
    pos = np.asarray(pos)
    S, D = x.shape
    T = int(txt_off[-1])
    out = np.empty_like(x)
    lse = np.empty((H, S))
    for b in range(len(txt_off) - 1):
        rows = np.concatenate([np.arange(txt_off[b], txt_off[b + 1]),
                               T + np.arange(img_off[b], img_off[b + 1])]).astype(np.int64)
        n_txt = int(txt_off[b + 1] - txt_off[b])
        if single is not None:
            o, l_ = single_block(x[rows], pos[rows], single, H)
        else:
            o, l_ = double_block(x[rows], pos[rows], n_txt, w_txt, w_img, H)
        out[rows] = o
        lse[:, rows] = l_
    return out, lse
