"""Spatiotemporal token importance (paper Section 3.3), fp64.

Test infrastructure: used only by tests, the smoke check and the CPU baseline.
"""
from __future__ import annotations

import numpy as np


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def joint_lse(q, k_all, row_chunk: int = 1024):
    """Log-sum-exp of each query's logits over the joint key set.

    Section 3.3.1, Eq. dit_attn: the attention weights are the softmax of
    P = Q K^T / sqrt(d_h) over all keys of the joint sequence.  For image query
    i in head h this returns lse[h, i] = log sum_j exp(P[h, i, j]), natural
    log, j over every key row of ``k_all``.

    q: [N, H, d]; k_all: [Nk, H, d] (text, then reference, then image keys).
    Returns [H, N] fp64.
    """
    q, k_all = _f64(q), _f64(k_all)
    N, H, d = q.shape
    out = np.empty((H, N))
    scale = 1.0 / np.sqrt(d)
    for h in range(H):
        kh = k_all[:, h, :]
        for r0 in range(0, N, row_chunk):
            p = (q[r0:r0 + row_chunk, h, :] @ kh.T) * scale
            m = p.max(axis=1, keepdims=True)
            out[h, r0:r0 + row_chunk] = m[:, 0] + np.log(np.exp(p - m).sum(axis=1))
    return out


def spatial_importance(q, k_txt, row_lse):
    """Spatial importance A_i (Section 3.3.1, Eq. spatial with Eq. dit_attn).

    A_i = (1/|H|) sum_h sum_{j < L} alpha_ij^(h), where alpha is the joint
    softmax restricted to image rows and text columns.  With the joint
    log-sum-exp given, alpha_ij^(h) = exp(q_ih . k_jh / sqrt(d) - lse[h, i]).

    Readings: the softmax denominator runs over the joint key set (text,
    reference and image keys), as Eq. dit_attn takes the softmax of the full
    P before selecting the image->text block; all heads are averaged
    uniformly; q and k are taken after the model's QK-normalisation and RoPE.

    q: [N, H, d]; k_txt: [L, H, d]; row_lse: [H, N].  Returns A [N] fp64.
    """
    q, k_txt, row_lse = _f64(q), _f64(k_txt), _f64(row_lse)
    N, H, d = q.shape
    scale = 1.0 / np.sqrt(d)
    acc = np.zeros(N)
    for h in range(H):
        p = (q[:, h, :] @ k_txt[:, h, :].T) * scale          # [N, L]
        acc += np.exp(p - row_lse[h][:, None]).sum(axis=1)
    return acc / H


def spatial_importance_bruteforce(q, k_all, L: int):
    """A_i from the full per-head softmax over ``k_all`` (text keys first).

    Forms the whole attention matrix, normalises each row, keeps the first L
    columns and averages over heads (Eq. spatial, Eq. dit_attn) without a
    precomputed log-sum-exp.  Small inputs only.
    """
    q, k_all = _f64(q), _f64(k_all)
    N, H, d = q.shape
    acc = np.zeros(N)
    for h in range(H):
        p = (q[:, h, :] @ k_all[:, h, :].T) / np.sqrt(d)
        p = np.exp(p - p.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        acc += p[:, :L].sum(axis=1)
    return acc / H


def text_attention_mass(q, k_all, L: int, row_chunk: int = 1024):
    """Per-head image-to-text attention mass (Eq. spatial before the head
    mean, with the softmax of Eq. dit_attn over the joint key set).

    mass[h, i] = sum_{j < L} softmax_j(q_ih . k_jh / sqrt(d)), the softmax
    taken over every row of ``k_all`` (text keys first).  q: [N, H, d];
    k_all: [Nk, H, d].  Returns [H, N] fp64.
    """
    q, k_all = _f64(q), _f64(k_all)
    N, H, d = q.shape
    out = np.empty((H, N))
    scale = 1.0 / np.sqrt(d)
    for h in range(H):
        kh = k_all[:, h, :]
        for r0 in range(0, N, row_chunk):
            p = (q[r0:r0 + row_chunk, h, :] @ kh.T) * scale
            e = np.exp(p - p.max(axis=1, keepdims=True))
            out[h, r0:r0 + row_chunk] = e[:, :L].sum(axis=1) / e.sum(axis=1)
    return out


def step_variance(snapshots):
    """Temporal importance V_i (Section 3.3.2, Eqs. zbar and step_var).

    snapshots: [N_T, N, D_f], the token features at N_T consecutive steps.
    zbar = mean over steps; V_i = mean over channels of the unbiased
    (divisor N_T - 1) variance across steps.  Returns [N] fp64.
    """
    z = _f64(snapshots)
    n_t = z.shape[0]
    if n_t < 2:
        raise ValueError("step variance needs at least two snapshots")
    zbar = z.mean(axis=0)
    var = ((z - zbar[None]) ** 2).sum(axis=0) / (n_t - 1)
    return var.mean(axis=1)


def minmax_normalise(x, eps: float):
    """Min-max normalisation of Section 3.3.3: (x - min) / (max - min + eps).

    The paper does not print eps; the default used across this project is
    1e-8 (a constant score vector then maps to all zeros).
    """
    x = _f64(x)
    lo, hi = x.min(), x.max()
    return (x - lo) / (hi - lo + eps)


def joint_score(a, v, alpha: float, eps: float):
    """Fused score S_i = alpha * A_hat_i + (1 - alpha) * V_hat_i (Eq. joint)."""
    return alpha * minmax_normalise(a, eps) + (1.0 - alpha) * minmax_normalise(v, eps)


def score(latent_q, text_k, row_lse, feat_t, feat_prev, alpha: float, eps: float = 1e-8):
    """The scoring stage: (S as fp32, A fp64, V fp64).

    The two snapshots are the previous and the current step (N_T = 2).  The
    fused score is returned rounded to fp32, the type the selection sorts on.
    """
    a = spatial_importance(latent_q, text_k, row_lse)
    v = step_variance(np.stack([_f64(feat_prev), _f64(feat_t)]))
    s = joint_score(a, v, alpha, eps)
    return s.astype(np.float32), a, v


def score_from_mass(mass_sum, count: int, snapshots, alpha: float, eps: float = 1e-8):
    """The scoring stage from aggregated attention masses: (S fp32, A, V).

    mass_sum: [H, N], the sum of ``count`` per-head text masses (probes of
    several blocks or steps, Section 3.3.1); A is their mean over heads and
    probes.  snapshots: [N_T, N, D_f] for the step variance (Section 3.3.2).
    """
    mass_sum = _f64(mass_sum)
    a = mass_sum.sum(axis=0) / (mass_sum.shape[0] * count)
    v = step_variance(snapshots)
    s = joint_score(a, v, alpha, eps)
    return s.astype(np.float32), a, v
