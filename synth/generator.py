"""Seeded synthetic inputs shared by the GPU path and the oracle.

Every tensor is drawn in fp64 from its own PCG64 stream,
``numpy.random.default_rng([seed, tensor_id])``, and rounded to the workload's
storage type (fp32, or fp32 then bf16, round-to-nearest-even at each step).
The returned arrays are float32 holding exactly the values both sides see;
a bf16 array converts to torch.bfloat16 without further rounding.

Distributions (the paper's Figure 2 motivates the long tail of the temporal
signal; nothing here is trained):
  * hidden states, low-res latent, text and reference tokens: N(0, 1);
  * previous-step features: feat_prev = feat_t + eps_i * z_i with z ~ N(0, 1)
    and a per-token eps_i ~ LogNormal(-2, 1);
  * post-norm/RoPE queries and keys used for scoring: N(0, 1);
  * projection weights: N(0, std) with std = 0.02 or 1/sqrt(fan_in);
    biases and modulation shifts/scales N(0, 0.02); gates and RMSNorm
    gains 1 + N(0, 0.02).

This module holds no arithmetic of the method itself.
"""
from __future__ import annotations

import numpy as np

from .configs import Workload

# Fixed stream ids per named tensor.
_TID = {
    "text": 1, "ref": 2, "lowres": 3, "feat_t": 4, "z": 5, "eps": 6,
    "latent_q": 7, "text_k": 8, "latent_k": 9, "ref_k": 10,
    "x_block": 11, "sel_perm": 12, "scores_dup": 13,
}


def rng(seed: int, tensor_id: int) -> np.random.Generator:
    return np.random.default_rng([seed, tensor_id])


def _bf16_rne_u32(x32: np.ndarray) -> np.ndarray:
    """float32 bits rounded to bf16 (RNE), left in the low 16 bits of uint32
    (computed in place on one temporary: weights run to 10^8 elements)."""
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    r = u >> np.uint32(16)
    r &= np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r >>= np.uint32(16)
    return r


def to_bf16_bits(x32: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of float32 values rounded to bf16 (RNE)."""
    return _bf16_rne_u32(x32).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round fp64 draws to the storage type; returns float32."""
    x32 = np.asarray(x, dtype=np.float64).astype(np.float32)
    if dtype == "f32":
        return x32
    if dtype == "bf16":
        r = _bf16_rne_u32(x32)
        r <<= np.uint32(16)
        return r.view(np.float32)
    raise ValueError(dtype)


def normal(seed: int, tid: int, shape, dtype: str, std: float = 1.0,
           mean: float = 0.0) -> np.ndarray:
    g = rng(seed, tid)
    x = g.standard_normal(size=shape)
    if std != 1.0:
        x *= std
    if mean != 0.0:
        x += mean
    return round_to(x, dtype)


def feature_pair(seed: int, N: int, Df: int, dtype: str):
    """(feat_t, feat_prev, eps): consecutive-step features with per-token drift."""
    feat_t = normal(seed, _TID["feat_t"], (N, Df), dtype)
    z = rng(seed, _TID["z"]).standard_normal(size=(N, Df))
    eps = rng(seed, _TID["eps"]).lognormal(mean=-2.0, sigma=1.0, size=N)
    feat_prev = round_to(feat_t.astype(np.float64) + eps[:, None] * z, dtype)
    return feat_t, feat_prev, eps


def score_inputs(w: Workload) -> dict:
    """Inputs of the scoring stage (all [rows, H, d] or [rows, D_f])."""
    s, dt = w.seed, w.dtype
    feat_t, feat_prev, eps = feature_pair(s, w.N, w.Df, dt)
    return {
        "latent_q": normal(s, _TID["latent_q"], (w.N, w.H, w.d), dt),
        "text_k": normal(s, _TID["text_k"], (w.L, w.H, w.d), dt),
        "latent_k": normal(s, _TID["latent_k"], (w.N, w.H, w.d), dt),
        "ref_k": normal(s, _TID["ref_k"], (w.R, w.H, w.d), dt),
        "feat_t": feat_t,
        "feat_prev": feat_prev,
        "eps": eps,
    }


def layout_inputs(w: Workload, feat_t: np.ndarray | None = None) -> dict:
    """Low-res latent, high-res features of the previous step, text and ref rows.

    When the temporal features are the hidden states (D_f == D), the high-res
    features of the previous step are the same array as feat_t.
    """
    s, dt = w.seed, w.dtype
    if feat_t is not None and feat_t.shape == (w.N, w.D):
        highres = feat_t
    else:
        highres = normal(s, _TID["feat_t"] + 100, (w.N, w.D), dt)
    return {
        "lowres": normal(s, _TID["lowres"], (w.N_lr, w.D), dt),
        "highres_prev": highres,
        "text": normal(s, _TID["text"], (w.L, w.D), dt),
        "ref": normal(s, _TID["ref"], (w.R, w.D), dt),
    }


def prefix_positions(w: Workload) -> np.ndarray:
    """Position ids (frame, row, col) of the always-kept prefix rows.

    Text rows sit at (0, 0, 0); reference-image rows at (1, r, c) on a grid
    W_hr wide, in raster order.
    """
    pos = np.zeros((w.LR, 3), dtype=np.int32)
    if w.R:
        i = np.arange(w.R)
        pos[w.L:, 0] = 1
        pos[w.L:, 1] = i // w.W_hr
        pos[w.L:, 2] = i % w.W_hr
    return pos


# ---------------------------------------------------------------------------
# Block weights (PyTorch Linear layout: W[out, in]).

DOUBLE_PARAMS = ("mod", "w_qkv", "b_qkv", "g_q", "g_k", "w_o", "b_o",
                 "w_mlp1", "b_mlp1", "w_mlp2", "b_mlp2")
SINGLE_PARAMS = ("mod", "w_in", "b_in", "g_q", "g_k", "w_out", "b_out")


def _wstd(w: Workload, fan_in: int) -> float:
    return w.weight_std if w.weight_std is not None else 1.0 / np.sqrt(fan_in)


def _mod(seed: int, tid: int, n_vec: int, D: int, dtype: str) -> np.ndarray:
    """Modulation vectors: (shift, scale, gate) triples; gates centred at 1."""
    x = rng(seed, tid).standard_normal(size=(n_vec, D)) * 0.02
    x[2::3] += 1.0
    return round_to(x, dtype)


def double_stream_weights(w: Workload, block: int, stream: int) -> dict:
    """Weights of one stream (0 text, 1 image) of double block ``block``."""
    D, d, dt, s = w.D, w.d, w.dtype, w.seed
    F = w.mlp_ratio * D
    base = 1000 + 200 * block + 100 * stream
    return {
        "mod": _mod(s, base + 0, 6, D, dt),
        "w_qkv": normal(s, base + 1, (3 * D, D), dt, _wstd(w, D)),
        "b_qkv": normal(s, base + 2, (3 * D,), dt, 0.02),
        "g_q": normal(s, base + 3, (d,), dt, 0.02, 1.0),
        "g_k": normal(s, base + 4, (d,), dt, 0.02, 1.0),
        "w_o": normal(s, base + 5, (D, D), dt, _wstd(w, D)),
        "b_o": normal(s, base + 6, (D,), dt, 0.02),
        "w_mlp1": normal(s, base + 7, (F, D), dt, _wstd(w, D)),
        "b_mlp1": normal(s, base + 8, (F,), dt, 0.02),
        "w_mlp2": normal(s, base + 9, (D, F), dt, _wstd(w, F)),
        "b_mlp2": normal(s, base + 10, (D,), dt, 0.02),
    }


def single_block_weights(w: Workload, block: int) -> dict:
    D, d, dt, s = w.D, w.d, w.dtype, w.seed
    F = w.mlp_ratio * D
    base = 100000 + 100 * block
    return {
        "mod": _mod(s, base + 0, 3, D, dt),
        "w_in": normal(s, base + 1, (3 * D + F, D), dt, _wstd(w, D)),
        "b_in": normal(s, base + 2, (3 * D + F,), dt, 0.02),
        "g_q": normal(s, base + 3, (d,), dt, 0.02, 1.0),
        "g_k": normal(s, base + 4, (d,), dt, 0.02, 1.0),
        "w_out": normal(s, base + 5, (D, D + F), dt, _wstd(w, D + F)),
        "b_out": normal(s, base + 6, (D,), dt, 0.02),
    }


LATENT_CHANNELS = 64  # FLUX's packed latent: 16 channels x a 2x2 patch


def sampler_weights(w: Workload, C: int = LATENT_CHANNELS) -> dict:
    """The model's latent embedder (C -> D) and output layer (D -> C) around
    the blocks: embed_w [D, C], embed_b [D], final_mod [2, D] (shift; scale),
    final_w [C, D], final_b [C]."""
    D, dt, s = w.D, w.dtype, w.seed
    base = 300000
    return {
        "embed_w": normal(s, base + 1, (D, C), dt, _wstd(w, C)),
        "embed_b": normal(s, base + 2, (D,), dt, 0.02),
        "final_mod": _mod(s, base + 3, 2, D, dt),
        "final_w": normal(s, base + 4, (C, D), dt, _wstd(w, D)),
        "final_b": normal(s, base + 5, (C,), dt, 0.02),
    }


def selected_latents(w: Workload, k: int, C: int = LATENT_CHANNELS, tid_offset: int = 0) -> np.ndarray:
    """Latents of k selected tokens [k, C] ~ N(0, 1) (a noisy latent)."""
    return normal(w.seed, 300100 + tid_offset, (k, C), w.dtype)


def block_input(w: Workload, n_rows: int, tid_offset: int = 0) -> np.ndarray:
    """A stand-alone block input [n_rows, D] ~ N(0, 1)."""
    return normal(w.seed, _TID["x_block"] + tid_offset, (n_rows, w.D), w.dtype)


def random_selection(w: Workload, k: int, tid_offset: int = 0) -> np.ndarray:
    """k distinct high-res indices in ascending order (a stand-in selection)."""
    g = rng(w.seed, _TID["sel_perm"] + tid_offset)
    return np.sort(g.permutation(w.N)[:k]).astype(np.int32)


def random_lowres_selection(w: Workload, k: int, tid_offset: int = 0) -> np.ndarray:
    """k distinct low-res indices in ascending order (a stand-in selection at
    the low-res granularity of the mixed-resolution sequence)."""
    g = rng(w.seed, _TID["sel_perm"] + 50 + tid_offset)
    return np.sort(g.permutation(w.N_lr)[:k]).astype(np.int32)


def tiebreak_noise(seed: int, n: int, std: float = 1e-6) -> np.ndarray:
    """Seeded Gaussian perturbation for the selection's tie-break, fp32."""
    g = rng(seed, _TID["scores_dup"] + 1)
    return (g.standard_normal(size=n) * std).astype(np.float32)


def quantised_scores(seed: int, n: int, levels: int) -> np.ndarray:
    """fp32 scores with heavy duplicates: ``levels`` distinct values in [0, 1)."""
    g = rng(seed, _TID["scores_dup"])
    return (g.integers(0, levels, size=n) / float(levels)).astype(np.float32)
