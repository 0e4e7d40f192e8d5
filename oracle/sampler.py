"""Around the path: the Stage-2 denoising step on the selected tokens.

TEST INFRASTRUCTURE ONLY (see the package docstring).  fp64 NumPy.

Section 3.1 integrates the flow-matching ODE with Euler steps (Eq. euler):
the latent moves by the velocity times the signed step dt.  In Stage 2
(Section 3.2) only the selected tokens are denoised, so the update applies to
their rows alone; the model's velocity for those rows comes from the blocks
through its output layer.  The latent embedder and the output layer are the
model's, not the paper's: here FLUX-style, a linear map into the hidden width,
and a modulated layer norm followed by a linear map back to the latent
channels (the same layer norm as the block's).
"""
import numpy as np

from .block import layer_norm


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def linear(x, w, b=None):
    """x w^T + b: x [M, K], w [N, K], b [N] or None."""
    y = _f64(x) @ _f64(w).T
    return y if b is None else y + _f64(b)


def final_layer(x, shift, scale, w, b=None):
    """Output layer: LN(x) (1 + scale) + shift, then the linear map to the
    latent channels.  x [M, D], shift / scale [D], w [C, D], b [C]."""
    h = layer_norm(x) * (1.0 + _f64(scale)) + _f64(shift)
    return linear(h, w, b)


def euler_update(z, v, dt: float):
    """One step of Eq. euler: z + dt v (dt negative from t = 1 towards 0)."""
    return _f64(z) + float(dt) * _f64(v)


def euler_integrate(z0, velocity, t0: float, t1: float, n_steps: int):
    """n_steps uniform Euler steps of dz/dt = velocity(z, t) from t0 to t1."""
    z = _f64(z0)
    dt = (t1 - t0) / n_steps
    t = t0
    for _ in range(n_steps):
        z = euler_update(z, velocity(z, t), dt)
        t += dt
    return z


# ---------------------------------------------------------------------------
# The three-stage dynamic-resolution sampler of Section 3.2 (Fig. 3a), on
# random weights: Stage 1 denoises the low-resolution latent and, over its
# last N_T steps, collects the latent snapshots and the blocks' text
# attention mass; Stage 2 scores and selects K = floor(rho M') low-res
# tokens, expands them 2x2 and keeps the rest at low resolution in one
# mixed sequence, re-injects coordinate-bound noise and denoises it; Stage 3
# expands the remaining tokens, re-injects the noise, reorders by coordinate
# and denoises the full grid.  Readings (the paper defers them to prior
# practice or leaves them open): a uniform time grid t_i = 1 - i / n over the
# n = N_1 + N_T + N_2 + N_3 steps; the blocks' modulation does not depend on
# t (random weights); the mass is summed over every double block of each
# collection step; the clean estimate at a stage boundary is x - t v with the
# last velocity; re-injection is oracle.noise.reinject at the boundary's t.

def timesteps(n_steps: int):
    """t_0 = 1 > t_1 > ... > t_n = 0, uniform (Eq. euler's Delta t_i < 0)."""
    return np.linspace(1.0, 0.0, n_steps + 1)


def run_blocks(x, pos, n_txt: int, doubles, singles, H: int, collect: bool = False):
    """The block stack on x [S, D] (positions pos [S, 3], real): the double
    blocks (each a (w_txt, w_img) pair), then the single blocks.  With
    collect, also the per-head text mass of every row summed over the double
    blocks, each taken on that block's own normalised, rotated q and k
    (Section 3.3.1).  Returns (x, mass [H, S] or None)."""
    from .block import block_qk, double_block, single_block
    from .importance import text_attention_mass
    x = _f64(x)
    mass = np.zeros((H, x.shape[0])) if collect else None
    for wt, wi in doubles:
        if collect:
            q, k = block_qk(x, pos, n_txt, wt, wi, H)
            mass += text_attention_mass(q, k, n_txt)
        x, _ = double_block(x, pos, n_txt, wt, wi, H)
    for ws in singles:
        x, _ = single_block(x, pos, ws, H)
    return x, mass


def denoise_step(z, prefix, pos, sw: dict, doubles, singles, H: int, dt: float, collect: bool = False):
    """One Euler step (Eq. euler) of the image latents z [n, C] behind the
    prefix rows [L, D]: h = embed(z), the blocks on [prefix; h] at pos, the
    velocity from the output layer on the image rows, z + dt v.  Returns
    (z_next, v, mass [H, L + n] or None)."""
    L = np.asarray(prefix).shape[0]
    x = np.concatenate([_f64(prefix), linear(z, sw["embed_w"], sw["embed_b"])])
    x, mass = run_blocks(x, pos, L, doubles, singles, H, collect)
    mod = _f64(sw["final_mod"])
    v = final_layer(x[L:], mod[0], mod[1], sw["final_w"], sw["final_b"])
    return euler_update(z, v, dt), v, mass


def lowres_positions(H_lr: int, W_lr: int):
    """(0, r, c) for the low-res grid in raster order (Stage 1's tokens)."""
    r = np.arange(H_lr * W_lr)
    return np.stack([np.zeros_like(r), r // W_lr, r % W_lr], axis=1).astype(np.int32)


def stage1(prefix, prefix_pos, sw, doubles, singles, H: int, H_lr: int, W_lr: int, C: int, seed: int, t,
           n1: int, nt: int, z0=None):
    """Stage 1: the low-res latent from the downsampled initial noise (or z0),
    n1 + nt Euler steps; over the last nt, the snapshots (the latent after
    each step) and the text mass of the image rows summed over the double
    blocks.  Returns (z, v_last, snapshots [nt, M', C], mass [H, M'], count)."""
    from .noise import block_noise
    Mp = H_lr * W_lr
    L = np.asarray(prefix).shape[0]
    z = block_noise(np.arange(Mp), W_lr, C, seed) if z0 is None else _f64(z0)
    pos = np.concatenate([np.asarray(prefix_pos), lowres_positions(H_lr, W_lr)])
    snaps, mass = [], np.zeros((H, Mp))
    v = None
    for i in range(n1 + nt):
        collect = i >= n1
        z, v, m = denoise_step(z, prefix, pos, sw, doubles, singles, H, t[i + 1] - t[i], collect)
        if collect:
            snaps.append(z.copy())
            mass += m[:, L:]
    return z, v, np.stack(snaps), mass, nt * len(doubles)


def transition12(z, v, t_s: float, mass, count: int, snapshots, K: int, H_lr: int, W_lr: int, C: int, seed: int,
                 alpha: float, eps: float = 1e-8, idx=None):
    """Stage 1 -> 2: score the M' tokens from the collected signals (Eqs.
    spatial, step_var, joint), select the top K (Eq. topk; or take idx),
    form the clean estimate z - t_s v, build the mixed sequence (selected
    tokens expanded 2x2, the rest kept) and re-inject the coordinate-bound
    noise at t_s.  Returns (scores fp32, idx, z_mix [4K + M' - K, C], pos
    in half units, children)."""
    from .importance import score_from_mass
    from .noise import halfunit_noise, reinject
    from .relayout import gather_mixed
    from .selection import select_topk
    s, _, _ = score_from_mass(mass, count, snapshots, alpha, eps)
    if idx is None:
        idx = select_topk(s, K)
    x0 = euler_update(z, v, -t_s)
    body, pos, children = gather_mixed(x0, None, idx, H_lr, W_lr)
    z_mix = reinject(body, halfunit_noise(pos, 2 * W_lr, C, seed), t_s)
    return s, np.asarray(idx), z_mix, pos, children


def stage_steps(z, prefix, pos, sw, doubles, singles, H: int, t, i0: int, n: int, pos_scale: float = 1.0):
    """n Euler steps from t[i0] on the sequence [prefix; embed(z)] at
    positions pos * pos_scale.  Returns (z, v_last)."""
    pos = np.asarray(pos, dtype=np.float64) * pos_scale
    v = None
    for i in range(i0, i0 + n):
        z, v, _ = denoise_step(z, prefix, pos, sw, doubles, singles, H, t[i + 1] - t[i])
    return z, v


def transition23(z_mix, v, t_s: float, idx, children, H_lr: int, W_lr: int, C: int, seed: int):
    """Stage 2 -> 3: the clean estimate z_mix - t_s v, expanded rows to their
    pixels, kept rows to their low-res slots, the kept tokens expanded by 2x
    nearest upsampling around the expanded ones, the coordinate-bound noise
    re-injected at t_s; rows in raster order.  Returns z [N, C]."""
    from .noise import pixel_noise, reinject
    from .relayout import gather_upsample, scatter_mixed
    Mp = H_lr * W_lr
    x0 = euler_update(z_mix, v, -t_s)
    canvas, state = scatter_mixed(x0, idx, 0, H_lr, W_lr, np.zeros((4 * Mp, C)), np.zeros((Mp, C)))
    _, _, full = gather_upsample(state, canvas, None, children, H_lr, W_lr)
    return reinject(full, pixel_noise(np.arange(4 * Mp), C, seed), t_s)


def highres_positions(H_hr: int, W_hr: int):
    r = np.arange(H_hr * W_hr)
    return np.stack([np.zeros_like(r), r // W_hr, r % W_hr], axis=1).astype(np.int32)
