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
