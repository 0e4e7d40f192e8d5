"""Pins of the oracle's sampler-side pieces: the Euler rule of Eq. euler
(Section 3.1), the latent embedder and the output layer around the blocks.

The Euler pins use closed forms of the ODE and of the Euler recurrence; the
output layer is pinned by layer-norm invariants and a hand-worked row; the
linear map by an explicit loop on a tiny case."""
import math

import numpy as np
import pytest

import oracle


def test_euler_linear_ode_closed_form_and_first_order():
    # dz/dt = lam z from t = 1 to t = 0: Euler gives (1 + lam dt)^n z0 exactly,
    # and the error against exp(-lam) z0 shrinks like dt (first order).
    lam, z0 = 0.7, np.array([1.0, -2.0, 0.5])
    errs = []
    for n in (8, 16, 32, 64):
        z = oracle.euler_integrate(z0, lambda z, t: lam * z, 1.0, 0.0, n)
        np.testing.assert_allclose(z, (1.0 - lam / n) ** n * z0, rtol=1e-13)
        errs.append(np.abs(z - math.exp(-lam) * z0).max())
    ratios = [errs[i] / errs[i + 1] for i in range(3)]
    assert all(1.8 < r < 2.2 for r in ratios), ratios


def test_euler_straight_flow_reaches_the_data():
    # Rectified flow: x_t = (1 - t) x0 + t noise has the constant velocity
    # noise - x0, so Euler from the noise at t = 1 lands on x0 at t = 0 in any
    # number of steps (dt = -1/n).
    g = np.random.default_rng(0)
    x0, noise = g.standard_normal((5, 4)), g.standard_normal((5, 4))
    for n in (1, 3, 28):
        z = oracle.euler_integrate(noise, lambda z, t: noise - x0, 1.0, 0.0, n)
        np.testing.assert_allclose(z, x0, atol=1e-12)


def test_euler_update_sign_and_zero_step():
    z, v = np.array([1.0, 2.0]), np.array([10.0, -4.0])
    np.testing.assert_array_equal(oracle.euler_update(z, v, 0.0), z)
    np.testing.assert_allclose(oracle.euler_update(z, v, -0.25), [-1.5, 3.0])


def test_linear_explicit_loop():
    g = np.random.default_rng(1)
    x, w, b = g.standard_normal((3, 5)), g.standard_normal((4, 5)), g.standard_normal(4)
    want = np.zeros((3, 4))
    for m in range(3):
        for n in range(4):
            want[m, n] = b[n] + sum(x[m, k] * w[n, k] for k in range(5))
    np.testing.assert_allclose(oracle.linear(x, w, b), want, rtol=1e-13)
    np.testing.assert_allclose(oracle.linear(x, np.eye(5)), x)


def test_final_layer_hand_worked_row():
    # Row (1, 2, 3, 4): mean 2.5, biased variance 1.25, so LN = (-1.5, -0.5,
    # 0.5, 1.5) / sqrt(1.25 + 1e-6); identity map, no modulation.
    x = np.array([[1.0, 2.0, 3.0, 4.0]])
    got = oracle.final_layer(x, np.zeros(4), np.zeros(4), np.eye(4))
    np.testing.assert_allclose(got[0], np.array([-1.5, -0.5, 0.5, 1.5]) / math.sqrt(1.25 + 1e-6), rtol=1e-12)


def test_final_layer_invariants():
    g = np.random.default_rng(2)
    D, C = 16, 8
    x = g.standard_normal((6, D)) * 3.0
    shift, scale = g.standard_normal(D), g.standard_normal(D)
    w, b = g.standard_normal((C, D)), g.standard_normal(C)
    y = oracle.final_layer(x, shift, scale, w, b)
    # Per-row shift and positive scale of the input leave the layer norm unchanged.
    np.testing.assert_allclose(oracle.final_layer(x * 2.5 + g.standard_normal((6, 1)), shift, scale, w, b), y,
                               rtol=1e-5, atol=1e-6)
    # scale = -1 removes the normalised term: every row maps to w shift + b.
    flat = oracle.final_layer(x, shift, -np.ones(D), w, b)
    np.testing.assert_allclose(flat, np.broadcast_to(w @ shift + b, flat.shape), rtol=1e-12)
    # Identity map, no modulation: rows of zero mean and (nearly) unit variance.
    h = oracle.final_layer(x, np.zeros(D), np.zeros(D), np.eye(D))
    np.testing.assert_allclose(h.mean(axis=1), 0.0, atol=1e-12)
    np.testing.assert_allclose(h.var(axis=1), 1.0, rtol=1e-5)
