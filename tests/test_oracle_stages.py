"""Pins of the oracle's three-stage sampler (Section 3.2 around the hot
path): time grid, the collected text mass, the Euler step, and the two
stage transitions with their coordinate-bound noise."""
import numpy as np

import oracle
from oracle import sampler as sp
from synth import configs as C
from synth import generator as G

W = C.TINY_F32.replace(D=64, H=2, d=32, L=6, H_lr=4, W_lr=3)   # tiny: hidden 64, 2 heads, 4x3 -> 8x6


def _model(w, n_double=1, n_single=1, Cc=8):
    doubles = [(G.double_stream_weights(w, b, 0), G.double_stream_weights(w, b, 1)) for b in range(n_double)]
    singles = [G.single_block_weights(w, b) for b in range(n_single)]
    sw = G.sampler_weights(w, Cc)
    return doubles, singles, sw


def test_timesteps():
    t = sp.timesteps(8)
    assert t[0] == 1.0 and t[-1] == 0.0 and t.size == 9
    np.testing.assert_allclose(np.diff(t), -0.125, rtol=1e-12)


def test_collected_mass_with_constant_keys_is_the_text_fraction():
    # Zero key projections give all-zero keys after the norm: every softmax
    # row is uniform, so each head's text mass is L / S for every row.
    w = W
    doubles, singles, _ = _model(w, n_double=2, n_single=0)
    for wt, wi in doubles:
        for s in (wt, wi):
            s["w_qkv"] = s["w_qkv"].copy()
            s["w_qkv"][w.D:2 * w.D] = 0.0
            s["b_qkv"] = s["b_qkv"].copy()
            s["b_qkv"][w.D:2 * w.D] = 0.0
    S = 20
    x = G.block_input(w, S)
    pos = np.zeros((S, 3), np.int32)
    _, mass = sp.run_blocks(x, pos, w.L, doubles, singles, w.H, collect=True)
    np.testing.assert_allclose(mass, 2 * w.L / S, rtol=1e-12)      # two blocks summed


def test_euler_step_is_linear_in_dt():
    w = W
    doubles, singles, sw = _model(w)
    z = G.normal(w.seed, 900, (12, 8), "f32")
    prefix = G.block_input(w, w.L, 3)
    pos = np.concatenate([np.zeros((w.L, 3), np.int32), sp.lowres_positions(4, 3)])
    z0, v0, _ = sp.denoise_step(z, prefix, pos, sw, doubles, singles, w.H, 0.0)
    np.testing.assert_array_equal(z0, z)
    z1, v1, _ = sp.denoise_step(z, prefix, pos, sw, doubles, singles, w.H, -0.25)
    np.testing.assert_array_equal(v1, v0)                     # the velocity does not depend on dt
    np.testing.assert_allclose(z1 - z, -0.25 * v0, rtol=1e-12, atol=1e-14)


def test_transitions_without_noise_give_the_nearest_upsampling():
    # t_s = 0 and v = 0: expanding the selected tokens, keeping the rest, then
    # expanding those too rebuilds the 2x nearest upsampling of the low-res
    # latent, whatever the selection.
    H_lr, W_lr, Cc = 4, 3, 8
    z = G.normal(1, 901, (H_lr * W_lr, Cc), "f32")
    want = np.repeat(np.repeat(z.reshape(H_lr, W_lr, Cc), 2, 0), 2, 1).reshape(-1, Cc)
    for idx in (np.array([], np.int64), np.array([0, 5, 11]), np.arange(12)):
        body, pos, children = oracle.gather_mixed(z, None, idx, H_lr, W_lr)
        z_hr = sp.transition23(body, np.zeros_like(body), 0.0, idx, children, H_lr, W_lr, Cc, seed=5)
        np.testing.assert_array_equal(z_hr, want)


def test_noise_is_the_same_field_in_both_stages():
    # Pure noise at both boundaries (t = 1): a pixel's noise in the mixed
    # sequence equals its noise on the full grid, and a kept token's noise is
    # the scaled mean of its four pixels' noise there.
    H_lr, W_lr, Cc, seed, K = 4, 3, 8, 17, 5
    Mp = H_lr * W_lr
    snaps = G.normal(2, 902, (2, Mp, Cc), "f32")
    mass = np.abs(G.normal(2, 903, (2, Mp), "f32"))
    z = snaps[-1]
    s, idx, z_mix, pos, children = sp.transition12(z, np.zeros_like(z), 1.0, mass, 1, snaps, K, H_lr, W_lr, Cc,
                                                   seed, alpha=0.5)
    z_hr = sp.transition23(z_mix, np.zeros_like(z_mix), 1.0, idx, children, H_lr, W_lr, Cc, seed)
    W_hr = 2 * W_lr
    for j, (Y, X) in enumerate(pos[:, 1:]):
        if Y % 2 == 0:
            np.testing.assert_array_equal(z_mix[j], z_hr[(Y // 2) * W_hr + X // 2])
        else:
            r, c = (Y - 1) // 4, (X - 1) // 4
            kids = [(2 * r + a) * W_hr + 2 * c + b for a in (0, 1) for b in (0, 1)]
            np.testing.assert_allclose(z_mix[j], z_hr[kids].mean(axis=0) * 2.0, rtol=1e-12, atol=1e-12)
    assert idx.size == K and np.all(np.diff(idx) > 0)
    np.testing.assert_array_equal(idx, oracle.select_topk(s, K))


def test_three_stages_run_end_to_end():
    w = W
    doubles, singles, sw = _model(w)
    n1, nt, n2, n3 = 1, 2, 1, 1
    t = sp.timesteps(n1 + nt + n2 + n3)
    prefix = G.block_input(w, w.L, 4)
    ppos = np.zeros((w.L, 3), np.int32)
    H_lr, W_lr, Cc, K = 4, 3, 8, 4
    z, v, snaps, mass, count = sp.stage1(prefix, ppos, sw, doubles, singles, w.H, H_lr, W_lr, Cc, 3, t, n1, nt)
    assert snaps.shape == (nt, 12, Cc) and count == nt * len(doubles)
    np.testing.assert_array_equal(snaps[-1], z)
    assert np.all(mass >= 0) and np.all(mass <= count + 1e-12)
    s, idx, z_mix, pos, children = sp.transition12(z, v, t[n1 + nt], mass, count, snaps, K, H_lr, W_lr, Cc, 3, 0.5)
    assert z_mix.shape == (3 * K + 12, Cc)
    z2, v2 = sp.stage_steps(z_mix, prefix, np.concatenate([2 * ppos, pos]), sw, doubles, singles, w.H, t,
                            n1 + nt, n2, pos_scale=0.5)
    z_hr = sp.transition23(z2, v2, t[n1 + nt + n2], idx, children, H_lr, W_lr, Cc, 3)
    z3, _ = sp.stage_steps(z_hr, prefix, np.concatenate([ppos, sp.highres_positions(8, 6)]), sw, doubles, singles,
                           w.H, t, n1 + nt + n2, n3)
    assert z3.shape == (48, Cc) and np.all(np.isfinite(z3))


def test_clean_estimate_uses_the_last_velocity():
    # A velocity that points exactly at a zero clean latent (v = z / t) leaves
    # only the re-injected noise: t times the coordinate-bound field.
    H_lr, W_lr, Cc, seed, K, t_s = 4, 3, 8, 23, 4, 0.375
    Mp = H_lr * W_lr
    z = G.normal(3, 904, (Mp, Cc), "f32").astype(np.float64)
    snaps = np.stack([z, z + 0.1])
    mass = np.ones((2, Mp))
    _, idx, z_mix, pos, children = sp.transition12(z, z / t_s, t_s, mass, 1, snaps, K, H_lr, W_lr, Cc, seed, 0.5)
    np.testing.assert_allclose(z_mix, t_s * oracle.halfunit_noise(pos, 2 * W_lr, Cc, seed), rtol=1e-12, atol=1e-12)
    z_hr = sp.transition23(z_mix, z_mix / t_s, t_s, idx, children, H_lr, W_lr, Cc, seed)
    np.testing.assert_allclose(z_hr, t_s * oracle.pixel_noise(np.arange(4 * Mp), Cc, seed), rtol=1e-12, atol=1e-12)


def test_stage1_collects_the_image_rows_of_the_last_steps():
    w = W
    doubles, singles, sw = _model(w, n_double=2, n_single=0)
    t = sp.timesteps(4)
    prefix = G.block_input(w, w.L, 6)
    ppos = np.zeros((w.L, 3), np.int32)
    z, v, snaps, mass, count = sp.stage1(prefix, ppos, sw, doubles, singles, w.H, 4, 3, 8, 3, t, 2, 2)
    # Recompute the four steps one by one: the last two steps' image-row masses, summed.
    zz = oracle.block_noise(np.arange(12), 3, 8, 3)
    pos = np.concatenate([ppos, sp.lowres_positions(4, 3)])
    want = np.zeros_like(mass)
    for i in range(4):
        zz, _, m = sp.denoise_step(zz, prefix, pos, sw, doubles, singles, w.H, t[i + 1] - t[i], collect=True)
        if i >= 2:
            want += m[:, w.L:]
            np.testing.assert_array_equal(snaps[i - 2], zz)
    np.testing.assert_allclose(mass, want, rtol=1e-12)
    assert count == 4
