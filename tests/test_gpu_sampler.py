"""Parity of the sampler-side pieces around the path (Stage 2 of Section 3.2
with the Euler rule of Eq. euler): the latent embedder, the output layer, the
Euler update, and whole Stage-2 steps through SelectedEuler, each stage
checked against the oracle on the GPU's own inputs of that stage."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17995_amd.step import SelectedEuler
from synth import configs as C
from synth import generator as G

from _gpu import assert_close, dev, double_weights_dev, host

pytestmark = pytest.mark.gpu

CASES = [(C.TINY_F32, 37), (C.TINY_BF16, 37), (C.TINY_F32_RAGGED, 5), (C.FLUX_1024, C.FLUX_1024.k)]
IDS = ["f32", "bf16", "f32_ragged", "flux_1024"]


@pytest.mark.parametrize("w,k", CASES, ids=IDS)
def test_linear_embedder(gpu, w, k):
    sw = G.sampler_weights(w)
    z = G.selected_latents(w, k)
    out = torch.full((k, w.D), 7.0, dtype=torch.float32 if w.dtype == "f32" else torch.bfloat16, device="cuda")
    gpu.avits_linear(dev(z, w.dtype), dev(sw["embed_w"], w.dtype), dev(sw["embed_b"], w.dtype), out)
    torch.cuda.synchronize()
    assert_close(host(out), oracle.linear(z, sw["embed_w"], sw["embed_b"]), w.dtype, "embed")


@pytest.mark.parametrize("w,k", CASES, ids=IDS)
def test_final_layer(gpu, w, k):
    sw = G.sampler_weights(w)
    x = G.block_input(w, k, 9)
    # A strong modulation as well as the generator's near-identity one.
    g = np.random.default_rng(w.seed)
    for mod in (sw["final_mod"], G.round_to(g.standard_normal((2, w.D)) * 0.5, w.dtype)):
        out = torch.full((k, 64), 7.0, dtype=torch.float32 if w.dtype == "f32" else torch.bfloat16, device="cuda")
        gpu.avits_final_layer(dev(x, w.dtype), dev(mod, w.dtype), dev(sw["final_w"], w.dtype),
                              dev(sw["final_b"], w.dtype), out)
        torch.cuda.synchronize()
        ref = oracle.final_layer(x, mod[0], mod[1], sw["final_w"], sw["final_b"])
        assert_close(host(out), ref, w.dtype, "final layer")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n", [8, 1003, 1229 * 64])
def test_euler_update(gpu, dtype, n):
    g = np.random.default_rng(n)
    z = G.round_to(g.standard_normal(n), dtype)
    v = G.round_to(g.standard_normal(n) * 3.0, dtype)
    dt = float(np.float32(-1.0 / 28.0))  # the step as the entry point receives it (fp32)
    t = dev(z, dtype)
    gpu.avits_euler_update(t, dev(v, dtype), dt)
    torch.cuda.synchronize()
    ref = oracle.euler_update(z, v, dt)
    got = host(t)
    if dtype == "f32":
        np.testing.assert_allclose(got, ref, rtol=2 ** -23)     # one fp32 rounding (fma)
    else:  # the fp32 fma, then one rounding to bf16: within one bf16 ulp of the exact value
        assert np.all(np.abs(got - ref) <= np.abs(ref) * 2.0 ** -7 + 1e-30)
    t0 = dev(z, dtype)
    gpu.avits_euler_update(t0, dev(v, dtype), 0.0)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(t0), z)


@pytest.mark.parametrize("base", [C.TINY_F32, C.TINY_BF16, C.TINY_BF16_REF], ids=lambda w: w.name)
def test_selected_euler_steps(gpu, base):
    """Three Stage-2 steps on the selected tokens (one double and one single
    block), then the scatter into the latent canvas; every stage of every step
    is checked on the GPU's inputs of that stage (fp32: the max-abs 1e-4 bar)."""
    w = base
    k, L, R, C_ = w.k, w.L, w.R, G.LATENT_CHANNELS
    sw = G.sampler_weights(w)
    wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
    ws = G.single_block_weights(w, 0)
    doubles = [gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=double_weights_dev(wt, w.dtype),
                                img=double_weights_dev(wi, w.dtype))]
    singles = [gpu.BlockWeights(gpu.BLOCK_SINGLE, single=double_weights_dev(ws, w.dtype))]
    idx = G.random_selection(w, k, 4)
    pos = np.concatenate([G.prefix_positions(w), oracle.selected_positions(idx, 2 * w.W_lr)]).astype(np.int32)
    lay = G.layout_inputs(w)
    prefix = np.concatenate([lay["text"], lay["ref"]])
    step = SelectedEuler(k, L, R, C_, w.D, w.H, w.mlp_ratio * w.D, doubles, singles, dev(sw["embed_w"], w.dtype),
                         dev(sw["embed_b"], w.dtype), dev(sw["final_mod"], w.dtype), dev(sw["final_w"], w.dtype),
                         dev(sw["final_b"], w.dtype), pos, torch.float32 if w.dtype == "f32" else torch.bfloat16)
    z = dev(G.selected_latents(w, k), w.dtype)
    t_prefix = dev(prefix, w.dtype)
    seen = {}

    def on_block(i, x_in, x_out):
        torch.cuda.synchronize()
        seen[i] = host(x_in)

    dts = [-0.3, -0.25, -0.2]  # exact in fp32 up to the rounding the oracle is given too
    for n, dt in enumerate(dts):
        z_before = host(z)
        step.step(z, t_prefix, dt, on_block=on_block)
        torch.cuda.synchronize()
        x0 = seen[0]
        np.testing.assert_array_equal(x0[:L + R], prefix, err_msg=f"step {n} prefix rows")
        assert_close(x0[L + R:], oracle.linear(z_before, sw["embed_w"], sw["embed_b"]), w.dtype, f"step {n} embed")
        ref1, _ = oracle.double_block(x0, pos, L, wt, wi, w.H)
        assert_close(seen[1], ref1, w.dtype, f"step {n} double block")
        last = host(step.last)
        ref2, _ = oracle.single_block(seen[1], pos, ws, w.H)
        assert_close(last, ref2, w.dtype, f"step {n} single block")
        v_ref = oracle.final_layer(last[L + R:], sw["final_mod"][0], sw["final_mod"][1], sw["final_w"],
                                   sw["final_b"])
        v = host(step.v)
        assert_close(v, v_ref, w.dtype, f"step {n} velocity")
        ref_z = oracle.euler_update(z_before, v, float(np.float32(dt)))
        # One rounding of the fp32 fma, then (bf16) one rounding to bf16.
        ulp = 2.0 ** -23 if w.dtype == "f32" else 2.0 ** -7
        assert np.all(np.abs(host(z) - ref_z) <= np.abs(ref_z) * ulp + 1e-30), f"step {n} update"
    canvas = dev(G.round_to(np.random.default_rng(3).standard_normal((w.N, C_)), w.dtype), w.dtype)
    before = host(canvas)
    step.finish(z, dev(idx), canvas)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(canvas), oracle.scatter(host(z), idx, 0, before))
