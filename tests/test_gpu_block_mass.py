"""avits_block_forward_ex: the text attention mass from the block's own
joint attention, per head each row's softmax share on the text keys (Eq. spatial with the softmax of Eq. dit_attn), taken inside the block's
attention pass, against the oracle's text mass of the block's own normalised,
rotated q and k (oracle.block_qk then oracle.text_attention_mass).

The block output with the mass requested is bit-identical to the plain
block; the accumulate flag adds to the buffer (two calls give twice one);
forced key-piece plans (the combine kernel merging the pieces' text sums)
give the same mass; the FLUX 1024^2 block (whose attention runs its overrun
units in key pieces) is checked on every row.  The fused Stage-3 scatter
is bit-identical to the block followed by avits_scatter.
"""
import numpy as np
import pytest
import torch

import oracle
from synth import configs as C
from synth import generator as G

from _gpu import assert_close, dev, double_weights_dev, host

pytestmark = pytest.mark.gpu


def _inputs(w, n_txt, n_img, seed):
    x = G.block_input(w, n_txt + n_img, seed)
    g = np.random.default_rng(2000 + seed)
    pos = np.zeros((n_txt + n_img, 3), np.int32)
    pos[n_txt:, 1] = g.integers(0, w.H_hr, n_img)
    pos[n_txt:, 2] = g.integers(0, w.W_hr, n_img)
    return x, pos


def _weights(gpu, w, kind):
    if kind == "double":
        wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
        bw = gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=double_weights_dev(wt, w.dtype),
                              img=double_weights_dev(wi, w.dtype))
        return bw, dict(w_txt=wt, w_img=wi)
    ws = G.single_block_weights(w, 0)
    return gpu.BlockWeights(gpu.BLOCK_SINGLE, single=double_weights_dev(ws, w.dtype)), dict(single=ws)


def _oracle_mass(w, x, pos, n_txt, ow):
    if "single" in ow:
        q, k = oracle.block_qk(x, pos, n_txt, None, None, w.H, single=ow["single"])
    else:
        q, k = oracle.block_qk(x, pos, n_txt, ow["w_txt"], ow["w_img"], w.H)
    return oracle.text_attention_mass(q, k, n_txt)


def _run(gpu, w, bw, x, pos, n_txt, accumulate_twice=False):
    S = x.shape[0]
    t_x, t_pos = dev(x, w.dtype), dev(pos)
    plain = torch.empty_like(t_x)
    gpu.avits_block_forward(t_x, plain, t_pos, n_txt, S - n_txt, bw, w.H)
    out = torch.empty_like(t_x)
    lse = torch.empty(w.H, S, device="cuda")
    mass = torch.full((w.H, S), float("nan"), device="cuda")
    gpu.avits_block_forward_ex(t_x, out, t_pos, n_txt, S - n_txt, bw, w.H, lse_out=lse, mass_out=mass)
    torch.cuda.synchronize()
    res = {"plain": host(plain), "out": host(out), "lse": host(lse), "mass": host(mass)}
    if accumulate_twice:
        gpu.avits_block_forward_ex(t_x, out, t_pos, n_txt, S - n_txt, bw, w.H, mass_out=mass, mass_accumulate=True)
        torch.cuda.synchronize()
        res["mass2"] = host(mass)
    return res


@pytest.mark.parametrize("kind", ["double", "single"])
@pytest.mark.parametrize("w", [C.TINY_F32, C.TINY_BF16, C.TINY_BF16_REF, C.TINY_F32_RAGGED],
                         ids=lambda w: w.name)
def test_block_mass_tiny(gpu, w, kind):
    n_txt, n_img = w.L, w.R + w.k
    x, pos = _inputs(w, n_txt, n_img, seed=3)
    bw, ow = _weights(gpu, w, kind)
    r = _run(gpu, w, bw, x, pos, n_txt, accumulate_twice=True)
    np.testing.assert_array_equal(r["out"], r["plain"])      # the mass leaves the block untouched
    ref = _oracle_mass(w, x, pos, n_txt, ow)
    assert_close(r["mass"], ref, w.dtype, "block text mass")
    assert np.abs(r["mass"] - ref).max() < (1e-4 if w.dtype == "f32" else 2e-3)
    np.testing.assert_array_equal(r["mass2"], 2.0 * r["mass"])   # accumulate adds the same value
    # Softmax shares: inside [0, 1].
    assert np.all(r["mass"] >= 0.0) and np.all(r["mass"] <= 1.0 + 1e-6)


@pytest.mark.parametrize("cfg", ["0,2", "0,3", "3,4", "7,2"])
@pytest.mark.parametrize("kind", ["double", "single"])
def test_block_mass_key_pieces(gpu, monkeypatch, kind, cfg):
    monkeypatch.setenv("AVITS_ATTN_SPLIT", cfg)
    w = C.TINY_BF16
    n_txt, n_img = 40, 555     # 10 attention units, 10 key tiles: the text keys end inside the first tile
    x, pos = _inputs(w, n_txt, n_img, seed=11)
    bw, ow = _weights(gpu, w, kind)
    r = _run(gpu, w, bw, x, pos, n_txt)
    ref = _oracle_mass(w, x, pos, n_txt, ow)
    assert_close(r["mass"], ref, "bf16", "block text mass (key pieces)")
    assert np.abs(r["mass"] - ref).max() < 2e-3


def test_block_mass_degenerate(gpu):
    # No text rows: the mass is 0 everywhere; only text rows: 1 everywhere.
    w = C.TINY_BF16
    bw, _ = _weights(gpu, w, "double")
    for n_txt, n_img in ((0, 77), (40, 0)):
        x, pos = _inputs(w, n_txt, n_img, seed=5)
        r = _run(gpu, w, bw, x, pos, n_txt)
        want = 0.0 if n_txt == 0 else 1.0
        assert np.abs(r["mass"] - want).max() < 1e-5, (n_txt, n_img)


@pytest.mark.slow
def test_block_mass_flux_1024(gpu):
    w = C.FLUX_1024
    n_txt, n_img = w.L, w.k
    x, pos = _inputs(w, n_txt, n_img, seed=1)
    bw, ow = _weights(gpu, w, "double")
    r = _run(gpu, w, bw, x, pos, n_txt)
    np.testing.assert_array_equal(r["out"], r["plain"])
    ref = _oracle_mass(w, x, pos, n_txt, ow)
    assert_close(r["mass"], ref, w.dtype, "block text mass")
    assert np.abs(r["mass"] - ref).max() < 2e-3


# ---------------------------------------------------------------------------
# The Stage-3 scatter fused into the block's last projection
# (avits_block_forward_ex with scatter_idx / canvas): canvas and block output
# bit-identical to the block followed by avits_scatter, whatever the GEMM plan
# of that projection (split-K with its reduce kernel, unsplit, 128-wide).

def _fused_vs_two_calls(gpu, w, kind, k, seed=13):
    n_txt, n_img = w.L, w.R + w.k
    x, pos = _inputs(w, n_txt, n_img, seed)
    bw, _ = _weights(gpu, w, kind)
    S = n_txt + n_img
    t_x, t_pos = dev(x, w.dtype), dev(pos)
    g = np.random.default_rng(seed)
    idx = np.sort(g.permutation(w.N)[:k]).astype(np.int32)
    canvas0 = dev(G.block_input(w, w.N, seed + 1), w.dtype)
    c1, c2 = canvas0.clone(), canvas0.clone()
    o1, o2 = torch.empty_like(t_x), torch.empty_like(t_x)
    t_idx = dev(idx)
    gpu.avits_block_forward(t_x, o1, t_pos, n_txt, n_img, bw, w.H)
    if k:
        gpu.avits_scatter(o1, t_idx, S - k, c1)
    gpu.avits_block_forward_ex(t_x, o2, t_pos, n_txt, n_img, bw, w.H, scatter_idx=t_idx if k else None,
                               canvas=c2 if k else None)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(o2), host(o1))
    np.testing.assert_array_equal(host(c2), host(c1))


@pytest.mark.parametrize("plan", [None, "256,3", "256,1", "128,1"])
@pytest.mark.parametrize("kind", ["double", "single"])
@pytest.mark.parametrize("w", [C.TINY_F32, C.TINY_BF16, C.TINY_BF16_REF], ids=lambda w: w.name)
def test_block_fused_scatter(gpu, monkeypatch, w, kind, plan):
    if plan:
        monkeypatch.setenv("AVITS_GEMM_TILE_gemm_mlp_out", plan)
        monkeypatch.setenv("AVITS_GEMM_TILE_gemm_single_out", plan)
    for k in sorted({0, 1, w.k}):
        _fused_vs_two_calls(gpu, w, kind, k)


@pytest.mark.slow
def test_block_fused_scatter_flux_1024(gpu):
    _fused_vs_two_calls(gpu, C.FLUX_1024, "double", C.FLUX_1024.k)
