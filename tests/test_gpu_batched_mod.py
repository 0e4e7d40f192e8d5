"""avits_block_forward_batched_ex: several images through one block pass,
each with its own modulation vectors (images at different timesteps, whose
timestep reaches every block through the modulation; Section 3.2 runs each
image on its own schedule).  Image b's rows are checked against the oracle
block run with image b's modulation (each image its own joint sequence, as
Section 3.3.1 defines it); changing one image's modulation changes that
image's rows only (bit for bit elsewhere); mod_stride 0 is
avits_block_forward_batched bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
from synth import configs as C
from synth import generator as G

from _gpu import assert_close, dev, double_weights_dev, host

pytestmark = pytest.mark.gpu


def _layout(txt, img):
    txt_off = np.concatenate([[0], np.cumsum(txt)]).astype(int).tolist()
    img_off = np.concatenate([[0], np.cumsum(img)]).astype(int).tolist()
    return txt_off, img_off


def _inputs(w, n_txt, n_img, seed):
    x = G.block_input(w, n_txt + n_img, seed)
    g = np.random.default_rng(3000 + seed)
    pos = np.zeros((n_txt + n_img, 3), np.int32)
    pos[n_txt:, 1] = g.integers(0, w.H_hr, n_img)
    pos[n_txt:, 2] = g.integers(0, w.W_hr, n_img)
    return x, pos


def _per_image_mods(base, B, seed, dtype):
    """B modulation blocks [B, n_vec, D] around `base` (shifts and scales
    moved by N(0, 0.3), gates by N(0, 0.3) around theirs), bf16-rounded."""
    g = np.random.default_rng(seed)
    return np.stack([G.round_to(base + g.normal(0.0, 0.3, base.shape), dtype) for _ in range(B)])


def _rows_of(b, txt_off, img_off):
    T = txt_off[-1]
    return np.concatenate([np.arange(txt_off[b], txt_off[b + 1]), T + np.arange(img_off[b], img_off[b + 1])])


def _setup(gpu, w, kind, B, seed):
    if kind == "double":
        wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
        mt, mi = _per_image_mods(wt["mod"], B, seed, w.dtype), _per_image_mods(wi["mod"], B, seed + 1, w.dtype)
        dt, di = double_weights_dev(wt, w.dtype), double_weights_dev(wi, w.dtype)
        dt["mod"], di["mod"] = dev(mt.reshape(-1, w.D), w.dtype), dev(mi.reshape(-1, w.D), w.dtype)
        bw = gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=dt, img=di)
        stride = 6 * w.D

        def oracle_image(x, pos, txt_off, img_off, b):
            out, lse = oracle.block_batched(x, pos, txt_off, img_off, w.H, dict(wt, mod=mt[b]), dict(wi, mod=mi[b]))
            return out, lse
        return bw, stride, oracle_image, (dt, di)
    ws_ = G.single_block_weights(w, 0)
    ms = _per_image_mods(ws_["mod"], B, seed, w.dtype)
    ds = double_weights_dev(ws_, w.dtype)
    ds["mod"] = dev(ms.reshape(-1, w.D), w.dtype)
    bw = gpu.BlockWeights(gpu.BLOCK_SINGLE, single=ds)

    def oracle_image(x, pos, txt_off, img_off, b):
        return oracle.block_batched(x, pos, txt_off, img_off, w.H, single=dict(ws_, mod=ms[b]))
    return bw, 3 * w.D, oracle_image, (ds,)


@pytest.mark.parametrize("kind", ["double", "single"])
def test_block_batched_per_image_modulation(gpu, kind):
    w = C.TINY_BF16
    txt, img = [32, 0, 7, 129], [200, 77, 1, 64]
    txt_off, img_off = _layout(txt, img)
    B = len(txt)
    x, pos = _inputs(w, txt_off[-1], img_off[-1], seed=31)
    bw, stride, oracle_image, keep = _setup(gpu, w, kind, B, seed=41)
    t_x, t_pos = dev(x, w.dtype), dev(pos)
    out = torch.empty_like(t_x)
    lse = torch.empty(w.H, x.shape[0], device="cuda")
    gpu.avits_block_forward_batched_ex(t_x, out, t_pos, txt_off, img_off, bw, w.H, stride, lse_out=lse)
    torch.cuda.synchronize()
    got, got_lse = host(out), host(lse)
    for b in range(B):
        rows = _rows_of(b, txt_off, img_off)
        ref, ref_lse = oracle_image(x, pos, txt_off, img_off, b)
        assert_close(got[rows] - x[rows], ref[rows] - x[rows], w.dtype, f"image {b} block update ({kind})")
        assert_close(got_lse[:, rows], ref_lse[:, rows], w.dtype, f"image {b} lse ({kind})")
    # mod_stride 0: every image takes image 0's modulation, exactly the
    # shared-modulation entry point.
    o0, o1 = torch.empty_like(t_x), torch.empty_like(t_x)
    gpu.avits_block_forward_batched_ex(t_x, o0, t_pos, txt_off, img_off, bw, w.H, 0)
    gpu.avits_block_forward_batched(t_x, o1, t_pos, txt_off, img_off, bw, w.H)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(o0), host(o1))
    assert not np.array_equal(host(o0), got)   # the per-image modulation did change the result


@pytest.mark.parametrize("kind", ["double", "single"])
def test_per_image_modulation_touches_its_own_rows(gpu, kind):
    # Moving image 2's modulation changes image 2's rows only.
    w = C.TINY_BF16
    txt, img = [16, 9, 24], [40, 130, 3]
    txt_off, img_off = _layout(txt, img)
    B = len(txt)
    x, pos = _inputs(w, txt_off[-1], img_off[-1], seed=5)
    bw, stride, _, devw = _setup(gpu, w, kind, B, seed=7)
    t_x, t_pos = dev(x, w.dtype), dev(pos)
    o1, o2 = torch.empty_like(t_x), torch.empty_like(t_x)
    gpu.avits_block_forward_batched_ex(t_x, o1, t_pos, txt_off, img_off, bw, w.H, stride)
    for d in devw:
        blk = d["mod"].view(B, -1, w.D)
        blk[2] = (blk[2].float() * 1.5 + 0.1).to(blk.dtype)
    gpu.avits_block_forward_batched_ex(t_x, o2, t_pos, txt_off, img_off, bw, w.H, stride)
    torch.cuda.synchronize()
    a, b2 = host(o1), host(o2)
    mine = _rows_of(2, txt_off, img_off)
    others = np.setdiff1d(np.arange(x.shape[0]), mine)
    np.testing.assert_array_equal(b2[others], a[others])
    assert not np.array_equal(b2[mine], a[mine])


@pytest.mark.slow
def test_per_image_modulation_flux_pair(gpu):
    # A CFG-style pair at the FLUX 1024^2 shape, each image at its own
    # timestep's modulation; every 16th row of both images against the oracle.
    w = C.FLUX_1024
    txt, img = [w.L, w.L], [w.k, w.k]
    txt_off, img_off = _layout(txt, img)
    x, pos = _inputs(w, txt_off[-1], img_off[-1], seed=11)
    bw, stride, _, _ = _setup(gpu, w, "double", 2, seed=13)
    t_x = dev(x, w.dtype)
    out = torch.empty_like(t_x)
    gpu.avits_block_forward_batched_ex(t_x, out, dev(pos), txt_off, img_off, bw, w.H, stride)
    torch.cuda.synchronize()
    got = host(out)
    wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
    mt, mi = _per_image_mods(wt["mod"], 2, 13, w.dtype), _per_image_mods(wi["mod"], 2, 14, w.dtype)
    for b in range(2):
        rows = _rows_of(b, txt_off, img_off)
        n_txt = txt[b]
        sub = rows[::16]
        local = np.searchsorted(rows, sub)
        ref, _ = oracle.double_block(x[rows], pos[rows], n_txt, dict(wt, mod=mt[b]), dict(wi, mod=mi[b]), w.H,
                                     rows=local)
        assert_close(got[sub] - x[sub], ref - x[sub], w.dtype, f"FLUX pair image {b}")
