"""avits_gather_upsample_ln: the gather that also writes the first stage of
the double block on the compacted rows, h = LN(row)(1 + scale1) + shift1
(text-stream vectors for the text rows, image-stream vectors for the
reference and selected rows; Section 3.3.1's block on the compacted
sequence).  Compact rows, positions and canvas equal avits_gather_upsample
bit for bit; h is checked against the oracle's modulated layer norm; and
the block started from h (avits_block_forward_ex h_in) equals the plain
block bit for bit, which pins h to the block's own first stage.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle.block import layer_norm
from synth import configs as C
from synth import generator as G

from _gpu import assert_close, dev, double_weights_dev, host

pytestmark = pytest.mark.gpu


def _case(gpu, w, k, n_txt=None, seed=0, alias=False):
    lay = G.layout_inputs(w)
    idx = G.random_selection(w, k, seed)
    prefix = np.concatenate([lay["text"], lay["ref"]])
    L = w.L if n_txt is None else n_txt
    t_low, t_high = dev(lay["lowres"], w.dtype), dev(lay["highres_prev"], w.dtype)
    t_pre = dev(prefix, w.dtype) if w.LR else None
    t_idx = dev(idx)
    wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
    dt, di = double_weights_dev(wt, w.dtype), double_weights_dev(wi, w.dtype)
    S = w.LR + k
    outs = []
    for fused in (False, True):
        compact = torch.full((S, w.D), 7.0, dtype=t_low.dtype, device="cuda")
        pos = torch.full((S, 3), -1, dtype=torch.int32, device="cuda")
        pos[:w.LR] = 0
        canvas = t_high.clone() if alias else torch.full_like(t_high, 7.0)
        high = canvas if alias else t_high
        if fused:
            h = torch.full((S, w.D), 3.0, dtype=t_low.dtype, device="cuda")
            gpu.avits_gather_upsample_ln(t_low, high, t_pre, t_idx, w.H_lr, w.W_lr, compact, pos[w.LR:], canvas, L,
                                         dt["mod"][0], dt["mod"][1], di["mod"][0], di["mod"][1], h)
        else:
            h = None
            gpu.avits_gather_upsample(t_low, high, t_pre, t_idx, w.H_lr, w.W_lr, compact, pos[w.LR:], canvas)
        outs.append((compact, pos, canvas, h))
    torch.cuda.synchronize()
    return outs, (wt, wi, dt, di), L


@pytest.mark.parametrize("w,k,n_txt", [(C.TINY_BF16, C.TINY_BF16.k, None), (C.TINY_BF16_REF, C.TINY_BF16_REF.k, None),
                                       (C.TINY_BF16_REF, 0, None), (C.TINY_BF16_REF, 5, 0),
                                       (C.TINY_BF16, C.TINY_BF16.N, None)],
                         ids=["tiny", "with_reference", "k0", "no_text_stream", "keep_all"])
@pytest.mark.parametrize("alias", [False, True], ids=["separate", "in_place"])
def test_gather_ln(gpu, w, k, n_txt, alias):
    (plain, fused), (wt, wi, dt, di), L = _case(gpu, w, k, n_txt, alias=alias)
    for a, b, what in zip(plain[:3], fused[:3], ("compact", "pos", "canvas")):
        np.testing.assert_array_equal(host(b), host(a), err_msg=what)
    compact = host(fused[0]).astype(np.float64)
    mt, mi = wt["mod"].astype(np.float64), wi["mod"].astype(np.float64)
    S = compact.shape[0]
    sh = np.where(np.arange(S)[:, None] < L, mt[0], mi[0])
    sc = np.where(np.arange(S)[:, None] < L, mt[1], mi[1])
    ref = layer_norm(compact) * (1.0 + sc) + sh
    assert_close(host(fused[3]), ref, w.dtype, "gathered rows' modulated layer norm")
    # The block started from h is the plain block, bit for bit.
    if S:
        bw = gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=dt, img=di)
        o1, o2 = torch.empty_like(fused[0]), torch.empty_like(fused[0])
        gpu.avits_block_forward(fused[0], o1, fused[1], L, S - L, bw, w.H)
        gpu.avits_block_forward_ex(fused[0], o2, fused[1], L, S - L, bw, w.H, h_in=fused[3])
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(o2), host(o1))


@pytest.mark.slow
def test_gather_ln_flux_1024(gpu):
    w = C.FLUX_1024
    (plain, fused), (wt, wi, dt, di), L = _case(gpu, w, w.k, seed=1, alias=True)
    for a, b in zip(plain[:3], fused[:3]):
        assert torch.equal(a, b)
    bw = gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=dt, img=di)
    S = fused[0].shape[0]
    o1, o2 = torch.empty_like(fused[0]), torch.empty_like(fused[0])
    gpu.avits_block_forward(fused[0], o1, fused[1], L, S - L, bw, w.H)
    gpu.avits_block_forward_ex(fused[0], o2, fused[1], L, S - L, bw, w.H, h_in=fused[3])
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)
    rows = np.arange(0, S, 7)
    compact = host(fused[0])[rows].astype(np.float64)
    mt, mi = wt["mod"].astype(np.float64), wi["mod"].astype(np.float64)
    sh = np.where(rows[:, None] < L, mt[0], mi[0])
    sc = np.where(rows[:, None] < L, mt[1], mi[1])
    assert_close(host(fused[3])[rows], layer_norm(compact) * (1.0 + sc) + sh, w.dtype, "FLUX rows' layer norm")


def test_gather_ln_rejects(gpu):
    w = C.TINY_BF16
    lay = G.layout_inputs(w)
    low, high = dev(lay["lowres"], w.dtype), dev(lay["highres_prev"], w.dtype)
    pre = dev(lay["text"], w.dtype)
    idx = dev(G.random_selection(w, 4, 0))
    compact = torch.empty(w.L + 4, w.D, dtype=low.dtype, device="cuda")
    pos = torch.empty(4, 3, dtype=torch.int32, device="cuda")
    vec = torch.zeros(w.D, dtype=low.dtype, device="cuda")
    with pytest.raises(gpu.AvitsError):   # h aliasing compact
        gpu.avits_gather_upsample_ln(low, high, pre, idx, w.H_lr, w.W_lr, compact, pos, high, w.L, vec, vec, vec, vec,
                                     compact)
    with pytest.raises(gpu.AvitsError):   # n_txt beyond the prefix
        gpu.avits_gather_upsample_ln(low, high, pre, idx, w.H_lr, w.W_lr, compact, pos, high, w.L + 1, vec, vec, vec,
                                     vec, torch.empty_like(compact))
    wf = C.TINY_F32
    layf = G.layout_inputs(wf)
    lowf, highf = dev(layf["lowres"], wf.dtype), dev(layf["highres_prev"], wf.dtype)
    cf = torch.empty(wf.L + 4, wf.D, device="cuda")
    vf = torch.zeros(wf.D, device="cuda")
    with pytest.raises(gpu.AvitsError):   # bf16 only
        gpu.avits_gather_upsample_ln(lowf, highf, dev(layf["text"], wf.dtype), dev(G.random_selection(wf, 4, 0)),
                                     wf.H_lr, wf.W_lr, cf, pos, highf, wf.L, vf, vf, vf, vf, torch.empty_like(cf))
