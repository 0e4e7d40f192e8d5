"""A selective step over several images at once (a CFG pair and a third
prompt with nothing selected): each image scored on its own (one launch per
image, or one launch over the stacked images), one selection
launch over all of them, one block pass over the rows packed by stream, and
each image's canvas updated from its own rows.  Every stage is checked
against the oracle on the GPU's inputs of that stage: indices, gathered rows,
positions and canvases bit-exact; scores and block outputs within the parity
bar.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17995_amd.step import BatchedStep, StepShape
from synth import configs as C
from synth import generator as G

from _gpu import assert_close, dev, double_weights_dev, host

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("stacked", ["none", "score", "all"], ids=["per_image", "score_stacked", "all_stacked"])
@pytest.mark.parametrize("base", [C.TINY_BF16, C.TINY_BF16_REF], ids=lambda w: w.name)
def test_batched_step(gpu, base, stacked):
    ws = [base, base.replace(seed=base.seed + 1, rho=0.45), base.replace(seed=base.seed + 2)]
    ks = [ws[0].k, ws[1].k, 0]
    Bn = len(ws)
    wt, wi = G.double_stream_weights(base, 0, 0), G.double_stream_weights(base, 0, 1)
    bw = gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=double_weights_dev(wt, base.dtype),
                          img=double_weights_dev(wi, base.dtype))
    shape = StepShape(N=base.N, H_lr=base.H_lr, W_lr=base.W_lr, L=base.L, R=base.R, k=0, D=base.D, H=base.H,
                      D_f=base.Df, mlp_hidden=base.mlp_ratio * base.D)
    step = BatchedStep(shape, ks, bw, dev(G.prefix_positions(base)), torch.bfloat16, alpha=base.alpha)
    si = [G.score_inputs(w) for w in ws]
    lay = [G.layout_inputs(w, s["feat_t"]) for w, s in zip(ws, si)]
    lse = [oracle.joint_lse(s["latent_q"], np.concatenate([s["text_k"], s["ref_k"], s["latent_k"]])) for s in si]
    canvases = [dev(l["highres_prev"], base.dtype) for l in lay]
    score_in = [[dev(s["latent_q"], base.dtype) for s in si], [dev(s["text_k"], base.dtype) for s in si],
                [dev(x) for x in lse], canvases, [dev(s["feat_prev"], base.dtype) for s in si]]
    lay_in = [[dev(l["lowres"], base.dtype) for l in lay], canvases, [dev(l["text"], base.dtype) for l in lay],
              [dev(l["ref"], base.dtype) for l in lay]]
    if stacked != "none":  # one scoring launch over the stacked images (feat_t: a copy of the canvases)
        score_in = [torch.stack(t) for t in score_in]
    if stacked == "all":   # one gather and one scatter launch for all images, canvases stacked
        lay_in = [torch.stack(t) if t[0].numel() else None for t in lay_in]
        canvases = lay_in[1]
    step.run(*score_in, *lay_in)
    torch.cuda.synchronize()
    scores, idx_all = step.scores.cpu().numpy(), step.idx.cpu().numpy()
    x, pos, x_out = host(step.x), step.pos.cpu().numpy(), host(step.x_out)
    T, R = step.txt_off[-1], base.R
    for b in range(Bn):
        s_b = scores[b * base.N:(b + 1) * base.N]
        s_ref, _, _ = oracle.score(si[b]["latent_q"], si[b]["text_k"], lse[b].astype(np.float32), si[b]["feat_t"],
                                   si[b]["feat_prev"], base.alpha, base.eps_minmax)
        assert_close(s_b, s_ref, base.dtype, f"image {b} scores")
        idx = idx_all[step.out_off[b]:step.out_off[b + 1]]
        np.testing.assert_array_equal(idx, oracle.select_topk(s_b, ks[b]), err_msg=f"image {b} selection")
        np.testing.assert_array_equal(x[step.txt_off[b]:step.txt_off[b + 1]], lay[b]["text"])
        compact, pos_sel, canvas = oracle.gather_upsample(lay[b]["lowres"], lay[b]["highres_prev"],
                                                          lay[b]["ref"] if R else None, idx, base.H_lr, base.W_lr)
        a0 = T + step.img_off[b]
        np.testing.assert_array_equal(x[a0:a0 + R + ks[b]], compact, err_msg=f"image {b} gathered rows")
        np.testing.assert_array_equal(pos[a0 + R:a0 + R + ks[b]], pos_sel)
        np.testing.assert_array_equal(pos[a0:a0 + R], G.prefix_positions(base)[base.L:])
        np.testing.assert_array_equal(host(canvases[b]), oracle.scatter(x_out[a0:a0 + R + ks[b]], idx, R, canvas),
                                      err_msg=f"image {b} canvas")
    # The block over the packed rows, from the GPU's own gathered input.
    ref, _ = oracle.block_batched(x, pos, step.txt_off, step.img_off, base.H, wt, wi)
    for b in range(Bn):
        rows = np.concatenate([np.arange(step.txt_off[b], step.txt_off[b + 1]),
                               T + np.arange(step.img_off[b], step.img_off[b + 1])])
        assert_close(x_out[rows] - x[rows], ref[rows] - x[rows], base.dtype, f"image {b} block update")
