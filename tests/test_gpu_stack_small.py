"""A small selective stack (3 double + 2 single blocks, 3 steps) through
StackStep, with the query/key scorer and with the fused route (text mass
from the joint-softmax pass, probes of one or two double blocks).  Each step
is checked on the GPU's own inputs of that stage, as the full-size stack
test does: probe masses and scores within the bar, the selection bit-exact,
gather and scatter bit-exact, every block teacher-forced."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17995_amd.step import StackStep, StepShape
from synth import configs as C
from synth import generator as G

from _gpu import assert_close, dev, double_weights_dev, host

pytestmark = pytest.mark.gpu

W = C.TINY_BF16.replace(name="tiny_bf16_stack", n_double=3, n_single=2, steps=3)


@pytest.mark.parametrize("fused,probes", [(False, (0,)), (True, (0,)), (True, (0, 2))],
                         ids=["qk", "fused", "fused_2probes"])
def test_small_stack_recurrence(gpu, fused, probes):
    w = W
    x0, x_m1, _ = G.feature_pair(w.seed, w.N, w.D, w.dtype)
    lay = G.layout_inputs(w, x0)
    dw = [(G.double_stream_weights(w, b, 0), G.double_stream_weights(w, b, 1)) for b in range(w.n_double)]
    sw = [G.single_block_weights(w, b) for b in range(w.n_single)]
    doubles = [gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=double_weights_dev(t, w.dtype), img=double_weights_dev(i, w.dtype))
               for t, i in dw]
    singles = [gpu.BlockWeights(gpu.BLOCK_SINGLE, single=double_weights_dev(x, w.dtype)) for x in sw]
    shape = StepShape(N=w.N, H_lr=w.H_lr, W_lr=w.W_lr, L=w.L, R=w.R, k=w.k, D=w.D, H=w.H, D_f=w.D,
                      mlp_hidden=w.mlp_ratio * w.D)
    step = StackStep(shape, doubles, singles, G.prefix_positions(w), torch.bfloat16, alpha=w.alpha, eps=w.eps_minmax,
                     fused=fused, probe_blocks=probes)
    text, lowres = dev(lay["text"], "bf16"), dev(lay["lowres"], "bf16")
    X = [dev(x_m1, "bf16"), dev(x0, "bf16")]
    img_pos = step.img_pos.cpu().numpy()
    pos_all = np.concatenate([np.zeros((w.L, 3), np.int32), img_pos])
    for s in range(1, w.steps + 1):
        x_prev, x_prev2 = host(X[-1]), host(X[-2])
        canvas = torch.empty_like(X[-1])
        outs, snap = {}, {}

        def on_block(i, x_in, x_out):
            torch.cuda.synchronize()
            if i == 0:
                snap["canvas"] = host(canvas)
                snap["compact"] = host(x_in)
            outs[i] = (host(x_in), host(x_out))

        step.run(X[-1], X[-2], lowres, text, canvas, on_block=on_block)
        torch.cuda.synchronize()
        scores = step.scores.cpu().numpy()
        idx = step.idx.cpu().numpy()
        # Scores from the oracle's probes of the GPU's X_{s-1}.
        if fused:
            mass = np.zeros((w.H, w.N))
            for b in probes:
                q, k = oracle.block_qk(np.concatenate([lay["text"], x_prev]), pos_all, w.L, dw[b][0], dw[b][1], w.H)
                mass += oracle.text_attention_mass(q[w.L:], k, w.L)
            assert_close(host(step.mass), mass, "bf16", f"step {s} probe mass")
            s_ref, _, _ = oracle.score_from_mass(mass, len(probes), np.stack([x_prev2, x_prev]), w.alpha,
                                                 w.eps_minmax)
        else:
            q, k = oracle.block_qk(np.concatenate([lay["text"], x_prev]), pos_all, w.L, dw[0][0], dw[0][1], w.H)
            s_ref, _, _ = oracle.score(q[w.L:], k[:w.L], oracle.joint_lse(q[w.L:], k), x_prev, x_prev2, w.alpha,
                                       w.eps_minmax)
        assert_close(scores, s_ref, "bf16", f"step {s} scores")
        np.testing.assert_array_equal(idx, oracle.select_topk(scores, w.k), err_msg=f"step {s} select")
        compact, pos, cv = oracle.gather_upsample(lay["lowres"], x_prev, lay["text"], idx, w.H_lr, w.W_lr)
        np.testing.assert_array_equal(snap["compact"], compact)
        np.testing.assert_array_equal(snap["canvas"], cv)
        pos_s = step.pos.cpu().numpy()
        for i, (x_in, x_out) in outs.items():
            if i < w.n_double:
                ref, _ = oracle.double_block(x_in, pos_s, w.L, dw[i][0], dw[i][1], w.H)
            else:
                ref, _ = oracle.single_block(x_in, pos_s, sw[i - w.n_double], w.H)
            assert_close(x_out, ref, "bf16", f"step {s} block {i}")
            assert_close(x_out - x_in, ref - x_in, "bf16", f"step {s} block {i} update")
        last = outs[w.n_double + w.n_single - 1][1]
        np.testing.assert_array_equal(host(canvas), oracle.scatter(last, idx, w.L, snap["canvas"]))
        X = [X[-1], canvas]
