"""The FLUX-shaped selective stack: 19 double + 38 single blocks, 4 denoising
steps at 1024^2 (512 text tokens, 32x32 -> 64x64, k = 1229 per step).

Recurrence (one image, the text re-fed unchanged every step; no embedders,
final layer or sampler update):
  probe   double block 0's first stage on [T; X_{s-1}] -> q_img, k_all
  lse     joint log-sum-exp of q_img over k_all
  score   A from (q_img, k_txt, lse); V from (X_{s-1}, X_{s-2}); alpha = 0.5
  select  k = 1229
  gather  compact = [T; X_{s-1}[idx]], canvas = X_{s-1} on idx, up(X_lr) elsewhere
  blocks  19 double, then 38 single, on the 1741 compacted rows
  scatter X_s = canvas with the last block's image rows written back
X_0 and X_{-1} are the seeded feature pair (X_{-1} = X_0 + eps_i z_i).

Every stage is checked on the GPU's own inputs of that stage (teacher
forcing): probe rows, LSE rows and scores within the parity bar; the
selection bit-exact against the oracle's selection of the GPU's scores and,
against the oracle's own probe -> LSE -> scores, different only at the
selection boundary; gather and scatter bit-exact; every block of step 1 and
seven blocks of steps 2-4 on sampled rows.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from paper_2608_17995_amd.step import StackStep, StepShape
from synth import configs as C
from synth import generator as G

from _gpu import assert_close, dev, host, rel_l2

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

W = C.FLUX_STACK
LATER_BLOCKS = (0, 1, 9, 18, 19, 37, 56)   # blocks checked at steps 2..4


def _bits(wd):
    return {k: G.to_bf16_bits(v) for k, v in wd.items()}


def _f32(bits):
    return {k: G.bf16_bits_to_f32(v) for k, v in bits.items()}


def _to_dev(bits):
    return {k: torch.from_numpy(v.view(np.int16)).view(torch.bfloat16).cuda() for k, v in bits.items()}


def _gen(job):
    kind, b = job
    if kind == "d":
        return job, (_bits(G.double_stream_weights(W, b, 0)), _bits(G.double_stream_weights(W, b, 1)))
    return job, _bits(G.single_block_weights(W, b))


def _sample_rows(S, L, seed):
    g = np.random.default_rng(seed)
    return np.unique(np.concatenate([np.arange(8), np.arange(L - 4, L), g.integers(L, S, 48), np.arange(S - 4, S)]))


def _update_bar(out, ref, x):
    """rel-L2 bar for the block update (out - x): 1e-2 plus twice the share of
    the update that rounding the output to bf16 alone can account for."""
    ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 1e-30))) - 7)
    floor = np.linalg.norm(ulp) / np.sqrt(12.0) / max(np.linalg.norm(ref - x), 1e-30)
    return 1e-2 + 2.0 * floor


@pytest.fixture(scope="module")
def stack(gpu):
    w = W
    print(f"\n[stack] {w.name}: {w.n_double} double + {w.n_single} single blocks, {w.steps} steps, "
          f"N={w.N} k={w.k} S={w.S}", flush=True)
    x0, x_m1, _ = G.feature_pair(w.seed, w.N, w.D, w.dtype)
    lay = G.layout_inputs(w, x0)
    jobs = [("d", b) for b in range(w.n_double)] + [("s", b) for b in range(w.n_single)]
    host_w = {}
    with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
        for job, bits in ex.map(_gen, jobs):
            host_w[job] = bits
    doubles = [gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=_to_dev(host_w[("d", b)][0]), img=_to_dev(host_w[("d", b)][1]))
               for b in range(w.n_double)]
    singles = [gpu.BlockWeights(gpu.BLOCK_SINGLE, single=_to_dev(host_w[("s", b)])) for b in range(w.n_single)]
    print("[stack] weights on device", flush=True)
    shape = StepShape(N=w.N, H_lr=w.H_lr, W_lr=w.W_lr, L=w.L, R=w.R, k=w.k, D=w.D, H=w.H, D_f=w.D,
                      mlp_hidden=w.mlp_ratio * w.D)
    step = StackStep(shape, doubles, singles, G.prefix_positions(w), torch.bfloat16, alpha=w.alpha, eps=w.eps_minmax)
    text, lowres = dev(lay["text"], "bf16"), dev(lay["lowres"], "bf16")
    X = [dev(x_m1, "bf16"), dev(x0, "bf16")]
    xs_host = [x_m1, x0]
    steps = []
    for s in range(1, w.steps + 1):
        canvas = torch.empty_like(X[-1])
        rec = {"outs": {}}
        check = range(w.n_double + w.n_single) if s == 1 else LATER_BLOCKS

        def on_block(i, x_in, x_out, rec=rec, check=check, canvas=canvas):
            if i == 0:
                torch.cuda.synchronize()
                rec["canvas_gather"] = host(canvas)
                rec["compact"] = host(step.compact)
            if i in check or i + 1 in check:
                torch.cuda.synchronize()
                rec["outs"][i] = host(x_out)

        step.run(X[-1], X[-2], lowres, text, canvas, on_block=on_block)
        torch.cuda.synchronize()
        rec.update(q_img=host(step.q_img), k_all=host(step.k_all), lse=host(step.lse),
                   scores=step.scores.cpu().numpy(), idx=step.idx.cpu().numpy(), pos=step.pos.cpu().numpy(),
                   x_prev=xs_host[-1], x_prev2=xs_host[-2], x_new=host(canvas), check=tuple(check))
        steps.append(rec)
        X = [X[-1], canvas]
        xs_host = [xs_host[-1], rec["x_new"]]
        print(f"[stack] step {s} done", flush=True)
    return {"w": w, "host_w": host_w, "text": lay["text"], "lowres": lay["lowres"], "steps": steps,
            "img_pos": step.img_pos.cpu().numpy()}


def test_stack_probe_rows(stack):
    w, hw = stack["w"], stack["host_w"]
    wt0, wi0 = _f32(hw[("d", 0)][0]), _f32(hw[("d", 0)][1])
    rows = np.unique(np.concatenate([np.arange(8), np.random.default_rng(3).integers(0, w.N, 56), [w.N - 1]]))
    trows = np.array([0, 1, 2, w.L // 2, w.L - 1])
    for s, rec in enumerate(stack["steps"], 1):
        q, k = oracle.block_qk(rec["x_prev"][rows], stack["img_pos"][rows], 0, None, wi0, w.H)
        assert_close(rec["q_img"][rows], q.reshape(len(rows), -1), "bf16", f"step {s} probe q")
        assert_close(rec["k_all"][w.L + rows], k.reshape(len(rows), -1), "bf16", f"step {s} probe k (image)")
        _, kt = oracle.block_qk(stack["text"][trows], np.zeros((len(trows), 3), np.int32), len(trows), wt0, None, w.H)
        assert_close(rec["k_all"][trows], kt.reshape(len(trows), -1), "bf16", f"step {s} probe k (text)")


def test_stack_lse_and_scores(stack):
    w = stack["w"]
    rows = np.unique(np.concatenate([np.arange(8), np.random.default_rng(4).integers(0, w.N, 56), [w.N - 1]]))
    for s, rec in enumerate(stack["steps"], 1):
        q = rec["q_img"].reshape(w.N, w.H, w.d)
        k_all = rec["k_all"].reshape(-1, w.H, w.d)
        ref = oracle.joint_lse(q[rows], k_all)
        assert np.abs(rec["lse"][:, rows] - ref).max() < 2e-3, f"step {s} lse"
        s_ref, _, _ = oracle.score(q, k_all[:w.L], rec["lse"], rec["x_prev"], rec["x_prev2"], w.alpha, w.eps_minmax)
        assert np.abs(rec["scores"] - s_ref).max() < 1e-4, f"step {s} scores"


def test_stack_select(stack):
    w, hw = stack["w"], stack["host_w"]
    wt0, wi0 = _f32(hw[("d", 0)][0]), _f32(hw[("d", 0)][1])
    pos = np.concatenate([np.zeros((w.L, 3), np.int32), stack["img_pos"]])
    for s, rec in enumerate(stack["steps"], 1):
        idx = rec["idx"]
        np.testing.assert_array_equal(idx, oracle.select_topk(rec["scores"], w.k), err_msg=f"step {s}")
        # The oracle's own probe, LSE and scores on this step's input: the two
        # selections may differ only at the selection boundary.
        q, k = oracle.block_qk(np.concatenate([stack["text"], rec["x_prev"]]), pos, w.L, wt0, wi0, w.H)
        lse = oracle.joint_lse(q[w.L:], k)
        s_ref, _, _ = oracle.score(q[w.L:], k[:w.L], lse, rec["x_prev"], rec["x_prev2"], w.alpha, w.eps_minmax)
        own = set(oracle.select_topk(s_ref, w.k).tolist())
        got = set(idx.tolist())
        kth = np.sort(s_ref.astype(np.float64))[::-1][w.k - 1]
        tol = 1e-2 * float(s_ref.max() - s_ref.min())
        bad = [i for i in got ^ own if abs(float(s_ref[i]) - kth) > tol]
        print(f"[stack] step {s}: {len(got ^ own)} boundary swaps, scores rel-L2 {rel_l2(rec['scores'], s_ref):.2e}")
        assert not bad, (s, bad[:8])
        assert rel_l2(rec["scores"], s_ref) < 1e-2


def test_stack_gather_scatter_bitexact(stack):
    w = stack["w"]
    for s, rec in enumerate(stack["steps"], 1):
        compact, pos, canvas = oracle.gather_upsample(stack["lowres"], rec["x_prev"], stack["text"], rec["idx"],
                                                      w.H_lr, w.W_lr)
        np.testing.assert_array_equal(rec["compact"], compact, err_msg=f"step {s} compact")
        np.testing.assert_array_equal(rec["pos"][w.L:], pos, err_msg=f"step {s} pos")
        np.testing.assert_array_equal(rec["canvas_gather"], canvas, err_msg=f"step {s} canvas")
        last = w.n_double + w.n_single - 1
        ref = oracle.scatter(rec["outs"][last], rec["idx"], w.L, rec["canvas_gather"])
        np.testing.assert_array_equal(rec["x_new"], ref, err_msg=f"step {s} scatter")


def test_stack_blocks_teacher_forced(stack):
    w, hw = stack["w"], stack["host_w"]
    worst = 0.0
    for s, rec in enumerate(stack["steps"], 1):
        rows = _sample_rows(w.S, w.L, 100 + s)
        for i in rec["check"]:
            x_in = rec["compact"] if i == 0 else rec["outs"][i - 1]
            if i < w.n_double:
                wt, wi = _f32(hw[("d", i)][0]), _f32(hw[("d", i)][1])
                ref, _ = oracle.double_block(x_in, rec["pos"], w.L, wt, wi, w.H, rows=rows)
            else:
                ref, _ = oracle.single_block(x_in, rec["pos"], _f32(hw[("s", i - w.n_double)]), w.H, rows=rows)
            out, x = rec["outs"][i][rows], x_in[rows]
            assert_close(out, ref, "bf16", f"step {s} block {i} x_out")
            err = rel_l2(out - x, ref - x)
            bar = _update_bar(out, ref, x)
            worst = max(worst, err / bar)
            assert err <= bar, f"step {s} block {i}: update rel-L2 {err:.3e} > {bar:.3e}"
    print(f"[stack] worst update error / bar = {worst:.3f}")
