"""Parity of the mixed-resolution Stage-2 path (Section 3.2): selection at
low-res granularity, the selected tokens expanded 2x2, the others kept at low
resolution in the same sequence, the block run with half-unit RoPE positions,
and the inverse re-layout.  Layouts, positions and children indices must
match the oracle bit for bit; block outputs within the parity bar.
"""
import numpy as np
import pytest
import torch

import oracle
from synth import configs as C
from synth import generator as G

from _gpu import assert_close, dev, double_weights_dev, host

TINY = [C.TINY_F32, C.TINY_BF16, C.TINY_BF16_REF, C.TINY_F32_RAGGED]
IDS = [w.name for w in TINY]

pytestmark = pytest.mark.gpu


def _mixed_rows(w, K):
    return 4 * K + w.N_lr - K


def _gather_mixed(gpu, w, K, mode, seed=0, children=True):
    lay = G.layout_inputs(w)
    idx = G.random_lowres_selection(w, K, seed)
    prefix = np.concatenate([lay["text"], lay["ref"]])
    t_low = dev(lay["lowres"], w.dtype)
    rows = _mixed_rows(w, K)
    compact = torch.full((w.LR + rows, w.D), 7.0, dtype=t_low.dtype, device="cuda")
    pos = torch.full((rows, 3), -1, dtype=torch.int32, device="cuda")
    ch = torch.full((4 * K,), -1, dtype=torch.int32, device="cuda") if children else None
    gpu.avits_gather_mixed(t_low, dev(prefix, w.dtype) if w.LR else None, dev(idx) if K else None,
                           w.H_lr, w.W_lr, compact, pos, ch, mode=mode)
    torch.cuda.synchronize()
    ref = oracle.gather_mixed(lay["lowres"], prefix, idx, w.H_lr, w.W_lr, "nearest" if mode == 0 else "bilinear")
    return (host(compact), host(pos), host(ch) if children else None), ref, idx, lay


@pytest.mark.parametrize("w", TINY, ids=IDS)
def test_gather_mixed_nearest_bitexact(gpu, w):
    K = C.mixed_keep_count(w.rho, w.N_lr)
    (compact, pos, ch), (rc, rp, rch), _, _ = _gather_mixed(gpu, w, K, 0)
    np.testing.assert_array_equal(compact, rc)
    np.testing.assert_array_equal(pos, rp)
    np.testing.assert_array_equal(ch, rch)


@pytest.mark.parametrize("w", [C.TINY_BF16, C.TINY_F32_RAGGED], ids=["bf16", "f32_ragged"])
@pytest.mark.parametrize("frac", [0.0, 0.37, 1.0], ids=["none", "some", "all"])
def test_gather_mixed_keep_fractions(gpu, w, frac):
    K = C.mixed_keep_count(frac, w.N_lr)
    (compact, pos, ch), (rc, rp, rch), _, lay = _gather_mixed(gpu, w, K, 0, seed=7)
    np.testing.assert_array_equal(compact, rc)
    np.testing.assert_array_equal(pos, rp)
    np.testing.assert_array_equal(ch, rch)
    if K == 0:
        np.testing.assert_array_equal(compact[w.LR:], lay["lowres"])
    if K == w.N_lr:
        np.testing.assert_array_equal(ch, np.arange(w.N))


@pytest.mark.parametrize("w", [C.TINY_BF16, C.TINY_F32], ids=["bf16", "f32"])
def test_gather_mixed_bilinear(gpu, w):
    K = C.mixed_keep_count(w.rho, w.N_lr)
    (compact, pos, ch), (rc, rp, rch), _, _ = _gather_mixed(gpu, w, K, 1, seed=3, children=False)
    np.testing.assert_array_equal(pos, rp)
    np.testing.assert_array_equal(compact[:w.LR], rc[:w.LR])
    np.testing.assert_array_equal(compact[w.LR + 4 * K:], rc[w.LR + 4 * K:])   # kept rows are copies
    got, want = compact[w.LR:w.LR + 4 * K], rc[w.LR:w.LR + 4 * K]
    if w.dtype == "bf16":
        # fp32 interpolation of bf16 values, one final rounding: within one bf16 ulp.
        assert np.all(np.abs(got - want) <= np.abs(want) * 2.0 ** -7 + 1e-30)
    else:
        assert np.abs(got - want).max() < 1e-5


@pytest.mark.parametrize("w", TINY, ids=IDS)
def test_scatter_mixed_bitexact(gpu, w):
    K = C.mixed_keep_count(w.rho, w.N_lr)
    lay = G.layout_inputs(w)
    idx = G.random_lowres_selection(w, K, 5)
    out = G.block_input(w, w.LR + _mixed_rows(w, K), 6)
    t_canvas, t_state = dev(lay["highres_prev"], w.dtype), dev(lay["lowres"], w.dtype)
    gpu.avits_scatter_mixed(dev(out, w.dtype), dev(idx), w.H_lr, w.W_lr, w.LR, t_canvas, t_state)
    torch.cuda.synchronize()
    rc, rs = oracle.scatter_mixed(out, idx, w.LR, w.H_lr, w.W_lr, lay["highres_prev"], lay["lowres"])
    np.testing.assert_array_equal(host(t_canvas), rc)
    np.testing.assert_array_equal(host(t_state), rs)


def test_scatter_mixed_extremes(gpu):
    w = C.TINY_BF16
    lay = G.layout_inputs(w)
    for K in (0, w.N_lr):
        idx = G.random_lowres_selection(w, K, 9)
        out = G.block_input(w, _mixed_rows(w, K), 10 + K)
        t_canvas = dev(lay["highres_prev"], w.dtype) if K else None
        t_state = dev(lay["lowres"], w.dtype) if K < w.N_lr else None
        gpu.avits_scatter_mixed(dev(out, w.dtype), dev(idx) if K else None, w.H_lr, w.W_lr, 0, t_canvas, t_state)
        torch.cuda.synchronize()
        rc, rs = oracle.scatter_mixed(out, idx, 0, w.H_lr, w.W_lr, lay["highres_prev"], lay["lowres"])
        if K:
            np.testing.assert_array_equal(host(t_canvas), rc)
        else:
            np.testing.assert_array_equal(host(t_state), rs)


def _mixed_block(gpu, w, K, seed):
    """Double block on the mixed sequence (prefix positions doubled, pos_scale
    0.5) against the oracle block at the real-valued positions."""
    (compact, pos, _), _, idx, _ = _gather_mixed(gpu, w, K, 0, seed=seed, children=False)
    pos_all = np.concatenate([2 * G.prefix_positions(w), pos]).astype(np.int32)
    wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
    t_x = dev(compact, w.dtype)
    out = torch.empty_like(t_x)
    lse = torch.empty(w.H, compact.shape[0], device="cuda")
    bw = gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=double_weights_dev(wt, w.dtype), img=double_weights_dev(wi, w.dtype))
    gpu.avits_block_forward(t_x, out, dev(pos_all), w.L, compact.shape[0] - w.L, bw, w.H, lse_out=lse,
                            pos_scale=0.5)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.double_block(compact, pos_all / 2.0, w.L, wt, wi, w.H)
    return compact, host(out), host(lse), ref, ref_lse, idx


@pytest.mark.parametrize("w", TINY, ids=IDS)
def test_block_on_mixed_sequence(gpu, w):
    K = C.mixed_keep_count(w.rho, w.N_lr)
    x, out, lse, ref, ref_lse, _ = _mixed_block(gpu, w, K, seed=11)
    assert_close(out, ref, w.dtype, "x_out")
    assert_close(out - x, ref - x, w.dtype, "block update x_out - x_in")
    assert_close(lse, ref_lse, w.dtype, "lse")


def test_half_unit_positions_are_not_integer_positions(gpu):
    # The kept tokens' fractional positions matter: rounding them to the grid
    # changes the block output well beyond the parity bar.
    w = C.TINY_F32
    K = C.mixed_keep_count(w.rho, w.N_lr)
    x, out, _, _, _, idx = _mixed_block(gpu, w, K, seed=12)
    (_, pos, _), _, _, _ = _gather_mixed(gpu, w, K, 0, seed=12, children=False)
    pos_all = np.concatenate([2 * G.prefix_positions(w), pos]).astype(np.float64)
    wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
    snapped, _ = oracle.double_block(x, np.floor(pos_all / 2.0), w.L, wt, wi, w.H)
    assert np.abs(out - snapped).max() > 1e-2


def test_mixed_stage2_step(gpu):
    """One Stage-2 step end to end at low-res granularity: score the M' low-res
    tokens, select floor(rho M'), gather the mixed sequence, run a double block
    and a single block, and scatter; each stage checked against the oracle on
    the values the GPU stage consumed."""
    w = C.TINY_BF16
    Mp, K = w.N_lr, C.mixed_keep_count(w.rho, w.N_lr)
    g = np.random.default_rng(21)
    scores = g.random(Mp).astype(np.float32)
    idx = torch.empty(K, dtype=torch.int32, device="cuda")
    gpu.avits_select(dev(scores), K, idx)
    ref_idx = oracle.select_topk(scores, K)
    np.testing.assert_array_equal(host(idx), ref_idx)
    lay = G.layout_inputs(w)
    prefix = np.concatenate([lay["text"], lay["ref"]])
    rows = _mixed_rows(w, K)
    S = w.LR + rows
    compact = torch.empty(S, w.D, dtype=torch.bfloat16, device="cuda")
    pos = torch.empty(S, 3, dtype=torch.int32, device="cuda")
    pos[:w.LR] = dev(2 * G.prefix_positions(w))
    children = torch.empty(4 * K, dtype=torch.int32, device="cuda")
    t_low = dev(lay["lowres"], w.dtype)
    gpu.avits_gather_mixed(t_low, dev(prefix, w.dtype) if w.LR else None, idx, w.H_lr, w.W_lr, compact,
                           pos[w.LR:], children)
    wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
    ws = G.single_block_weights(w, 0)
    bd = gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=double_weights_dev(wt, w.dtype), img=double_weights_dev(wi, w.dtype))
    bs = gpu.BlockWeights(gpu.BLOCK_SINGLE, single=double_weights_dev(ws, w.dtype))
    mid, out = torch.empty_like(compact), torch.empty_like(compact)
    gpu.avits_block_forward(compact, mid, pos, w.L, S - w.L, bd, w.H, pos_scale=0.5)
    gpu.avits_block_forward(mid, out, pos, w.L, S - w.L, bs, w.H, pos_scale=0.5)
    canvas, state = dev(lay["highres_prev"], w.dtype), t_low.clone()
    gpu.avits_scatter_mixed(out, idx, w.H_lr, w.W_lr, w.LR, canvas, state)
    torch.cuda.synchronize()
    rc, rp, rch = oracle.gather_mixed(lay["lowres"], prefix, ref_idx, w.H_lr, w.W_lr)
    np.testing.assert_array_equal(host(compact), rc)
    np.testing.assert_array_equal(host(pos)[w.LR:], rp)
    np.testing.assert_array_equal(host(children), rch)
    p = host(pos) / 2.0
    r_mid, _ = oracle.double_block(rc, p, w.L, wt, wi, w.H)
    assert_close(host(mid), r_mid, w.dtype, "double block")
    r_out, _ = oracle.single_block(host(mid), p, ws, w.H)
    assert_close(host(out), r_out, w.dtype, "single block")
    ref_canvas, ref_state = oracle.scatter_mixed(host(out), ref_idx, w.LR, w.H_lr, w.W_lr, lay["highres_prev"],
                                                 lay["lowres"])
    np.testing.assert_array_equal(host(canvas), ref_canvas)
    np.testing.assert_array_equal(host(state), ref_state)
    # Stage 3 from that state: the kept tokens upsampled around the children.
    compact3 = torch.empty(4 * K, w.D, dtype=torch.bfloat16, device="cuda")
    pos3 = torch.empty(4 * K, 3, dtype=torch.int32, device="cuda")
    gpu.avits_gather_upsample(state, canvas, None, children, w.H_lr, w.W_lr, compact3, pos3, canvas)
    torch.cuda.synchronize()
    _, _, full = oracle.gather_upsample(ref_state, ref_canvas, None, rch, w.H_lr, w.W_lr)
    np.testing.assert_array_equal(host(canvas), full)


@pytest.mark.parametrize("probes", [(0,), (0, 1)], ids=["probe0", "probe01"])
def test_mixed_stage2_class(gpu, probes):
    """MixedStage2 over a 2 double + 1 single stack: the transition (probe at
    low res, N_T = 3 snapshots, select, gather) and two Stage-2 steps, each
    stage checked on the GPU's own inputs of that stage."""
    from paper_2608_17995_amd.step import MixedStage2
    w = C.TINY_BF16.replace(name="tiny_bf16_mixed", n_double=2, n_single=1)
    Mp, K = w.N_lr, C.mixed_keep_count(w.rho, w.N_lr)
    g = G.rng(w.seed, 900)
    z = G.round_to(g.standard_normal((Mp, w.D)), "bf16")
    snaps = [G.round_to(z + 0.1 * (3 - j) * g.standard_normal((Mp, w.D)), "bf16") for j in range(3)]
    lay = G.layout_inputs(w)
    prefix = np.concatenate([lay["text"], lay["ref"]])
    dw = [(G.double_stream_weights(w, b, 0), G.double_stream_weights(w, b, 1)) for b in range(w.n_double)]
    sw = [G.single_block_weights(w, b) for b in range(w.n_single)]
    doubles = [gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=double_weights_dev(t, w.dtype), img=double_weights_dev(i, w.dtype))
               for t, i in dw]
    singles = [gpu.BlockWeights(gpu.BLOCK_SINGLE, single=double_weights_dev(x, w.dtype)) for x in sw]
    m = MixedStage2(w.H_lr, w.W_lr, w.L, w.R, K, w.D, w.H, w.mlp_ratio * w.D, doubles, singles,
                    G.prefix_positions(w), torch.bfloat16, alpha=w.alpha, eps=w.eps_minmax, probe_blocks=probes)
    t_z = dev(z, "bf16")
    m.transition(t_z, [dev(s, "bf16") for s in snaps], dev(prefix, "bf16") if w.LR else None)
    torch.cuda.synchronize()
    # Probe at low-res grid positions; prefix at its own positions.
    r = np.arange(Mp)
    pos_lr = np.concatenate([G.prefix_positions(w), np.stack([0 * r, r // w.W_lr, r % w.W_lr], 1)])
    mass = np.zeros((w.H, Mp))
    for b in probes:
        q, k = oracle.block_qk(np.concatenate([prefix, z]), pos_lr, w.L, dw[b][0], dw[b][1], w.H)
        mass += oracle.text_attention_mass(q[w.LR:], k, w.L)
    assert_close(host(m.mass), mass, "bf16", "probe mass")
    s_ref, _, _ = oracle.score_from_mass(host(m.mass), len(probes), np.stack(snaps), w.alpha, w.eps_minmax)
    scores = m.scores.cpu().numpy()
    assert_close(scores, s_ref, "bf16", "scores")
    idx = m.idx.cpu().numpy()
    np.testing.assert_array_equal(idx, oracle.select_topk(scores, K))
    rc, rp, rch = oracle.gather_mixed(z, prefix, idx, w.H_lr, w.W_lr)
    np.testing.assert_array_equal(host(m.x), rc)
    np.testing.assert_array_equal(host(m.pos)[w.LR:], rp)
    np.testing.assert_array_equal(host(m.children), rch)
    p = host(m.pos) / 2.0
    np.testing.assert_array_equal(p[:w.LR], G.prefix_positions(w))
    for s in range(2):
        outs = {}

        def on_block(i, x_in, x_out):
            torch.cuda.synchronize()
            outs[i] = (host(x_in), host(x_out))

        m.step(on_block=on_block)
        torch.cuda.synchronize()
        for i, (x_in, x_out) in outs.items():
            if i < w.n_double:
                ref, _ = oracle.double_block(x_in, p, w.L, dw[i][0], dw[i][1], w.H)
            else:
                ref, _ = oracle.single_block(x_in, p, sw[i - w.n_double], w.H)
            assert_close(x_out - x_in, ref - x_in, "bf16", f"step {s} block {i} update")
        np.testing.assert_array_equal(host(m.x), outs[w.n_double + w.n_single - 1][1])
    canvas, state = dev(lay["highres_prev"], "bf16"), t_z.clone()
    m.leave(canvas, state)
    torch.cuda.synchronize()
    rcv, rst = oracle.scatter_mixed(host(m.x), idx, w.LR, w.H_lr, w.W_lr, lay["highres_prev"], z)
    np.testing.assert_array_equal(host(canvas), rcv)
    np.testing.assert_array_equal(host(state), rst)
