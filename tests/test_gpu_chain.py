"""A stack of blocks with each block's first stage written by the block
before it (avits_block_forward_ex h_next / h_in, step.run_chain): the
last projection's split-K reduce applies the next block's layer norm and
modulation to the rows it produces (or the LN kernel does, when the
projection is not split), bit for bit what the next block would compute
itself.  Checked: every block output of a chained stack equals the plain
stack's bit for bit (double -> double -> single -> single, bf16 and fp32,
forced split and unsplit last projections), with the fused scatter on the
same block, at the FLUX 1024^2 shape, and the argument checks.
"""
import numpy as np
import pytest
import torch

from synth import configs as C
from synth import generator as G

from _gpu import dev, double_weights_dev, host

pytestmark = pytest.mark.gpu


def _stack(gpu, w, n_double=2, n_single=2):
    blocks = []
    for b in range(n_double):
        wt, wi = G.double_stream_weights(w, b, 0), G.double_stream_weights(w, b, 1)
        blocks.append(gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=double_weights_dev(wt, w.dtype),
                                       img=double_weights_dev(wi, w.dtype)))
    for b in range(n_single):
        blocks.append(gpu.BlockWeights(gpu.BLOCK_SINGLE, single=double_weights_dev(G.single_block_weights(w, b),
                                                                                    w.dtype)))
    return blocks


def _inputs(w, S, seed):
    x = G.block_input(w, S, seed)
    g = np.random.default_rng(4000 + seed)
    pos = np.zeros((S, 3), np.int32)
    pos[w.L:, 1] = g.integers(0, w.H_hr, S - w.L)
    pos[w.L:, 2] = g.integers(0, w.W_hr, S - w.L)
    return x, pos


def _plain(gpu, w, blocks, t_x, t_pos):
    outs, cur = [], t_x
    S = t_x.shape[0]
    for bw in blocks:
        nxt = torch.empty_like(t_x)
        gpu.avits_block_forward(cur, nxt, t_pos, w.L, S - w.L, bw, w.H)
        outs.append(nxt)
        cur = nxt
    return outs


def _chained(gpu, w, blocks, t_x, t_pos):
    from paper_2608_17995_amd.step import run_chain
    S = t_x.shape[0]
    outs = [torch.empty_like(t_x) for _ in blocks]
    hbuf = [torch.full_like(t_x, 5.0) for _ in range(2)]
    ws = torch.empty(max(gpu.avits_block_workspace_bytes(b.kind, S, w.H, w.D // w.H, w.mlp_ratio * w.D,
                                                         gpu.BF16 if w.dtype == "bf16" else gpu.F32) for b in blocks),
                     dtype=torch.uint8, device="cuda")
    run_chain(blocks, t_x, lambda i: outs[i], hbuf, t_pos, w.L, S, w.H, ws)
    return outs


@pytest.mark.parametrize("plan", [None, "256,3", "256,1", "128,2"], ids=["auto", "split3", "unsplit", "w128_split2"])
@pytest.mark.parametrize("w", [C.TINY_BF16, C.TINY_F32], ids=lambda w: w.name)
def test_chained_stack_matches_plain(gpu, monkeypatch, w, plan):
    if plan:
        monkeypatch.setenv("AVITS_GEMM_TILE_gemm_mlp_out", plan)
        monkeypatch.setenv("AVITS_GEMM_TILE_gemm_single_out", plan)
    S = w.L + w.R + w.k
    x, pos = _inputs(w, S, seed=2)
    blocks = _stack(gpu, w)
    t_x, t_pos = dev(x, w.dtype), dev(pos)
    ref = _plain(gpu, w, blocks, t_x, t_pos)
    got = _chained(gpu, w, blocks, t_x, t_pos)
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(zip(got, ref)):
        np.testing.assert_array_equal(host(a), host(b), err_msg=f"block {i}")


def test_next_stage_with_fused_scatter(gpu):
    # One block writes the next block's first stage and scatters its image rows.
    w = C.TINY_BF16
    S = w.L + w.R + w.k
    x, pos = _inputs(w, S, seed=4)
    blocks = _stack(gpu, w, 2, 0)
    t_x, t_pos = dev(x, w.dtype), dev(pos)
    idx = dev(np.sort(np.random.default_rng(4).permutation(w.N)[:w.k]).astype(np.int32))
    canvas0 = dev(G.block_input(w, w.N, 9), w.dtype)
    c1, c2 = canvas0.clone(), canvas0.clone()
    o1, o2 = torch.empty_like(t_x), torch.empty_like(t_x)
    h = torch.empty_like(t_x)
    gpu.avits_block_forward(t_x, o1, t_pos, w.L, S - w.L, blocks[0], w.H)
    gpu.avits_scatter(o1, idx, S - w.k, c1)
    gpu.avits_block_forward_ex(t_x, o2, t_pos, w.L, S - w.L, blocks[0], w.H, scatter_idx=idx, canvas=c2, h_next=h,
                               next_weights=blocks[1])
    p1, p2 = torch.empty_like(t_x), torch.empty_like(t_x)
    gpu.avits_block_forward(o1, p1, t_pos, w.L, S - w.L, blocks[1], w.H)
    gpu.avits_block_forward_ex(o2, p2, t_pos, w.L, S - w.L, blocks[1], w.H, h_in=h)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(o2), host(o1))
    np.testing.assert_array_equal(host(c2), host(c1))
    np.testing.assert_array_equal(host(p2), host(p1))


@pytest.mark.slow
def test_chained_flux_1024(gpu):
    w = C.FLUX_1024
    S = w.S
    x, pos = _inputs(w, S, seed=6)
    blocks = _stack(gpu, w, 2, 1)
    t_x, t_pos = dev(x, w.dtype), dev(pos)
    ref = _plain(gpu, w, blocks, t_x, t_pos)
    got = _chained(gpu, w, blocks, t_x, t_pos)
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(zip(got, ref)):
        assert torch.equal(a, b), f"block {i}"


def test_chain_rejects(gpu):
    w = C.TINY_BF16
    S = w.L + w.R + w.k
    x, pos = _inputs(w, S, seed=1)
    blocks = _stack(gpu, w, 2, 0)
    t_x, t_pos = dev(x, w.dtype), dev(pos)
    out = torch.empty_like(t_x)
    with pytest.raises(gpu.AvitsError):   # h_next without the next block's weights
        gpu.avits_block_forward_ex(t_x, out, t_pos, w.L, S - w.L, blocks[0], w.H, h_next=torch.empty_like(t_x))
    with pytest.raises(gpu.AvitsError):   # h_next aliasing x_out
        gpu.avits_block_forward_ex(t_x, out, t_pos, w.L, S - w.L, blocks[0], w.H, h_next=out, next_weights=blocks[1])
