"""The coordinate-bound noise kernel and the three-stage sampler
(Section 3.2) on the GPU against the oracle.

Noise: the generator's 32-bit stream bit-exact (avits_noise_bits vs
oracle.pixel_noise_bits); the normals and the re-injection on raster rows,
half-unit positions and low-res rows within the parity bar.

Sampler: ThreeStageSampler on a tiny model (2 double + 1 single blocks,
hidden 256, 16x16 -> 32x32, 64 latent channels, K = 64) with every stage
teacher-forced: the oracle runs each stage from the GPU's state after the
previous one.  Stage 1's latents, snapshots and collected mass, the
transition's scores, selection (bit-exact against the oracle's selection of
the GPU's scores), mixed positions and children (bit-exact) and re-injected
latents, Stage 2, the Stage 2 -> 3 expansion with its noise, and Stage 3,
each within the bar.  A free-running fp32 run checks the oracle's own
selection against the GPU's (different only at the selection boundary).
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import sampler as sp
from paper_2608_17995_amd.step import ThreeStageSampler
from synth import configs as C
from synth import generator as G

from _gpu import assert_close, dev, double_weights_dev, host

pytestmark = pytest.mark.gpu

CH = 64   # latent channels


@pytest.mark.parametrize("seed", [0, 5, (7 << 32) | 12345])
def test_noise_bits_bitexact(gpu, seed):
    first, n = 1000, 3001
    bits = torch.empty(n, CH, dtype=torch.int32, device="cuda")
    gpu.avits_noise_bits(first, bits, seed)
    torch.cuda.synchronize()
    got = bits.cpu().numpy().view(np.uint32)
    np.testing.assert_array_equal(got, oracle.pixel_noise_bits(np.arange(first, first + n), CH, seed))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("t", [1.0, 0.3, 0.0])
def test_noise_reinject_rows(gpu, dtype, t):
    H_lr, W_lr, seed = 6, 5, 99
    H_hr, W_hr = 2 * H_lr, 2 * W_lr
    N, Mp = H_hr * W_hr, H_lr * W_lr
    g = np.random.default_rng(4)
    # raster rows of the high-res grid
    x = G.round_to(g.standard_normal((N, CH)), dtype)
    tx = dev(x, dtype)
    gpu.avits_noise_reinject(tx, t, seed, H_hr, W_hr)
    ref = oracle.reinject(x, oracle.pixel_noise(np.arange(N), CH, seed), t)
    assert_close(host(tx), ref, dtype, f"raster rows t={t}")
    # low-res rows (the downsampled field)
    y = G.round_to(g.standard_normal((Mp, CH)), dtype)
    ty = dev(y, dtype)
    gpu.avits_noise_reinject(ty, t, seed, H_hr, W_hr, rows_kind=gpu.NOISE_LOWRES)
    ref = oracle.reinject(y, oracle.block_noise(np.arange(Mp), W_lr, CH, seed), t)
    assert_close(host(ty), ref, dtype, f"low-res rows t={t}")
    # rows at half-unit positions: the mixed sequence of a random selection
    idx = np.sort(g.permutation(Mp)[:7])
    _, pos, _ = oracle.gather_mixed(np.zeros((Mp, 8)), None, idx, H_lr, W_lr)
    z = G.round_to(g.standard_normal((pos.shape[0], CH)), dtype)
    tz = dev(z, dtype)
    gpu.avits_noise_reinject(tz, t, seed, H_hr, W_hr, pos=dev(pos))
    torch.cuda.synchronize()
    ref = oracle.reinject(z, oracle.halfunit_noise(pos, W_hr, CH, seed), t)
    assert_close(host(tz), ref, dtype, f"half-unit rows t={t}")
    if t == 0.0:
        np.testing.assert_array_equal(host(tz), z)


def test_positions_kernels(gpu):
    pos = torch.empty(77, 3, dtype=torch.int32, device="cuda")
    gpu.avits_grid_positions(pos, 9, frame=1, scale=4, offset=1)
    r = np.arange(77)
    np.testing.assert_array_equal(pos.cpu().numpy(), np.stack([np.ones(77), 4 * (r // 9) + 1, 4 * (r % 9) + 1], 1))
    src = torch.from_numpy(np.arange(30, dtype=np.int32).reshape(10, 3)).cuda()
    dst = torch.empty_like(src)
    gpu.avits_scale_positions(src, 2, dst)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(dst.cpu().numpy(), 2 * np.arange(30).reshape(10, 3))


# ---------------------------------------------------------------------------
# The sampler.

def _model(w):
    doubles = [(G.double_stream_weights(w, b, 0), G.double_stream_weights(w, b, 1)) for b in range(2)]
    singles = [G.single_block_weights(w, 0)]
    sw = G.sampler_weights(w, CH)
    return doubles, singles, sw


def _setup(gpu, w, K, steps):
    doubles, singles, sw = _model(w)
    bw_d = [gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=double_weights_dev(a, w.dtype), img=double_weights_dev(b, w.dtype))
            for a, b in doubles]
    bw_s = [gpu.BlockWeights(gpu.BLOCK_SINGLE, single=double_weights_dev(s, w.dtype)) for s in singles]
    sw_dev = {k: dev(v, w.dtype) for k, v in sw.items()}
    prefix = G.block_input(w, w.L, 21)
    ppos = G.prefix_positions(w)
    n1, nt, n2, n3 = steps
    samp = ThreeStageSampler(w.H_lr, w.W_lr, w.L, CH, w.D, w.H, w.mlp_ratio * w.D, bw_d, bw_s, sw_dev, dev(ppos), K,
                             n1, nt, n2, n3, torch.float32 if w.dtype == "f32" else torch.bfloat16, seed=w.seed + 31,
                             alpha=w.alpha)
    return samp, (doubles, singles, sw), prefix, ppos


@pytest.mark.parametrize("w", [C.TINY_F32, C.TINY_BF16], ids=["f32", "bf16"])
def test_three_stages_teacher_forced(gpu, w):
    K = C.mixed_keep_count(w.rho, w.N_lr)
    steps = (2, 2, 2, 2)
    samp, (doubles, singles, sw), prefix, ppos = _setup(gpu, w, K, steps)
    n1, nt, n2, n3 = steps
    t = sp.timesteps(sum(steps))
    seed, Cc, H_lr, W_lr = samp.seed, CH, w.H_lr, w.W_lr
    tp = dev(prefix, w.dtype)
    print(f"\n[three-stage] {w.name}: M'={w.N_lr} K={K} S1={samp.S1} S2={samp.S2} S3={samp.S3}", flush=True)

    # Stage 1 from the downsampled noise.
    samp.stage1(tp)
    torch.cuda.synchronize()
    z1, v1 = host(samp.z1), host(samp.v1)
    snaps = np.stack([host(z) for z in samp.snaps])
    mass = host(samp.mass)[:, w.L:]
    rz1, rv1, rsn, rmass, count = sp.stage1(prefix, ppos, sw, doubles, singles, w.H, H_lr, W_lr, Cc, seed, t, n1, nt)
    assert count == nt * len(doubles)
    assert_close(z1, rz1, w.dtype, "stage-1 latent")
    assert_close(snaps, rsn, w.dtype, "stage-1 snapshots")
    assert_close(mass, rmass, w.dtype, "collected text mass")
    assert_close(v1, rv1, w.dtype, "stage-1 last velocity")

    # Transition 1 -> 2 on the GPU's Stage-1 state.
    samp.transition12()
    torch.cuda.synchronize()
    scores, idx = samp.scores.cpu().numpy(), samp.idx[:K].cpu().numpy()
    t_s = t[n1 + nt]
    rs, _, rzm, rpos, rch = sp.transition12(z1, v1, t_s, mass, count, snaps, K, H_lr, W_lr, Cc, seed, w.alpha,
                                            w.eps_minmax, idx=idx)
    assert np.abs(scores - rs).max() < 1e-4
    np.testing.assert_array_equal(idx, oracle.select_topk(scores, K))
    np.testing.assert_array_equal(samp.pos2[w.L:].cpu().numpy(), rpos)
    np.testing.assert_array_equal(samp.pos2[:w.L].cpu().numpy(), 2 * ppos)
    np.testing.assert_array_equal(samp.children[:4 * K].cpu().numpy(), rch)
    z2 = host(samp.z2)
    assert_close(z2, rzm, w.dtype, "mixed sequence after re-injection")

    # Stage 2 on the GPU's mixed sequence.
    samp.stage2(tp)
    torch.cuda.synchronize()
    z2b, v2 = host(samp.z2), host(samp.v2)
    rz2, rv2 = sp.stage_steps(z2, prefix, np.concatenate([2 * ppos, rpos]), sw, doubles, singles, w.H, t, n1 + nt,
                              n2, pos_scale=0.5)
    assert_close(z2b, rz2, w.dtype, "stage-2 latent")
    assert_close(v2, rv2, w.dtype, "stage-2 last velocity")

    # Transition 2 -> 3 and Stage 3.
    samp.transition23()
    torch.cuda.synchronize()
    z3 = host(samp.z3)
    rz3 = sp.transition23(z2b, v2, t[n1 + nt + n2], idx, rch, H_lr, W_lr, Cc, seed)
    assert_close(z3, rz3, w.dtype, "full grid after re-injection")
    samp.stage3(tp)
    torch.cuda.synchronize()
    rz4, _ = sp.stage_steps(z3, prefix, np.concatenate([ppos, sp.highres_positions(w.H_hr, w.W_hr)]), sw, doubles,
                            singles, w.H, t, n1 + nt + n2, n3)
    assert_close(host(samp.z3), rz4, w.dtype, "final latent")


@pytest.mark.parametrize("K", [0, 256])
def test_three_stages_degenerate_keep(gpu, K):
    # K = 0 keeps every token at low resolution through Stage 2; K = M'
    # expands them all: both run, and Stage 3 starts from the right grid.
    w = C.TINY_F32
    steps = (1, 2, 1, 1)
    samp, (doubles, singles, sw), prefix, ppos = _setup(gpu, w, K, steps)
    tp = dev(prefix, w.dtype)
    samp.stage1(tp)
    samp.transition12()
    samp.stage2(tp)
    torch.cuda.synchronize()
    z2b, v2 = host(samp.z2), host(samp.v2)
    idx = samp.idx[:K].cpu().numpy()
    ch = samp.children[:4 * K].cpu().numpy()
    samp.transition23()
    torch.cuda.synchronize()
    t = sp.timesteps(sum(steps))
    rz3 = sp.transition23(z2b, v2, t[4], idx, ch, w.H_lr, w.W_lr, CH, samp.seed)
    assert_close(host(samp.z3), rz3, w.dtype, f"full grid after re-injection, K={K}")


def test_three_stages_free_running_f32(gpu):
    w = C.TINY_F32
    K = C.mixed_keep_count(w.rho, w.N_lr)
    steps = (2, 2, 2, 2)
    samp, (doubles, singles, sw), prefix, ppos = _setup(gpu, w, K, steps)
    n1, nt, n2, n3 = steps
    samp.run(dev(prefix, w.dtype))
    torch.cuda.synchronize()
    t = sp.timesteps(sum(steps))
    seed = samp.seed
    z1, v1, snaps, mass, count = sp.stage1(prefix, ppos, sw, doubles, singles, w.H, w.H_lr, w.W_lr, CH, seed, t,
                                           n1, nt)
    s, idx, zm, pos, ch = sp.transition12(z1, v1, t[n1 + nt], mass, count, snaps, K, w.H_lr, w.W_lr, CH, seed,
                                          w.alpha, w.eps_minmax)
    got = set(samp.idx[:K].cpu().numpy().tolist())
    ref = set(idx.tolist())
    kth = np.sort(s.astype(np.float64))[::-1][K - 1]
    for i in got ^ ref:
        assert abs(float(s[i]) - kth) <= 1e-4, (i, float(s[i]), kth)
    if got == ref:
        z2, v2 = sp.stage_steps(zm, prefix, np.concatenate([2 * ppos, pos]), sw, doubles, singles, w.H, t, n1 + nt, n2,
                                pos_scale=0.5)
        z3 = sp.transition23(z2, v2, t[n1 + nt + n2], idx, ch, w.H_lr, w.W_lr, CH, seed)
        z4, _ = sp.stage_steps(z3, prefix, np.concatenate([ppos, sp.highres_positions(w.H_hr, w.W_hr)]), sw, doubles,
                               singles, w.H, t, n1 + nt + n2, n3)
        assert_close(host(samp.z3), z4, "f32", "free-running final latent")
