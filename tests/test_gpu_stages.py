"""Stage-by-stage parity of the HIP path against the oracle on identical inputs.

Each stage's oracle runs on exactly the values the GPU stage consumed (the
GPU's own upstream outputs copied to the host), so indices and layouts must
match bit for bit and floats within the parity bar.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from synth import configs as C
from synth import generator as G

from _gpu import assert_close, dev, double_weights_dev, host, rel_l2

TINY = [C.TINY_F32, C.TINY_BF16, C.TINY_BF16_REF, C.TINY_F32_RAGGED]
IDS = [w.name for w in TINY]

pytestmark = pytest.mark.gpu


def _k_all(si):
    return np.concatenate([si["text_k"], si["ref_k"], si["latent_k"]])


def _lse_gpu(gpu, w, si):
    lse = torch.empty(w.H, w.N, device="cuda")
    gpu.avits_joint_lse(dev(si["latent_q"], w.dtype), dev(_k_all(si), w.dtype), lse)
    return lse


@pytest.mark.parametrize("w", TINY, ids=IDS)
def test_joint_lse(gpu, w):
    si = G.score_inputs(w)
    lse = _lse_gpu(gpu, w, si)
    torch.cuda.synchronize()
    ref = oracle.joint_lse(si["latent_q"], _k_all(si))
    assert_close(host(lse), ref, w.dtype, "joint_lse")
    assert np.abs(host(lse) - ref).max() < 1e-3


@pytest.mark.parametrize("w", TINY, ids=IDS)
def test_score(gpu, w):
    si = G.score_inputs(w)
    lse = _lse_gpu(gpu, w, si)
    S = torch.empty(w.N, device="cuda")
    A = torch.empty(w.N, device="cuda")
    V = torch.empty(w.N, device="cuda")
    gpu.avits_score(dev(si["latent_q"], w.dtype), dev(si["text_k"], w.dtype), lse, dev(si["feat_t"], w.dtype),
                    dev(si["feat_prev"], w.dtype), w.alpha, w.eps_minmax, S, A, V)
    torch.cuda.synchronize()
    s_ref, a_ref, v_ref = oracle.score(si["latent_q"], si["text_k"], host(lse), si["feat_t"], si["feat_prev"],
                                       w.alpha, w.eps_minmax)
    assert_close(host(A), a_ref, w.dtype, "A")
    assert_close(host(V), v_ref, w.dtype, "V")
    assert_close(host(S), s_ref, w.dtype, "S")
    # fp32 arithmetic on both bf16 and fp32 inputs: the fused score is tight either way.
    assert np.abs(host(S) - s_ref).max() < 1e-4
    np.testing.assert_allclose(host(A), a_ref, rtol=1e-4)
    np.testing.assert_allclose(host(V), v_ref, rtol=1e-4)


def _score_select_case(gpu, w, k, scores_override=None):
    si = G.score_inputs(w)
    lse = _lse_gpu(gpu, w, si)
    args = [dev(si["latent_q"], w.dtype), dev(si["text_k"], w.dtype), lse, dev(si["feat_t"], w.dtype),
            dev(si["feat_prev"], w.dtype), w.alpha, w.eps_minmax]
    S1, A1, V1 = (torch.empty(w.N, device="cuda") for _ in range(3))
    S2, A2, V2 = (torch.full((w.N,), float("nan"), device="cuda") for _ in range(3))
    idx1 = torch.empty(k, dtype=torch.int32, device="cuda")
    idx2 = torch.full((k,), -1, dtype=torch.int32, device="cuda")
    gpu.avits_score(*args, S1, A1, V1)
    if k:
        gpu.avits_select(S1, k, idx1)
    gpu.avits_score_select(*args, S2, k, idx2, A2, V2)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(S2.cpu().numpy(), S1.cpu().numpy())
    np.testing.assert_array_equal(A2.cpu().numpy(), A1.cpu().numpy())
    np.testing.assert_array_equal(V2.cpu().numpy(), V1.cpu().numpy())
    np.testing.assert_array_equal(idx2.cpu().numpy(), idx1.cpu().numpy())
    np.testing.assert_array_equal(idx2.cpu().numpy(), oracle.select_topk(S2.cpu().numpy(), k))


@pytest.mark.parametrize("w", TINY, ids=IDS)
def test_score_select_matches_the_two_calls(gpu, w):
    # The fused call writes the same scores and raw terms, bit for bit, and
    # the selection of them; every k regime (none, a few, the workload's, all).
    for k in sorted({0, 1, w.k, w.N - 1, w.N}):
        _score_select_case(gpu, w, k)


@pytest.mark.parametrize("lr", [(32, 32), (64, 64), (40, 51)], ids=["N4096", "N16384", "N8160"])
def test_score_select_sizes(gpu, lr):
    # Up to the one-workgroup limit, with a ragged size and the FLUX head layout shrunk to 2 heads.
    w = C.TINY_BF16.replace(H_lr=lr[0], W_lr=lr[1])
    _score_select_case(gpu, w, C.keep_count(0.3, w.N))


@pytest.mark.parametrize("w", [C.TINY_F32, C.TINY_BF16], ids=["f32", "bf16"])
def test_score_without_optional_outputs_and_small_feature_width(gpu, w):
    # D_f = 64 (the packed-latent reading of the snapshots); A/V outputs omitted.
    w = w.replace(D_f=64)
    si = G.score_inputs(w)
    lse = _lse_gpu(gpu, w, si)
    S = torch.empty(w.N, device="cuda")
    gpu.avits_score(dev(si["latent_q"], w.dtype), dev(si["text_k"], w.dtype), lse, dev(si["feat_t"], w.dtype),
                    dev(si["feat_prev"], w.dtype), w.alpha, w.eps_minmax, S)
    torch.cuda.synchronize()
    s_ref, _, _ = oracle.score(si["latent_q"], si["text_k"], host(lse), si["feat_t"], si["feat_prev"],
                               w.alpha, w.eps_minmax)
    assert np.abs(host(S) - s_ref).max() < 1e-4


@pytest.mark.parametrize("w", TINY, ids=IDS)
def test_score_batched(gpu, w):
    """Three images of one shape in one launch: each matches the oracle, and
    is bit-identical to avits_score on that image alone (own min-max)."""
    ws = [w, w.replace(seed=w.seed + 1), w.replace(seed=w.seed + 2)]
    si = [G.score_inputs(x) for x in ws]
    lse = [_lse_gpu(gpu, x, s) for x, s in zip(ws, si)]
    stack = lambda key: torch.stack([dev(s[key], w.dtype) for s in si])  # noqa: E731
    S = torch.empty(len(ws), w.N, device="cuda")
    A = torch.empty_like(S)
    V = torch.empty_like(S)
    gpu.avits_score_batched(stack("latent_q"), stack("text_k"), torch.stack(lse), stack("feat_t"),
                            stack("feat_prev"), w.alpha, w.eps_minmax, S, A, V)
    torch.cuda.synchronize()
    for b, (x, s) in enumerate(zip(ws, si)):
        s_ref, a_ref, v_ref = oracle.score(s["latent_q"], s["text_k"], host(lse[b]), s["feat_t"], s["feat_prev"],
                                           w.alpha, w.eps_minmax)
        assert_close(host(A[b]), a_ref, w.dtype, f"image {b} A")
        assert_close(host(V[b]), v_ref, w.dtype, f"image {b} V")
        assert np.abs(host(S[b]) - s_ref).max() < 1e-4
        one = torch.empty(w.N, device="cuda")
        gpu.avits_score(dev(s["latent_q"], w.dtype), dev(s["text_k"], w.dtype), lse[b], dev(s["feat_t"], w.dtype),
                        dev(s["feat_prev"], w.dtype), w.alpha, w.eps_minmax, one)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(S[b]), host(one), err_msg=f"image {b} vs its own launch")


def test_score_batched_flux_pair(gpu):
    """The CFG pair at the FLUX 1024^2 shape (N = 4096, L = 512, 24 heads):
    each image's scores are bit-identical to its own single-image launch,
    and a sample of rows matches the oracle."""
    w = C.FLUX_1024
    ws = [w, w.replace(seed=w.seed + 1)]
    si = [G.score_inputs(x) for x in ws]
    lse = [_lse_gpu(gpu, x, s) for x, s in zip(ws, si)]
    stack = lambda key: torch.stack([dev(s[key], w.dtype) for s in si])  # noqa: E731
    S = torch.empty(2, w.N, device="cuda")
    A = torch.empty_like(S)
    V = torch.empty_like(S)
    gpu.avits_score_batched(stack("latent_q"), stack("text_k"), torch.stack(lse), stack("feat_t"),
                            stack("feat_prev"), w.alpha, w.eps_minmax, S, A, V)
    rows = np.random.default_rng(5).choice(w.N, 64, replace=False)
    for b, s in enumerate(si):
        one = torch.empty(w.N, device="cuda")
        gpu.avits_score(dev(s["latent_q"], w.dtype), dev(s["text_k"], w.dtype), lse[b], dev(s["feat_t"], w.dtype),
                        dev(s["feat_prev"], w.dtype), w.alpha, w.eps_minmax, one)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(S[b]), host(one), err_msg=f"image {b}")
        _, a_ref, v_ref = oracle.score(s["latent_q"][rows], s["text_k"], host(lse[b])[:, rows], s["feat_t"][rows],
                                       s["feat_prev"][rows], w.alpha, w.eps_minmax)
        np.testing.assert_allclose(host(A[b])[rows], a_ref, rtol=1e-4, atol=1e-7)
        np.testing.assert_allclose(host(V[b])[rows], v_ref, rtol=1e-4)


def _select(gpu, scores_np, k):
    s = torch.from_numpy(np.ascontiguousarray(scores_np, dtype=np.float32)).cuda()
    idx = torch.full((max(k, 1),), -7, dtype=torch.int32, device="cuda")
    gpu.avits_select(s, k, idx[:k])
    torch.cuda.synchronize()
    return host(idx)[:k], host(idx)


@pytest.mark.parametrize("n,k", [(1, 1), (5, 2), (1000, 1), (1024, 256), (1025, 1024), (4096, 1229),
                                 (3001, 3001), (16384, 4915), (20000, 7)])
def test_select_random(gpu, n, k):
    s = np.random.default_rng(n * 7 + k).standard_normal(n).astype(np.float32)
    got, _ = _select(gpu, s, k)
    np.testing.assert_array_equal(got, oracle.select_topk(s, k))


@pytest.mark.parametrize("n,k,levels", [(4096, 1229, 8), (1000, 500, 2), (2048, 2047, 1), (777, 300, 3)])
def test_select_ties_lowest_index(gpu, n, k, levels):
    s = G.quantised_scores(n, n, levels)
    got, _ = _select(gpu, s, k)
    np.testing.assert_array_equal(got, oracle.select_topk(s, k))


def test_select_special_values_and_k0(gpu):
    s = np.array([np.nan, -0.0, 0.0, -np.inf, np.inf, np.nan, -1.0, 3.0, -0.0], dtype=np.float32)
    for k in range(len(s) + 1):
        got, _ = _select(gpu, s, k)
        np.testing.assert_array_equal(got, oracle.select_topk(s, k))
    # k = 0 writes nothing.
    _, raw = _select(gpu, s, 0)
    assert raw[0] == -7


# Above 16384 scores the selection runs grid-wide (histogram passes over many
# workgroups, chunked index-order emission).
@pytest.mark.parametrize("n,k", [(16385, 1), (16385, 16385), (65573, 19672), (1 << 20, 314573),
                                 (3_000_017, 900_005)])
def test_select_grid_random(gpu, n, k):
    g = np.random.default_rng(n + k)
    s = g.standard_normal(n).astype(np.float32)
    got, raw = _select(gpu, s, k)
    np.testing.assert_array_equal(got, oracle.select_topk(s, k))
    # Min-max-normalised scores share their top bits (one exponent for most
    # of [0.5, 1)): the histogram's concentrated-digit path.
    u = g.random(n).astype(np.float32) ** 0.25
    got, _ = _select(gpu, u, k)
    np.testing.assert_array_equal(got, oracle.select_topk(u, k))


@pytest.mark.parametrize("n,k,levels", [(100_003, 30_001, 8), (1 << 20, 524_288, 2), (70_000, 69_999, 1),
                                        (200_000, 123, 3)])
def test_select_grid_ties_lowest_index(gpu, n, k, levels):
    s = G.quantised_scores(n, n, levels)
    got, _ = _select(gpu, s, k)
    np.testing.assert_array_equal(got, oracle.select_topk(s, k))


def test_select_grid_special_values(gpu):
    n = 50_000
    g = np.random.default_rng(5)
    s = g.standard_normal(n).astype(np.float32)
    specials = np.array([np.nan, -0.0, 0.0, -np.inf, np.inf], dtype=np.float32)
    pos = g.integers(0, n, 5000)
    s[pos] = specials[g.integers(0, len(specials), 5000)]
    for k in (1, 37, 20_000, n - 3, n):
        buf = torch.full((n + 8,), -7, dtype=torch.int32, device="cuda")
        gpu.avits_select(torch.from_numpy(s).cuda(), k, buf[:k])
        torch.cuda.synchronize()
        raw = host(buf)
        np.testing.assert_array_equal(raw[:k], oracle.select_topk(s, k))
        assert np.all(raw[k:] == -7)  # nothing written past k


def test_select_grid_workspace(gpu):
    assert gpu.avits_select_workspace_bytes(16384) == 0
    assert gpu.avits_select_workspace_bytes(16385) > 0
    s = torch.rand(40_000, device="cuda")
    idx = torch.empty(10, dtype=torch.int32, device="cuda")
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(gpu.AvitsError) as e:
        gpu.avits_select(s, 10, idx, workspace=small)
    assert e.value.code == -3


# The paper's tie-break perturbation (Section 3.3): keys are the fp32 sums
# scores + delta; both paths (one workgroup, grid-wide).
@pytest.mark.parametrize("n,k,levels", [(4096, 1229, 8), (777, 300, 2), (16384, 4915, 3), (70_000, 21_000, 4),
                                        (1 << 20, 314573, 8)])
def test_select_perturbed(gpu, n, k, levels):
    s = G.quantised_scores(n, n, levels)
    d = G.tiebreak_noise(n, n)
    idx = torch.full((k,), -7, dtype=torch.int32, device="cuda")
    gpu.avits_select_perturbed(dev(s), dev(d), k, idx)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(idx), oracle.select_topk_perturbed(s, d, k))


@pytest.mark.parametrize("perturbed", [False, True], ids=["plain", "perturbed"])
def test_select_batched(gpu, perturbed):
    sizes = [4096, 1, 1000, 16384, 64, 4096, 257]
    ks = [1229, 1, 0, 4915, 64, 0, 100]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    s = G.quantised_scores(11, int(off[-1]), 6)
    d = G.tiebreak_noise(11, int(off[-1])) if perturbed else None
    idx = torch.full((sum(ks) + 4,), -7, dtype=torch.int32, device="cuda")
    gpu.avits_select_batched(dev(s), off.tolist(), ks, idx, delta=dev(d) if perturbed else None)
    torch.cuda.synchronize()
    raw = host(idx)
    np.testing.assert_array_equal(raw[:sum(ks)], oracle.select_topk_batched(s, off, ks, delta=d))
    assert np.all(raw[sum(ks):] == -7)
    # Element by element, the batched result equals the single selection.
    o = 0
    for b in range(len(sizes)):
        if ks[b]:
            one, _ = _select(gpu, s[off[b]:off[b + 1]] if d is None else
                             (s[off[b]:off[b + 1]] + d[off[b]:off[b + 1]]).astype(np.float32), ks[b])
            np.testing.assert_array_equal(raw[o:o + ks[b]], one)
        o += ks[b]


def _gather(gpu, w, k, mode, alias, seed=0):
    lay = G.layout_inputs(w)
    idx = G.random_selection(w, k, seed)
    prefix = np.concatenate([lay["text"], lay["ref"]])
    t_low, t_high = dev(lay["lowres"], w.dtype), dev(lay["highres_prev"], w.dtype)
    t_pre = dev(prefix, w.dtype) if w.LR else None
    t_idx = dev(idx)
    compact = torch.full((w.LR + k, w.D), 7.0, dtype=t_low.dtype, device="cuda")
    pos = torch.full((k, 3), -1, dtype=torch.int32, device="cuda")
    canvas = t_high if alias else torch.full_like(t_high, 7.0)
    gpu.avits_gather_upsample(t_low, t_high, t_pre, t_idx, w.H_lr, w.W_lr, compact, pos, canvas, mode=mode)
    torch.cuda.synchronize()
    ref = oracle.gather_upsample(lay["lowres"], lay["highres_prev"], prefix, idx, w.H_lr, w.W_lr,
                                 "nearest" if mode == 0 else "bilinear")
    return (host(compact), host(pos), host(canvas)), ref, idx


@pytest.mark.parametrize("w", TINY, ids=IDS)
@pytest.mark.parametrize("alias", [False, True], ids=["separate", "in_place"])
def test_gather_nearest_bitexact(gpu, w, alias):
    (compact, pos, canvas), (rc, rp, rcv), idx = _gather(gpu, w, w.k, 0, alias)
    np.testing.assert_array_equal(compact, rc)
    np.testing.assert_array_equal(pos, rp)
    np.testing.assert_array_equal(canvas, rcv)


@pytest.mark.parametrize("w", [C.TINY_BF16, C.TINY_F32], ids=["bf16", "f32"])
def test_gather_keep_none_and_all(gpu, w):
    for k in (0, w.N):
        (compact, pos, canvas), (rc, rp, rcv), _ = _gather(gpu, w, k, 0, False)
        np.testing.assert_array_equal(compact, rc)
        np.testing.assert_array_equal(canvas, rcv)
        if k == 0:  # pure upsampling
            np.testing.assert_array_equal(canvas, oracle.upsample_nearest(G.layout_inputs(w)["lowres"], w.H_lr, w.W_lr))
        else:       # dense fallback: every token keeps its high-res features
            np.testing.assert_array_equal(canvas, G.layout_inputs(w)["highres_prev"])


@pytest.mark.parametrize("w", [C.TINY_BF16, C.TINY_F32_RAGGED], ids=["bf16", "f32"])
def test_gather_bilinear(gpu, w):
    (compact, pos, canvas), (rc, rp, rcv), _ = _gather(gpu, w, w.k, 1, False)
    np.testing.assert_array_equal(compact, rc)
    np.testing.assert_array_equal(pos, rp)
    if w.dtype == "bf16":
        # fp32 interpolation of bf16 values, one final rounding: within one bf16 ulp.
        ulp = np.abs(rcv) * 2.0 ** -7 + 1e-30
        assert np.all(np.abs(canvas - rcv) <= ulp)
    else:
        assert np.abs(canvas - rcv).max() < 1e-5


@pytest.mark.parametrize("w", TINY, ids=IDS)
def test_scatter_bitexact(gpu, w):
    lay = G.layout_inputs(w)
    idx = G.random_selection(w, w.k, 3)
    out = G.block_input(w, w.S, 5)
    t_canvas = dev(lay["highres_prev"], w.dtype)
    gpu.avits_scatter(dev(out, w.dtype), dev(idx), w.LR, t_canvas)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(t_canvas), oracle.scatter(out, idx, w.LR, lay["highres_prev"]))


# Rows longer than one 8 KiB copy batch (64 lanes x 8 chunks of 16 bytes): a
# second batch plus a partial tail, so every lane-chunk bound of the row copy
# is taken.  fp32 D = 2304 is 9216 bytes per row (576 chunks: one full batch,
# 64 chunks more); bf16 D = 4160 is 8320 bytes (520 chunks: 8 more).
WIDE = [dataclasses.replace(C.TINY_F32_RAGGED, name="wide_f32_d2304", D=2304, H=3, d=768),
        dataclasses.replace(C.TINY_F32_RAGGED, name="wide_bf16_d4160", dtype="bf16", D=4160, H=5, d=832)]


@pytest.mark.parametrize("w", WIDE, ids=[w.name for w in WIDE])
def test_gather_and_scatter_wide_rows(gpu, w):
    for k, alias in ((w.k, False), (w.k, True), (0, False), (w.N, False)):
        (compact, pos, canvas), (rc, rp, rcv), _ = _gather(gpu, w, k, 0, alias)
        np.testing.assert_array_equal(compact, rc)
        np.testing.assert_array_equal(pos, rp)
        np.testing.assert_array_equal(canvas, rcv)
    lay = G.layout_inputs(w)
    idx = G.random_selection(w, w.k, 3)
    out = G.block_input(w, w.S, 5)
    t_canvas = dev(lay["highres_prev"], w.dtype)
    gpu.avits_scatter(dev(out, w.dtype), dev(idx), w.LR, t_canvas)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(t_canvas), oracle.scatter(out, idx, w.LR, lay["highres_prev"]))


@pytest.mark.parametrize("w", TINY, ids=IDS)
@pytest.mark.parametrize("mode,alias", [(0, False), (0, True), (1, False)], ids=["nearest", "nearest_in_place",
                                                                                 "bilinear"])
def test_gather_and_scatter_batched(gpu, w, mode, alias):
    """Three images in one launch each way (k_b = the workload's k, none, all
    N), their rows placed out of image order with gaps in one packed buffer:
    every image's rows, positions and canvas equal the oracle's for that image
    alone (bit-exact; bilinear bf16 within one ulp, as the single launch), and
    rows between the images are left untouched."""
    ws = [w.replace(seed=w.seed + i) for i in range(3)]
    ks = [w.k, 0, w.N]
    lays = [G.layout_inputs(x) for x in ws]
    idxs = [G.random_selection(x, k, 7 + i) for i, (x, k) in enumerate(zip(ws, ks))]
    R = w.R
    row_off = [R + ks[1] + 5 + R + ks[2] + 3, R + ks[2] + 3, 0]       # image 2 first, then 1, then 0
    rows = row_off[0] + R + ks[0] + 2
    idx_off = [0, ks[0], ks[0] + ks[1], sum(ks)]
    stack = lambda key: torch.stack([dev(l[key], w.dtype) for l in lays])  # noqa: E731
    low, high = stack("lowres"), stack("highres_prev")
    pre = stack("ref") if R else None
    idx = dev(np.concatenate(idxs).astype(np.int32)) if sum(ks) else torch.zeros(1, dtype=torch.int32, device="cuda")
    compact = torch.full((rows, w.D), 7.0, dtype=low.dtype, device="cuda")
    pos = torch.full((rows, 3), -1, dtype=torch.int32, device="cuda")
    canvas = high if alias else torch.full_like(high, 7.0)
    gpu.avits_gather_upsample_batched(low, high, pre, idx, idx_off, w.H_lr, w.W_lr, compact, row_off, pos, canvas,
                                      mode=mode)
    torch.cuda.synchronize()
    c, p, cv = host(compact), host(pos), host(canvas)
    touched = np.zeros(rows, bool)
    for b in range(3):
        rc, rp, rcv = oracle.gather_upsample(lays[b]["lowres"], lays[b]["highres_prev"], lays[b]["ref"] if R else None,
                                             idxs[b], w.H_lr, w.W_lr, "nearest" if mode == 0 else "bilinear")
        a0 = row_off[b]
        np.testing.assert_array_equal(c[a0:a0 + R + ks[b]], rc, err_msg=f"image {b} rows")
        np.testing.assert_array_equal(p[a0 + R:a0 + R + ks[b]], rp, err_msg=f"image {b} positions")
        if mode == 1 and w.dtype == "bf16":
            assert np.all(np.abs(cv[b] - rcv) <= np.abs(rcv) * 2.0 ** -7 + 1e-30), f"image {b} canvas"
        elif mode == 1:
            assert np.abs(cv[b] - rcv).max() < 1e-5, f"image {b} canvas"
        else:
            np.testing.assert_array_equal(cv[b], rcv, err_msg=f"image {b} canvas")
        touched[a0:a0 + R + ks[b]] = True
    assert np.all(c[~touched] == 7.0) and np.all(p[~touched] == -1)
    assert np.all(p[[row_off[b] + i for b in range(3) for i in range(R)]] == -1)  # prefix positions are the caller's

    # Scatter the packed rows back: each image's canvas gets its own rows.
    out = G.block_input(w, rows, 5)
    canv = stack("highres_prev")
    gpu.avits_scatter_batched(dev(out, w.dtype), idx, idx_off, [a + R for a in row_off], canv)
    torch.cuda.synchronize()
    for b in range(3):
        np.testing.assert_array_equal(host(canv[b]), oracle.scatter(out, idxs[b], row_off[b] + R,
                                                                    lays[b]["highres_prev"]), err_msg=f"image {b}")


def _block_inputs(w, n_txt, n_img, seed=0):
    x = G.block_input(w, n_txt + n_img, seed)
    g = np.random.default_rng(1000 + seed)
    pos = np.zeros((n_txt + n_img, 3), np.int32)
    pos[n_txt:, 0] = g.integers(0, 2, n_img)
    pos[n_txt:, 1] = g.integers(0, w.H_hr, n_img)
    pos[n_txt:, 2] = g.integers(0, w.W_hr, n_img)
    return x, pos


def _run_double(gpu, w, x, pos, n_txt, wt, wi):
    t_x = dev(x, w.dtype)
    out = torch.empty_like(t_x)
    lse = torch.empty(w.H, x.shape[0], device="cuda")
    bw = gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=double_weights_dev(wt, w.dtype), img=double_weights_dev(wi, w.dtype))
    gpu.avits_block_forward(t_x, out, dev(pos), n_txt, x.shape[0] - n_txt, bw, w.H, lse_out=lse)
    torch.cuda.synchronize()
    return host(out), host(lse)


@pytest.mark.parametrize("w", TINY, ids=IDS)
def test_double_block(gpu, w):
    n_txt, n_img = w.L, w.R + w.k
    x, pos = _block_inputs(w, n_txt, n_img)
    wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
    out, lse = _run_double(gpu, w, x, pos, n_txt, wt, wi)
    ref, ref_lse = oracle.double_block(x, pos, n_txt, wt, wi, w.H)
    assert_close(out, ref, w.dtype, "x_out")
    assert_close(out - x, ref - x, w.dtype, "block update x_out - x_in")
    assert_close(lse, ref_lse, w.dtype, "lse")


@pytest.mark.parametrize("n_txt,n_img", [(40, 0), (0, 77), (1, 1), (129, 130)])
def test_double_block_degenerate_streams(gpu, n_txt, n_img):
    w = C.TINY_BF16
    x, pos = _block_inputs(w, n_txt, n_img, seed=n_txt + n_img)
    wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
    out, lse = _run_double(gpu, w, x, pos, n_txt, wt, wi)
    ref, ref_lse = oracle.double_block(x, pos, n_txt, wt, wi, w.H)
    assert_close(out - x, ref - x, "bf16", "block update")
    assert_close(lse, ref_lse, "bf16", "lse")


@pytest.mark.parametrize("w", [C.TINY_F32, C.TINY_BF16], ids=["f32", "bf16"])
def test_single_block(gpu, w):
    S = w.L + w.k
    x, pos = _block_inputs(w, w.L, w.k, seed=9)
    ws = G.single_block_weights(w, 0)
    t_x = dev(x, w.dtype)
    out = torch.empty_like(t_x)
    lse = torch.empty(w.H, S, device="cuda")
    bw = gpu.BlockWeights(gpu.BLOCK_SINGLE, single=double_weights_dev(ws, w.dtype))
    gpu.avits_block_forward(t_x, out, dev(pos), w.L, w.k, bw, w.H, lse_out=lse)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.single_block(x, pos, ws, w.H)
    assert_close(host(out), ref, w.dtype, "x_out")
    assert_close(host(out) - x, ref - x, w.dtype, "block update")
    assert_close(host(lse), ref_lse, w.dtype, "lse")


# ---------------------------------------------------------------------------
# Load-balance forms, forced at small shapes through the tuning overrides:
# the attention's key pieces merged by the combine kernel, and the GEMM's
# split tail (the last tiles in k splits, reduced by a second kernel).  Each
# form must still give the oracle's block.

def _balanced_block(gpu, kind, seed):
    w = C.TINY_BF16
    n_txt, n_img = 40, 555  # 5 row blocks x 2 heads = 10 attention units, 10 key tiles
    x, pos = _block_inputs(w, n_txt, n_img, seed=seed)
    S = n_txt + n_img
    if kind == "double":
        wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
        bw = gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=double_weights_dev(wt, w.dtype), img=double_weights_dev(wi, w.dtype))
        ref, ref_lse = oracle.double_block(x, pos, n_txt, wt, wi, w.H)
    else:
        ws_ = G.single_block_weights(w, 0)
        bw = gpu.BlockWeights(gpu.BLOCK_SINGLE, single=double_weights_dev(ws_, w.dtype))
        ref, ref_lse = oracle.single_block(x, pos, ws_, w.H)
    t_x = dev(x, w.dtype)
    out = torch.empty_like(t_x)
    lse = torch.empty(w.H, S, device="cuda")
    gpu.avits_block_forward(t_x, out, dev(pos), n_txt, n_img, bw, w.H, lse_out=lse)
    torch.cuda.synchronize()
    assert_close(host(out) - x, ref - x, w.dtype, f"{kind} block update")
    assert_close(host(lse), ref_lse, w.dtype, f"{kind} lse")
    return host(out)


@pytest.mark.parametrize("cfg", ["0,1", "0,2", "0,3", "0,4", "3,2", "5,4", "9,3"])
@pytest.mark.parametrize("kind", ["double", "single"])
def test_attention_key_pieces(gpu, monkeypatch, kind, cfg):
    monkeypatch.setenv("AVITS_ATTN_SPLIT", cfg)
    _balanced_block(gpu, kind, seed=31)


@pytest.mark.parametrize("tail,tsp", [(1, 2), (3, 3), (7, 4), (100, 2)])
@pytest.mark.parametrize("kind", ["double", "single"])
def test_gemm_split_tail(gpu, monkeypatch, kind, tail, tsp):
    monkeypatch.setenv("AVITS_GEMM_TILE", f"256,1,8,1,{tail},{tsp}")
    _balanced_block(gpu, kind, seed=37)



def test_block_relayout_equivariance(gpu):
    # RoPE reads positions, not sequence slots: shuffling image rows with their
    # positions shuffles the outputs (bit-exact is not expected: summation order).
    w = C.TINY_BF16
    x, pos = _block_inputs(w, 16, 48, seed=4)
    wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
    out, _ = _run_double(gpu, w, x, pos, 16, wt, wi)
    perm = np.concatenate([np.arange(16), 16 + np.random.default_rng(2).permutation(48)])
    out2, _ = _run_double(gpu, w, x[perm], pos[perm], 16, wt, wi)
    assert rel_l2(out2 - x[perm], out[perm] - x[perm]) < 1e-2


@pytest.mark.parametrize("kind", ["double", "single"])
def test_block_batched(gpu, kind):
    # Several images through one block: rows packed by stream (text rows of
    # all images, then their image rows); attention within each image only.
    w = C.TINY_BF16
    txt = [32, 0, 7, 129]
    img = [200, 77, 1, 64]
    txt_off = np.concatenate([[0], np.cumsum(txt)]).astype(int).tolist()
    img_off = np.concatenate([[0], np.cumsum(img)]).astype(int).tolist()
    S = txt_off[-1] + img_off[-1]
    x, pos = _block_inputs(w, txt_off[-1], img_off[-1], seed=21)
    if kind == "double":
        wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
        bw = gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=double_weights_dev(wt, w.dtype), img=double_weights_dev(wi, w.dtype))
        ref, ref_lse = oracle.block_batched(x, pos, txt_off, img_off, w.H, wt, wi)
    else:
        ws_ = G.single_block_weights(w, 0)
        bw = gpu.BlockWeights(gpu.BLOCK_SINGLE, single=double_weights_dev(ws_, w.dtype))
        ref, ref_lse = oracle.block_batched(x, pos, txt_off, img_off, w.H, single=ws_)
    t_x = dev(x, w.dtype)
    out = torch.empty_like(t_x)
    lse = torch.empty(w.H, S, device="cuda")
    gpu.avits_block_forward_batched(t_x, out, dev(pos), txt_off, img_off, bw, w.H, lse_out=lse)
    torch.cuda.synchronize()
    got = host(out)
    T = txt_off[-1]
    for b in range(len(txt)):
        rows = np.concatenate([np.arange(txt_off[b], txt_off[b + 1]), T + np.arange(img_off[b], img_off[b + 1])])
        assert_close(got[rows] - x[rows], ref[rows] - x[rows], w.dtype, f"image {b} block update")
        assert_close(host(lse)[:, rows], ref_lse[:, rows], w.dtype, f"image {b} lse")
    # Changing one image's rows leaves the others' outputs bit for bit.
    x2 = x.copy()
    r3 = np.concatenate([np.arange(txt_off[3], txt_off[4]), T + np.arange(img_off[3], img_off[4])])
    x2[r3] = G.round_to(x2[r3] + 0.5, w.dtype)
    out2 = torch.empty_like(t_x)
    gpu.avits_block_forward_batched(dev(x2, w.dtype), out2, dev(pos), txt_off, img_off, bw, w.H)
    torch.cuda.synchronize()
    keep = np.setdiff1d(np.arange(S), r3)
    np.testing.assert_array_equal(host(out2)[keep], got[keep])


def _run_block_qk(gpu, w, x, pos, n_txt, bw):
    t_x = dev(x, w.dtype)
    q = torch.empty_like(t_x)
    k = torch.empty_like(t_x)
    gpu.avits_block_qk(t_x, dev(pos), n_txt, x.shape[0] - n_txt, bw, w.H, q, k)
    torch.cuda.synchronize()
    return host(q), host(k)


@pytest.mark.parametrize("w", TINY, ids=IDS)
def test_block_qk_probe(gpu, w):
    n_txt, n_img = w.L, w.R + w.k
    x, pos = _block_inputs(w, n_txt, n_img, seed=5)
    wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
    bw = gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=double_weights_dev(wt, w.dtype), img=double_weights_dev(wi, w.dtype))
    q, k = _run_block_qk(gpu, w, x, pos, n_txt, bw)
    rq, rk = oracle.block_qk(x, pos, n_txt, wt, wi, w.H)
    assert_close(q, rq.reshape(len(x), -1), w.dtype, "probe q")
    assert_close(k, rk.reshape(len(x), -1), w.dtype, "probe k")
    # The probe's q and k give the block's own attention normaliser.
    _, lse = _run_double(gpu, w, x, pos, n_txt, wt, wi)
    assert_close(lse, oracle.joint_lse(rq, rk), w.dtype, "block lse vs probe")


@pytest.mark.parametrize("n_txt,n_img", [(40, 0), (0, 77), (1, 1), (129, 130)])
def test_block_qk_probe_degenerate_streams(gpu, n_txt, n_img):
    w = C.TINY_BF16
    x, pos = _block_inputs(w, n_txt, n_img, seed=7 + n_txt)
    wt, wi = G.double_stream_weights(w, 0, 0), G.double_stream_weights(w, 0, 1)
    bw = gpu.BlockWeights(gpu.BLOCK_DOUBLE, txt=double_weights_dev(wt, w.dtype), img=double_weights_dev(wi, w.dtype))
    q, k = _run_block_qk(gpu, w, x, pos, n_txt, bw)
    rq, rk = oracle.block_qk(x, pos, n_txt, wt, wi, w.H)
    assert_close(q, rq.reshape(len(x), -1), "bf16", "probe q")
    assert_close(k, rk.reshape(len(x), -1), "bf16", "probe k")


@pytest.mark.parametrize("w", [C.TINY_F32, C.TINY_BF16], ids=["f32", "bf16"])
def test_block_qk_probe_single(gpu, w):
    x, pos = _block_inputs(w, w.L, w.k, seed=11)
    ws = G.single_block_weights(w, 0)
    bw = gpu.BlockWeights(gpu.BLOCK_SINGLE, single=double_weights_dev(ws, w.dtype))
    q, k = _run_block_qk(gpu, w, x, pos, w.L, bw)
    rq, rk = oracle.block_qk(x, pos, 0, None, None, w.H, single=ws)
    assert_close(q, rq.reshape(len(x), -1), w.dtype, "probe q")
    assert_close(k, rk.reshape(len(x), -1), w.dtype, "probe k")


# ---------------------------------------------------------------------------
# Text attention mass inside the statistics pass, and the score from it.

@pytest.mark.parametrize("w", TINY, ids=IDS)
def test_joint_attention_stats(gpu, w):
    si = G.score_inputs(w)
    k_all = _k_all(si)
    q, k = dev(si["latent_q"], w.dtype), dev(k_all, w.dtype)
    lse = torch.empty(w.H, w.N, device="cuda")
    mass = torch.full((w.H, w.N), 7.0, device="cuda")
    gpu.avits_joint_attention_stats(q, k, w.L, mass, lse=lse)
    torch.cuda.synchronize()
    assert_close(host(lse), oracle.joint_lse(si["latent_q"], k_all), w.dtype, "lse")
    ref = oracle.text_attention_mass(si["latent_q"], k_all, w.L)
    assert_close(host(mass), ref, w.dtype, "text mass")
    assert_close(host(mass).mean(axis=0), oracle.spatial_importance(si["latent_q"], si["text_k"],
                                                                   oracle.joint_lse(si["latent_q"], k_all)),
                 w.dtype, "head-mean mass = A")
    # Accumulation over two probes; the limits L = 0 and L = Nk.
    gpu.avits_joint_attention_stats(q, k, w.L, mass, accumulate=True)
    torch.cuda.synchronize()
    assert_close(host(mass), 2 * ref, w.dtype, "accumulated mass")
    gpu.avits_joint_attention_stats(q, k, 0, mass)
    gpu.avits_joint_attention_stats(q, k, k_all.shape[0], lse)  # lse buffer reused as a mass output
    torch.cuda.synchronize()
    assert np.all(host(mass) == 0.0)
    np.testing.assert_allclose(host(lse), 1.0, atol=1e-5)


@pytest.mark.parametrize("w", [C.TINY_F32, C.TINY_BF16, C.TINY_F32_RAGGED], ids=["f32", "bf16", "f32_ragged"])
@pytest.mark.parametrize("n_t", [2, 3, 5])
def test_score_from_mass(gpu, w, n_t):
    si = G.score_inputs(w)
    mass = oracle.text_attention_mass(si["latent_q"], _k_all(si), w.L).astype(np.float32)
    g = np.random.default_rng(n_t)
    snaps = [si["feat_prev"], si["feat_t"]]
    while len(snaps) < n_t:
        snaps.append(G.round_to(snaps[-1] + 0.1 * g.standard_normal(snaps[-1].shape), w.dtype))
    snaps = np.stack(snaps)
    s = torch.empty(w.N, device="cuda")
    a = torch.empty(w.N, device="cuda")
    v = torch.empty(w.N, device="cuda")
    gpu.avits_score_from_mass(dev(2 * mass), 2, [dev(z, w.dtype) for z in snaps], w.alpha, w.eps_minmax, s,
                              a_raw=a, v_raw=v)
    torch.cuda.synchronize()
    s_ref, a_ref, v_ref = oracle.score_from_mass(2 * mass.astype(np.float64), 2, snaps, w.alpha, w.eps_minmax)
    assert_close(host(a), a_ref, w.dtype, "A")
    assert_close(host(v), v_ref, w.dtype, "V")
    assert_close(host(s), s_ref, w.dtype, "S")
    assert np.abs(host(s) - s_ref).max() < 1e-4


@pytest.mark.parametrize("w", [C.TINY_BF16, C.TINY_BF16_REF], ids=["bf16", "bf16_ref"])
def test_fused_mass_score_matches_query_key_score(gpu, w):
    # The statistics pass + score_from_mass and the LSE + query/key scorer are
    # two GPU routes to the same scores.
    si = G.score_inputs(w)
    k_all = _k_all(si)
    q = dev(si["latent_q"], w.dtype)
    lse = torch.empty(w.H, w.N, device="cuda")
    mass = torch.empty(w.H, w.N, device="cuda")
    gpu.avits_joint_attention_stats(q, dev(k_all, w.dtype), w.L, mass, lse=lse)
    s1 = torch.empty(w.N, device="cuda")
    gpu.avits_score_from_mass(mass, 1, [dev(si["feat_prev"], w.dtype), dev(si["feat_t"], w.dtype)], w.alpha,
                              w.eps_minmax, s1)
    s2 = torch.empty(w.N, device="cuda")
    gpu.avits_score(q, dev(si["text_k"], w.dtype), lse, dev(si["feat_t"], w.dtype), dev(si["feat_prev"], w.dtype),
                    w.alpha, w.eps_minmax, s2)
    torch.cuda.synchronize()
    assert np.abs(host(s1) - host(s2)).max() < 1e-4
