"""Pins of the oracle's MMDiT block (joint attention, Section 3.3.1).

Library special cases (torch CPU fp64 functional ops), closed forms of RoPE,
and a scalar pure-Python brute force written independently (complex-number
RoPE, explicit loops, math.fsum).
"""
import cmath
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import block as ob
from synth import Workload, generator


def _t(x):
    return torch.from_numpy(np.asarray(x, dtype=np.float64))


def test_layer_norm_matches_torch():
    x = np.random.default_rng(0).standard_normal((7, 33)) * 3 + 1
    np.testing.assert_allclose(oracle.layer_norm(x), F.layer_norm(_t(x), (33,), eps=1e-6).numpy(), atol=1e-13)


def test_rms_norm_matches_torch():
    g = np.random.default_rng(1)
    x, w = g.standard_normal((5, 3, 16)), g.standard_normal(16)
    ref = F.rms_norm(_t(x), (16,), weight=_t(w), eps=1e-6).numpy()
    np.testing.assert_allclose(oracle.rms_norm(x, w), ref, atol=1e-13)


def test_gelu_matches_torch_and_limits():
    x = np.linspace(-8, 8, 401)
    np.testing.assert_allclose(oracle.gelu_tanh(x), F.gelu(_t(x), approximate="tanh").numpy(), atol=1e-15)
    assert oracle.gelu_tanh(np.array([0.0]))[0] == 0.0
    assert abs(oracle.gelu_tanh(np.array([30.0]))[0] - 30.0) < 1e-12
    assert abs(oracle.gelu_tanh(np.array([-30.0]))[0]) < 1e-12


@pytest.mark.parametrize("Sq,Sk,H,d", [(5, 7, 2, 8), (33, 20, 3, 16), (1, 1, 1, 4)])
def test_attention_matches_torch_sdpa(Sq, Sk, H, d):
    g = np.random.default_rng(Sq * 100 + Sk)
    q, k, v = g.standard_normal((Sq, H, d)), g.standard_normal((Sk, H, d)), g.standard_normal((Sk, H, d))
    o, lse = oracle.attention(q, k, v)
    tq, tk, tv = (_t(a).permute(1, 0, 2)[None] for a in (q, k, v))
    ref = F.scaled_dot_product_attention(tq, tk, tv)[0].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(o, ref, atol=1e-12)
    ref_lse = torch.logsumexp(torch.einsum("qhd,khd->hqk", _t(q), _t(k)) / math.sqrt(d), dim=-1).numpy()
    np.testing.assert_allclose(lse, ref_lse, atol=1e-12)


def test_rope_frequencies_hand_values():
    # d = 128 splits as (16, 56, 56): 8 frame pairs, then 28 row pairs, 28 col pairs.
    ang = oracle.rope_angles(np.array([[0, 1, 0], [0, 0, 3], [2, 0, 0]]), 128)
    assert ang.shape == (3, 64)
    np.testing.assert_array_equal(ang[0, :8], 0.0)
    np.testing.assert_allclose(ang[0, 8:36], [10000.0 ** (-2 * m / 56) for m in range(28)], rtol=1e-15)
    np.testing.assert_array_equal(ang[0, 36:], 0.0)
    np.testing.assert_allclose(ang[1, 36:], [3 * 10000.0 ** (-2 * m / 56) for m in range(28)], rtol=1e-15)
    np.testing.assert_allclose(ang[2, :8], [2 * 10000.0 ** (-2 * m / 16) for m in range(8)], rtol=1e-15)
    assert ob.rope_axes(64) == (8, 28, 28)


def test_rope_identity_norm_and_relative_position():
    g = np.random.default_rng(3)
    d = 64
    x = g.standard_normal((4, 2, d))
    np.testing.assert_array_equal(oracle.apply_rope(x, oracle.rope_angles(np.zeros((4, 3)), d)), x)
    pos = g.integers(0, 50, size=(4, 3))
    y = oracle.apply_rope(x, oracle.rope_angles(pos, d))
    # Each pair keeps its norm.
    np.testing.assert_allclose(np.hypot(y[..., 0::2], y[..., 1::2]), np.hypot(x[..., 0::2], x[..., 1::2]), atol=1e-13)
    # <R(p) q, R(p') k> depends only on p - p'.
    q, k = g.standard_normal((1, 1, d)), g.standard_normal((1, 1, d))
    def dot(pq, pk):
        a = oracle.apply_rope(q, oracle.rope_angles(np.array([pq]), d))
        b = oracle.apply_rope(k, oracle.rope_angles(np.array([pk]), d))
        return float((a * b).sum())
    assert abs(dot([1, 5, 9], [0, 2, 4]) - dot([3, 13, 7], [2, 10, 2])) < 1e-12
    assert abs(dot([1, 5, 9], [0, 2, 4]) - dot([1, 5, 9], [0, 2, 5])) > 1e-6


def test_rope_matches_complex_rotation():
    g = np.random.default_rng(4)
    x = g.standard_normal((3, 1, 32))
    pos = np.array([[0, 7, 2], [1, 0, 0], [0, 3, 30]])
    y = oracle.apply_rope(x, oracle.rope_angles(pos, 32))
    xc = torch.view_as_complex(_t(x).reshape(3, 1, 16, 2).contiguous())
    ang = []
    for p in pos:
        row = []
        for a, n in enumerate((4, 14, 14)):
            row += [p[a] * 10000.0 ** (-2 * m / n) for m in range(n // 2)]
        ang.append(row)
    rot = torch.polar(torch.ones(3, 16, dtype=torch.float64), _t(np.array(ang)))[:, None, :]
    ref = torch.view_as_real(xc * rot).reshape(3, 1, 32).numpy()
    np.testing.assert_allclose(y, ref, atol=1e-13)


# ---------------------------------------------------------------------------
# Scalar brute force of both block kinds.

def _vec_ln(v, eps=1e-6):
    n = len(v)
    mu = math.fsum(v) / n
    var = math.fsum((a - mu) ** 2 for a in v) / n
    return [(a - mu) / math.sqrt(var + eps) for a in v]


def _matvec(W, b, v):
    return [math.fsum(W[o][i] * v[i] for i in range(len(v))) + b[o] for o in range(len(W))]


def _gelu(a):
    return 0.5 * a * (1 + math.tanh(math.sqrt(2 / math.pi) * (a + 0.044715 * a ** 3)))


def _rope_head(vals, p, d):
    axes = (d // 8, 7 * d // 16, 7 * d // 16)
    out, m0 = [], 0
    for a, n in enumerate(axes):
        for m in range(n // 2):
            z = complex(vals[2 * (m0 + m)], vals[2 * (m0 + m) + 1])
            z *= cmath.exp(1j * p[a] * 10000.0 ** (-2 * m / n))
            out += [z.real, z.imag]
        m0 += n // 2
    return out


def _rms(vals, g, eps=1e-6):
    r = math.sqrt(math.fsum(a * a for a in vals) / len(vals) + eps)
    return [a / r * gg for a, gg in zip(vals, g)]


def _heads(vec, H, d):
    return [vec[h * d:(h + 1) * d] for h in range(H)]


def _attend(Q, K, V, H, d):
    """Q[i][h], K[j][h], V[j][h] lists -> O[i] flat, LSE[h][i]."""
    O, LSE = [], [[0.0] * len(Q) for _ in range(H)]
    for i in range(len(Q)):
        oi = []
        for h in range(H):
            logits = [math.fsum(Q[i][h][c] * K[j][h][c] for c in range(d)) / math.sqrt(d) for j in range(len(K))]
            m = max(logits)
            e = [math.exp(a - m) for a in logits]
            z = math.fsum(e)
            LSE[h][i] = m + math.log(z)
            oi += [math.fsum(e[j] * V[j][h][c] for j in range(len(K))) / z for c in range(d)]
        O.append(oi)
    return O, LSE


def _brute_double(x, pos, n_txt, wt, wi, H):
    S, D = len(x), len(x[0])
    d = D // H
    Q, K, V = [], [], []
    for i in range(S):
        w = wt if i < n_txt else wi
        mod = w["mod"]
        h = [a * (1 + s) + t for a, s, t in zip(_vec_ln(x[i]), mod[1], mod[0])]
        qkv = _matvec(w["w_qkv"], w["b_qkv"], h)
        Q.append([_rope_head(_rms(hq, w["g_q"]), pos[i], d) for hq in _heads(qkv[:D], H, d)])
        K.append([_rope_head(_rms(hk, w["g_k"]), pos[i], d) for hk in _heads(qkv[D:2 * D], H, d)])
        V.append(_heads(qkv[2 * D:], H, d))
    O, LSE = _attend(Q, K, V, H, d)
    out = []
    for i in range(S):
        w = wt if i < n_txt else wi
        mod = w["mod"]
        att = _matvec(w["w_o"], w["b_o"], O[i])
        y = [a + g * b for a, g, b in zip(x[i], mod[2], att)]
        h2 = [a * (1 + s) + t for a, s, t in zip(_vec_ln(y), mod[4], mod[3])]
        m = [_gelu(a) for a in _matvec(w["w_mlp1"], w["b_mlp1"], h2)]
        mlp = _matvec(w["w_mlp2"], w["b_mlp2"], m)
        out.append([a + g * b for a, g, b in zip(y, mod[5], mlp)])
    return np.array(out), np.array(LSE)


def _brute_single(x, pos, w, H):
    S, D = len(x), len(x[0])
    d = D // H
    Q, K, V, M = [], [], [], []
    mod = w["mod"]
    for i in range(S):
        h = [a * (1 + s) + t for a, s, t in zip(_vec_ln(x[i]), mod[1], mod[0])]
        t = _matvec(w["w_in"], w["b_in"], h)
        Q.append([_rope_head(_rms(hq, w["g_q"]), pos[i], d) for hq in _heads(t[:D], H, d)])
        K.append([_rope_head(_rms(hk, w["g_k"]), pos[i], d) for hk in _heads(t[D:2 * D], H, d)])
        V.append(_heads(t[2 * D:3 * D], H, d))
        M.append([_gelu(a) for a in t[3 * D:]])
    O, LSE = _attend(Q, K, V, H, d)
    out = []
    for i in range(S):
        y = _matvec(w["w_out"], w["b_out"], O[i] + M[i])
        out.append([a + g * b for a, g, b in zip(x[i], mod[2], y)])
    return np.array(out), np.array(LSE)


_TINY = Workload("brute", "f32", D=64, H=2, d=32, L=2, R=0, H_lr=2, W_lr=2, rho=0.5,
                 alpha=0.5, weight_std=0.3, seed=77, mlp_ratio=2)


def _lists(w):
    return {k: np.asarray(v, dtype=np.float64).tolist() for k, v in w.items()}


def _tiny_inputs(S=6):
    x = generator.block_input(_TINY, S)
    pos = np.array([[0, 0, 0], [0, 0, 0], [0, 0, 1], [0, 2, 3], [1, 1, 0], [0, 3, 3]][:S], dtype=np.int32)
    return x, pos


def test_double_block_matches_scalar_bruteforce():
    x, pos = _tiny_inputs()
    wt = generator.double_stream_weights(_TINY, 0, 0)
    wi = generator.double_stream_weights(_TINY, 0, 1)
    out, lse = oracle.double_block(x, pos, 2, wt, wi, 2)
    ref, ref_lse = _brute_double(x.astype(float).tolist(), pos.tolist(), 2, _lists(wt), _lists(wi), 2)
    np.testing.assert_allclose(out, ref, atol=1e-11)
    np.testing.assert_allclose(lse, ref_lse, atol=1e-11)


def test_single_block_matches_scalar_bruteforce():
    x, pos = _tiny_inputs()
    w = generator.single_block_weights(_TINY, 0)
    out, lse = oracle.single_block(x, pos, w, 2)
    ref, ref_lse = _brute_single(x.astype(float).tolist(), pos.tolist(), _lists(w), 2)
    np.testing.assert_allclose(out, ref, atol=1e-11)
    np.testing.assert_allclose(lse, ref_lse, atol=1e-11)


def test_row_subsets_match_full():
    w = _TINY.replace(D=128, H=2, d=64, mlp_ratio=4)
    x = generator.block_input(w, 11)
    pos = np.random.default_rng(5).integers(0, 9, size=(11, 3)).astype(np.int32)
    wt, wi = generator.double_stream_weights(w, 0, 0), generator.double_stream_weights(w, 0, 1)
    full, lse = oracle.double_block(x, pos, 4, wt, wi, 2)
    rows = np.array([0, 3, 4, 10])
    part, plse = oracle.double_block(x, pos, 4, wt, wi, 2, rows=rows)
    np.testing.assert_allclose(part, full[rows], atol=1e-12)
    np.testing.assert_allclose(plse, lse[:, rows], atol=1e-12)
    ws = generator.single_block_weights(w, 0)
    full, lse = oracle.single_block(x, pos, ws, 2)
    part, plse = oracle.single_block(x, pos, ws, 2, rows=rows)
    np.testing.assert_allclose(part, full[rows], atol=1e-12)


def test_zero_gates_are_identity_and_image_permutation_equivariance():
    w = _TINY.replace(D=128, H=2, d=64, mlp_ratio=4)
    x = generator.block_input(w, 9)
    pos = np.random.default_rng(6).integers(0, 9, size=(9, 3)).astype(np.int32)
    wt, wi = generator.double_stream_weights(w, 0, 0), generator.double_stream_weights(w, 0, 1)
    z = {k: v.copy() for k, v in wt.items()}
    zi = {k: v.copy() for k, v in wi.items()}
    z["mod"][[2, 5]] = 0.0
    zi["mod"][[2, 5]] = 0.0
    out, _ = oracle.double_block(x, pos, 3, z, zi, 2)
    np.testing.assert_array_equal(out, x.astype(np.float64))
    # Shuffling image rows together with their positions shuffles the outputs.
    out, lse = oracle.double_block(x, pos, 3, wt, wi, 2)
    perm = np.concatenate([np.arange(3), 3 + np.random.default_rng(7).permutation(6)])
    out2, lse2 = oracle.double_block(x[perm], pos[perm], 3, wt, wi, 2)
    np.testing.assert_allclose(out2, out[perm], atol=1e-12)
    np.testing.assert_allclose(lse2, lse[:, perm], atol=1e-12)
    # The text stream does not see positions of image rows beyond their relative offsets:
    # moving every image row by the same grid offset leaves the text outputs' attention to
    # them unchanged only if text is also moved; with text fixed at 0 it changes.
    shifted = pos.copy()
    shifted[3:, 1] += 1
    out3, _ = oracle.double_block(x, shifted, 3, wt, wi, 2)
    assert np.abs(out3[:3] - out[:3]).max() > 1e-9


def test_single_block_zero_gate_identity():
    w = _TINY.replace(D=128, H=2, d=64, mlp_ratio=4)
    x = generator.block_input(w, 5)
    pos = np.zeros((5, 3), np.int32)
    ws = generator.single_block_weights(w, 0)
    ws["mod"][2] = 0.0
    out, _ = oracle.single_block(x, pos, ws, 2)
    np.testing.assert_array_equal(out, x.astype(np.float64))


def _brute_qk(x, pos, n_txt, wt, wi, H, wname="w_qkv", bname="b_qkv"):
    """Per-row scalar statement of the block's first stage: LN + modulation,
    the q / k projections, RMSNorm and complex-number RoPE."""
    S, D = len(x), len(x[0])
    d = D // H
    Q, K = [], []
    for i in range(S):
        w = wt if i < n_txt else wi
        mod = w["mod"]
        h = [a * (1 + s) + t for a, s, t in zip(_vec_ln(x[i]), mod[1], mod[0])]
        t = _matvec(w[wname][:2 * D], w[bname][:2 * D], h)
        Q.append([v for hq in _heads(t[:D], H, d) for v in _rope_head(_rms(hq, w["g_q"]), pos[i], d)])
        K.append([v for hk in _heads(t[D:], H, d) for v in _rope_head(_rms(hk, w["g_k"]), pos[i], d)])
    return np.array(Q).reshape(S, H, d), np.array(K).reshape(S, H, d)


def test_block_qk_matches_scalar_bruteforce():
    x, pos = _tiny_inputs()
    wt = generator.double_stream_weights(_TINY, 0, 0)
    wi = generator.double_stream_weights(_TINY, 0, 1)
    q, k = oracle.block_qk(x, pos, 2, wt, wi, 2)
    rq, rk = _brute_qk(x.astype(float).tolist(), pos.tolist(), 2, _lists(wt), _lists(wi), 2)
    np.testing.assert_allclose(q, rq, atol=1e-12)
    np.testing.assert_allclose(k, rk, atol=1e-12)
    ws = generator.single_block_weights(_TINY, 0)
    q, k = oracle.block_qk(x, pos, 0, None, None, 2, single=ws)
    rq, rk = _brute_qk(x.astype(float).tolist(), pos.tolist(), 0, _lists(ws), _lists(ws), 2, "w_in", "b_in")
    np.testing.assert_allclose(q, rq, atol=1e-12)
    np.testing.assert_allclose(k, rk, atol=1e-12)


def test_block_qk_softmax_normaliser_is_the_blocks():
    # The probe's queries and keys give exactly the block's attention LSE, and
    # with every position zero the rotation drops out (pure RMSNorm * g rows).
    w = _TINY.replace(D=128, H=2, d=64, mlp_ratio=4)
    x = generator.block_input(w, 9)
    pos = np.stack([np.zeros(9), np.arange(9) % 3, np.arange(9) // 3], axis=1).astype(np.int32)
    wt, wi = generator.double_stream_weights(w, 0, 0), generator.double_stream_weights(w, 0, 1)
    q, k = oracle.block_qk(x, pos, 4, wt, wi, 2)
    _, lse = oracle.double_block(x, pos, 4, wt, wi, 2)
    np.testing.assert_allclose(oracle.joint_lse(q, k), lse, atol=1e-12)
    q0, _ = oracle.block_qk(x, np.zeros_like(pos), 4, wt, wi, 2)
    g = np.stack([np.asarray(wt["g_q"], float)] * 4 + [np.asarray(wi["g_q"], float)] * 5)[:, None, :]
    np.testing.assert_allclose(np.sqrt(((q0 / g) ** 2).mean(-1)), np.ones((9, 2)), atol=1e-6)


# ---------------------------------------------------------------------------
# Several images through one block, rows packed by stream.

def _brute_double_packed(x, pos, is_txt, seg, wt, wi, H):
    """Scalar double block on the packed rows: stream weights by is_txt[i],
    attention of row i restricted to the rows j with seg[j] == seg[i]."""
    S, D = len(x), len(x[0])
    d = D // H
    Q, K, V = [], [], []
    for i in range(S):
        w = wt if is_txt[i] else wi
        mod = w["mod"]
        h = [a * (1 + s) + t for a, s, t in zip(_vec_ln(x[i]), mod[1], mod[0])]
        qkv = _matvec(w["w_qkv"], w["b_qkv"], h)
        Q.append([_rope_head(_rms(hq, w["g_q"]), pos[i], d) for hq in _heads(qkv[:D], H, d)])
        K.append([_rope_head(_rms(hk, w["g_k"]), pos[i], d) for hk in _heads(qkv[D:2 * D], H, d)])
        V.append(_heads(qkv[2 * D:], H, d))
    O, LSE = [None] * S, [[0.0] * S for _ in range(H)]
    for i in range(S):
        js = [j for j in range(S) if seg[j] == seg[i]]
        o, l_ = _attend([Q[i]], [K[j] for j in js], [V[j] for j in js], H, d)
        O[i] = o[0]
        for h in range(H):
            LSE[h][i] = l_[h][0]
    out = []
    for i in range(S):
        w = wt if is_txt[i] else wi
        mod = w["mod"]
        att = _matvec(w["w_o"], w["b_o"], O[i])
        y = [a + g * b for a, g, b in zip(x[i], mod[2], att)]
        h2 = [a * (1 + s) + t for a, s, t in zip(_vec_ln(y), mod[4], mod[3])]
        m = [_gelu(a) for a in _matvec(w["w_mlp1"], w["b_mlp1"], h2)]
        mlp = _matvec(w["w_mlp2"], w["b_mlp2"], m)
        out.append([a + g * b for a, g, b in zip(y, mod[5], mlp)])
    return np.array(out), np.array(LSE)


def test_block_batched_matches_masked_bruteforce():
    # Three images: (text, image) rows (2, 2), (0, 1), (1, 2); text rows first.
    txt_off, img_off = [0, 2, 2, 3], [0, 2, 3, 5]
    S = txt_off[-1] + img_off[-1]
    x = generator.block_input(_TINY, S, 3)
    pos = np.array([[0, 0, 0], [0, 0, 0], [0, 0, 0], [0, 1, 2], [0, 3, 3], [0, 2, 2], [1, 1, 0], [0, 0, 1]],
                   dtype=np.int32)
    is_txt = [True] * 3 + [False] * 5
    seg = [0, 0, 2] + [0, 0, 1, 2, 2]
    wt = generator.double_stream_weights(_TINY, 0, 0)
    wi = generator.double_stream_weights(_TINY, 0, 1)
    out, lse = oracle.block_batched(x, pos, txt_off, img_off, 2, wt, wi)
    ref, ref_lse = _brute_double_packed(x.astype(float).tolist(), pos.tolist(), is_txt, seg, _lists(wt), _lists(wi), 2)
    np.testing.assert_allclose(out, ref, atol=1e-11)
    np.testing.assert_allclose(lse, ref_lse, atol=1e-11)
    # One image reduces to the plain block; images do not see each other.
    o1, l1 = oracle.block_batched(x[[0, 1, 3, 4]], pos[[0, 1, 3, 4]], [0, 2], [0, 2], 2, wt, wi)
    p1, pl1 = oracle.double_block(x[[0, 1, 3, 4]], pos[[0, 1, 3, 4]], 2, wt, wi, 2)
    np.testing.assert_array_equal(o1, p1)
    np.testing.assert_array_equal(l1, pl1)
    x2 = x.copy()
    x2[[2, 6, 7]] += 1.0   # image 2's rows
    out2, _ = oracle.block_batched(x2, pos, txt_off, img_off, 2, wt, wi)
    np.testing.assert_array_equal(out2[[0, 1, 3, 4, 5]], out[[0, 1, 3, 4, 5]])


def test_block_batched_single_kind():
    txt_off, img_off = [0, 1, 3], [0, 2, 3]
    S = 6
    x = generator.block_input(_TINY, S, 4)
    pos, _ = _tiny_inputs(S)[1], None
    w = generator.single_block_weights(_TINY, 0)
    out, lse = oracle.block_batched(x, pos, txt_off, img_off, 2, single=w)
    # Image 1 = text row 1..2 and image row 5; image 0 = text row 0 and image rows 3, 4.
    for rows in ([0, 3, 4], [1, 2, 5]):
        ref, ref_lse = _brute_single(x[rows].astype(float).tolist(), pos[rows].tolist(), _lists(w), 2)
        np.testing.assert_allclose(out[rows], ref, atol=1e-11)
        np.testing.assert_allclose(lse[:, rows], ref_lse, atol=1e-11)
