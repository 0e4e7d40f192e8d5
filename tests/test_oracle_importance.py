"""Pins of the oracle's scoring stage (Section 3.3) to things other than itself."""
import math
import statistics

import numpy as np
import pytest
import scipy.special

import oracle


def _tiny(seed=0, N=5, H=2, d=4, L=3, extra=4):
    g = np.random.default_rng(seed)
    q = g.standard_normal((N, H, d))
    k_txt = g.standard_normal((L, H, d))
    k_rest = g.standard_normal((extra, H, d))
    return q, k_txt, k_rest


def _bruteforce_A(q, k_all, L):
    """Pure-Python: per head, softmax over every key, mass on the first L keys."""
    N, H, d = q.shape
    out = []
    for i in range(N):
        heads = []
        for h in range(H):
            logits = [math.fsum(q[i, h, c] * k_all[j, h, c] for c in range(d)) / math.sqrt(d)
                      for j in range(k_all.shape[0])]
            m = max(logits)
            e = [math.exp(x - m) for x in logits]
            z = math.fsum(e)
            heads.append(math.fsum(e[:L]) / z)
        out.append(math.fsum(heads) / H)
    return np.array(out)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_spatial_matches_pure_python_softmax(seed):
    q, k_txt, k_rest = _tiny(seed)
    k_all = np.concatenate([k_txt, k_rest])
    lse = oracle.joint_lse(q, k_all)
    a = oracle.spatial_importance(q, k_txt, lse)
    ref = _bruteforce_A(q, k_all, k_txt.shape[0])
    np.testing.assert_allclose(a, ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(oracle.spatial_importance_bruteforce(q, k_all, 3), ref, atol=1e-12)


def test_joint_lse_matches_scipy_logsumexp():
    q, k_txt, k_rest = _tiny(3, N=7, H=3, d=8, L=5, extra=6)
    k_all = np.concatenate([k_txt, k_rest])
    lse = oracle.joint_lse(q, k_all)
    for h in range(3):
        logits = q[:, h, :] @ k_all[:, h, :].T / math.sqrt(8)
        np.testing.assert_allclose(lse[h], scipy.special.logsumexp(logits, axis=1), atol=1e-12)


def test_row_mass_sums_to_one():
    # Text mass + the mass of every other key = 1 (softmax rows sum to 1).
    q, k_txt, k_rest = _tiny(4, N=9, H=3, d=8, L=4, extra=7)
    k_all = np.concatenate([k_txt, k_rest])
    lse = oracle.joint_lse(q, k_all)
    a_txt = oracle.spatial_importance(q, k_txt, lse)
    a_rest = oracle.spatial_importance(q, k_rest, lse)
    np.testing.assert_allclose(a_txt + a_rest, 1.0, atol=1e-13)
    # All keys counted as "text": A == 1 exactly up to rounding.
    np.testing.assert_allclose(oracle.spatial_importance(q, k_all, lse), 1.0, atol=1e-13)


def test_equal_logits_give_text_fraction():
    # Zero keys: every logit is 0, so each key holds 1/(L+R+N) of the mass.
    N, H, d, L, R = 6, 2, 8, 3, 5
    q = np.random.default_rng(5).standard_normal((N, H, d))
    k_txt = np.zeros((L, H, d))
    k_all = np.zeros((L + R + N, H, d))
    lse = oracle.joint_lse(q, k_all)
    np.testing.assert_allclose(lse, np.log(L + R + N), atol=1e-14)
    np.testing.assert_allclose(oracle.spatial_importance(q, k_txt, lse), L / (L + R + N), atol=1e-15)


def test_text_permutation_invariance_and_row_equivariance():
    q, k_txt, k_rest = _tiny(6, N=8, H=2, d=8, L=6, extra=5)
    k_all = np.concatenate([k_txt, k_rest])
    lse = oracle.joint_lse(q, k_all)
    a = oracle.spatial_importance(q, k_txt, lse)
    perm = np.random.default_rng(7).permutation(6)
    np.testing.assert_allclose(oracle.spatial_importance(q, k_txt[perm], lse), a, atol=1e-14)
    kperm = np.random.default_rng(8).permutation(k_all.shape[0])
    np.testing.assert_allclose(oracle.joint_lse(q, k_all[kperm]), lse, atol=1e-13)
    rperm = np.random.default_rng(9).permutation(8)
    np.testing.assert_allclose(
        oracle.spatial_importance(q[rperm], k_txt, lse[:, rperm]), a[rperm], atol=1e-14)


def test_step_variance_two_snapshots_closed_form():
    g = np.random.default_rng(10)
    a, b = g.standard_normal((7, 11)), g.standard_normal((7, 11))
    v = oracle.step_variance(np.stack([a, b]))
    # N_T = 2: the unbiased variance of {a, b} is (a - b)^2 / 2.
    np.testing.assert_allclose(v, ((a - b) ** 2).sum(axis=1) / (2 * 11), atol=1e-14)
    np.testing.assert_allclose(v, np.var(np.stack([a, b]), axis=0, ddof=1).mean(axis=1), atol=1e-14)


def test_step_variance_general_nt_against_statistics():
    g = np.random.default_rng(11)
    z = g.standard_normal((5, 4, 3))
    v = oracle.step_variance(z)
    for i in range(4):
        per_c = [statistics.variance([float(z[t, i, c]) for t in range(5)]) for c in range(3)]
        assert abs(v[i] - math.fsum(per_c) / 3) < 1e-13


def test_step_variance_invariances():
    g = np.random.default_rng(12)
    z = g.standard_normal((3, 6, 5))
    v = oracle.step_variance(z)
    np.testing.assert_allclose(oracle.step_variance(z + 3.25), v, atol=1e-13)    # shift
    np.testing.assert_allclose(oracle.step_variance(2.0 * z), 4.0 * v, atol=1e-13)  # scale
    np.testing.assert_array_equal(oracle.step_variance(np.stack([z[0], z[0]])), 0.0)


def test_generator_drift_gives_expected_variance():
    # feat_prev = feat_t + eps_i z_i  =>  V_i = eps_i^2 mean_c(z^2) / 2 (before rounding).
    g = np.random.default_rng(13)
    ft = g.standard_normal((50, 64))
    z = g.standard_normal((50, 64))
    eps = g.lognormal(-2, 1, size=50)
    v = oracle.step_variance(np.stack([ft + eps[:, None] * z, ft]))
    np.testing.assert_allclose(v, eps ** 2 * (z ** 2).mean(axis=1) / 2, rtol=1e-10)


def test_minmax_and_fuse_hand_example():
    # a = [1, 2, 3] -> [0, .5, 1]; v = [3, 1, 2] -> [1, 0, .5]; alpha = .5.
    s = oracle.joint_score(np.array([1.0, 2, 3]), np.array([3.0, 1, 2]), 0.5, 0.0)
    np.testing.assert_allclose(s, [0.5, 0.25, 0.75], atol=1e-15)
    s = oracle.joint_score(np.array([1.0, 2, 3]), np.array([3.0, 1, 2]), 0.25, 0.0)
    np.testing.assert_allclose(s, [0.75, 0.125, 0.625], atol=1e-15)


def test_minmax_range_and_constant():
    x = np.random.default_rng(14).standard_normal(100)
    y = oracle.minmax_normalise(x, 1e-8)
    assert y.min() == 0.0 and y[np.argmin(x)] == 0.0
    assert 0.0 <= y.max() < 1.0
    np.testing.assert_array_equal(oracle.minmax_normalise(np.full(10, 2.5), 1e-8), 0.0)


def test_alpha_extremes_select_by_one_signal():
    g = np.random.default_rng(15)
    a, v = g.random(200), g.random(200)
    top = lambda x, k: set(np.argsort(-x, kind="stable")[:k])  # noqa: E731
    assert top(oracle.joint_score(a, v, 1.0, 1e-8), 30) == top(a, 30)
    assert top(oracle.joint_score(a, v, 0.0, 1e-8), 30) == top(v, 30)


def test_score_wrapper_composes_stages():
    q, k_txt, k_rest = _tiny(16, N=12, H=2, d=8, L=3, extra=12)
    lse = oracle.joint_lse(q, np.concatenate([k_txt, k_rest]))
    g = np.random.default_rng(17)
    ft, fp = g.standard_normal((12, 5)), g.standard_normal((12, 5))
    s, a, v = oracle.score(q, k_txt, lse, ft, fp, 0.4)
    assert s.dtype == np.float32
    np.testing.assert_allclose(a, _bruteforce_A(q, np.concatenate([k_txt, k_rest]), 3), atol=1e-12)
    np.testing.assert_allclose(v, ((ft - fp) ** 2).sum(1) / 10, atol=1e-14)
    an = (a - a.min()) / (a.max() - a.min() + 1e-8)
    vn = (v - v.min()) / (v.max() - v.min() + 1e-8)
    np.testing.assert_array_equal(s, (0.4 * an + 0.6 * vn).astype(np.float32))


def _bruteforce_mass(q, k_all, L):
    """Pure-Python per-head text mass: softmax over every key, sum of the first L."""
    N, H, d = q.shape
    out = np.zeros((H, N))
    for i in range(N):
        for h in range(H):
            logits = [math.fsum(q[i, h, c] * k_all[j, h, c] for c in range(d)) / math.sqrt(d)
                      for j in range(k_all.shape[0])]
            m = max(logits)
            e = [math.exp(x - m) for x in logits]
            out[h, i] = math.fsum(e[:L]) / math.fsum(e)
    return out


@pytest.mark.parametrize("seed", [0, 5])
def test_text_mass_matches_pure_python_and_limits(seed):
    q, k_txt, k_rest = _tiny(seed, N=6, H=3, d=4, L=3, extra=5)
    k_all = np.concatenate([k_txt, k_rest])
    mass = oracle.text_attention_mass(q, k_all, 3)
    np.testing.assert_allclose(mass, _bruteforce_mass(q, k_all, 3), atol=1e-12)
    # Head mean is the spatial importance; L = 0 and L = Nk are the limits.
    np.testing.assert_allclose(mass.mean(axis=0), _bruteforce_A(q, k_all, 3), atol=1e-12)
    np.testing.assert_array_equal(oracle.text_attention_mass(q, k_all, 0), np.zeros((3, 6)))
    np.testing.assert_allclose(oracle.text_attention_mass(q, k_all, 8), np.ones((3, 6)), atol=1e-15)
    # Zero keys: every logit equal, so the mass is L / Nk exactly.
    np.testing.assert_allclose(oracle.text_attention_mass(q, np.zeros_like(k_all), 3), np.full((3, 6), 3 / 8),
                               atol=1e-15)


def test_score_from_mass_aggregates_probes_and_snapshots():
    g = np.random.default_rng(9)
    H, N, Df = 4, 50, 12
    m1, m2 = g.random((H, N)), g.random((H, N))
    snaps = g.standard_normal((5, N, Df))
    s, a, v = oracle.score_from_mass(m1 + m2, 2, snaps, 0.3, 1e-8)
    # A: the plain average over heads and the two probes, element by element.
    ref_a = np.array([math.fsum(list(m1[:, i]) + list(m2[:, i])) / (2 * H) for i in range(N)])
    np.testing.assert_allclose(a, ref_a, atol=1e-14)
    # V: the unbiased variance over the five steps, averaged over channels.
    ref_v = np.array([statistics.fmean(statistics.variance(snaps[:, i, c]) for c in range(Df)) for i in range(N)])
    np.testing.assert_allclose(v, ref_v, atol=1e-12)
    np.testing.assert_array_equal(s, oracle.joint_score(ref_a, ref_v, 0.3, 1e-8).astype(np.float32))
    # One probe and two snapshots: the same score as the query/key form.
    q, k_txt, k_rest = _tiny(2, N=7, H=2, d=4, L=3, extra=6)
    k_all = np.concatenate([k_txt, k_rest])
    lse = oracle.joint_lse(q, k_all)
    f0, f1 = g.standard_normal((7, 6)), g.standard_normal((7, 6))
    s_qk, a_qk, v_qk = oracle.score(q, k_txt, lse, f1, f0, 0.5)
    s_m, a_m, v_m = oracle.score_from_mass(oracle.text_attention_mass(q, k_all, 3), 1, np.stack([f0, f1]), 0.5)
    np.testing.assert_allclose(a_m, a_qk, atol=1e-13)
    np.testing.assert_allclose(v_m, v_qk, atol=1e-13)
    np.testing.assert_allclose(s_m, s_qk, atol=1e-6)
