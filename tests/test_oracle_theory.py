"""Pins of the distortion theory (Theorem 1, Lemma 1, softmax ray derivatives)."""
import numpy as np
import pytest

from oracle import theory


@pytest.mark.parametrize("seed", range(3))
def test_ray_derivatives_match_finite_differences(seed):
    rng = np.random.default_rng(seed)
    s = rng.standard_normal(9) * 2
    al = rng.standard_normal(9)
    th = 0.37
    eps = 1e-4
    f = lambda t: theory.ray_derivatives(s, al, t)   # noqa: E731
    g0, g1, g2, g3 = f(th)
    gp, gm = f(th + eps), f(th - eps)
    np.testing.assert_allclose(g1, (gp[0] - gm[0]) / (2 * eps), rtol=1e-6, atol=1e-10)
    np.testing.assert_allclose(g2, (gp[1] - gm[1]) / (2 * eps), rtol=1e-6, atol=1e-10)
    np.testing.assert_allclose(g3, (gp[2] - gm[2]) / (2 * eps), rtol=1e-5, atol=1e-9)


def test_expansion_terms_sum_to_zero_and_match_taylor():
    rng = np.random.default_rng(4)
    s = rng.standard_normal(12)
    al = 1e-3 * rng.standard_normal(12)
    da, da1, da2, r = theory.delta_a_expansion(s, al)
    assert abs(da1.sum()) < 1e-17 and abs(da2.sum()) < 1e-17 and abs(da.sum()) < 1e-15
    _, g1, g2, _ = theory.ray_derivatives(s, al, 0.0)
    np.testing.assert_allclose(da1, g1, rtol=1e-12)
    np.testing.assert_allclose(da2, 0.5 * g2, rtol=1e-12)
    # The remainder is third order: shrinking alpha by 10 shrinks r by ~1000.
    r2 = theory.delta_a_expansion(s, al / 10)[3]
    ratio = np.abs(r).sum() / np.abs(r2).sum()
    assert 700 < ratio < 1300


@pytest.mark.parametrize("scale", [0.05, 0.5, 2.0])
def test_lemma1_tail_bound_pathwise(scale):
    rng = np.random.default_rng(5)
    for _ in range(200):
        t = int(rng.integers(2, 30))
        s = rng.standard_normal(t) * 3
        al = rng.uniform(-1, 1, t) * scale
        a0 = np.abs(al).max()
        r = theory.delta_a_expansion(s, al)[3]
        assert np.abs(r).max() <= 7 * a0 ** 3 + 1e-15
        assert np.abs(r).sum() <= 7 * a0 ** 3 + 1e-15


def _tiny_problem(seed):
    rng = np.random.default_rng(seed)
    t, d, dout = 8, 6, 5
    q = rng.standard_normal(d)
    k = rng.standard_normal((t, d))
    v = rng.standard_normal((t, d))
    w_o = rng.standard_normal((d, dout)) / np.sqrt(d)
    return q, k, v, w_o


def test_theorem1_decomposition_monte_carlo():
    """E||o - o^||^2 = D_K + D_V + R with R of higher order: the relative gap shrinks
    as the quantization step halves, and the K-V cross term vanishes."""
    q, k, v, w_o = _tiny_problem(6)
    rng = np.random.default_rng(60)
    gaps = []
    for half in (0.1, 0.05, 0.025):
        var = np.full(k.shape, half ** 2 / 3)          # uniform on [-half, half]
        d_k, d_v = theory.leading_distortion(q, k, v, w_o, var, var)
        mc = theory.monte_carlo_distortion(q, k, v, w_o, half, half, 400000, rng)
        lead = d_k + d_v
        gaps.append(abs(mc["d_emp"] - lead) / lead)
        # the K-V cross term E[E_K . E_V] is exactly zero in expectation
        assert abs(mc["cross_kv"]) <= 4 * mc["cross_kv_se"] + 1e-3 * lead
        assert mc["lemma_max_ratio"] <= 7 and mc["lemma_sum_ratio"] <= 7
    assert gaps[-1] < 0.02
    assert gaps[0] > gaps[-1]


def test_factorized_key_distortion_identity():
    q, k, v, w_o = _tiny_problem(7)
    var_c = np.random.default_rng(8).uniform(0.001, 0.01, size=k.shape[1])
    full = np.broadcast_to(var_c, k.shape)
    d_k, _ = theory.leading_distortion(q, k, v, w_o, full, np.zeros_like(full))
    assert d_k == pytest.approx(theory.factorized_key_distortion(q, k, v, w_o, var_c), rel=1e-12)


def test_centered_variance_identity_monte_carlo():
    """E[(alpha_l - abar)^2] = (1 - 2 a_l) E[alpha_l^2] + sum_m a_m^2 E[alpha_m^2]
    (App. A, eq. centered-var) for independent zero-mean logit perturbations."""
    rng = np.random.default_rng(9)
    t = 6
    a = theory.softmax(rng.standard_normal(t))
    sd = rng.uniform(0.5, 2.0, t)
    al = rng.uniform(-1, 1, size=(400000, t)) * sd * np.sqrt(3)
    abar = al @ a
    emp = ((al - abar[:, None]) ** 2).mean(axis=0)
    pred = (1 - 2 * a) * sd ** 2 + np.sum(a ** 2 * sd ** 2)
    np.testing.assert_allclose(emp, pred, rtol=0.01)


def test_output_error_terms_sum_to_the_output_change():
    """o^ - o = E_K + E_V + E_x exactly (the decomposition of the output error, Sec. 4),
    with the attention weights perturbed through the keys and the values perturbed directly;
    each term is also checked against its own definition evaluated elementwise."""
    q, k, v, w_o = _tiny_problem(11)
    rng = np.random.default_rng(12)
    dk = 0.05 * rng.standard_normal(k.shape)
    dv = 0.05 * rng.standard_normal(v.shape)
    a = theory.softmax(k @ q)
    a_hat = theory.softmax((k + dk) @ q)
    da = a_hat - a
    o = (a @ v) @ w_o
    o_hat = (a_hat @ (v + dv)) @ w_o
    e_k, e_v, e_x = theory.output_error_terms(a, da, v, dv, w_o)
    np.testing.assert_allclose(e_k + e_v + e_x, o_hat - o, rtol=1e-12, atol=1e-14)
    t = len(a)
    np.testing.assert_allclose(e_k, sum(da[i] * (v[i] @ w_o) for i in range(t)), rtol=1e-12)
    np.testing.assert_allclose(e_v, sum(a[i] * (dv[i] @ w_o) for i in range(t)), rtol=1e-12)
    np.testing.assert_allclose(e_x, sum(da[i] * (dv[i] @ w_o) for i in range(t)), rtol=1e-12)
    # E_x is second order: halving both perturbations quarters it
    a_h = theory.softmax((k + dk / 2) @ q)
    _, _, e_x2 = theory.output_error_terms(a, a_h - a, v, dv / 2, w_o)
    assert np.linalg.norm(e_x2) < 0.3 * np.linalg.norm(e_x)
