"""Pins of the oracle's aggregation (Eq. 2-4, layer-sequential EMA, Proposition 1, Corollary 1)."""
import numpy as np
import pytest

from conftest import read_golden
from oracle import CUMULATIVE, EMA, SINGLE_STEP, fold_layers, select_keep


def test_layer_weights_golden():
    g = read_golden("ema_layer_weights.txt")
    alpha, K = float(g["alpha"]), int(g["layers"])
    # probe each weight with one-hot inputs: token 0 = prior, token l = layer l
    u0 = np.zeros(K + 1)
    u0[0] = 1.0
    s_layers = np.zeros((K, K + 1))
    for l in range(K):
        s_layers[l, l + 1] = 1.0
    u = fold_layers(u0, s_layers, alpha)
    assert abs(u[0] - float(g["prior"])) < 1e-15
    for l in range(1, K + 1):
        assert abs(u[l] - float(g[f"layer_{l}"])) < 1e-15, l
    assert abs(u.sum() - 1.0) < 1e-15


@pytest.mark.parametrize("alpha,K,T", [(0.9, 32, 3), (0.8, 28, 2), (0.9, 2, 16), (0.3, 5, 7)])
def test_constant_scores_closed_form(alpha, K, T):
    """Fixed cache, constant score c every layer and step: u_T = c (1 - alpha^(KT)) + alpha^(KT) u_0
    (Proposition 1 proof's expansion applied to K*T layer updates)."""
    rng = np.random.default_rng(K * T)
    n = 9
    c = rng.random(n)
    u0 = rng.random(n)
    u = u0
    for _ in range(T):
        u = fold_layers(u, np.broadcast_to(c, (K, n)), alpha)
    a = alpha ** (K * T)
    np.testing.assert_allclose(u, c * (1 - a) + a * u0, rtol=1e-12)


def test_mass_conservation_fixed_cache():
    """Scores that are distributions keep sum(u) = 1 - alpha^(KT) (1 - sum u_0)."""
    rng = np.random.default_rng(5)
    alpha, K, T, n = 0.9, 4, 5, 13
    u = np.zeros(n)
    for _ in range(T):
        s = rng.random((K, n))
        s /= s.sum(axis=1, keepdims=True)
        u = fold_layers(u, s, alpha)
    assert abs(u.sum() - (1 - alpha ** (K * T))) < 1e-13


def test_alpha_zero_keeps_last_layer_only():
    """Sec. 5.1: alpha = 0 retains only the last processed layer; equals the single-step rule (Eq. 2)."""
    rng = np.random.default_rng(9)
    s = rng.random((6, 10))
    u0 = rng.random(10)
    np.testing.assert_array_equal(fold_layers(u0, s, 0.0), s[-1])
    np.testing.assert_array_equal(fold_layers(u0, s, 0.5, SINGLE_STEP), s[-1])


def test_cumulative_rule():
    """Eq. 3 never forgets: with distributions as scores every layer adds exactly one unit of mass, the result
    is independent of alpha and of the layer order, and it dominates the EMA state of the same inputs."""
    rng = np.random.default_rng(11)
    s = rng.random((3, 8))
    s /= s.sum(axis=1, keepdims=True)
    u0 = rng.random(8)
    u = fold_layers(u0, s, 0.9, CUMULATIVE)
    assert abs(u.sum() - (u0.sum() + 3)) < 1e-13
    np.testing.assert_allclose(u, fold_layers(u0, s[::-1], 0.1, CUMULATIVE), rtol=1e-14)
    assert np.all(u >= fold_layers(u0, s, 0.9, EMA))


def test_momentum_perturbation_golden():
    g = read_golden("momentum_perturbation.txt")
    alpha, rel = float(g["alpha"]), float(g["relative_perturbation"])
    base = np.array([0.5])
    u_a = fold_layers(np.zeros(1), [base], alpha)
    u_b = fold_layers(np.zeros(1), [base * (1 + rel)], alpha)
    assert abs((u_b - u_a)[0] / base[0] - float(g["relative_effect"])) < 1e-15


def test_prop1_variance_monte_carlo():
    """Proposition 1(b): i.i.d. scores of variance sigma^2 give Var[mu_T] = (1-a)(1-a^(2T))/(1+a) sigma^2
    with one aggregate update per step and mu_0 = 0; the expected value is (1 - a^T) s_bar (part (a))."""
    g = read_golden("prop1_bounds.txt")
    alpha = float(g["alpha"])
    rng = np.random.default_rng(2024)
    tokens, sigma, mean = 400_000, 0.3, 1.0
    for T, key in ((1, "single_variance_factor_T1"), (2, "single_variance_factor_T2"), (40, None)):
        u = np.zeros(tokens)
        for _ in range(T):
            u = fold_layers(u, [mean + sigma * rng.standard_normal(tokens)], alpha)
        factor = (1 - alpha) * (1 - alpha ** (2 * T)) / (1 + alpha)
        if key:
            assert abs(factor - float(g[key])) < 1e-15
        var = u.var()
        # sampling error of a variance estimate ~ sqrt(2/N) relative
        assert abs(var / (factor * sigma ** 2) - 1) < 6 * np.sqrt(2 / tokens)
        assert abs(u.mean() - (1 - alpha ** T) * mean) < 6 * np.sqrt(var / tokens)
        # the gap of two independent tokens stays under the bound of part (b)
        assert 2 * var <= float(g["gap_variance_factor"]) * sigma ** 2 * (1 + 6 * np.sqrt(2 / tokens))


def test_cor1_uniform_scaling_invisible_to_ranking():
    """Corollary 1: uniform positive scaling of every score leaves the retained set unchanged (m_0 = 0)."""
    rng = np.random.default_rng(17)
    n, K, B = 60, 4, 12
    pos = np.arange(n)
    u1 = np.zeros(n)
    u2 = np.zeros(n)
    for _ in range(6):
        s = rng.random((K, n))
        u1 = fold_layers(u1, s, 0.8)
        u2 = fold_layers(u2, 3.7 * s, 0.8)
    np.testing.assert_array_equal(select_keep(u1, pos, B), select_keep(u2, pos, B))


def test_unknown_rule_rejected():
    with pytest.raises(ValueError):
        fold_layers(np.zeros(2), [np.zeros(2)], 0.5, "bogus")
    assert EMA == "ema"
