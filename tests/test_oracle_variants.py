"""Pins of the oracle's scorer perturbations of Sec. 5.1 (VNorm, entropy weighting): closed forms,
reductions to plain attention, and the order-preservation properties the paper states."""
import math

import numpy as np

from oracle import (Cache, Params, evict_step, fold_layers, layer_scores, layer_scores_variant,
                    normalized_entropy, select_keep, value_norm_weights)


def _inputs(seed, hq=4, hkv=2, n=12, d=8):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((hq, d)), rng.standard_normal((hkv, n, d)) * 1.3,
            rng.standard_normal((hkv, n, d)), np.arange(n))


def test_vnorm_factor_closed_form():
    """Rows (3, 4) and (0, 1) have norms 5 and 1: factors 5/3 and 1/3."""
    nu = value_norm_weights(np.array([[3.0, 4.0], [0.0, 1.0]]))
    np.testing.assert_allclose(nu, [5 / 3, 1 / 3], rtol=1e-15)
    np.testing.assert_array_equal(value_norm_weights(np.zeros((3, 2))), np.ones(3))


def test_vnorm_with_equal_norms_is_plain_attention():
    """Values of equal norm (random directions scaled to 2): every factor is 1, the score is Eq. 1's."""
    q, k, v, pos = _inputs(1)
    v = 2.0 * v / np.linalg.norm(v, axis=-1, keepdims=True)
    np.testing.assert_allclose(layer_scores_variant(q, k, v, pos, 11, 0.5, 4, True, False),
                               layer_scores(q, k, pos, 11, 0.5, 4), rtol=1e-13)


def test_vnorm_single_kv_head_scales_each_token():
    """One KV head: s_vnorm(i) = s(i) * |v_i| / mean_j |v_j| exactly (the factor leaves the head sum)."""
    q, k, v, pos = _inputs(2, hq=3, hkv=1)
    norms = np.array([math.sqrt(sum(x * x for x in row)) for row in v[0]])
    np.testing.assert_allclose(layer_scores_variant(q, k, v, pos, 0, 0.0, 0, True, False),
                               layer_scores(q, k, pos, 0, 0.0, 0) * norms / norms.mean(), rtol=1e-13)


def test_vnorm_per_kv_head_factor():
    """Scaling all value rows of KV head 1 by 7 changes nothing: the factor is mean-normalised per KV head."""
    q, k, v, pos = _inputs(3)
    base = layer_scores_variant(q, k, v, pos, 0, 0.0, 0, True, False)
    v2 = v.copy()
    v2[1] *= 7.0
    np.testing.assert_allclose(layer_scores_variant(q, k, v2, pos, 0, 0.0, 0, True, False), base, rtol=1e-13)


def test_entropy_closed_forms():
    np.testing.assert_allclose(normalized_entropy(np.full(8, 1 / 8)), 1.0, rtol=1e-15)
    p = 0.2
    h2 = -(p * math.log(p) + (1 - p) * math.log(1 - p)) / math.log(2)
    np.testing.assert_allclose(normalized_entropy(np.array([p, 1 - p])), h2, rtol=1e-14)
    assert normalized_entropy(np.array([1.0, 0.0, 0.0])) == 0.0
    assert normalized_entropy(np.array([0.3])) == 1.0


def test_entropy_weighting_is_a_uniform_scale_of_the_layer():
    """Entropy weighting multiplies the whole layer by the normalised entropy of its attention: ratios are
    constant, the within-layer order is unchanged (Sec. 5.1), and identical keys (uniform attention) give
    a factor of exactly 1."""
    q, k, v, pos = _inputs(4)
    plain = layer_scores(q, k, pos, 11, 0.5, 4)
    ent = layer_scores_variant(q, k, v, pos, 11, 0.5, 4, False, True)
    ratio = ent / plain
    np.testing.assert_allclose(ratio, ratio[0], rtol=1e-13)
    assert 0.0 < ratio[0] < 1.0
    np.testing.assert_allclose(ratio[0], normalized_entropy(plain), rtol=1e-13)
    np.testing.assert_array_equal(np.argsort(-ent, kind="stable"), np.argsort(-plain, kind="stable"))
    kk = np.broadcast_to(k[:, :1], k.shape).copy()
    np.testing.assert_allclose(layer_scores_variant(q, kk, v, pos, 0, 0.0, 0, False, True),
                               layer_scores(q, kk, pos, 0, 0.0, 0), rtol=1e-14)


def test_entropy_uses_attention_before_vnorm():
    q, k, v, pos = _inputs(5)
    both = layer_scores_variant(q, k, v, pos, 11, 0.5, 4, True, True)
    vn = layer_scores_variant(q, k, v, pos, 11, 0.5, 4, True, False)
    np.testing.assert_allclose(both, vn * normalized_entropy(layer_scores(q, k, pos, 11, 0.5, 4)), rtol=1e-13)


def test_entropy_single_layer_keeps_the_retention_set():
    """One layer from a zero prior: entropy weighting scales u uniformly, so the top-B set is unchanged
    (the Corollary 1 argument)."""
    rng = np.random.default_rng(6)
    L, b, hkv, cap, d, n = 1, 1, 2, 40, 8, 30
    k = rng.standard_normal((L, b, hkv, cap, d)).astype(np.float32)
    v = rng.standard_normal((L, b, hkv, cap, d)).astype(np.float32)
    q = rng.standard_normal((L, b, 4, d)).astype(np.float32)
    kn = rng.standard_normal((L, b, hkv, d)).astype(np.float32)
    res = {}
    for ent in (False, True):
        c = Cache(k.copy(), v.copy(), np.zeros((b, cap)), np.arange(cap)[None].copy(), n, "f32")
        res[ent] = evict_step(c, q, kn, kn, 1, n, Params(alpha=0.8, budget=9, entropy=ent))
    np.testing.assert_array_equal(res[True].keep, res[False].keep)
    ratio = res[True].s_layers / res[False].s_layers
    np.testing.assert_allclose(ratio, ratio.flat[0], rtol=1e-13)


def test_vnorm_changes_rankings_only_through_values():
    """VNorm is a per-token reweighting: with K = 1 and a zero prior the retained set is the top B of
    s(i) * factor(i), computed here from the plain score."""
    rng = np.random.default_rng(7)
    L, b, hkv, cap, d, n = 1, 1, 1, 40, 8, 30
    k = rng.standard_normal((L, b, hkv, cap, d)).astype(np.float32)
    v = (rng.standard_normal((L, b, hkv, cap, d)) * rng.uniform(0.2, 3.0, (1, 1, 1, cap, 1))).astype(np.float32)
    q = rng.standard_normal((L, b, 2, d)).astype(np.float32)
    kn = rng.standard_normal((L, b, hkv, d)).astype(np.float32)
    c = Cache(k.copy(), v.copy(), np.zeros((b, cap)), np.arange(cap)[None].copy(), n, "f32")
    res = evict_step(c, q, kn, kn, 1, n, Params(alpha=0.8, budget=9, vnorm=True))
    kf = np.concatenate([k[0, 0, 0, :n], kn[0, 0]], axis=0).astype(np.float64)[None]
    vf = np.concatenate([v[0, 0, 0, :n], kn[0, 0]], axis=0).astype(np.float64)
    s = layer_scores(q[0, 0].astype(np.float64), kf, None, 0, 0.0, 0)
    norms = np.sqrt((vf * vf).sum(axis=1))
    u = fold_layers(np.zeros(n + 1), [s * norms / norms.mean()], 0.8)
    np.testing.assert_array_equal(res.keep[0], select_keep(u, np.arange(n + 1), 9))
