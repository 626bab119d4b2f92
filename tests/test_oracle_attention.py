"""Pins of the oracle's decode attention output (the softmax of Eq. 1 applied to V), used by the fused
attention + score path.  Every pin is a closed form or an invariant, not the oracle's own formula."""
import math

import numpy as np
import pytest

from oracle import Cache, Params, attention_output, evict_step, layer_scores


def _rng(seed):
    return np.random.default_rng(seed)


def test_identical_keys_give_the_mean_value():
    """Equal logits: a = 1/n, so o_h is the plain mean of its KV head's value rows."""
    rng = _rng(1)
    hq, hkv, n, d = 4, 2, 7, 8
    keys = np.broadcast_to(rng.standard_normal(d), (hkv, n, d)).copy()
    vals = rng.standard_normal((hkv, n, d))
    o, scale = attention_output(rng.standard_normal((hq, d)), keys, vals)
    for h in range(hq):
        np.testing.assert_allclose(o[h], vals[h // 2].mean(axis=0), rtol=0, atol=1e-15)
        np.testing.assert_allclose(scale[h], np.abs(vals[h // 2]).mean(axis=0), rtol=0, atol=1e-15)


def test_two_tokens_closed_form():
    """Two rows: a_1 = 1 / (1 + exp(z_2 - z_1)) (logistic), o = a_1 v_1 + (1 - a_1) v_2."""
    rng = _rng(2)
    d = 16
    q = rng.standard_normal((1, d))
    keys = rng.standard_normal((1, 2, d))
    vals = rng.standard_normal((1, 2, d))
    z1, z2 = (float(np.dot(keys[0, i], q[0])) / 4.0 for i in range(2))  # sqrt(16) = 4
    a1 = 1.0 / (1.0 + math.exp(z2 - z1))
    o, _ = attention_output(q, keys, vals)
    np.testing.assert_allclose(o[0], a1 * vals[0, 0] + (1 - a1) * vals[0, 1], rtol=1e-14, atol=1e-15)


def test_constant_values_and_group_mapping():
    """Rows of KV head g all equal c_g: every query head h returns exactly c_{h // G} (weights sum to 1),
    which pins the GQA head-to-KV-head mapping."""
    rng = _rng(3)
    hq, hkv, n, d = 6, 3, 11, 4
    c = rng.standard_normal((hkv, d))
    vals = np.repeat(c[:, None, :], n, axis=1)
    o, _ = attention_output(rng.standard_normal((hq, d)), rng.standard_normal((hkv, n, d)), vals)
    for h in range(hq):
        np.testing.assert_allclose(o[h], c[h // 2], rtol=1e-14)


def test_dominant_key_selects_its_value():
    """One logit 60 above the rest: o equals that row's value to exp(-60) ~ 1e-26."""
    rng = _rng(4)
    n, d = 9, 4
    q = np.zeros((1, d))
    q[0, 0] = 1.0
    keys = np.zeros((1, n, d))
    keys[0, 5, 0] = 120.0  # logit 120 / sqrt(4) = 60
    vals = rng.standard_normal((1, n, d))
    o, _ = attention_output(q, keys, vals)
    np.testing.assert_allclose(o[0], vals[0, 5], rtol=1e-15, atol=1e-15)


def test_recency_bias_closed_form():
    """Identical keys, bias beta on the w newest positions: those rows weigh e^beta / (w e^beta + n - w)."""
    rng = _rng(5)
    n, d, w, beta = 10, 8, 3, 0.5
    keys = np.broadcast_to(rng.standard_normal(d), (1, n, d)).copy()
    vals = rng.standard_normal((1, n, d))
    pos = np.arange(100, 100 + n)
    cur = int(pos[-1])
    o, _ = attention_output(rng.standard_normal((1, d)), keys, vals, pos, cur, beta, w)
    den = w * math.exp(beta) + (n - w)
    wts = np.where(pos >= cur - (w - 1), math.exp(beta), 1.0) / den
    np.testing.assert_allclose(o[0], wts @ vals[0], rtol=1e-14)


def test_linear_in_values_and_row_order_free():
    rng = _rng(6)
    hq, hkv, n, d = 4, 1, 13, 8
    q = rng.standard_normal((hq, d))
    keys = rng.standard_normal((hkv, n, d))
    v1, v2 = rng.standard_normal((2, hkv, n, d))
    o1, _ = attention_output(q, keys, v1)
    o2, _ = attention_output(q, keys, v2)
    o12, _ = attention_output(q, keys, v1 - 2.5 * v2)
    np.testing.assert_allclose(o12, o1 - 2.5 * o2, rtol=1e-12, atol=1e-14)
    perm = rng.permutation(n)
    op, _ = attention_output(q, keys[:, perm], v1[:, perm])
    np.testing.assert_allclose(op, o1, rtol=1e-12, atol=1e-14)


def test_head_mean_of_outputs_is_the_score_weighted_value():
    """One KV head: (1/H) sum_h o_h = sum_i s(i) v(i) with s the pooled score of Eq. 1 -- ties the attention
    output to the score the eviction uses."""
    rng = _rng(7)
    hq, n, d = 5, 17, 8
    q = rng.standard_normal((hq, d))
    keys = rng.standard_normal((1, n, d))
    vals = rng.standard_normal((1, n, d))
    pos = np.arange(n)
    o, _ = attention_output(q, keys, vals, pos, n - 1, 0.5, 4)
    s = layer_scores(q, keys, pos, n - 1, 0.5, 4)
    np.testing.assert_allclose(o.mean(axis=0), s @ vals[0], rtol=1e-12, atol=1e-14)


def test_convex_combination_bounds():
    """o is a convex combination of its KV head's value rows: elementwise between their min and max, and
    |o| <= scale <= max |v|."""
    rng = _rng(8)
    vals = rng.standard_normal((2, 20, 8))
    o, scale = attention_output(rng.standard_normal((4, 8)), rng.standard_normal((2, 20, 8)) * 3, vals)
    for h in range(4):
        g = h // 2
        assert np.all(o[h] >= vals[g].min(axis=0) - 1e-15) and np.all(o[h] <= vals[g].max(axis=0) + 1e-15)
        assert np.all(np.abs(o[h]) <= scale[h] + 1e-15)
        assert np.all(scale[h] <= np.abs(vals[g]).max(axis=0) + 1e-15)


def test_evict_step_attends_after_append_before_eviction():
    """The step's attention sees the appended token (it can dominate) and all n + 1 rows, even the one
    evicted by the same step."""
    rng = _rng(9)
    L, b, hkv, cap, d = 1, 1, 1, 8, 4
    k = np.zeros((L, b, hkv, cap, d), dtype=np.float32)
    v = rng.standard_normal((L, b, hkv, cap, d)).astype(np.float32)
    cache = Cache(k, v, np.zeros((b, cap)), np.arange(cap)[None].repeat(b, 0), 5, "f32")
    q = np.zeros((L, b, 1, d), dtype=np.float32)
    q[..., 0] = 1.0
    k_new = np.zeros((L, b, hkv, d), dtype=np.float32)
    k_new[..., 0] = 80.0  # logit 40 on the new token
    v_new = rng.standard_normal((L, b, hkv, d)).astype(np.float32)
    res = evict_step(cache, q, k_new, v_new, 1, 5, Params(alpha=0.5, budget=3), attention=True)
    np.testing.assert_allclose(res.o[0, 0, 0], v_new[0, 0, 0].astype(np.float64), rtol=1e-12)
    assert res.o.shape == (L, b, 1, d)
    no_attn = evict_step(Cache(k, v, np.zeros((b, cap)), np.arange(cap)[None].repeat(b, 0), 5, "f32"), q, k_new,
                         v_new, 1, 5, Params(alpha=0.5, budget=3))
    assert no_attn.o is None


@pytest.mark.parametrize("bad", [(4, 3)])
def test_group_mismatch_rejected(bad):
    hq, hkv = bad
    with pytest.raises(ValueError):
        attention_output(np.zeros((hq, 2)), np.zeros((hkv, 1, 2)), np.zeros((hkv, 1, 2)))
