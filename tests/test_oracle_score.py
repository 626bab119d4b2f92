"""Pins of the oracle's scoring step (Eq. 1, GQA pooling, scaled logits, recency bias) against facts that do
not depend on the oracle itself: closed forms, exact special cases and brute force on tiny inputs."""
import math

import numpy as np
import pytest
import scipy.special

from conftest import read_golden
from oracle import head_attention, layer_scores


def _rand(rng, *shape):
    return rng.standard_normal(shape)


@pytest.mark.parametrize("hq,hkv,n,d", [(4, 2, 7, 64), (8, 8, 33, 16), (28, 4, 19, 128), (32, 8, 50, 128)])
def test_probabilities_sum_to_one(hq, hkv, n, d):
    rng = np.random.default_rng(hq * 1000 + n)
    q, keys = _rand(rng, hq, d), _rand(rng, hkv, n, d)
    for h in range(hq):
        a = head_attention(q[h], keys[h // (hq // hkv)])
        assert np.all(a > 0)
        assert abs(a.sum() - 1.0) < 1e-12
    s = layer_scores(q, keys)
    # mean over H_q heads of distributions is a distribution; dividing by H_kv instead would give G.
    assert abs(s.sum() - 1.0) < 1e-12


def test_identical_keys_give_uniform_scores():
    rng = np.random.default_rng(1)
    n, d = 37, 64
    row = _rand(rng, d)
    keys = np.broadcast_to(row, (2, n, d)).copy()
    s = layer_scores(_rand(rng, 4, d), keys)
    assert np.all(s == s[0])
    assert abs(s[0] - 1.0 / n) < 1e-15


def test_two_token_closed_form():
    g = read_golden("two_token_softmax.txt")
    d = int(g["head_dim"])
    gap = float(g["raw_gap"])
    q = np.zeros(d)
    q[0] = 1.0
    keys = np.zeros((1, 2, d))
    keys[0, 0, 0] = gap + 0.25        # q.k1 - q.k2 = gap
    keys[0, 1, 0] = 0.25
    s = layer_scores(q[None], keys)
    assert abs(s[0] - float(g["p_first"])) < 1e-15
    assert abs(s[1] - float(g["p_second"])) < 1e-15


def test_gqa_group_mapping():
    """Query heads 0..G-1 read KV head 0 and G..2G-1 read KV head 1 (contiguous groups).  Only heads 0 and 1
    carry a strong query, aligned with a key planted in KV head 0 at slot 3; heads 2 and 3 attend
    uniformly.  The closed form below fails under an interleaved mapping (h % H_kv)."""
    d, n = 16, 9
    keys = np.zeros((2, n, d))
    keys[0, 3, 0] = 1.0
    keys[1, 5, 1] = 1.0
    q = np.zeros((4, d))
    q[0, 0] = q[1, 0] = 80.0            # logit gap 80 / 4 = 20 on KV head 0's slot 3
    s = layer_scores(q, keys)
    e = math.exp(20.0)
    p_hot = e / (e + n - 1)
    expect = np.full(n, (2 * (1 - p_hot) / (n - 1) + 2.0 / n) / 4)
    expect[3] = (2 * p_hot + 2.0 / n) / 4
    np.testing.assert_allclose(s, expect, rtol=1e-13, atol=0)


def test_recency_bias_window_boundary():
    """Identical keys; the bias applies to positions >= cur - (W - 1) only."""
    d, n, w, bias = 8, 6, 3, 0.5
    keys = np.ones((1, n, d))
    pos = np.array([0, 10, 17, 18, 19, 20])
    cur = 20                               # window covers 18, 19, 20 (17 is just outside)
    a = head_attention(np.ones(d), keys[0], pos, cur, bias, w)
    lo = 1.0 / (3 + 3 * math.exp(bias))
    np.testing.assert_allclose(a, [lo, lo, lo, lo * math.exp(bias), lo * math.exp(bias), lo * math.exp(bias)],
                               rtol=1e-14)


def test_brute_force_tiny():
    """Pure-Python loops with math.exp, against scipy's softmax, against the oracle."""
    rng = np.random.default_rng(7)
    hq, hkv, n, d = 6, 3, 5, 4
    q, keys = _rand(rng, hq, d), _rand(rng, hkv, n, d)
    pos = np.arange(n) * 3
    cur, bias, win = 12, 0.7, 2
    brute = [0.0] * n
    for h in range(hq):
        g = h // (hq // hkv)
        logits = []
        for i in range(n):
            dot = sum(q[h][j] * keys[g][i][j] for j in range(d)) / math.sqrt(d)
            if pos[i] >= cur - (win - 1):
                dot += bias
            logits.append(dot)
        ref = scipy.special.softmax(np.array(logits))
        mx = max(logits)
        tot = sum(math.exp(x - mx) for x in logits)
        for i in range(n):
            p = math.exp(logits[i] - mx) / tot
            assert abs(p - ref[i]) < 1e-15
            brute[i] += p / hq
    s = layer_scores(q, keys, pos, cur, bias, win)
    np.testing.assert_allclose(s, brute, rtol=1e-13)


def test_dominating_key_takes_all_mass():
    d, n = 32, 11
    rng = np.random.default_rng(3)
    keys = _rand(rng, 1, n, d) * 0.01
    q = np.zeros((2, d))
    q[:, 5] = 1.0
    keys[0, 4, 5] = 1e4
    s = layer_scores(q, keys)
    assert s[4] > 1 - 1e-12
