"""Pins of the oracle's rank-trace diagnostics (appendix "Mechanistic Diagnostics"): hand-built sets with
known intersections, the closed-form EMA churn of a steady step (k = B), and Jaccard identities."""
import math

import numpy as np

from oracle import Cache, Params, RankTraceState, evict_step, rank_trace_counts, trace_metrics


def test_hand_built_sets():
    """Positions 10..15; raw top-3 = {12, 14, 15}, u top-3 = {10, 12, 13}, evicted = {11, 14}; the previous
    step's sets were R' = {12, 13, 99} and E' = {10, 12, 13}."""
    pos = np.array([10, 11, 12, 13, 14, 15])
    raw = np.array([0.1, 0.0, 0.5, 0.2, 0.6, 0.4])
    u = np.array([0.9, 0.1, 0.8, 0.7, 0.3, 0.2])
    keep = np.array([1, 0, 1, 1, 0, 1], dtype=bool)
    st = RankTraceState(raw={12, 13, 99}, ema={10, 12, 13})
    c = rank_trace_counts(st, raw, u, pos, keep, 3)
    assert c == dict(r=3, e=3, has_prev=1, rr=1, ee=3, re=1, rev=1, rp=3, ep=3)
    m = trace_metrics(c)
    assert math.isclose(m["raw_churn"], 1 - 1 / 5) and m["ema_churn"] == 0.0
    assert math.isclose(m["raw_ema_jaccard"], 1 / 5) and math.isclose(m["raw_top_evicted"], 1 / 3)
    assert st.raw == {12, 14, 15} and st.ema == {10, 12, 13}


def test_ties_keep_lower_position_and_first_step():
    pos = np.array([7, 3, 5])
    st = RankTraceState()
    c = rank_trace_counts(st, np.ones(3), np.ones(3), pos, np.ones(3, dtype=bool), 2)
    assert st.raw == {3, 5} == st.ema
    assert c["has_prev"] == 0 and c["rr"] == 0 and c["re"] == 2 and c["rev"] == 0
    m = trace_metrics(c)
    assert math.isnan(m["raw_churn"]) and math.isnan(m["ema_churn"]) and m["raw_ema_jaccard"] == 1.0


def test_steady_ema_churn_closed_form():
    """k = B on steady steps (B cached + 1 new): E_t is the retained set, so consecutive sets share B - 1
    tokens when an old token is evicted (churn 2 / (B + 1)) and all B when the new one is (churn 0)."""
    rng = np.random.default_rng(3)
    L, b, hkv, d, B = 2, 1, 2, 8, 12
    cap = B + 2
    k = rng.standard_normal((L, b, hkv, cap, d)).astype(np.float32)
    v = rng.standard_normal((L, b, hkv, cap, d)).astype(np.float32)
    cache = Cache(k, v, np.zeros((b, cap)), np.arange(cap)[None].copy(), B, "f32")
    st = RankTraceState()
    p = Params(alpha=0.7, budget=B)
    seen = set()
    for t in range(1, 9):
        q = rng.standard_normal((L, b, 4, d)).astype(np.float32)
        kn = rng.standard_normal((L, b, hkv, d)).astype(np.float32)
        res = evict_step(cache, q, kn, kn, t, 100 + t, p)
        c = rank_trace_counts(st, res.raw[0], res.u_pre[0], res.pos_pre[0], res.keep[0], B)
        assert c["r"] == c["e"] == B and c["rev"] in (0, 1)
        if c["has_prev"]:
            new_kept = bool(res.keep[0, -1])
            assert c["ee"] == (B - 1 if new_kept else B)
            churn = trace_metrics(c)["ema_churn"]
            assert math.isclose(churn, 2 / (B + 1) if new_kept else 0.0, abs_tol=1e-15)
            seen.add(new_kept)
        # the raw score is the layer mean of the plain scores, a distribution over the n tokens
        assert abs(res.raw[0].sum() - 1) < 1e-12
    assert seen  # at least one step compared with its predecessor


def test_jaccard_identities():
    c = dict(r=4, e=4, has_prev=1, rr=4, ee=0, re=4, rev=0, rp=4, ep=6)
    m = trace_metrics(c)
    assert m["raw_churn"] == 0.0 and m["ema_churn"] == 1.0 and m["raw_ema_jaccard"] == 1.0
    assert m["raw_top_evicted"] == 0.0
