"""Pins of the oracle's decode step: refresh schedule (Eq. 5, Score-Free box), new-token initialisation
(Appendix, new-token insertion), stale-ranking eviction, budget formula, invariants over whole runs."""
import numpy as np
import pytest

from conftest import read_golden, read_golden_rows
from oracle import Cache, Params, budget_from_ratio, evict_step, refresh_due, to_f64
from workload import TINY, Workload, raw_numpy


def _cache(cfg, seed=None):
    w = Workload(cfg, seed=seed)
    st = w.prefill()
    c = Cache(raw_numpy(st["k"]), raw_numpy(st["v"]), st["u"].numpy().astype(np.float64),
              st["pos"].numpy().astype(np.int64), st["n"], cfg.dtype)
    return w, c


def _params(cfg, **kw):
    base = dict(alpha=cfg.alpha, budget=cfg.budget, refresh_period=cfg.refresh_period,
                score_free=cfg.score_free, nonrefresh_init=cfg.nonrefresh_init,
                recency_bias=cfg.recency_bias, recency_window=cfg.recency_window)
    base.update(kw)
    return Params(**base)


def _run(cfg, params, steps, seed=None):
    w, c = _cache(cfg, seed)
    results = []
    for t in range(1, steps + 1):
        si = w.step_inputs(t)
        r = evict_step(c, raw_numpy(si["q"]), raw_numpy(si["k_new"]), raw_numpy(si["v_new"]), t,
                       si["new_pos"], params)
        results.append(r)
    return c, results


SMALL = TINY.scaled(batch=2, layers=3, prefill_len=96, budget=17, steps=10)


def test_refresh_sets_golden():
    g = read_golden("refresh_sets.txt")
    for key, period, sf in (("r1", 1, False), ("r4", 4, False), ("r8", 8, False), ("score_free", 7, True)):
        want = [int(x) for x in g[key].split()]
        got = [t for t in range(1, 17) if refresh_due(t, period, sf)]
        assert got == want, key
    with pytest.raises(ValueError):
        refresh_due(0, 1, False)


def test_budget_formula_golden():
    for L0, rho, B in read_golden_rows("budgets.txt"):
        assert budget_from_ratio(int(L0), float(rho)) == int(B)


def test_to_f64_bf16_exact():
    bits = np.array([0x3F80, 0xBF80, 0x4049, 0x0000, 0x7F7F, 0x0001], dtype=np.uint16)
    np.testing.assert_array_equal(to_f64(bits, "bf16"), [1.0, -1.0, 3.140625, 0.0, 3.3895313892515355e38,
                                                         9.183549615799121e-41])


def test_full_vs_period_one_bit_identical():
    c1, r1 = _run(SMALL, _params(SMALL, refresh_period=1), 6)
    c2, _ = _run(SMALL, _params(SMALL, refresh_period=1, nonrefresh_init="min"), 6)
    assert all(r.refreshed for r in r1)
    np.testing.assert_array_equal(c1.u, c2.u)            # init policy is irrelevant when every step refreshes
    np.testing.assert_array_equal(c1.k, c2.k)


@pytest.mark.parametrize("init", ["mean", "min"])
def test_long_period_equals_score_free(init):
    T = 8
    ca, ra = _run(SMALL, _params(SMALL, refresh_period=T + 5, nonrefresh_init=init), T)
    cb, rb = _run(SMALL, _params(SMALL, score_free=True, nonrefresh_init=init), T)
    for a, b in zip(ra, rb):
        np.testing.assert_array_equal(a.keep, b.keep)
    np.testing.assert_array_equal(ca.u, cb.u)
    np.testing.assert_array_equal(ca.pos, cb.pos)


def test_step_one_identical_across_schedules():
    outs = []
    for kw in (dict(), dict(refresh_period=4), dict(score_free=True)):
        c, r = _run(SMALL, _params(SMALL, **kw), 1)
        outs.append((c.u.copy(), c.pos.copy(), r[0].keep))
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            np.testing.assert_array_equal(a, b)


def test_nonrefresh_keeps_old_utilities_and_inits_new_token():
    w, c = _cache(SMALL)
    p = _params(SMALL, refresh_period=4, nonrefresh_init="mean")
    si = w.step_inputs(1)
    evict_step(c, raw_numpy(si["q"]), raw_numpy(si["k_new"]), raw_numpy(si["v_new"]), 1, si["new_pos"], p)
    u_before = c.u[:, :c.n].copy()
    si = w.step_inputs(2)
    r = evict_step(c, raw_numpy(si["q"]), raw_numpy(si["k_new"]), raw_numpy(si["v_new"]), 2, si["new_pos"], p)
    assert not r.refreshed
    np.testing.assert_array_equal(r.u_pre[:, :-1], u_before)                  # stale ranking, bit-identical
    np.testing.assert_allclose(r.u_pre[:, -1], u_before.mean(axis=1), rtol=1e-15)
    assert r.s_layers is None


def test_min_init_new_token_evicted_at_once():
    """With the 'min' policy the new token ties the current minimum and loses the tie (highest position)."""
    w, c = _cache(SMALL)
    p = _params(SMALL, score_free=True, nonrefresh_init="min")
    for t in range(1, 6):
        si = w.step_inputs(t)
        r = evict_step(c, raw_numpy(si["q"]), raw_numpy(si["k_new"]), raw_numpy(si["v_new"]), t,
                       si["new_pos"], p)
        if t > 1:
            assert not r.keep[:, -1].any()
            assert all(len(d) == 0 for d, _ in r.moves)


def _hand_cache(u_vals, budget):
    n = len(u_vals)
    k = np.zeros((1, 1, 1, n + 1, 4), dtype=np.float32)
    k[0, 0, 0, :n, 0] = np.arange(n)
    return Cache(k, k.copy(), np.concatenate([u_vals, [0.0]])[None].astype(np.float64),
                 np.arange(n + 1, dtype=np.int64)[None] * 2, n, "f32")


def test_new_token_evicted_same_step_under_mean_when_it_ties():
    """Mean init over equal utilities equals every old utility; the newcomer (highest position) loses."""
    c = _hand_cache(np.full(5, 0.2), 5)
    p = Params(alpha=0.9, budget=5, score_free=True, nonrefresh_init="mean")
    z = np.zeros((1, 1, 1, 4), dtype=np.float32)
    r = evict_step(c, np.zeros((1, 1, 1, 4), np.float32), z + 7, z, 2, 100, p)
    assert r.u_pre[0, -1] == 0.2 and not r.keep[0, -1]
    assert c.n == 5 and 100 not in c.pos[0, :5]


def test_new_token_survives_under_mean_when_a_token_is_below():
    c = _hand_cache(np.array([0.5, 0.01, 0.3, 0.09, 0.1]), 5)
    p = Params(alpha=0.9, budget=5, score_free=True, nonrefresh_init="mean")
    z = np.zeros((1, 1, 1, 4), dtype=np.float32)
    r = evict_step(c, np.zeros((1, 1, 1, 4), np.float32), z + 7, z, 2, 100, p)
    assert abs(r.u_pre[0, -1] - 0.2) < 1e-15 and r.keep[0, -1]
    # the lowest-utility token (slot 1) is evicted and the newcomer's row fills its slot
    assert c.pos[0, 1] == 100 and c.k[0, 0, 0, 1, 0] == 7 and c.u[0, 1] == r.u_pre[0, -1]


def test_tiny_run_invariants():
    cfg = TINY
    c, res = _run(cfg, _params(cfg), cfg.steps)
    for t, r in enumerate(res, start=1):
        assert r.n_scored == (cfg.prefill_len + 1 if t == 1 else cfg.budget + 1)
        assert r.keep.sum(axis=1).tolist() == [cfg.budget] * cfg.batch
        # every per-layer score is a distribution over the n cached tokens
        np.testing.assert_allclose(r.s_layers.sum(axis=2), 1.0, rtol=1e-12)
    assert c.n == cfg.budget
    for b in range(cfg.batch):
        p = c.pos[b, :c.n]
        assert len(set(p.tolist())) == c.n
        assert np.all(c.u[b, :c.n] > 0)
    # the newest token's key row must sit wherever its position went
    w = Workload(cfg)
    last = w.step_inputs(cfg.steps)
    where = np.nonzero(c.pos[0, :c.n] == last["new_pos"])[0]
    if len(where):
        np.testing.assert_array_equal(c.k[:, 0, :, where[0], :], raw_numpy(last["k_new"])[:, 0])


def test_keep_override_must_be_valid():
    w, c = _cache(SMALL)
    si = w.step_inputs(1)
    bad = np.ones((SMALL.batch, SMALL.prefill_len + 1), dtype=bool)
    with pytest.raises(ValueError):
        evict_step(c, raw_numpy(si["q"]), raw_numpy(si["k_new"]), raw_numpy(si["v_new"]), 1, si["new_pos"],
                   _params(SMALL), keep_override=bad)
