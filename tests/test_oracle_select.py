"""Pins of the oracle's top-B selection (Sec. 3 eviction rule, ties to the lower position) and hole-fill
compaction: brute force on tiny inputs plus invariants."""
import numpy as np
from hypothesis import given, settings
from hypothesis import strategies as st

from oracle import compact_rows, holefill_moves, select_keep


def _brute_keep(u, pos, B):
    order = sorted(range(len(u)), key=lambda i: (-u[i], pos[i]))
    keep = [False] * len(u)
    for i in order[:B]:
        keep[i] = True
    return np.array(keep)


@settings(max_examples=300, deadline=None)
@given(st.integers(1, 40).flatmap(lambda n: st.tuples(
    st.lists(st.sampled_from([0.0, 0.125, 0.25, 0.5, 1.0, 1e-30, 3.0]), min_size=n, max_size=n),
    st.permutations(list(range(100, 100 + n))),
    st.integers(1, n + 3))))
def test_select_matches_brute_force(case):
    u, pos, B = case
    u = np.array(u)
    pos = np.array(pos)
    keep = select_keep(u, pos, B)
    np.testing.assert_array_equal(keep, _brute_keep(u, pos, B))
    assert keep.sum() == min(B, len(u))
    if keep.sum() < len(u):
        kept = [(u[i], -pos[i]) for i in range(len(u)) if keep[i]]
        dropped = [(u[i], -pos[i]) for i in range(len(u)) if not keep[i]]
        assert min(kept) > max(dropped)


def test_all_equal_keeps_lowest_positions():
    n, B = 50, 7
    pos = np.random.default_rng(0).permutation(n) + 1000
    keep = select_keep(np.full(n, 0.02), pos, B)
    assert set(pos[keep]) == set(range(1000, 1007))


def test_under_budget_keeps_everything():
    keep = select_keep(np.array([0.1, 0.0, 0.3]), np.array([5, 6, 7]), 3)
    assert keep.all()


@settings(max_examples=300, deadline=None)
@given(st.integers(1, 60).flatmap(lambda n: st.tuples(
    st.lists(st.booleans(), min_size=n, max_size=n), st.integers(1, n))))
def test_holefill_invariants(case):
    flags, B = case
    n = len(flags)
    keep = np.zeros(n, dtype=bool)
    # force exactly min(B, n) kept by taking the first min(B,n) True-preferring slots of a random order
    rng = np.random.default_rng(n * 131 + B)
    order = sorted(range(n), key=lambda i: (not flags[i], rng.random()))
    keep[order[:min(B, n)]] = True
    k = min(B, n)
    dst, src = holefill_moves(keep, B)
    assert len(dst) == len(src) == int(keep[k:].sum())          # minimal: only kept rows beyond k move
    assert np.all(dst < k) and np.all(src >= k)                  # hazard-free
    assert np.all(np.diff(dst) > 0) and np.all(np.diff(src) > 0)
    rows = np.arange(n) * 10 + 3                                  # row payload = its original slot
    out = compact_rows(rows, keep, B)
    assert sorted(out[:k]) == sorted(rows[keep])                  # rows [0, k) hold exactly the kept rows
    np.testing.assert_array_equal(out[:k][keep[:k]], rows[:k][keep[:k]])   # kept rows below k stay put
