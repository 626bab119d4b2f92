"""Multi-step GPU parity of kv_evict_step against the oracle in lockstep, on the five workloads at sizes the
oracle finishes in seconds (same GQA shapes, dtypes, schedules and input laws; fewer tokens and layers).

Per step: per-layer scores and the compacted utilities within 1e-3 relative; retention sets equal outside
the 1e-4 band around the B-th utility; positions and compacted K/V rows bit-exact.  When the GPU takes an
equally valid in-band decision, the oracle adopts it (its own float64 utilities kept) so the runs stay
comparable; such flips are counted and reported."""
import numpy as np
import pytest
import torch

from oracle import evict_step
from parity import assert_close, check_norm_cache, lockstep_adopter, oracle_cache, oracle_params, to_device
from workload import LLAMA8B, LLAMA8B_LAZY, QWEN, SCOREFREE128K, TINY, Workload, raw_numpy

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2609_03515_amd.binding")


def run_lockstep(cfg, steps, seed=None, rule="ema", vnorm=False, entropy=False, merge=0, norm_cache=False):
    w = Workload(cfg, seed=seed)
    cap = max(cfg.prefill_len, cfg.budget) + 1          # room for the cache to grow up to B + 1
    st = w.prefill(capacity=cap)
    oc = oracle_cache(st, cfg.dtype)
    dev = to_device(st)
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cap, cfg.dtype)
    params = B.make_params(cfg.alpha, cfg.budget, cfg.refresh_period, cfg.score_free, cfg.nonrefresh_init,
                           cfg.recency_bias, cfg.recency_window, rule, vnorm=vnorm, entropy=entropy,
                           score_merge=merge)
    op = oracle_params(cfg, rule=rule, vnorm=vnorm, entropy=entropy)
    ws = B.workspace(shape, cap)
    n = st["n"]
    norms = None
    if norm_cache:   # VNorm's value-norm cache, filled once from the prefill, then kept by the steps
        norms = torch.full((cfg.layers, cfg.batch, cfg.n_kv_heads, cap), -1.0, device="cuda")
        if n > 0:
            B.kv_value_norms(shape, n, dev["v"], norms)
    flips = 0
    for t in range(1, steps + 1):
        si = w.step_inputs(t)
        sig = to_device(si)
        keep = torch.zeros(cfg.batch, cap, dtype=torch.uint8, device="cuda")
        s_out = torch.full((cfg.layers, cfg.batch, n + 1), -1.0, device="cuda")
        n_out = B.kv_evict_step(shape, params, t, n, si["new_pos"], sig["q"], sig["k_new"], sig["v_new"],
                                dev["k"], dev["v"], dev["u"], dev["pos"], ws, keep_out=keep, s_out=s_out,
                                v_norms=norms)
        torch.cuda.synchronize()
        q_raw, kn_raw, vn_raw = raw_numpy(si["q"]), raw_numpy(si["k_new"]), raw_numpy(si["v_new"])
        keep_g = keep.cpu().numpy()[:, : n + 1].astype(bool)
        step_flips = []
        ref = evict_step(oc, q_raw, kn_raw, vn_raw, t, si["new_pos"], op,
                         keep_override=lockstep_adopter(keep_g, cfg.budget, f"{cfg.name} t={t}", step_flips))
        assert n_out == ref.n_out == min(cfg.budget, n + 1)
        flips += sum(step_flips)
        if ref.refreshed:
            assert_close(s_out.cpu().numpy(), ref.s_layers, f"{cfg.name} t={t} scores")
        n = n_out
        assert_close(dev["u"][:, :n].cpu().numpy(), oc.u[:, :n], f"{cfg.name} t={t} utilities")
        np.testing.assert_array_equal(dev["pos"][:, :n].cpu().numpy(), oc.pos[:, :n])
        np.testing.assert_array_equal(raw_numpy(dev["k"])[:, :, :, :n], oc.k[:, :, :, :n])
        np.testing.assert_array_equal(raw_numpy(dev["v"])[:, :, :, :n], oc.v[:, :, :, :n])
        if norms is not None:
            check_norm_cache(B, shape, dev["v"], norms, n, oc.v, cfg.dtype, f"{cfg.name} t={t}")
        print(f"{cfg.name} t={t} refresh={ref.refreshed} n={n} in-band flips so far={flips}", flush=True)
    return flips


CASES = {
    "tiny": (TINY, TINY.steps),
    "llama8b_reduced": (LLAMA8B.scaled(batch=2, layers=4, prefill_len=1200, budget=120), 6),
    "llama8b_split_step1": (LLAMA8B.scaled(batch=1, layers=2, prefill_len=6000, budget=600), 3),
    "lazy_r4_min": (LLAMA8B_LAZY.scaled(batch=2, layers=3, prefill_len=800, budget=80), 10),
    "lazy_r4_mean": (LLAMA8B_LAZY.scaled(batch=2, layers=3, prefill_len=800, budget=80, nonrefresh_init="mean"), 10),
    "lazy_r8_min": (LLAMA8B_LAZY.scaled(batch=2, layers=3, prefill_len=800, budget=80, refresh_period=8), 12),
    "scorefree_min": (SCOREFREE128K.scaled(batch=2, layers=3, prefill_len=3000, budget=300), 12),
    "scorefree_mean": (SCOREFREE128K.scaled(batch=2, layers=3, prefill_len=3000, budget=300,
                                            nonrefresh_init="mean"), 12),
    "qwen_reduced": (QWEN.scaled(batch=3, layers=3, prefill_len=1000, budget=250), 5),
    "qwen_split_step1": (QWEN.scaled(batch=1, layers=2, prefill_len=3000, budget=750), 3),
    # step 1 over 20,001 tokens at batch 2: the multi-workgroup selection and its compaction plan
    "scorefree_wide_select": (SCOREFREE128K.scaled(batch=2, layers=2, prefill_len=20000, budget=2000), 4),
    "under_budget": (TINY.scaled(prefill_len=40, budget=45), 8),
    # Lazy steps that first only append (cache under budget), then evict one token each
    "lazy_under_budget": (LLAMA8B_LAZY.scaled(batch=2, layers=2, prefill_len=40, budget=44, nonrefresh_init="mean"), 9),
    "lazy_under_budget_min": (LLAMA8B_LAZY.scaled(batch=2, layers=2, prefill_len=40, budget=44), 9),
    # an empty cache: the first refresh steps score only the newcomer (no cached row is read), then evict
    "empty_start": (TINY.scaled(prefill_len=0, budget=3), 8),
    "lazy_empty_start": (LLAMA8B_LAZY.scaled(batch=2, layers=2, prefill_len=0, budget=4, nonrefresh_init="mean"), 10),
}


@pytest.mark.parametrize("name", list(CASES))
def test_evict_step_lockstep(name):
    cfg, steps = CASES[name]
    print(f"lockstep case {name}: {cfg}", flush=True)
    flips = run_lockstep(cfg, steps)
    print(f"{name}: in-band flips {flips}", flush=True)


@pytest.mark.parametrize("rule", ["single", "cumulative"])
def test_aggregation_rules(rule):
    cfg = LLAMA8B.scaled(batch=1, layers=3, prefill_len=500, budget=50)
    run_lockstep(cfg, 4, rule=rule)


VARIANT_CASES = {
    "tiny": (TINY, 5),
    "llama8b_reduced": (LLAMA8B.scaled(batch=2, layers=3, prefill_len=1200, budget=120), 4),
    "llama8b_split_step1": (LLAMA8B.scaled(batch=1, layers=2, prefill_len=6000, budget=600), 2),
    "qwen_reduced": (QWEN.scaled(batch=2, layers=2, prefill_len=1000, budget=250), 3),
    "lazy_r4_mean": (LLAMA8B_LAZY.scaled(batch=2, layers=2, prefill_len=800, budget=80, nonrefresh_init="mean"), 6),
}


@pytest.mark.parametrize("vnorm,entropy", [(True, False), (False, True), (True, True)],
                         ids=["vnorm", "entropy", "both"])
@pytest.mark.parametrize("name", list(VARIANT_CASES))
def test_scorer_variants_lockstep(name, vnorm, entropy):
    """Sec. 5.1 scorer perturbations through kv_evict_step, in lockstep with the oracle."""
    cfg, steps = VARIANT_CASES[name]
    run_lockstep(cfg, steps, vnorm=vnorm, entropy=entropy)


NORM_CACHE_CASES = {
    "tiny": (TINY, 6),
    "llama8b_reduced": (LLAMA8B.scaled(batch=2, layers=3, prefill_len=1200, budget=120), 5),
    "llama8b_split_step1": (LLAMA8B.scaled(batch=1, layers=2, prefill_len=6000, budget=600), 3),
    "qwen_reduced": (QWEN.scaled(batch=2, layers=2, prefill_len=1000, budget=250), 4),
    "lazy_r4_min": (LLAMA8B_LAZY.scaled(batch=2, layers=2, prefill_len=800, budget=80), 9),
    "lazy_r4_mean": (LLAMA8B_LAZY.scaled(batch=2, layers=2, prefill_len=800, budget=80, nonrefresh_init="mean"), 9),
    "scorefree_mean": (SCOREFREE128K.scaled(batch=2, layers=2, prefill_len=3000, budget=300,
                                            nonrefresh_init="mean"), 8),
    "lazy_under_budget": (LLAMA8B_LAZY.scaled(batch=2, layers=2, prefill_len=40, budget=44, nonrefresh_init="mean"), 9),
    "empty_start": (TINY.scaled(prefill_len=0, budget=3), 6),
}


@pytest.mark.parametrize("vnorm,entropy", [(True, False), (True, True), (False, False)],
                         ids=["vnorm", "vnorm_entropy", "plain"])
@pytest.mark.parametrize("name", list(NORM_CACHE_CASES))
def test_value_norm_cache_lockstep(name, vnorm, entropy):
    """VNorm from the value-norm cache (Sec. 5.1; a value row's norm is computed once, when it is cached):
    kv_evict_step in lockstep with the oracle, the cache checked after every step (every append, placement
    and compaction keeps each norm beside its row), on steady steps (three kernels plus the norms' mean),
    first steps, non-refresh steps under both priors and caches under budget; "plain" keeps the cache without
    VNorm."""
    cfg, steps = NORM_CACHE_CASES[name]
    run_lockstep(cfg, steps, vnorm=vnorm, entropy=entropy, norm_cache=True)


def test_vnorm_fused_into_the_merged_scorer_lockstep():
    """VNorm applied inside the multi-slab scorer (Sec. 5.1): a steady step given the value-norm cache, with the
    planned merge above one (1,024 slabs over 256 CUs plan two KV heads per workgroup), weights each KV head's
    group sums by norm / mean before the item adds them; in lockstep with the oracle over the first step (the
    five-kernel path) and four steady steps, the norm cache checked after every step."""
    cfg = LLAMA8B.scaled(batch=4, layers=32, prefill_len=400, budget=300)
    cap = cfg.prefill_len + 1
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cap, cfg.dtype)
    plain = B.make_params(cfg.alpha, cfg.budget, 1, False, "mean", cfg.recency_bias, cfg.recency_window)
    if B.kv_score_merge(shape, cfg.budget + 1, plain) < 2:
        pytest.skip("this device plans one KV head per scoring workgroup at this shape")
    run_lockstep(cfg, 5, vnorm=True, norm_cache=True)


@pytest.mark.parametrize("init", ["min", "mean"])
def test_nonrefresh_newcomer_kept_on_position_tie(init):
    """Non-refresh step where the newcomer survives: under the min prior it ties the lowest utility, and the
    cached token holding that utility has a higher position than the newcomer (positions need not grow), so
    that token is evicted and the newcomer's rows must land in its slot."""
    cfg = LLAMA8B_LAZY.scaled(batch=2, layers=3, prefill_len=60, budget=60, nonrefresh_init=init)
    w = Workload(cfg)
    cap = cfg.prefill_len + 1
    st = w.prefill(capacity=cap)
    rng = np.random.default_rng(5)
    u = rng.uniform(0.1, 1.0, (cfg.batch, cap))
    low = [7, 33]                                   # per sequence: the unique minimum
    for b, j in enumerate(low):
        u[b, j] = 0.01
    st["u"] = torch.tensor(u, dtype=torch.float32)
    pos = np.tile(np.arange(cap, dtype=np.int64) * 10, (cfg.batch, 1))
    pos[0, low[0]] = 10_000                          # higher than the newcomer's position below
    pos[1, low[1]] = 10_000
    st["pos"] = torch.tensor(pos, dtype=torch.int32)
    oc = oracle_cache(st, cfg.dtype)
    dev = to_device(st)
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cap, cfg.dtype)
    params = B.make_params(cfg.alpha, cfg.budget, 4, False, init, cfg.recency_bias, cfg.recency_window)
    ws = B.workspace(shape, cap)
    si = w.step_inputs(2)
    new_pos = 5_000
    keep = torch.zeros(cfg.batch, cap, dtype=torch.uint8, device="cuda")
    sig = to_device(si)
    n_out = B.kv_evict_step(shape, params, 2, st["n"], new_pos, sig["q"], sig["k_new"], sig["v_new"], dev["k"],
                            dev["v"], dev["u"], dev["pos"], ws, keep_out=keep)
    torch.cuda.synchronize()
    ref = evict_step(oc, raw_numpy(si["q"]), raw_numpy(si["k_new"]), raw_numpy(si["v_new"]), 2, new_pos,
                     oracle_params(cfg, refresh_period=4, nonrefresh_init=init))
    assert n_out == ref.n_out == cfg.budget
    np.testing.assert_array_equal(keep.cpu().numpy()[:, : cfg.budget + 1].astype(bool), ref.keep)
    if init == "min":
        assert not ref.keep[0, low[0]] and not ref.keep[1, low[1]] and ref.keep[:, -1].all()
    assert_close(dev["u"][:, :n_out].cpu().numpy(), oc.u[:, :n_out], f"{init} utilities")
    np.testing.assert_array_equal(dev["pos"][:, :n_out].cpu().numpy(), oc.pos[:, :n_out])
    np.testing.assert_array_equal(raw_numpy(dev["k"])[:, :, :, :n_out], oc.k[:, :, :, :n_out])
    np.testing.assert_array_equal(raw_numpy(dev["v"])[:, :, :, :n_out], oc.v[:, :, :, :n_out])


MERGE_CASES = {
    "llama8b_reduced": (LLAMA8B.scaled(batch=2, layers=3, prefill_len=1200, budget=120), 4),
    "llama8b_split_step1": (LLAMA8B.scaled(batch=1, layers=2, prefill_len=6000, budget=600), 3),
    "qwen_reduced": (QWEN.scaled(batch=2, layers=2, prefill_len=1000, budget=250), 3),
    "tiny": (TINY, 5),
}


@pytest.mark.parametrize("name,merge,entropy", [
    ("llama8b_reduced", 2, False), ("llama8b_reduced", 4, True), ("llama8b_reduced", 8, False),
    ("llama8b_split_step1", 8, False), ("qwen_reduced", 2, False), ("qwen_reduced", 4, True),
    ("tiny", 2, False)])
def test_merged_scoring_lockstep(name, merge, entropy):
    """Scoring workgroups that cover several KV heads of one (layer, sequence) and add their group sums in
    LDS before writing them (the first step of the split case: teams of chunks exchanging their statistics
    that add the sums of 8 KV heads over consecutive rounds)."""
    cfg, steps = MERGE_CASES[name]
    run_lockstep(cfg, steps, entropy=entropy, merge=merge)


@pytest.mark.parametrize("merge,entropy", [(0, False), (1, False), (2, False), (4, False), (8, False), (0, True)])
def test_first_step_exchange_teams_lockstep(merge, entropy):
    """A first step over slabs too long for one workgroup: chunks that exchange their softmax statistics, in
    teams that score `merge` KV heads of a (layer, sequence) in consecutive rounds and add their group sums in
    LDS (0: the planned merge, 4 for 8 KV heads), then a steady step; in lockstep with the oracle (also with
    entropy weighting, taken from the merged rows)."""
    cfg = LLAMA8B.scaled(batch=2, layers=3, prefill_len=12000, budget=1200)
    cap = cfg.prefill_len + 1
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cap, cfg.dtype)
    params = B.make_params(cfg.alpha, cfg.budget, 1, False, "mean", cfg.recency_bias, cfg.recency_window,
                           entropy=entropy, score_merge=merge)
    info = B.kv_score_plan(shape, cap, params)
    assert info.path == B.KV_PATH_EXCHANGE and info.chunks > 1, (info.path, info.chunks)
    assert info.merge == (merge or 4)
    assert B.kv_score_merge(shape, cap, params) == info.merge
    run_lockstep(cfg, 2, entropy=entropy, merge=merge)


@pytest.mark.parametrize("cfg,chunks,merge", [(LLAMA8B, 16, 4), (SCOREFREE128K, 61, 4), (QWEN, 4, 4)],
                         ids=["llama8b_32k", "scorefree_128k", "qwen_8k"])
def test_first_step_plans_of_the_benchmark_shapes(cfg, chunks, merge):
    """The planner's first-step choices at the benchmark's shapes on an MI355X (256 CUs): the exchange path,
    42.5 KiB chunks of logits and item sums for groups of 4 (16 chunks per 32k slab, 61 per 128k slab), 80 KiB
    for Qwen's padded group of 8, and teams of 4 KV heads; VNorm keeps one row per KV head (52 KiB chunks)."""
    n = cfg.prefill_len + 1
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.capacity, cfg.dtype)
    info = B.kv_score_plan(shape, n, B.make_params(cfg.alpha, cfg.budget, 1))
    assert (info.path, info.chunks, info.merge) == (B.KV_PATH_EXCHANGE, chunks, merge)
    vn = B.kv_score_plan(shape, n, B.make_params(cfg.alpha, cfg.budget, 1, vnorm=True))
    assert vn.path == B.KV_PATH_EXCHANGE and vn.merge == 1


@pytest.mark.parametrize("cfg,merge", [(LLAMA8B, 4), (QWEN, 2)], ids=["llama8b_32k", "qwen_8k"])
def test_steady_step_plans_of_the_benchmark_shapes(cfg, merge):
    """The planner's steady-step choices at the benchmark's shapes on an MI355X: one workgroup per item of
    `merge` KV heads with its logits in LDS (8B: 512 items of 4, two per CU; Qwen-shaped: 1,792 items of 2)."""
    n = cfg.budget + 1
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, n, cfg.dtype)
    info = B.kv_score_plan(shape, n, B.make_params(cfg.alpha, cfg.budget, 1))
    assert (info.path, info.chunks, info.merge) == (B.KV_PATH_LDS, 1, merge)


def test_first_step_exchange_teams_several_items_each():
    """Exchange teams that score more than one item: 40,001 tokens make 19 chunks per slab, so an MI355X holds
    768 / 19 = 40 teams at once for the 48 items of 4 KV heads (2 sequences x 12 layers x 2 blocks); eight
    teams go on to a second item.  In lockstep with the oracle."""
    cfg = LLAMA8B.scaled(batch=2, layers=12, prefill_len=40000, budget=4000)
    cap = cfg.prefill_len + 1
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cap, cfg.dtype)
    params = B.make_params(cfg.alpha, cfg.budget, 1, False, "mean", cfg.recency_bias, cfg.recency_window)
    info = B.kv_score_plan(shape, cap, params)
    assert (info.path, info.merge) == (B.KV_PATH_EXCHANGE, 4) and info.chunks >= 16, (info.path, info.chunks)
    run_lockstep(cfg, 2)


@pytest.mark.parametrize("cfg", [LLAMA8B.scaled(batch=2, layers=3, prefill_len=300, budget=60),
                                 QWEN.scaled(batch=3, layers=2, prefill_len=200, budget=50)],
                         ids=["llama8b_reduced", "qwen_reduced"])
def test_steps_without_keep_out_leave_identical_caches(cfg):
    """kv_evict_step with and without keep_out (the benchmark's call) leaves bit-identical caches, utilities and
    positions: the decision writes are the only difference between the two launches."""
    w = Workload(cfg)
    cap = cfg.prefill_len + 1
    st = to_device(w.prefill(capacity=cap))
    other = {k: (v.clone() if isinstance(v, torch.Tensor) else v) for k, v in st.items()}
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cap, cfg.dtype)
    params = B.make_params(cfg.alpha, cfg.budget, 1, False, "mean", cfg.recency_bias, cfg.recency_window)
    ws = B.workspace(shape, cap)
    n1 = n2 = st["n"]
    for t in range(1, 7):
        sig = to_device(w.step_inputs(t))
        keep = torch.zeros(cfg.batch, cap, dtype=torch.uint8, device="cuda")
        n1 = B.kv_evict_step(shape, params, t, n1, sig["new_pos"], sig["q"], sig["k_new"], sig["v_new"], st["k"],
                             st["v"], st["u"], st["pos"], ws, keep_out=keep)
        n2 = B.kv_evict_step(shape, params, t, n2, sig["new_pos"], sig["q"], sig["k_new"], sig["v_new"],
                             other["k"], other["v"], other["u"], other["pos"], ws)
        torch.cuda.synchronize()
        assert n1 == n2 == min(cfg.budget, (cfg.prefill_len if t == 1 else cfg.budget) + 1)
        assert int(keep[:, : (cfg.prefill_len if t == 1 else cfg.budget) + 1].sum()) == cfg.batch * n1
        for name in ("u", "pos"):
            assert torch.equal(st[name][:, :n1], other[name][:, :n1]), (t, name)
        for name in ("k", "v"):
            assert torch.equal(st[name][:, :, :, :n1], other[name][:, :, :, :n1]), (t, name)
        print(f"{cfg.name} t={t}: identical with and without keep_out", flush=True)


def test_cache_wrapper_matches_entry_point():
    """evict_step(cache, q, k_new, v_new, t, params) is kv_evict_step on the cache's buffers: over refresh and
    non-refresh steps (Lazy R = 4, mean prior) both leave bit-identical buffers and row counts."""
    cfg = LLAMA8B_LAZY.scaled(batch=2, layers=3, prefill_len=800, budget=80, nonrefresh_init="mean")
    w = Workload(cfg, seed=7)
    cap = cfg.prefill_len + 1
    st = w.prefill(capacity=cap)
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cap, cfg.dtype)
    params = B.make_params(cfg.alpha, cfg.budget, cfg.refresh_period, cfg.score_free, cfg.nonrefresh_init,
                           cfg.recency_bias, cfg.recency_window)
    a, b = to_device(st), to_device(st)
    cache = B.KvCache(shape, b["k"], b["v"], b["u"], b["pos"], st["n"], B.workspace(shape, cap))
    ws, n = B.workspace(shape, cap), st["n"]
    for t in range(1, 7):
        si = w.step_inputs(t)
        sig = to_device(si)
        n = B.kv_evict_step(shape, params, t, n, si["new_pos"], sig["q"], sig["k_new"], sig["v_new"], a["k"],
                            a["v"], a["u"], a["pos"], ws)
        assert B.evict_step(cache, sig["q"], sig["k_new"], sig["v_new"], t, params, si["new_pos"]) == n
        assert cache.n == n <= cfg.budget
        torch.cuda.synchronize()
        for key in ("k", "v", "u", "pos"):
            assert torch.equal(a[key][..., :n] if key in ("u", "pos") else a[key][:, :, :, :n],
                               b[key][..., :n] if key in ("u", "pos") else b[key][:, :, :, :n]), (t, key)
