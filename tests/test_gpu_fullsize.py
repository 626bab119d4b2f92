"""GPU parity at the workloads' full sizes, in the launch configuration the benchmark times.

The GPU runs every sequence of the batch; the float64 oracle follows sampled sequences one by one (sequences
are independent, so each sampled sequence is checked exactly as if it were alone).  Per step and sampled
sequence: per-layer scores and compacted utilities within 1e-3 relative, retention sets equal outside the
1e-4 band (lockstep adoption inside it), positions and compacted K/V rows bit-exact."""
import gc

import numpy as np
import pytest
import torch

from oracle import Cache, evict_step
from parity import assert_close, lockstep_adopter, oracle_params
from workload import LLAMA8B, QWEN, SCOREFREE128K, Workload, raw_numpy

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2609_03515_amd.binding")


def _oracle_seq(st, b, dtype):
    return Cache(raw_numpy(st["k"][:, b:b + 1]), raw_numpy(st["v"][:, b:b + 1]),
                 st["u"][b:b + 1].cpu().numpy().astype(np.float64),
                 st["pos"][b:b + 1].cpu().numpy().astype(np.int64), st["n"], dtype)


def run_sampled(cfg, plan, samples):
    """plan: list of (t, overrides of the workload's schedule)."""
    w = Workload(cfg, device="cuda")
    st = w.prefill()
    cap = cfg.capacity
    oc = {b: _oracle_seq(st, b, cfg.dtype) for b in samples}
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cap, cfg.dtype)
    ws = B.workspace(shape, cap)
    n = st["n"]
    flips = 0
    for t, over in plan:
        sched = dict(refresh_period=cfg.refresh_period, score_free=cfg.score_free,
                     nonrefresh_init=cfg.nonrefresh_init)
        sched.update(over)
        params = B.make_params(cfg.alpha, cfg.budget, sched["refresh_period"], sched["score_free"],
                               sched["nonrefresh_init"], cfg.recency_bias, cfg.recency_window)
        op = oracle_params(cfg, **sched)
        si = w.step_inputs(t)
        keep = torch.zeros(cfg.batch, cap, dtype=torch.uint8, device="cuda")
        s_out = torch.empty((cfg.layers, cfg.batch, n + 1), device="cuda")
        print(f"{cfg.name} t={t} {sched} n_in={n}", flush=True)
        n_out = B.kv_evict_step(shape, params, t, n, si["new_pos"], si["q"], si["k_new"], si["v_new"],
                                st["k"], st["v"], st["u"], st["pos"], ws, keep_out=keep, s_out=s_out)
        torch.cuda.synchronize()
        assert n_out == min(cfg.budget, n + 1)
        for b in samples:
            keep_g = keep[b:b + 1, : n + 1].cpu().numpy().astype(bool)
            step_flips = []
            ref = evict_step(oc[b], raw_numpy(si["q"][:, b:b + 1]), raw_numpy(si["k_new"][:, b:b + 1]),
                             raw_numpy(si["v_new"][:, b:b + 1]), t, si["new_pos"], op,
                             keep_override=lockstep_adopter(keep_g, cfg.budget, f"{cfg.name} t={t} seq {b}",
                                                            step_flips))
            flips += sum(step_flips)
            if ref.refreshed:
                assert_close(s_out[:, b].cpu().numpy(), ref.s_layers[:, 0], f"{cfg.name} t={t} seq {b} scores")
            assert_close(st["u"][b, :n_out].cpu().numpy(), oc[b].u[0, :n_out], f"{cfg.name} t={t} seq {b} u")
            np.testing.assert_array_equal(st["pos"][b, :n_out].cpu().numpy(), oc[b].pos[0, :n_out])
            np.testing.assert_array_equal(raw_numpy(st["k"][:, b, :, :n_out]), oc[b].k[:, 0, :, :n_out])
            np.testing.assert_array_equal(raw_numpy(st["v"][:, b, :, :n_out]), oc[b].v[:, 0, :, :n_out])
        n = n_out
        print(f"{cfg.name} t={t} ok, n={n}, in-band flips so far {flips}", flush=True)
    del st, ws
    gc.collect()
    torch.cuda.empty_cache()
    return flips


def test_llama8b_32k_full_refresh_then_lazy():
    """First step over all 32,769 tokens (split scorer, ~2,950 moved rows per slab), two steady full-refresh
    steps (the benchmarked step), then Lazy R = 4 with the min prior: non-refresh steps 4, 6-8 and refresh
    steps 5 and 9."""
    plan = [(1, {}), (2, {}), (3, {})] + [(t, dict(refresh_period=4, nonrefresh_init="min")) for t in range(4, 10)]
    run_sampled(LLAMA8B, plan, samples=(0, 7))


def test_scorefree_128k():
    """Score-Free at 131,073 scored tokens, then append-and-evict steps on the frozen ranking (min prior)."""
    plan = [(t, {}) for t in range(1, 6)]
    run_sampled(SCOREFREE128K, plan, samples=(1,))


def test_qwen_8k():
    """Qwen-style GQA 7 with Student-t keys: first step (split scorer), then steady full-refresh steps."""
    plan = [(t, {}) for t in range(1, 4)]
    run_sampled(QWEN, plan, samples=(0, 31))


def test_llama8b_32k_next_rows_full_size():
    """The rows the benchmark times beyond the headline, at the 8B / 32k shape on sampled sequences: step 1,
    then fused decode steps (attention per layer, then in one call; outputs against the oracle's attention),
    a VNorm + entropy step and a rank-traced step (k = B)."""
    from oracle import RankTraceState, rank_trace_counts, select_keep
    from parity import assert_o, check_keep

    cfg = LLAMA8B
    samples = (0, 7)
    w = Workload(cfg, device="cuda")
    st = w.prefill()
    cap = cfg.capacity
    oc = {b: _oracle_seq(st, b, cfg.dtype) for b in samples}
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cap, cfg.dtype)
    ws = B.workspace(shape, cap)
    max_pos = cfg.prefill_len + 16
    tstate = torch.zeros(B.kv_rank_trace_state_bytes(cfg.batch, max_pos) // 4, dtype=torch.int32, device="cuda")
    counts = torch.zeros(cfg.batch, B.KV_TRACE_COUNTS, dtype=torch.int32, device="cuda")
    rk = torch.zeros(cfg.batch, cap, dtype=torch.uint8, device="cuda")
    rt = B.make_rank_trace(cfg.budget, max_pos, tstate, counts, raw_keep=rk)
    ostate = {b: RankTraceState() for b in samples}
    n = st["n"]
    plan = [(1, "step", {}), (2, "fused_per_layer", {}), (3, "fused_all", {}),
            (4, "step", dict(vnorm=True, entropy=True)), (5, "traced", {}), (6, "traced", {})]
    for t, mode, var in plan:
        params = B.make_params(cfg.alpha, cfg.budget, 1, False, "mean", cfg.recency_bias, cfg.recency_window, **var)
        op = oracle_params(cfg, refresh_period=1, score_free=False, nonrefresh_init="mean", **var)
        si = w.step_inputs(t)
        keep = torch.zeros(cfg.batch, cap, dtype=torch.uint8, device="cuda")
        s_out = torch.empty((cfg.layers, cfg.batch, n + 1), device="cuda")
        o = None
        print(f"8B next rows t={t} {mode} {var} n_in={n}", flush=True)
        if mode.startswith("fused"):
            B.kv_append(shape, params, t, n, si["new_pos"], si["k_new"], si["v_new"], st["k"], st["v"], st["u"],
                        st["pos"])
            o = torch.empty_like(si["q"])
            if mode == "fused_per_layer":
                for l in range(cfg.layers):
                    B.kv_attend_score(shape, l, 1, n + 1, si["q"][l], st["k"], st["v"], st["pos"], si["new_pos"],
                                      cfg.recency_bias, cfg.recency_window, 1, o[l], ws)
            else:
                B.kv_attend_score(shape, 0, cfg.layers, n + 1, si["q"], st["k"], st["v"], st["pos"], si["new_pos"],
                                  cfg.recency_bias, cfg.recency_window, 1, o, ws)
            n_out = B.kv_evict_finish(shape, params, t, n + 1, st["k"], st["v"], st["u"], st["pos"], ws,
                                      keep_out=keep, s_out=s_out)
        else:
            n_out = B.kv_evict_step(shape, params, t, n, si["new_pos"], si["q"], si["k_new"], si["v_new"], st["k"],
                                    st["v"], st["u"], st["pos"], ws, keep_out=keep, s_out=s_out,
                                    rank_trace=rt if mode == "traced" else None)
        torch.cuda.synchronize()
        assert n_out == min(cfg.budget, n + 1)
        c = counts.cpu().numpy()
        for b in samples:
            keep_g = keep[b:b + 1, : n + 1].cpu().numpy().astype(bool)
            ref = evict_step(oc[b], raw_numpy(si["q"][:, b:b + 1]), raw_numpy(si["k_new"][:, b:b + 1]),
                             raw_numpy(si["v_new"][:, b:b + 1]), t, si["new_pos"], op,
                             keep_override=lockstep_adopter(keep_g, cfg.budget, f"t={t} seq {b}", []),
                             attention=o is not None)
            what = f"8B t={t} {mode} seq {b}"
            if o is not None:
                assert_o(o[:, b:b + 1], ref.o, ref.o_scale, cfg.dtype, what + " attention")
            assert_close(s_out[:, b].cpu().numpy(), ref.s_layers[:, 0], what + " scores")
            assert_close(st["u"][b, :n_out].cpu().numpy(), oc[b].u[0, :n_out], what + " u")
            np.testing.assert_array_equal(st["pos"][b, :n_out].cpu().numpy(), oc[b].pos[0, :n_out])
            np.testing.assert_array_equal(raw_numpy(st["k"][:, b, :, :n_out]), oc[b].k[:, 0, :, :n_out])
            np.testing.assert_array_equal(raw_numpy(st["v"][:, b, :, :n_out]), oc[b].v[:, 0, :, :n_out])
            if mode == "traced":
                rk_g = rk[b, : n + 1].cpu().numpy().astype(bool)
                check_keep(rk_g, select_keep(ref.raw[0], ref.pos_pre[0], cfg.budget), ref.raw[0], cfg.budget,
                           what + " raw top-k")
                cr = rank_trace_counts(ostate[b], ref.raw[0], ref.u_pre[0], ref.pos_pre[0], ref.keep[0], cfg.budget,
                                       raw_keep=rk_g, ema_keep=ref.keep[0])
                assert list(c[b]) == [1, cr["r"], cr["e"], cr["has_prev"], cr["rr"], cr["ee"], cr["re"], cr["rev"],
                                      cr["rp"], cr["ep"]], (what, list(c[b]))
        n = n_out
        print(f"8B next rows t={t} ok", flush=True)
    del st, ws
    gc.collect()
    torch.cuda.empty_cache()
