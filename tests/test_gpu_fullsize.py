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
