"""GPU parity of the rank-trace diagnostics (appendix "Mechanistic Diagnostics") against the oracle.

Both traced top-k decisions are checked like the retention decision (exact size, equal outside the 1e-4
band around the k-th value of the oracle's float64 scores) and then adopted by the oracle; the ten counts
per sequence and step must then be equal exactly (integer set arithmetic on the same sets).  The eviction
itself runs in lockstep as in the step tests."""
import numpy as np
import pytest
import torch

from oracle import RankTraceState, evict_step, rank_trace_counts, select_keep, trace_metrics
from parity import check_keep, lockstep_adopter, oracle_cache, oracle_params, to_device
from workload import LLAMA8B, LLAMA8B_LAZY, TINY, Workload, raw_numpy

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2609_03515_amd.binding")


def run_trace(cfg, steps, k, fused=False, max_pos=None, expect_oob=False):
    w = Workload(cfg)
    cap = max(cfg.prefill_len, cfg.budget) + 1
    st = w.prefill(capacity=cap)
    oc = oracle_cache(st, cfg.dtype)
    dev = to_device(st)
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cap, cfg.dtype)
    params = B.make_params(cfg.alpha, cfg.budget, cfg.refresh_period, cfg.score_free, cfg.nonrefresh_init,
                           cfg.recency_bias, cfg.recency_window)
    op = oracle_params(cfg)
    ws = B.workspace(shape, cap)
    max_pos = max_pos or cfg.prefill_len + steps + 8
    state = torch.zeros(B.kv_rank_trace_state_bytes(cfg.batch, max_pos) // 4, dtype=torch.int32, device="cuda")
    counts = torch.full((cfg.batch, B.KV_TRACE_COUNTS), -7, dtype=torch.int32, device="cuda")
    rk = torch.zeros(cfg.batch, cap, dtype=torch.uint8, device="cuda")
    ek = torch.zeros_like(rk)
    rt = B.make_rank_trace(k, max_pos, state, counts, rk, ek)
    ostate = [RankTraceState() for _ in range(cfg.batch)]
    n = st["n"]
    metrics = []
    for t in range(1, steps + 1):
        si = w.step_inputs(t)
        sig = to_device(si)
        keep = torch.zeros(cfg.batch, cap, dtype=torch.uint8, device="cuda")
        print(f"{cfg.name} t={t} k={k} fused={fused} n_in={n}", flush=True)
        if fused:
            refresh = (t - 1) % cfg.refresh_period == 0 and (not cfg.score_free or t == 1)
            B.kv_append(shape, params, t, n, si["new_pos"], sig["k_new"], sig["v_new"], dev["k"], dev["v"],
                        dev["u"], dev["pos"])
            o = torch.empty_like(sig["q"])
            B.kv_attend_score(shape, 0, cfg.layers, n + 1, sig["q"], dev["k"], dev["v"], dev["pos"], si["new_pos"],
                              cfg.recency_bias, cfg.recency_window, refresh, o, ws)
            n_out = B.kv_evict_finish(shape, params, t, n + 1, dev["k"], dev["v"], dev["u"], dev["pos"], ws,
                                      keep_out=keep, rank_trace=rt)
        else:
            n_out = B.kv_evict_step(shape, params, t, n, si["new_pos"], sig["q"], sig["k_new"], sig["v_new"],
                                    dev["k"], dev["v"], dev["u"], dev["pos"], ws, keep_out=keep, rank_trace=rt)
        torch.cuda.synchronize()
        keep_g = keep.cpu().numpy()[:, : n + 1].astype(bool)
        ref = evict_step(oc, raw_numpy(si["q"]), raw_numpy(si["k_new"]), raw_numpy(si["v_new"]), t, si["new_pos"],
                         op, keep_override=lockstep_adopter(keep_g, cfg.budget, f"{cfg.name} t={t}", []))
        c = counts.cpu().numpy()
        if not ref.refreshed:
            assert np.all(c[:, 0] == 0), c
        elif expect_oob:
            assert np.all(c[:, 0] == -2), c
        else:
            rk_g = rk.cpu().numpy()[:, : n + 1].astype(bool)
            ek_g = ek.cpu().numpy()[:, : n + 1].astype(bool)
            for b in range(cfg.batch):
                what = f"{cfg.name} t={t} b={b}"
                check_keep(rk_g[b], select_keep(ref.raw[b], ref.pos_pre[b], k), ref.raw[b], k, what + " raw top-k")
                check_keep(ek_g[b], select_keep(ref.u_pre[b], ref.pos_pre[b], k), ref.u_pre[b], k,
                           what + " EMA top-k")
                cr = rank_trace_counts(ostate[b], ref.raw[b], ref.u_pre[b], ref.pos_pre[b], ref.keep[b], k,
                                       raw_keep=rk_g[b], ema_keep=ek_g[b])
                want = [1, cr["r"], cr["e"], cr["has_prev"], cr["rr"], cr["ee"], cr["re"], cr["rev"], cr["rp"],
                        cr["ep"]]
                assert list(c[b]) == want, (what, list(c[b]), want)
                metrics.append(trace_metrics(cr))
        n = n_out
    return metrics


CASES = {
    "tiny_kB": (TINY, 8, TINY.budget, False),
    "llama8b_reduced_kB": (LLAMA8B.scaled(batch=2, layers=3, prefill_len=1200, budget=120), 5, 120, False),
    "llama8b_reduced_k30": (LLAMA8B.scaled(batch=2, layers=3, prefill_len=1200, budget=120), 5, 30, False),
    # bitmaps too large for LDS (positions < 300,000): the statistics work on them in global memory
    "lazy_r4_min": (LLAMA8B_LAZY.scaled(batch=2, layers=2, prefill_len=800, budget=80), 9, 80, False),
    "fused_tiny_kB": (TINY, 6, TINY.budget, True),
    "fused_llama8b_reduced_k40": (LLAMA8B.scaled(batch=2, layers=3, prefill_len=1200, budget=120), 4, 40, True),
}


@pytest.mark.parametrize("name", list(CASES))
def test_rank_trace_lockstep(name):
    cfg, steps, k, fused = CASES[name]
    m = run_trace(cfg, steps, k, fused, max_pos=300_000 if name == "lazy_r4_min" else None)
    steady = [x["ema_churn"] for x in m[cfg.batch:]]
    print(f"{name}: EMA churn {np.nanmean(steady):.4g}, raw churn {np.nanmean([x['raw_churn'] for x in m]):.4g}")


def test_rank_trace_positions_out_of_range():
    """A bitmap too small for the positions flags the step instead of writing out of range."""
    run_trace(TINY, 2, TINY.budget, max_pos=100, expect_oob=True)
