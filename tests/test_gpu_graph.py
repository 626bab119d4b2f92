"""Eviction steps captured into a HIP graph (through torch.cuda.CUDAGraph on the caller's stream) and
replayed: every replay from the same starting state must leave exactly the state the eager calls leave.
The launch-bound Lazy / Score-Free steps are what a serving loop would capture.  Replays are interleaved with
eager work and host synchronisation, and every replay is checked (not only the first)."""
import pytest
import torch

from workload import LLAMA8B_LAZY, TINY, Workload

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2609_03515_amd.binding")


def _state(st):
    return {k: v.clone() for k, v in st.items() if isinstance(v, torch.Tensor)}


def _restore(dst, src):
    for k, v in src.items():
        dst[k].copy_(v)


@pytest.mark.parametrize("cfg,period,steps", [(LLAMA8B_LAZY.scaled(batch=2, layers=3, prefill_len=600, budget=60), 4, 8),
                                              (TINY, 1, 4)], ids=["lazy_r4", "tiny_full"])
def test_graph_replay_matches_eager(cfg, period, steps):
    w = Workload(cfg)
    cap = cfg.prefill_len + 1
    st = {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in w.prefill(capacity=cap).items()}
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cap, cfg.dtype)
    params = B.make_params(cfg.alpha, cfg.budget, period, False, cfg.nonrefresh_init, cfg.recency_bias,
                           cfg.recency_window)
    ws = B.workspace(shape, cap)
    ins = [{k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in w.step_inputs(t).items()}
           for t in range(1, steps + 2)]
    # step 1 eagerly (compacts the prefill), then the cycle to capture starts from a steady cache
    n = B.kv_evict_step(shape, params, 1, st["n"], ins[0]["new_pos"], ins[0]["q"], ins[0]["k_new"],
                        ins[0]["v_new"], st["k"], st["v"], st["u"], st["pos"], ws)
    start = _state(st)

    def cycle():
        m = n
        for t in range(2, steps + 2):
            si = ins[t - 1]
            m = B.kv_evict_step(shape, params, t, m, si["new_pos"], si["q"], si["k_new"], si["v_new"], st["k"],
                                st["v"], st["u"], st["pos"], ws)
        return m

    cycle()                              # eager reference (also loads every kernel before capture)
    torch.cuda.synchronize()
    ref = _state(st)
    _restore(st, start)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        cycle()
    for rep in range(3):
        _restore(st, start)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for key in ("k", "v", "u", "pos"):
            assert torch.equal(st[key][..., :n] if key in ("u", "pos") else st[key][..., :n, :],
                               ref[key][..., :n] if key in ("u", "pos") else ref[key][..., :n, :]), (rep, key)
        _ = (st["u"] * 2).sum().item()   # eager work between replays
