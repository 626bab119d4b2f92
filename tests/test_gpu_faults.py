"""The long-slab scorer's bounded wait reports a give-up instead of folding an incomplete softmax.

Slabs too long for one workgroup's LDS are scored in chunks that exchange their per-head (max, sum) pairs and
wait, for a bounded time, for their peers' words.  A chunk that gives up must leave a visible trace: NaN
scores and the workspace's sticky fault word.  The give-up is forced from the host with a wait limit of 0
(no chunk polls, so none waits: every kernel runs to its end), then the default limit is restored and the
same call must again match the float64 oracle with a clear fault word."""
import numpy as np
import pytest
import torch

from oracle import Cache, Params, evict_step, fold_layers, layer_scores, to_f64
from parity import assert_close, lockstep_adopter
from workload import TINY, Workload, raw_numpy

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2609_03515_amd.binding")


def _case(n=20001, batch=2, layers=2, hq=16, hkv=4):
    cfg = TINY.scaled(name="fault", batch=batch, layers=layers, n_q_heads=hq, n_kv_heads=hkv, head_dim=128,
                      dtype="bf16", prefill_len=n, budget=n // 10, heavy_frac=0.02, recency_bias=0.5,
                      recency_window=64)
    w = Workload(cfg, seed=4242)
    st = w.prefill()
    shape = B.make_shape(batch, layers, hq, hkv, 128, cfg.capacity, "bf16")
    return cfg, w, st, shape


class _WaitLimit:
    """Sets the exchange wait limit for a block and restores the default afterwards, even on failure."""

    def __init__(self, polls):
        self.polls = polls

    def __enter__(self):
        B.kv_set_exchange_wait_limit(self.polls)

    def __exit__(self, *exc):
        B.kv_set_exchange_wait_limit(-1)
        return False


def test_exchange_give_up_is_reported_by_kv_score_ema():
    cfg, w, st, shape = _case()
    n = st["n"]
    p = B.make_params(0.9, cfg.budget)
    info = B.kv_score_plan(shape, n, p)
    # chunks in teams that add the group sums of the 4 KV heads: one give-up poisons the team's whole row
    assert (info.path, info.merge) == (B.KV_PATH_EXCHANGE, 4) and info.chunks > 1, (info.path, info.chunks)
    print(f"fault case: n={n}, {info.chunks} chunks per slab, teams of {info.merge} KV heads", flush=True)
    ws = B.workspace(shape, n)
    si = w.step_inputs(1)
    q, k, pos = si["q"].cuda(), st["k"].cuda(), st["pos"].cuda()
    cur = si["new_pos"]

    def score(u, s_out):
        B.kv_score_ema(shape, n, q, k, pos, cur, 0.9, cfg.recency_bias, cfg.recency_window, u, s_out, ws)
        torch.cuda.synchronize()

    # forced give-up: every chunk reports, and its scores are NaN rather than a partial softmax
    u_bad = torch.zeros(cfg.batch, cfg.capacity, device="cuda")
    s_bad = torch.zeros((cfg.layers, cfg.batch, n), device="cuda")
    with _WaitLimit(0):
        score(u_bad, s_bad)
    assert B.faults(ws) == B.KV_FAULT_EXCHANGE_TIMEOUT
    assert torch.isnan(s_bad).all(), "a chunk that gave up must not leave plausible scores"
    assert torch.isnan(u_bad[:, :n]).all()

    # the word is sticky: a later good call does not clear it
    u_ok = torch.zeros(cfg.batch, cfg.capacity, device="cuda")
    s_ok = torch.full((cfg.layers, cfg.batch, n), -1.0, device="cuda")
    score(u_ok, s_ok)
    assert B.faults(ws, clear=True) == B.KV_FAULT_EXCHANGE_TIMEOUT
    assert B.faults(ws) == 0

    # with the default limit the call matches the oracle and raises nothing
    score(u_ok.zero_(), s_ok)
    assert B.faults(ws) == 0
    k_raw, q_raw, pos_np = raw_numpy(st["k"]), raw_numpy(si["q"]), st["pos"].numpy()
    for b in range(cfg.batch):
        s_ref = np.stack([layer_scores(to_f64(q_raw[l, b], "bf16"), to_f64(k_raw[l, b, :, :n], "bf16"),
                                       pos_np[b, :n], cur, cfg.recency_bias, cfg.recency_window)
                          for l in range(cfg.layers)])
        assert_close(s_ok[:, b].cpu().numpy(), s_ref, f"seq {b} scores")
        assert_close(u_ok[b, :n].cpu().numpy(), fold_layers(np.zeros(n), s_ref, 0.9), f"seq {b} utilities")


def test_exchange_give_up_is_reported_by_the_first_step():
    cfg, w, st, shape = _case(batch=1)
    n_in = st["n"]
    p = B.make_params(cfg.alpha, cfg.budget, recency_bias=cfg.recency_bias, recency_window=cfg.recency_window)
    assert B.kv_score_plan(shape, n_in + 1, p).path == B.KV_PATH_EXCHANGE
    si = {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in w.step_inputs(1).items()}

    def first_step(polls):
        dev = {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in st.items()}
        ws = B.workspace(shape, cfg.capacity)
        keep = torch.zeros(cfg.batch, cfg.capacity, dtype=torch.uint8, device="cuda")
        with _WaitLimit(polls):
            n_out = B.kv_evict_step(shape, p, 1, n_in, si["new_pos"], si["q"], si["k_new"], si["v_new"], dev["k"],
                                    dev["v"], dev["u"], dev["pos"], ws, keep_out=keep)
        torch.cuda.synchronize()
        return dev, keep, n_out, B.faults(ws)

    _, _, n_out, fault = first_step(0)
    assert n_out == cfg.budget
    assert fault == B.KV_FAULT_EXCHANGE_TIMEOUT, "the step's invalid scores must be reported"

    dev, keep, n_out, fault = first_step(-1)
    assert fault == 0
    oc = Cache(raw_numpy(st["k"]), raw_numpy(st["v"]), st["u"].numpy().astype(np.float64),
               st["pos"].numpy().astype(np.int64), n_in, "bf16")
    op = Params(alpha=cfg.alpha, budget=cfg.budget, recency_bias=cfg.recency_bias, recency_window=cfg.recency_window)
    cpu_in = w.step_inputs(1)
    ref = evict_step(oc, raw_numpy(cpu_in["q"]), raw_numpy(cpu_in["k_new"]), raw_numpy(cpu_in["v_new"]), 1,
                     si["new_pos"], op,
                     keep_override=lockstep_adopter(keep.cpu().numpy().astype(bool), cfg.budget, "first step", []))
    assert_close(dev["u"][:, :n_out].cpu().numpy(), oc.u[:, :n_out], "utilities after the first step")
    np.testing.assert_array_equal(raw_numpy(dev["k"])[:, :, :, :n_out], oc.k[:, :, :, :n_out])
    assert ref.n_out == n_out
