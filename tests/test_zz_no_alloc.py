"""kv_evict_step_static (no workspace: the library's static per-device scratch) against kv_evict_step.

Two calls in a row through the C ABI, the second on a smaller input, each compared with kv_evict_step on an
identical copy of the same state: the cache, utilities, positions, retention decision and per-layer scores
must be bit-identical (the same kernels run on the same inputs; only the scratch differs).  The second call
also shows that what the first left in the shared scratch does not leak into its results."""
import pytest
import torch

from workload import LLAMA8B, QWEN, TINY, Workload

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2609_03515_amd.binding")


def _state(cfg, rows):
    w = Workload(cfg, device="cuda")
    st = w.steady_state(rows=rows, capacity=rows + 1)
    return w, st


def _copy(st):
    return {k: (v.clone() if isinstance(v, torch.Tensor) else v) for k, v in st.items()}


def _compare(cfg, w, st, t, params, what, norm_cache=False):
    cap = st["k"].shape[3]
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cap, cfg.dtype)
    si = w.step_inputs(t)
    n_in = st["n"]
    if norm_cache:   # the value-norm cache, filled from the cached rows, is part of the state both sides keep
        st = dict(st, norms=torch.full((cfg.layers, cfg.batch, cfg.n_kv_heads, cap), -1.0, device="cuda"))
        B.kv_value_norms(shape, n_in, st["v"], st["norms"])
    a, b = _copy(st), _copy(st)
    outs = []
    for side, fn in (("workspace", B.kv_evict_step), ("static", B.kv_evict_step_static)):
        d = a if side == "workspace" else b
        keep = torch.full((cfg.batch, cap), 7, dtype=torch.uint8, device="cuda")
        s_out = torch.full((cfg.layers, cfg.batch, n_in + 1), -1.0, device="cuda")
        args = (shape, params, t, n_in, si["new_pos"], si["q"], si["k_new"], si["v_new"], d["k"], d["v"], d["u"],
                d["pos"])
        if side == "workspace":
            n_out = fn(*args, B.workspace(shape, n_in + 1), keep_out=keep, s_out=s_out, v_norms=d.get("norms"))
        else:
            n_out = fn(*args, keep_out=keep, s_out=s_out, v_norms=d.get("norms"))
        torch.cuda.synchronize()
        outs.append((n_out, keep, s_out))
    assert outs[0][0] == outs[1][0] == min(params.budget, n_in + 1), what
    n_out = outs[0][0]
    assert torch.equal(outs[0][1], outs[1][1]), f"{what}: retention decision"
    assert torch.equal(outs[0][2], outs[1][2]), f"{what}: per-layer scores"
    assert torch.equal(a["u"][:, :n_out], b["u"][:, :n_out]), f"{what}: utilities"
    assert torch.equal(a["pos"][:, :n_out], b["pos"][:, :n_out]), f"{what}: positions"
    assert torch.equal(a["k"][:, :, :, :n_out], b["k"][:, :, :, :n_out]), f"{what}: keys"
    assert torch.equal(a["v"][:, :, :, :n_out], b["v"][:, :, :, :n_out]), f"{what}: values"
    if norm_cache:
        assert torch.equal(a["norms"][..., :n_out], b["norms"][..., :n_out]), f"{what}: value norms"


def test_static_scratch_matches_workspace_variant_on_two_calls():
    # call 1: the 8B-shaped steady full-refresh step (batch 8, 32 layers, B + 1 = 3,278 tokens scored)
    cfg = LLAMA8B
    w, st = _state(cfg, cfg.budget)
    p = B.make_params(cfg.alpha, cfg.budget, 1, False, "mean", cfg.recency_bias, cfg.recency_window)
    print("no-alloc call 1: 8B steady step, batch 8, n = 3,278", flush=True)
    _compare(cfg, w, st, 2, p, "8B steady step")
    del w, st
    torch.cuda.empty_cache()
    # call 2, smaller: a Qwen-shaped cache of 500 tokens at batch 4 (one eviction, GQA 7, no recency bias)
    cfg = QWEN.scaled(batch=4, budget=500)
    w, st = _state(cfg, 500)
    p = B.make_params(cfg.alpha, cfg.budget)
    print("no-alloc call 2: Qwen-shaped steady step, batch 4, n = 501", flush=True)
    _compare(cfg, w, st, 2, p, "Qwen-shaped small step")


def test_static_scratch_other_step_kinds():
    """A non-refresh step (Lazy, mean prior), a VNorm refresh step, and the Tiny first step (select + move)."""
    cfg = LLAMA8B.scaled(batch=2, layers=4)
    w, st = _state(cfg, cfg.budget)
    lazy = B.make_params(cfg.alpha, cfg.budget, 4, False, "mean", cfg.recency_bias, cfg.recency_window)
    print("no-alloc: Lazy non-refresh step", flush=True)
    _compare(cfg, w, st, 3, lazy, "non-refresh step")
    vn = B.make_params(cfg.alpha, cfg.budget, 1, False, "mean", cfg.recency_bias, cfg.recency_window, vnorm=True,
                       entropy=True)
    print("no-alloc: VNorm + entropy refresh step", flush=True)
    _compare(cfg, w, st, 2, vn, "VNorm + entropy step")
    print("no-alloc: VNorm + entropy refresh step from the value-norm cache", flush=True)
    _compare(cfg, w, st, 2, vn, "VNorm step, norm cache", norm_cache=True)
    cfg = TINY
    w = Workload(cfg, device="cuda")
    st = w.prefill()
    print("no-alloc: Tiny first step", flush=True)
    _compare(cfg, w, st, 1, B.make_params(cfg.alpha, cfg.budget), "Tiny first step")
