"""Kernels write only inside the buffers they are given.

Every device buffer a call receives — the K and V caches, u, pos, the retention mask, the per-layer scores,
the step's inputs (q, k_new, v_new), the attention output, the rank trace's state, counts and masks, and the
workspace — sits between two 4 KiB guard bands filled with a byte pattern.  At the 8B / 32k shape the test
runs the path's step kinds one after another on the same cache (decode step 1 over 32,769 tokens with the
chunk-exchange scorer, the multi-workgroup selection and the row moves; a steady refresh step; non-refresh
steps under both priors; a decode step around per-layer attention calls; a VNorm + entropy + rank-traced step;
the separate entry points) and checks after each call that every guard still holds its pattern."""
import math

import pytest
import torch

from workload import LLAMA8B, Workload

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2609_03515_amd.binding")

GUARD = 4096  # bytes on each side (keeps the 256-byte alignment of the buffer between them)


class Guarded:
    """A device buffer of `shape` between two patterned guard bands."""

    registry = []

    def __init__(self, name, shape, dtype):
        self.name = name
        nbytes = math.prod(shape) * torch.tensor([], dtype=dtype).element_size()
        self.raw = torch.empty(GUARD + nbytes + GUARD, dtype=torch.uint8, device="cuda")
        self.pattern = (torch.arange(GUARD, device="cuda") * 37 + len(name)) % 251
        self.pattern = self.pattern.to(torch.uint8)
        self.raw[:GUARD] = self.pattern
        self.raw[GUARD + nbytes:] = self.pattern
        self.t = self.raw[GUARD:GUARD + nbytes].view(dtype).view(shape)
        Guarded.registry.append(self)

    def intact(self):
        return bool(torch.equal(self.raw[:GUARD], self.pattern) and torch.equal(self.raw[-GUARD:], self.pattern))


def check_guards(after):
    torch.cuda.synchronize()
    bad = [g.name for g in Guarded.registry if not g.intact()]
    assert not bad, f"after {after}: guard bands overwritten around {bad}"
    print(f"guards intact after {after}", flush=True)


def test_guard_bands_untouched_at_full_size():
    Guarded.registry = []
    cfg = LLAMA8B
    cap, L, b, hq, hkv, d = cfg.capacity, cfg.layers, cfg.batch, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    bf = torch.bfloat16
    w = Workload(cfg, device="cuda")
    st = w.prefill()
    k = Guarded("k", (L, b, hkv, cap, d), bf)
    v = Guarded("v", (L, b, hkv, cap, d), bf)
    k.t.copy_(st["k"])
    v.t.copy_(st["v"])
    del st["k"], st["v"]
    torch.cuda.empty_cache()
    u = Guarded("u", (b, cap), torch.float32)
    pos = Guarded("pos", (b, cap), torch.int32)
    u.t.copy_(st["u"])
    pos.t.copy_(st["pos"])
    keep = Guarded("keep", (b, cap), torch.uint8)
    q = Guarded("q", (L, b, hq, d), bf)
    k_new = Guarded("k_new", (L, b, hkv, d), bf)
    v_new = Guarded("v_new", (L, b, hkv, d), bf)
    o = Guarded("o", (L, b, hq, d), bf)
    shape = B.make_shape(b, L, hq, hkv, d, cap, cfg.dtype)
    ws = Guarded("workspace", (B.kv_workspace_bytes(shape, cap),), torch.uint8)
    B.kv_fault_status(ws.t, None, clear=True)
    check_guards("set-up")
    n = st["n"]

    def inputs(t):
        si = w.step_inputs(t)
        q.t.copy_(si["q"])
        k_new.t.copy_(si["k_new"])
        v_new.t.copy_(si["v_new"])
        return si["new_pos"]

    def params(R=1, init="mean", **kw):
        return B.make_params(cfg.alpha, cfg.budget, R, False, init, cfg.recency_bias, cfg.recency_window, **kw)

    def step(t, p, **kw):
        nonlocal n
        new_pos = inputs(t)
        s_out = Guarded(f"s_out t={t}", (L, b, n + 1), torch.float32)   # [layers][batch][n] for this n
        n = B.kv_evict_step(shape, p, t, n, new_pos, q.t, k_new.t, v_new.t, k.t, v.t, u.t, pos.t, ws.t,
                            keep_out=keep.t, s_out=s_out.t, rank_trace=kw.get("rank_trace"))

    step(1, params())
    assert n == cfg.budget
    check_guards("decode step 1 over 32,769 tokens")
    step(2, params())
    check_guards("a steady refresh step")
    step(3, params(4, "mean"))
    check_guards("a non-refresh step, mean prior")
    step(4, params(4, "min"))
    check_guards("a non-refresh step, min prior")

    # decode step around the model's attention: append, one attention call per layer, finish
    t = 5
    p = params(4, "mean")
    new_pos = inputs(t)
    B.kv_append(shape, p, t, n, new_pos, k_new.t, v_new.t, k.t, v.t, u.t, pos.t)
    for l in range(L):
        B.kv_attend_score(shape, l, 1, n + 1, q.t[l], k.t, v.t, pos.t, new_pos, cfg.recency_bias,
                          cfg.recency_window, B.KV_EMIT_SCORES, o.t[l], ws.t)
    n = B.kv_evict_finish(shape, p, t, n + 1, k.t, v.t, u.t, pos.t, ws.t, keep_out=keep.t)
    check_guards("a fused decode step (per-layer attention)")

    max_pos = cfg.prefill_len + 64
    tstate = Guarded("trace_state", (B.kv_rank_trace_state_bytes(b, max_pos) // 4,), torch.int32)
    tstate.t.zero_()
    counts = Guarded("trace_counts", (b, B.KV_TRACE_COUNTS), torch.int32)
    raw_keep = Guarded("raw_keep", (b, cap), torch.uint8)
    ema_keep = Guarded("ema_keep", (b, cap), torch.uint8)
    rt = B.make_rank_trace(40, max_pos, tstate.t, counts.t, raw_keep=raw_keep.t, ema_keep=ema_keep.t)
    step(6, params(vnorm=True, entropy=True), rank_trace=rt)
    check_guards("a VNorm + entropy step with a rank trace (k = 40)")

    # the separate entry points on the same buffers
    new_pos = inputs(7)
    s_out = Guarded("s_out kv_score_ema", (L, b, n), torch.float32)
    B.kv_score_ema(shape, n, q.t, k.t, pos.t, new_pos, cfg.alpha, cfg.recency_bias, cfg.recency_window, u.t,
                   s_out.t, ws.t)
    B.kv_topk_select(shape, n, cfg.budget - 7, u.t, pos.t, keep.t, ws.t)
    B.kv_compact(shape, n, cfg.budget - 7, keep.t, k.t, v.t, u.t, pos.t, ws.t)
    check_guards("kv_score_ema, kv_topk_select and kv_compact")
    assert B.faults(ws.t) == 0
