"""GPU parity of the fused decode attention + score path (kv_append, kv_attend_score, kv_evict_finish).

The attention output of every layer, sequence and query head is compared with the oracle's float64
attention: |o_gpu - o_ref| <= 1e-3 * sum_i a(i) |v(i)| (the scale of the weighted sum, which bounds its
rounding; 1e-3 is the probability tolerance of the scores) + 2^-8 |o_ref| when the output is rounded to bf16.
The scores, utilities, retention sets and compacted rows follow the same rules as the separate-pass step
(scores/utilities 1e-3 relative, retention equal outside the 1e-4 band with lockstep adoption, positions and
K/V rows bit-exact)."""
import zlib

import numpy as np
import pytest
import torch

from oracle import attention_output, evict_step, layer_scores, refresh_due, to_f64
from parity import assert_close, assert_o, check_norm_cache, lockstep_adopter, oracle_cache, oracle_params, to_device
from workload import LLAMA8B, LLAMA8B_LAZY, QWEN, TINY, Workload, raw_numpy

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2609_03515_amd.binding")

def attend_layers(shape, cfg, n, q, k, v, pos, cur_pos, emit, ws, per_layer):
    o = torch.empty_like(q)
    if per_layer:
        for l in range(cfg.layers):
            B.kv_attend_score(shape, l, 1, n, q[l], k, v, pos, cur_pos, cfg.recency_bias, cfg.recency_window,
                              emit, o[l], ws)
    else:
        B.kv_attend_score(shape, 0, cfg.layers, n, q, k, v, pos, cur_pos, cfg.recency_bias, cfg.recency_window,
                          emit, o, ws)
    return o


def run_fused_lockstep(cfg, steps, per_layer, vnorm=False, entropy=False, emit_norms=False, merge=0,
                       norm_cache=False):
    w = Workload(cfg)
    cap = max(cfg.prefill_len, cfg.budget) + 1
    st = w.prefill(capacity=cap)
    oc = oracle_cache(st, cfg.dtype)
    dev = to_device(st)
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cap, cfg.dtype)
    params = B.make_params(cfg.alpha, cfg.budget, cfg.refresh_period, cfg.score_free, cfg.nonrefresh_init,
                           cfg.recency_bias, cfg.recency_window, vnorm=vnorm, entropy=entropy,
                           norms_emitted=emit_norms, score_merge=merge)
    op = oracle_params(cfg, vnorm=vnorm, entropy=entropy)
    ws = B.workspace(shape, cap)
    n = st["n"]
    norms = None
    if norm_cache:
        norms = torch.full((cfg.layers, cfg.batch, cfg.n_kv_heads, cap), -1.0, device="cuda")
        B.kv_value_norms(shape, n, dev["v"], norms)
    flips = 0
    for t in range(1, steps + 1):
        si = w.step_inputs(t)
        sig = to_device(si)
        refresh = refresh_due(t, cfg.refresh_period, cfg.score_free)
        print(f"{cfg.name} t={t} refresh={refresh} per_layer={per_layer} n_in={n}", flush=True)
        B.kv_append(shape, params, t, n, si["new_pos"], sig["k_new"], sig["v_new"], dev["k"], dev["v"], dev["u"],
                    dev["pos"], v_norms=norms)
        emit = (B.KV_EMIT_SCORES | (B.KV_EMIT_VNORMS if emit_norms else 0)) if refresh else 0
        o = attend_layers(shape, cfg, n + 1, sig["q"], dev["k"], dev["v"], dev["pos"], si["new_pos"], emit, ws,
                          per_layer)
        keep = torch.zeros(cfg.batch, cap, dtype=torch.uint8, device="cuda")
        s_out = torch.full((cfg.layers, cfg.batch, n + 1), -1.0, device="cuda")
        n_out = B.kv_evict_finish(shape, params, t, n + 1, dev["k"], dev["v"], dev["u"], dev["pos"], ws,
                                  keep_out=keep, s_out=s_out, v_norms=norms)
        torch.cuda.synchronize()
        keep_g = keep.cpu().numpy()[:, : n + 1].astype(bool)
        step_flips = []
        ref = evict_step(oc, raw_numpy(si["q"]), raw_numpy(si["k_new"]), raw_numpy(si["v_new"]), t, si["new_pos"],
                         op, keep_override=lockstep_adopter(keep_g, cfg.budget, f"{cfg.name} t={t}", step_flips),
                         attention=True)
        assert n_out == ref.n_out == min(cfg.budget, n + 1)
        flips += sum(step_flips)
        assert_o(o, ref.o, ref.o_scale, cfg.dtype, f"{cfg.name} t={t} attention")
        if ref.refreshed:
            assert_close(s_out.cpu().numpy(), ref.s_layers, f"{cfg.name} t={t} scores")
        n = n_out
        assert_close(dev["u"][:, :n].cpu().numpy(), oc.u[:, :n], f"{cfg.name} t={t} utilities")
        np.testing.assert_array_equal(dev["pos"][:, :n].cpu().numpy(), oc.pos[:, :n])
        np.testing.assert_array_equal(raw_numpy(dev["k"])[:, :, :, :n], oc.k[:, :, :, :n])
        np.testing.assert_array_equal(raw_numpy(dev["v"])[:, :, :, :n], oc.v[:, :, :, :n])
        if norms is not None:
            check_norm_cache(B, shape, dev["v"], norms, n, oc.v, cfg.dtype, f"{cfg.name} t={t}")
    return flips


CASES = {
    "tiny": (TINY, 6),
    "llama8b_reduced": (LLAMA8B.scaled(batch=2, layers=3, prefill_len=1200, budget=120), 4),
    "llama8b_split_step1": (LLAMA8B.scaled(batch=1, layers=2, prefill_len=6000, budget=600), 2),
    "lazy_r4_min": (LLAMA8B_LAZY.scaled(batch=2, layers=2, prefill_len=800, budget=80), 6),
    "qwen_reduced": (QWEN.scaled(batch=2, layers=2, prefill_len=1000, budget=250), 3),
}


@pytest.mark.parametrize("per_layer", [True, False], ids=["per_layer", "all_layers"])
@pytest.mark.parametrize("name", list(CASES))
def test_fused_step_lockstep(name, per_layer):
    cfg, steps = CASES[name]
    flips = run_fused_lockstep(cfg, steps, per_layer)
    print(f"{name}: in-band flips {flips}")


@pytest.mark.parametrize("emit_norms", [False, True], ids=["norms_from_v", "norms_emitted"])
@pytest.mark.parametrize("name", ["tiny", "llama8b_reduced", "llama8b_split_step1", "qwen_reduced"])
def test_fused_step_scorer_variants(name, emit_norms):
    """VNorm + entropy weighting on the fused path: the perturbations are applied by kv_evict_finish to the
    scores the attention emitted, with the value norms either read from V by the finish or emitted by the
    attention's V pass (one and several chunks per slab)."""
    cfg, steps = CASES[name]
    run_fused_lockstep(cfg, steps, per_layer=True, vnorm=True, entropy=True, emit_norms=emit_norms)
    if emit_norms:
        run_fused_lockstep(cfg, 2, per_layer=False, vnorm=True, entropy=False, emit_norms=True)


@pytest.mark.parametrize("per_layer", [True, False], ids=["per_layer", "all_layers"])
@pytest.mark.parametrize("name", ["tiny", "llama8b_reduced", "llama8b_split_step1", "lazy_r4_min", "qwen_reduced"])
def test_fused_step_value_norm_cache(name, per_layer):
    """VNorm + entropy on the fused path with the value-norm cache: kv_append caches the newcomer's norm, the
    finish reads the cached norms (neither the attention nor the finish reads V for them) and keeps the cache
    through the placement and the compaction."""
    cfg, steps = CASES[name]
    run_fused_lockstep(cfg, steps, per_layer, vnorm=True, entropy=True, norm_cache=True)


@pytest.mark.parametrize("name,merge", [("llama8b_reduced", 4), ("llama8b_split_step1", 8), ("qwen_reduced", 2)])
def test_fused_step_merged_fold(name, merge):
    """The finish folds the attention's per-KV-head scores in the blocks a merging scorer would add (one and
    several chunks per slab)."""
    cfg, steps = CASES[name]
    run_fused_lockstep(cfg, steps, per_layer=True, entropy=True, merge=merge)


# ---- one call on random inputs over the supported geometries -------------------------------------------
GEOMS = [  # (dtype, head_dim, n_q, n_kv, n)
    ("bf16", 128, 32, 8, 1), ("bf16", 128, 32, 8, 15), ("bf16", 128, 32, 8, 256), ("bf16", 128, 32, 8, 257),
    ("bf16", 128, 32, 8, 3278), ("bf16", 128, 8, 8, 700), ("bf16", 128, 16, 8, 700), ("bf16", 128, 28, 4, 2049),
    ("bf16", 128, 16, 2, 300), ("bf16", 128, 16, 1, 520), ("bf16", 64, 8, 8, 333), ("bf16", 64, 16, 4, 1000),
    ("bf16", 64, 16, 2, 999), ("f32", 64, 4, 2, 513), ("f32", 128, 4, 4, 600), ("f32", 128, 8, 2, 1025),
    ("f32", 64, 16, 1, 200), ("bf16", 128, 32, 8, 5200),  # LDS limit: more than 5120 rows per chunk
    ("bf16", 128, 10, 2, 701), ("bf16", 128, 24, 2, 611), ("bf16", 64, 12, 2, 803),  # groups 5, 12, 6
]


@pytest.mark.parametrize("dtype,d,hq,hkv,n", GEOMS)
def test_attend_geometries(dtype, d, hq, hkv, n):
    L, b = 2, 2
    gen = torch.Generator(device="cpu").manual_seed(zlib.crc32(repr((dtype, d, hq, hkv, n)).encode()))
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    cap = n + 3
    k = (torch.randn(L, b, hkv, cap, d, generator=gen) * 1.5).to(tdt)
    v = torch.randn(L, b, hkv, cap, d, generator=gen).to(tdt)
    q = torch.randn(L, b, hq, d, generator=gen).to(tdt)
    pos = torch.randperm(4 * cap, generator=gen)[:cap].to(torch.int32).repeat(b, 1).contiguous()
    cur = int(pos[0, :n].max())
    bias, window = 0.5, 64
    shape = B.make_shape(b, L, hq, hkv, d, cap, dtype)
    ws = B.workspace(shape, n)
    dk, dv, dq, dpos = k.cuda(), v.cuda(), q.cuda(), pos.cuda()
    print(f"attend {dtype} d={d} hq={hq} hkv={hkv} n={n}", flush=True)
    o_all = torch.empty_like(dq)
    B.kv_attend_score(shape, 0, L, n, dq, dk, dv, dpos, cur, bias, window, 1, o_all, ws)
    u = torch.zeros(b, cap, device="cuda")
    s_out = torch.empty(L, b, n, device="cuda")
    params = B.make_params(0.5, n, recency_bias=bias, recency_window=window)
    assert B.kv_evict_finish(shape, params, 1, n, dk, dv, u, dpos, ws, s_out=s_out) == n
    o_one = torch.empty_like(dq)
    for l in range(L):
        B.kv_attend_score(shape, l, 1, n, dq[l], dk, dv, dpos, cur, bias, window, 0, o_one[l], ws)
    torch.cuda.synchronize()
    kr, vr, qr = raw_numpy(k), raw_numpy(v), raw_numpy(q)
    pr = pos.numpy().astype(np.int64)
    o_ref = np.zeros((L, b, hq, d))
    sc = np.zeros_like(o_ref)
    s_ref = np.zeros((L, b, n))
    for l in range(L):
        for bb in range(b):
            keys = to_f64(kr[l, bb, :, :n], dtype)
            ql = to_f64(qr[l, bb], dtype)
            o_ref[l, bb], sc[l, bb] = attention_output(ql, keys, to_f64(vr[l, bb, :, :n], dtype), pr[bb, :n], cur,
                                                       bias, window)
            s_ref[l, bb] = layer_scores(ql, keys, pr[bb, :n], cur, bias, window)
    assert_o(o_all, o_ref, sc, dtype, "all layers in one call")
    assert_o(o_one, o_ref, sc, dtype, "one call per layer")
    assert_close(s_out.cpu().numpy(), s_ref, "scores from the attention")


@pytest.mark.parametrize("merge,entropy", [(0, False), (1, False), (2, False), (4, False), (8, False), (4, True)],
                         ids=["auto", "merge1", "merge2", "merge4", "merge8", "merge4_entropy"])
def test_fused_scores_equal_separate_pass_bitwise(merge, entropy):
    """With one chunk per slab the attention computes its scores with the scorer's arithmetic in the same
    order, so the fused step and kv_evict_step leave bit-identical utilities and caches; also when the scorer
    adds the group sums of several KV heads in one workgroup (the finish adds the attention's per-KV-head rows
    in the same blocks), and with entropy weighting (computed from those sums)."""
    cfg = LLAMA8B.scaled(batch=8, layers=16, prefill_len=500, budget=400)
    w = Workload(cfg)
    cap = cfg.prefill_len + 1
    st = to_device(w.prefill(capacity=cap))
    st2 = {k: (v.clone() if isinstance(v, torch.Tensor) else v) for k, v in st.items()}
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cap, cfg.dtype)
    params = B.make_params(cfg.alpha, cfg.budget, 1, False, "mean", cfg.recency_bias, cfg.recency_window,
                           entropy=entropy, score_merge=merge)
    ws = B.workspace(shape, cap)
    n = st["n"]
    si = to_device(w.step_inputs(1))
    s1 = torch.empty(cfg.layers, cfg.batch, n + 1, device="cuda")
    s2 = torch.empty_like(s1)
    n1 = B.kv_evict_step(shape, params, 1, n, si["new_pos"], si["q"], si["k_new"], si["v_new"], st["k"], st["v"],
                         st["u"], st["pos"], ws, s_out=s1)
    B.kv_append(shape, params, 1, n, si["new_pos"], si["k_new"], si["v_new"], st2["k"], st2["v"], st2["u"],
                st2["pos"])
    o = torch.empty_like(si["q"])
    B.kv_attend_score(shape, 0, cfg.layers, n + 1, si["q"], st2["k"], st2["v"], st2["pos"], si["new_pos"],
                      cfg.recency_bias, cfg.recency_window, 1, o, ws)
    n2 = B.kv_evict_finish(shape, params, 1, n + 1, st2["k"], st2["v"], st2["u"], st2["pos"], ws, s_out=s2)
    torch.cuda.synchronize()
    assert n1 == n2 == cfg.budget
    assert torch.equal(s1, s2)
    assert torch.equal(st["u"], st2["u"]) and torch.equal(st["pos"], st2["pos"])
    assert torch.equal(st["k"], st2["k"]) and torch.equal(st["v"], st2["v"])


def test_attend_without_scores_leaves_other_layers_alone():
    """emit_scores = 0 writes no score: a later finish folds what the emitting calls left (here: layer 0
    emitted, layer 1 not, so layer 1's scores are the previous step's)."""
    cfg = TINY
    w = Workload(cfg)
    st = to_device(w.prefill())
    shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.capacity,
                         cfg.dtype)
    ws = B.workspace(shape, cfg.capacity)
    n = st["n"]
    si = to_device(w.step_inputs(1))
    params = B.make_params(cfg.alpha, n + 5)
    o = torch.empty_like(si["q"])
    B.kv_attend_score(shape, 0, 2, n, si["q"], st["k"], st["v"], st["pos"], 0, 0.0, 0, 1, o, ws)
    s_a = torch.empty(cfg.layers, cfg.batch, n, device="cuda")
    B.kv_evict_finish(shape, params, 1, n, st["k"], st["v"], st["u"].clone(), st["pos"], ws, s_out=s_a)
    q2 = torch.flip(si["q"], dims=[0]).contiguous()
    B.kv_attend_score(shape, 0, 1, n, q2[0], st["k"], st["v"], st["pos"], 0, 0.0, 0, 1, o[0], ws)
    B.kv_attend_score(shape, 1, 1, n, q2[1], st["k"], st["v"], st["pos"], 0, 0.0, 0, 0, o[1], ws)
    s_b = torch.empty_like(s_a)
    B.kv_evict_finish(shape, params, 1, n, st["k"], st["v"], st["u"].clone(), st["pos"], ws, s_out=s_b)
    torch.cuda.synchronize()
    assert torch.equal(s_b[1], s_a[1])          # layer 1 kept the first call's scores
    assert not torch.equal(s_b[0], s_a[0])      # layer 0 was re-scored with another query
