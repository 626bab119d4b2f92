"""GPU parity of each C entry point against the float64 oracle on the same seeded inputs.

Scores and utilities: |gpu - ref| <= 1e-3 |ref| + 1e-12.  Selection from identical float32 utilities and
compaction are integer/byte work and must match bit for bit."""
import numpy as np
import pytest
import torch

from oracle import compact_rows, fold_layers, layer_scores, select_keep, to_f64
from parity import assert_close
from workload import TINY, Workload, raw_numpy

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2609_03515_amd.binding")


def _cfg(dtype, d, hq, hkv, n, batch, layers, bias):
    return TINY.scaled(name="case", batch=batch, layers=layers, n_q_heads=hq, n_kv_heads=hkv, head_dim=d,
                       dtype=dtype, prefill_len=n, budget=max(1, n // 10), heavy_frac=0.05,
                       recency_bias=0.5 if bias else 0.0, recency_window=64 if bias else 0)


SCORE_CASES = [
    # dtype, d, Hq, Hkv, n, batch, layers, recency bias        (comment: path exercised)
    ("f32", 64, 4, 2, 513, 1, 2, False),      # Tiny shape, first step
    ("f32", 64, 4, 2, 52, 1, 2, False),       # Tiny shape, steady step (one partial tile)
    ("bf16", 128, 32, 8, 1000, 2, 3, True),   # Llama GQA 4, several tiles + ragged tail
    ("bf16", 128, 28, 4, 777, 2, 2, False),   # Qwen GQA 7 (padded group 8)
    ("bf16", 128, 8, 8, 300, 2, 2, True),     # no GQA (group 1)
    ("bf16", 64, 16, 2, 500, 1, 2, False),    # d = 64 bf16: 8 lanes per row, group 8
    ("bf16", 128, 32, 2, 400, 1, 2, True),    # group 16
    ("f32", 128, 8, 4, 333, 2, 2, False),     # f32 d = 128: two chunks per lane
    ("bf16", 128, 8, 2, 6000, 1, 2, True),    # group 4 beyond the LDS-resident limit: split path
    ("bf16", 128, 14, 2, 3000, 1, 2, False),  # group 7 split path
    ("f32", 64, 2, 1, 10500, 1, 1, False),    # f32 split path
    ("bf16", 128, 4, 1, 1, 1, 1, False),      # a single cached token
    ("bf16", 128, 8, 2, 40000, 1, 1, True),   # split path: 13 chunks exchanging their statistics
    ("bf16", 128, 32, 2, 14000, 1, 1, False),  # group 16, 11 chunks of 80 KiB exchanging their statistics
    ("bf16", 128, 32, 2, 24000, 1, 1, True),  # group 16, 19 chunks: too many to exchange, logits + finish
    ("bf16", 128, 10, 2, 701, 1, 2, True),    # group 5: three padded heads in the matrix-core tile
    ("bf16", 128, 24, 2, 509, 1, 2, False),   # group 12 (padded group 16)
    ("bf16", 64, 12, 2, 20001, 1, 1, True),   # group 6, d = 64: one line per row, chunks exchanging statistics
    ("f32", 128, 8, 4, 12000, 2, 2, True),    # f32 chunks exchanging statistics in teams of 4 KV heads
    ("bf16", 128, 16, 8, 15001, 1, 3, False),  # group 2, teams of 4 KV heads over a ragged last chunk
]


@pytest.mark.parametrize("case", SCORE_CASES, ids=lambda c: "-".join(map(str, c)))
def test_score_ema_parity(case):
    dtype, d, hq, hkv, n, batch, layers, bias = case
    cfg = _cfg(*case)
    print(f"score case {case}", flush=True)
    w = Workload(cfg, seed=1234 + n)
    st = w.prefill(capacity=n + 3, rows=n)
    si = w.step_inputs(1)
    cur = n - 1 + 5
    gen = torch.Generator().manual_seed(n)
    u0 = torch.rand(batch, n + 3, generator=gen) * 1e-3
    alpha = 0.85
    shape = B.make_shape(batch, layers, hq, hkv, d, n + 3, dtype)
    ws = B.workspace(shape, n)
    u_g = u0.cuda()
    s_out = torch.full((layers, batch, n), -1.0, device="cuda")
    B.kv_score_ema(shape, n, si["q"].cuda(), st["k"].cuda(), st["pos"].cuda(), cur, alpha, cfg.recency_bias,
                   cfg.recency_window, u_g, s_out, ws)
    torch.cuda.synchronize()
    k_raw, q_raw = raw_numpy(st["k"]), raw_numpy(si["q"])
    pos = st["pos"].numpy()
    s_ref = np.zeros((layers, batch, n))
    u_ref = np.zeros((batch, n))
    for b in range(batch):
        for l in range(layers):
            s_ref[l, b] = layer_scores(to_f64(q_raw[l, b], dtype), to_f64(k_raw[l, b, :, :n], dtype), pos[b, :n],
                                       cur, cfg.recency_bias, cfg.recency_window)
        u_ref[b] = fold_layers(u0[b, :n].double().numpy(), s_ref[:, b], alpha)
    assert_close(s_out.cpu().numpy(), s_ref, "per-layer scores")
    u_gpu = u_g.cpu()
    assert_close(u_gpu[:, :n].numpy(), u_ref, "utilities")
    assert torch.equal(u_gpu[:, n:], u0[:, n:]), "entries beyond n must stay untouched"


def _select_inputs(batch, n, pattern, seed):
    g = torch.Generator().manual_seed(seed)
    if pattern == "random":
        u = torch.rand(batch, n, generator=g)
    elif pattern == "ties":
        u = torch.randint(0, 7, (batch, n), generator=g).float() * 0.125
    elif pattern == "equal":
        u = torch.full((batch, n), 0.3)
    elif pattern == "tiny":
        u = torch.rand(batch, n, generator=g) * 1e-30   # denormal-range utilities keep their order
    else:
        raise ValueError(pattern)
    pos = torch.stack([torch.randperm(1 << 20, generator=g)[:n] for _ in range(batch)]).to(torch.int32)
    return u.contiguous(), pos.contiguous()


SELECT_CASES = [
    (3, 1000, 100, "random"), (3, 1000, 100, "ties"), (2, 1000, 100, "equal"), (2, 101, 100, "random"),
    (2, 101, 100, "ties"), (2, 101, 100, "equal"), (2, 50, 100, "random"), (2, 100, 100, "ties"),
    (2, 40000, 4000, "random"), (1, 40000, 4000, "ties"), (2, 3278, 3277, "random"), (2, 777, 1, "random"),
    (2, 777, 776, "ties"), (1, 5000, 123, "tiny"), (1, 1, 1, "random"),
    # long sequences in a small batch: the multi-workgroup selection (slices of every sequence)
    (4, 20000, 2000, "ties"), (2, 131073, 13107, "random"), (8, 32769, 3277, "equal"), (1, 16384, 16382, "random"),
    (3, 50000, 100, "tiny"), (2, 20000, 19998, "ties"),
    # the edges of that choice: 128 sequences still slice (4 per sequence), 129 do not; 16,383 tokens do not
    (128, 16384, 1638, "ties"), (129, 16384, 1638, "random"), (5, 16383, 1000, "random"), (5, 16384, 1000, "equal"),
]


@pytest.mark.parametrize("case", SELECT_CASES, ids=lambda c: "-".join(map(str, c)))
def test_topk_select_parity(case):
    batch, n, budget, pattern = case
    print(f"select case {case}", flush=True)
    u, pos = _select_inputs(batch, n, pattern, seed=n + budget)
    cap = n + 2
    shape = B.make_shape(batch, 1, 1, 1, 128, cap, "bf16")
    ws = B.workspace(shape, n)
    u_c = torch.zeros(batch, cap)
    u_c[:, :n] = u
    p_c = torch.zeros(batch, cap, dtype=torch.int32)
    p_c[:, :n] = pos
    keep = torch.full((batch, cap), 7, dtype=torch.uint8, device="cuda")
    B.kv_topk_select(shape, n, budget, u_c.cuda(), p_c.cuda(), keep, ws)
    keep = keep.cpu().numpy()
    for b in range(batch):
        ref = select_keep(u[b].double().numpy(), pos[b].numpy(), budget)
        np.testing.assert_array_equal(keep[b, :n].astype(bool), ref, err_msg=f"sequence {b}")
        assert np.all(keep[b, n:] == 7), "entries beyond n must stay untouched"


COMPACT_CASES = [(2, 2, 2, 128, "bf16", 500, 50), (1, 3, 4, 64, "f32", 300, 299), (2, 1, 1, 128, "bf16", 101, 100),
                 (1, 2, 2, 64, "bf16", 2000, 1900), (2, 2, 2, 128, "f32", 64, 8), (1, 1, 2, 128, "bf16", 5, 7)]


@pytest.mark.parametrize("case", COMPACT_CASES, ids=lambda c: "-".join(map(str, c)))
def test_compact_parity(case):
    batch, layers, hkv, d, dtype, n, budget = case
    print(f"compact case {case}", flush=True)
    cap = n + 4
    g = torch.Generator().manual_seed(n * 7 + budget)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    k = torch.randn(layers, batch, hkv, cap, d, generator=g).to(tdt)
    v = torch.randn(layers, batch, hkv, cap, d, generator=g).to(tdt)
    u = torch.rand(batch, cap, generator=g)
    pos = torch.stack([torch.randperm(10 * cap, generator=g)[:cap] for _ in range(batch)]).to(torch.int32)
    keep = torch.zeros(batch, cap, dtype=torch.uint8)
    kk = min(budget, n)
    for b in range(batch):
        keep[b, torch.randperm(n, generator=g)[:kk]] = 1
    shape = B.make_shape(batch, layers, 2 * hkv, hkv, d, cap, dtype)
    ws = B.workspace(shape, n)
    kg, vg, ug, pg = k.cuda(), v.cuda(), u.cuda(), pos.cuda()
    B.kv_compact(shape, n, budget, keep.cuda(), kg, vg, ug, pg, ws)
    torch.cuda.synchronize()
    kr, vr = raw_numpy(k), raw_numpy(v)
    kgr, vgr = raw_numpy(kg), raw_numpy(vg)
    for b in range(batch):
        kb = keep[b, :n].numpy().astype(bool)
        for l in range(layers):
            for h in range(hkv):
                want_k = compact_rows(kr[l, b, h, :n], kb, budget)
                want_v = compact_rows(vr[l, b, h, :n], kb, budget)
                np.testing.assert_array_equal(kgr[l, b, h, :kk], want_k[:kk])
                np.testing.assert_array_equal(vgr[l, b, h, :kk], want_v[:kk])
                np.testing.assert_array_equal(kgr[l, b, h, kk:], kr[l, b, h, kk:])   # untouched beyond k
        np.testing.assert_array_equal(ug.cpu()[b, :kk].numpy(), compact_rows(u[b, :n].numpy(), kb, budget)[:kk])
        np.testing.assert_array_equal(pg.cpu()[b, :kk].numpy(), compact_rows(pos[b, :n].numpy(), kb, budget)[:kk])
