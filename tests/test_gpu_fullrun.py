"""Whole runs at the workloads' full sizes, in lockstep with the float64 oracle on sampled sequences.

Each workload runs every decode step it defines, with the launch configuration the benchmark times:
* Llama-8B 32k: step 1 over 32,769 tokens, then steps 2..64 under full refresh (the benchmarked schedule) and
  under Lazy R = 4 and R = 8 (Eq. 5), each with the minimum prior (the workload's "last utility floor") and the
  paper's mean prior (appendix "New token insertion"), all continuing the same checked step 1;
* Score-Free 128k: step 1 over 131,073 tokens, then the 256 append-and-evict steps on the frozen ranking
  (Sec. 3.2 Score-Free box: "current mean momentum"), under both priors;
* Qwen-shaped: all 128 full-refresh steps (step 1 over 8,193 tokens, then 2,049 per step).
The GPU steps every sequence of the batch; the oracle follows sampled sequences (sequences are independent, so
each is checked exactly as if alone).  Every step: the decision equal outside the 1e-4 band (lockstep adoption
inside it, counted and printed), utilities within 1e-3 relative, positions bit-exact, per-layer scores on
refresh steps, and the K/V rows the step wrote bit-exact; every `full_every` steps and after the last one the
whole retained K/V of the sampled sequences bit-exact."""
import gc

import numpy as np
import pytest
import torch

from oracle import Cache, evict_step
from parity import assert_close, check_norm_cache, lockstep_adopter, oracle_params
from workload import LLAMA8B, QWEN, SCOREFREE128K, Workload, raw_numpy

pytestmark = pytest.mark.gpu

B = pytest.importorskip("paper_2609_03515_amd.binding")


def _oracle_seq(st, b, dtype):
    return Cache(raw_numpy(st["k"][:, b:b + 1]), raw_numpy(st["v"][:, b:b + 1]),
                 st["u"][b:b + 1].cpu().numpy().astype(np.float64),
                 st["pos"][b:b + 1].cpu().numpy().astype(np.int64), st["n"], dtype)


class Run:
    """GPU state of a whole batch plus oracle caches of sampled sequences, stepped in lockstep."""

    def __init__(self, cfg, samples, full_every):
        self.cfg, self.samples, self.full_every = cfg, samples, full_every
        self.w = Workload(cfg, device="cuda")
        self.st = self.w.prefill()
        self.oc = {b: _oracle_seq(self.st, b, cfg.dtype) for b in samples}
        self.shape = B.make_shape(cfg.batch, cfg.layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim,
                                  cfg.capacity, cfg.dtype)
        self.ws = B.workspace(self.shape, cfg.capacity)
        self.flips = 0
        self.norms = None   # VNorm's value-norm cache, when a run keeps one

    def step(self, t, sched, tag):
        cfg, st = self.cfg, self.st
        variants = {k: sched.get(k, False) for k in ("vnorm", "entropy")}
        params = B.make_params(cfg.alpha, cfg.budget, sched["refresh_period"], sched["score_free"],
                               sched["nonrefresh_init"], cfg.recency_bias, cfg.recency_window, **variants)
        op = oracle_params(cfg, **{k: v for k, v in sched.items() if k != "last"})
        si = self.w.step_inputs(t)
        n = st["n"]
        keep = torch.zeros(cfg.batch, cfg.capacity, dtype=torch.uint8, device="cuda")
        s_out = torch.empty((cfg.layers, cfg.batch, n + 1), device="cuda")
        n_out = B.kv_evict_step(self.shape, params, t, n, si["new_pos"], si["q"], si["k_new"], si["v_new"],
                                st["k"], st["v"], st["u"], st["pos"], self.ws, keep_out=keep, s_out=s_out,
                                v_norms=self.norms)
        torch.cuda.synchronize()
        assert n_out == min(cfg.budget, n + 1)
        full = t == 1 or t % self.full_every == 0 or t == sched["last"]
        for b in self.samples:
            keep_g = keep[b:b + 1, : n + 1].cpu().numpy().astype(bool)
            flips = []
            what = f"{tag} t={t} seq {b}"
            ref = evict_step(self.oc[b], raw_numpy(si["q"][:, b:b + 1]), raw_numpy(si["k_new"][:, b:b + 1]),
                             raw_numpy(si["v_new"][:, b:b + 1]), t, si["new_pos"], op,
                             keep_override=lockstep_adopter(keep_g, cfg.budget, what, flips))
            self.flips += sum(flips)
            oc = self.oc[b]
            if ref.refreshed:
                assert_close(s_out[:, b].cpu().numpy(), ref.s_layers[:, 0], what + " scores")
            assert_close(st["u"][b, :n_out].cpu().numpy(), oc.u[0, :n_out], what + " utilities")
            np.testing.assert_array_equal(st["pos"][b, :n_out].cpu().numpy(), oc.pos[0, :n_out], what + " positions")
            if full:
                rows = slice(0, n_out)
            else:   # the rows this step wrote: hole-fill destinations and the appended slot while under budget
                dst = list(ref.moves[0][0])
                if n + 1 <= cfg.budget:
                    dst.append(n)
                rows = np.array(sorted(set(int(r) for r in dst)), dtype=np.int64)
                if len(rows) == 0:
                    continue
                rows_t = torch.from_numpy(rows).cuda()
            for name in ("k", "v"):
                if full:
                    got = raw_numpy(st[name][:, b, :, rows])
                else:
                    got = raw_numpy(st[name][:, b].index_select(2, rows_t))
                want = getattr(oc, name)[:, 0][:, :, rows]
                assert np.array_equal(got, want), f"{what}: {name} rows differ ({'all' if full else rows[:8]})"
        if self.norms is not None and full:
            for b in self.samples:
                check_norm_cache(B, self.shape, st["v"], self.norms, n_out, None, cfg.dtype, f"{tag} t={t} seq {b}",
                                 b=b, v_ref_seq=self.oc[b].v[:, 0])
        st["n"] = n_out
        if t == 1 or t % 16 == 0 or t == sched["last"]:
            print(f"{tag} t={t} ok, n={n_out}, in-band flips so far {self.flips}", flush=True)

    def snapshot(self):
        """The live rows [0, n) of the GPU state and copies of the oracle caches.  The oracle caches are cut to
        n + 1 rows (the cache never holds more than B + 1 = n + 1 tokens after the first step), live ones too."""
        n = self.st["n"]
        st = self.st
        self.oc = {b: Cache(c.k[:, :, :, :n + 1].copy(), c.v[:, :, :, :n + 1].copy(), c.u[:, :n + 1].copy(),
                            c.pos[:, :n + 1].copy(), c.n, c.dtype) for b, c in self.oc.items()}
        gc.collect()
        return (n, st["k"][:, :, :, :n].clone(), st["v"][:, :, :, :n].clone(), st["u"][:, :n].clone(),
                st["pos"][:, :n].clone(), {b: c.copy() for b, c in self.oc.items()})

    def restore(self, snap):
        n, k, v, u, p, oc = snap
        st = self.st
        st["k"][:, :, :, :n] = k
        st["v"][:, :, :, :n] = v
        st["u"][:, :n] = u
        st["pos"][:, :n] = p
        st["n"] = n
        self.oc = {b: c.copy() for b, c in oc.items()}
        torch.cuda.synchronize()

    def close(self):
        del self.st, self.ws
        gc.collect()
        torch.cuda.empty_cache()


def _sched(cfg, last, **kw):
    s = dict(refresh_period=cfg.refresh_period, score_free=cfg.score_free, nonrefresh_init=cfg.nonrefresh_init)
    s.update(kw)
    s["last"] = last
    return s


@pytest.fixture(scope="module")
def llama_after_step1():
    cfg = LLAMA8B
    run = Run(cfg, samples=(0, 5), full_every=16)
    run.step(1, _sched(cfg, cfg.steps, refresh_period=1, nonrefresh_init="mean"), "8B step 1")
    snap = run.snapshot()
    yield run, snap
    run.close()


LLAMA_SCHEDULES = [(1, "mean"), (4, "min"), (4, "mean"), (8, "min"), (8, "mean")]


@pytest.mark.parametrize("period,init", LLAMA_SCHEDULES, ids=[f"R{r}-{i}" for r, i in LLAMA_SCHEDULES])
def test_llama8b_32k_all_64_steps(llama_after_step1, period, init):
    """Steps 2..64 after the shared, checked step 1: full refresh (63 refresh steps), Lazy R = 4 (15 more
    refresh steps) and R = 8 (7), each under the minimum and the mean prior."""
    run, snap = llama_after_step1
    run.restore(snap)
    cfg = run.cfg
    sched = _sched(cfg, cfg.steps, refresh_period=period, nonrefresh_init=init, score_free=False)
    for t in range(2, cfg.steps + 1):
        run.step(t, sched, f"8B R={period} {init}")


def test_llama8b_32k_vnorm_from_the_norm_cache(llama_after_step1):
    """VNorm + entropy steps at the 8B / 32k shape with the value-norm cache filled once (kv_value_norms) after
    the shared step 1: 16 full-refresh steps (the steady step's three kernels plus the norms' mean), then 16
    Lazy R = 4 steps under the mean prior; the cache itself is checked at every full comparison."""
    run, snap = llama_after_step1
    run.restore(snap)
    cfg = run.cfg
    run.norms = torch.full((cfg.layers, cfg.batch, cfg.n_kv_heads, cfg.capacity), -1.0, device="cuda")
    try:
        B.kv_value_norms(run.shape, run.st["n"], run.st["v"], run.norms)
        full = _sched(cfg, 33, refresh_period=1, nonrefresh_init="mean", score_free=False, vnorm=True, entropy=True)
        lazy = _sched(cfg, 33, refresh_period=4, nonrefresh_init="mean", score_free=False, vnorm=True, entropy=True)
        for t in range(2, 18):
            run.step(t, full, "8B VNorm norm cache R=1")
        for t in range(18, 34):
            run.step(t, lazy, "8B VNorm norm cache R=4 mean")
    finally:
        run.norms = None


@pytest.fixture(scope="module")
def scorefree_after_step1():
    cfg = SCOREFREE128K
    run = Run(cfg, samples=(1,), full_every=64)
    run.step(1, _sched(cfg, cfg.steps), "SF128k step 1")
    snap = run.snapshot()
    yield run, snap
    run.close()


@pytest.mark.parametrize("init", ["min", "mean"])
def test_scorefree_128k_all_257_steps(scorefree_after_step1, init):
    """The 256 append-and-evict steps after the shared step 1 over 131,073 tokens, on the frozen ranking."""
    run, snap = scorefree_after_step1
    run.restore(snap)
    cfg = run.cfg
    sched = _sched(cfg, cfg.steps, nonrefresh_init=init)
    for t in range(2, cfg.steps + 1):
        run.step(t, sched, f"SF128k {init}")


def test_qwen_8k_all_128_steps():
    """All 128 full-refresh steps of the Qwen-shaped workload (GQA 7, Student-t keys)."""
    cfg = QWEN
    run = Run(cfg, samples=(0, 31), full_every=32)
    try:
        sched = _sched(cfg, cfg.steps)
        for t in range(1, cfg.steps + 1):
            run.step(t, sched, "Qwen")
    finally:
        run.close()
