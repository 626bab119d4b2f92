"""Seeded synthetic decode workloads shaped like the paper's backbones.

This module only draws inputs: it holds none of the eviction method's arithmetic, and both the HIP path and
the float64 oracle consume the tensors it returns.  Nothing here reads a dataset or trained weights: the
paper evaluates on LongBench / LongBench-v2 / RULER contexts with Llama-3.1-8B and Qwen2.5-7B (Sec. 4); these
seeded Gaussian (or Student-t) activations with planted heavy hitters and a recency bias stand in for them.

Recipe (per configuration):
* queries, keys and values ~ N(0, 1) i.i.d.; keys ~ Student-t(nu = 4) for the Qwen-style shape;
* one heavy-hitter direction per (layer, KV head): a random unit vector scaled by d^(1/4); a heavy token's key
  gets +3 x direction and every query of that KV group gets +1 x direction, so a heavy key's expected logit
  (q.k / sqrt(d)) is raised by 3;
* heavy tokens: a seeded fraction of prefill positions per sequence (shared by all layers and heads); each
  decode token is heavy with the same probability;
* keys/values/queries are drawn in float32 and rounded to the storage dtype (bf16 or f32);
* positions 0..L0-1 for the prefill, L0 + t - 1 for the token appended at decode step t; utility 0.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass

import torch

BASE_SEED = 2609_03515


@dataclass(frozen=True)
class Config:
    name: str
    batch: int
    layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: str              # "f32" | "bf16"
    prefill_len: int
    budget: int
    alpha: float
    steps: int
    refresh_period: int = 1
    score_free: bool = False
    nonrefresh_init: str = "mean"
    heavy_frac: float = 0.02
    key_dist: str = "normal"  # "normal" | "student_t4"
    recency_bias: float = 0.0
    recency_window: int = 0
    seed_offset: int = 0

    @property
    def capacity(self) -> int:
        return self.prefill_len + 1

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    def scaled(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


# The five workloads: a tiny fp32 case, the Llama-3.1-8B shape (full refresh and Lazy), the Score-Free point
# at 128k context and a Qwen2.5-7B-like small-GQA shape.  GQA counts follow Sec. 4.2 (Llama: 8 KV heads x 4;
# Qwen: 4 KV heads x 7).
TINY = Config("tiny", 1, 2, 4, 2, 64, "f32", 512, 51, 0.9, 16, seed_offset=1)
LLAMA8B = Config("llama8b_32k", 8, 32, 32, 8, 128, "bf16", 32768, 3277, 0.9, 64,
                 recency_bias=0.5, recency_window=64, seed_offset=2)
LLAMA8B_LAZY = LLAMA8B.scaled(name="llama8b_32k_lazy", refresh_period=4, nonrefresh_init="min", seed_offset=3)
SCOREFREE128K = Config("llama8b_128k_scorefree", 2, 32, 32, 8, 128, "bf16", 131072, 13107, 0.9, 257,
                       score_free=True, nonrefresh_init="min", recency_bias=0.5, recency_window=64,
                       seed_offset=4)
QWEN = Config("qwen_8k", 32, 28, 28, 4, 128, "bf16", 8192, 2048, 0.8, 128, heavy_frac=0.05,
              key_dist="student_t4", seed_offset=5)
CONFIGS = {c.name: c for c in (TINY, LLAMA8B, LLAMA8B_LAZY, SCOREFREE128K, QWEN)}


def _gen(seed: int, *tags: int, device="cpu") -> torch.Generator:
    h = seed
    for t in tags:
        h = (h * 1_000_003 + int(t) + 7919) % (2 ** 62)
    g = torch.Generator(device=device)
    g.manual_seed(h)
    return g


# tags for the sub-streams
_T_DIR, _T_HEAVY, _T_K, _T_V, _T_Q, _T_KNEW, _T_VNEW, _T_HNEW, _T_POS, _T_U = range(10)


class Workload:
    """Draws the prefill cache and the per-step inputs of one configuration on one device."""

    def __init__(self, cfg: Config, seed: int | None = None, device="cpu"):
        self.cfg = cfg
        self.device = torch.device(device)
        self.seed = BASE_SEED + cfg.seed_offset if seed is None else int(seed)
        c = cfg
        g = _gen(self.seed, _T_DIR, device=self.device)
        dirs = torch.randn(c.layers, c.n_kv_heads, c.head_dim, generator=g, device=self.device)
        dirs = dirs / dirs.norm(dim=-1, keepdim=True)
        self.directions = dirs * (c.head_dim ** 0.25)            # [K, H_kv, d] float32

    # -- raw draws -------------------------------------------------------------------------------------
    def _keys(self, shape, g) -> torch.Tensor:
        z = torch.randn(*shape, generator=g, device=self.device)
        if self.cfg.key_dist == "student_t4":
            chi2 = torch.zeros_like(z)
            for _ in range(4):
                chi2 += torch.randn(*shape, generator=g, device=self.device) ** 2
            z = z / torch.sqrt(chi2 / 4.0)
        elif self.cfg.key_dist != "normal":
            raise ValueError(self.cfg.key_dist)
        return z

    def heavy_mask(self, rows: int, tag: int = _T_HEAVY, *extra) -> torch.Tensor:
        g = _gen(self.seed, tag, *extra, device=self.device)
        return torch.rand(self.cfg.batch, rows, generator=g, device=self.device) < self.cfg.heavy_frac

    # -- prefill cache -----------------------------------------------------------------------------------
    def prefill(self, capacity: int | None = None, rows: int | None = None):
        """K, V: [K, b, H_kv, cap, d] storage dtype; pos: [b, cap] int32; u: [b, cap] float32 (zeros);
        rows [0, L0) hold the prefill, the rest are zero."""
        c = self.cfg
        cap = c.capacity if capacity is None else capacity
        n = c.prefill_len if rows is None else rows
        if n + 1 > cap:
            raise ValueError("capacity must exceed the prefill length")
        dt = c.torch_dtype
        k = torch.zeros(c.layers, c.batch, c.n_kv_heads, cap, c.head_dim, dtype=dt, device=self.device)
        v = torch.zeros_like(k)
        heavy = self.heavy_mask(n).to(torch.float32)                               # [b, n]
        for l in range(c.layers):                                                  # layer by layer: bounded temporaries
            gk = _gen(self.seed, _T_K, l, device=self.device)
            gv = _gen(self.seed, _T_V, l, device=self.device)
            kl = self._keys((c.batch, c.n_kv_heads, n, c.head_dim), gk)
            kl += 3.0 * heavy[:, None, :, None] * self.directions[l][None, :, None, :]
            k[l, :, :, :n] = kl.to(dt)
            del kl
            v[l, :, :, :n] = torch.randn(c.batch, c.n_kv_heads, n, c.head_dim, generator=gv,
                                         device=self.device).to(dt)
        pos = torch.zeros(c.batch, cap, dtype=torch.int32, device=self.device)
        pos[:, :n] = torch.arange(n, dtype=torch.int32, device=self.device)
        u = torch.zeros(c.batch, cap, dtype=torch.float32, device=self.device)
        return {"k": k, "v": v, "pos": pos, "u": u, "n": n}

    # -- per-step inputs -------------------------------------------------------------------------------
    def step_inputs(self, t: int):
        """q: [K, b, H_q, d]; k_new, v_new: [K, b, H_kv, d]; new_pos = L0 + t - 1."""
        c = self.cfg
        dt = c.torch_dtype
        group = c.n_q_heads // c.n_kv_heads
        gq = _gen(self.seed, _T_Q, t, device=self.device)
        q = torch.randn(c.layers, c.batch, c.n_q_heads, c.head_dim, generator=gq, device=self.device)
        q += self.directions.repeat_interleave(group, dim=1)[:, None]
        gk = _gen(self.seed, _T_KNEW, t, device=self.device)
        kn = self._keys((c.layers, c.batch, c.n_kv_heads, c.head_dim), gk)
        heavy = self.heavy_mask(1, _T_HNEW, t).to(torch.float32)[:, 0]             # [b]
        kn += 3.0 * heavy[None, :, None, None] * self.directions[:, None]
        gv = _gen(self.seed, _T_VNEW, t, device=self.device)
        vn = torch.randn(c.layers, c.batch, c.n_kv_heads, c.head_dim, generator=gv, device=self.device)
        return {"q": q.to(dt), "k_new": kn.to(dt), "v_new": vn.to(dt), "new_pos": c.prefill_len + t - 1}

    # -- a steady-state cache drawn directly -------------------------------------------------------------
    def steady_state(self, rows: int | None = None, capacity: int | None = None):
        """A cache of `rows` (default B) tokens as it looks in the middle of decoding: keys/values drawn like
        the prefill, positions a sorted random subset of [0, L0) (the newest position always present),
        utilities positive and summing to about one (exp of a Gaussian, normalised)."""
        c = self.cfg
        n = c.budget if rows is None else rows
        cap = (n + 1) if capacity is None else capacity
        st = self.prefill(capacity=cap, rows=n)
        gp = _gen(self.seed, _T_POS, device=self.device)
        pos = torch.empty(c.batch, cap, dtype=torch.int32, device=self.device)
        pos.zero_()
        for b in range(c.batch):
            perm = torch.randperm(c.prefill_len - 1, generator=gp, device=self.device)[: n - 1]
            p = torch.sort(perm).values.to(torch.int32)
            pos[b, : n - 1] = p
            pos[b, n - 1] = c.prefill_len - 1
        gu = _gen(self.seed, _T_U, device=self.device)
        u = torch.exp(torch.randn(c.batch, n, generator=gu, device=self.device))
        u = u / u.sum(dim=1, keepdim=True)
        st["pos"] = pos
        st["u"] = torch.zeros(c.batch, cap, dtype=torch.float32, device=self.device)
        st["u"][:, :n] = u
        return st


def raw_numpy(t: torch.Tensor):
    """Storage bits for the oracle: bf16 as uint16 bit patterns, everything else as is."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view("uint16")
    return t.numpy()

