"""Helpers for GPU-vs-oracle parity tests: moving the same seeded inputs to both sides and comparing."""
from __future__ import annotations

import numpy as np
import torch

from oracle import Cache, Params, to_f64
from workload import raw_numpy

REL_TOL = 1e-3        # scores and utilities
O_REL = 1e-3          # attention outputs, relative to sum_i a(i) |v_i|
ABS_TOL = 1e-12
BAND = 1e-4           # retention sets may differ only for utilities this close to the B-th value


def oracle_cache(st: dict, dtype: str) -> Cache:
    return Cache(raw_numpy(st["k"]), raw_numpy(st["v"]), st["u"].detach().cpu().numpy().astype(np.float64),
                 st["pos"].detach().cpu().numpy().astype(np.int64), int(st["n"]), dtype)


def oracle_params(cfg, **kw) -> Params:
    base = dict(alpha=cfg.alpha, budget=cfg.budget, refresh_period=cfg.refresh_period,
                score_free=cfg.score_free, nonrefresh_init=cfg.nonrefresh_init,
                recency_bias=cfg.recency_bias, recency_window=cfg.recency_window)
    base.update(kw)
    return Params(**base)


def to_device(st: dict, device="cuda") -> dict:
    return {k: (v.to(device).contiguous() if isinstance(v, torch.Tensor) else v) for k, v in st.items()}


def assert_close(gpu, ref, what, rel=REL_TOL, abs_=ABS_TOL):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, (what, gpu.shape, ref.shape)
    err = np.abs(gpu - ref)
    lim = rel * np.abs(ref) + abs_
    bad = np.nonzero(err > lim)
    assert len(bad[0]) == 0, (f"{what}: {len(bad[0])} of {err.size} outside tolerance; worst rel "
                              f"{np.max(err / (np.abs(ref) + 1e-30)):.3e} at {tuple(b[0] for b in bad)}")


def band_mask(u_ref: np.ndarray, budget: int) -> np.ndarray:
    """Tokens whose reference utility lies within BAND (relative) of the B-th value."""
    n = len(u_ref)
    if n <= budget:
        return np.zeros(n, dtype=bool)
    tau = np.sort(u_ref)[::-1][budget - 1]
    return np.abs(u_ref - tau) <= BAND * abs(tau)


def check_keep(keep_gpu: np.ndarray, keep_ref: np.ndarray, u_ref: np.ndarray, budget: int, what: str) -> int:
    """Exact count; equality outside the rounding band.  Returns the number of in-band differences."""
    keep_gpu = np.asarray(keep_gpu, dtype=bool)
    keep_ref = np.asarray(keep_ref, dtype=bool)
    assert keep_gpu.sum() == keep_ref.sum() == min(budget, len(keep_ref)), (what, keep_gpu.sum(), keep_ref.sum())
    band = band_mask(u_ref, budget)
    diff = keep_gpu != keep_ref
    assert not np.any(diff & ~band), f"{what}: {int((diff & ~band).sum())} retention differences outside the band"
    return int(diff.sum())


def lockstep_adopter(keep_gpu_rows: np.ndarray, budget: int, what: str, counter: list):
    """keep_override callback for the oracle: checks the GPU's decision against the oracle's own (exact count,
    equal outside the band) and returns the GPU's mask, so both sides continue from the same retained set.
    Appends the number of in-band differences to `counter`."""
    def adopt(keep_ref, u_pre):
        n = keep_ref.shape[1]
        flips = 0
        for b in range(keep_ref.shape[0]):
            flips += check_keep(keep_gpu_rows[b, :n], keep_ref[b], u_pre[b], budget, f"{what} b={b}")
        counter.append(flips)
        return np.asarray(keep_gpu_rows[:, :n], dtype=bool)
    return adopt


def assert_o(o_gpu, o_ref, scale, dtype, what):
    """Attention outputs: |o_gpu - o_ref| <= 1e-3 * sum_i a(i)|v_i| (+ 2^-8 |o_ref| for a bf16 output)."""
    got = to_f64(raw_numpy(o_gpu), dtype)
    assert got.shape == o_ref.shape, (what, got.shape, o_ref.shape)
    lim = O_REL * scale + (2.0 ** -8 if dtype == "bf16" else 0.0) * np.abs(o_ref) + 1e-12
    err = np.abs(got - o_ref)
    bad = np.nonzero(err > lim)
    assert len(bad[0]) == 0, (f"{what}: {len(bad[0])} of {err.size} outputs outside tolerance; worst "
                              f"err/scale {np.max(err / (scale + 1e-30)):.3e} at {tuple(b[0] for b in bad)}")


def check_norm_cache(B, shape, v_dev, norms, n, v_ref_raw, dtype, what, b=None, v_ref_seq=None):
    """The value-norm cache's live rows [0, n): bit for bit the norms kv_value_norms recomputes from the GPU's V
    (one arithmetic produces every cached norm, so appends and moves must have kept each norm beside its row),
    and within 1e-5 relative of the float64 l2 norms of the oracle's V rows.  v_ref_raw: the oracle's V of the
    whole batch [K, b, H_kv, cap, d]; or, for sequence b only, v_ref_seq [K, H_kv, cap, d]."""
    fresh = torch.full_like(norms, -1.0)
    B.kv_value_norms(shape, n, v_dev, fresh)
    torch.cuda.synchronize()
    got = norms[..., :n] if b is None else norms[:, b, :, :n]
    want = fresh[..., :n] if b is None else fresh[:, b, :, :n]
    assert torch.equal(got, want), f"{what}: cached norms differ from the norms of the rows beside them"
    ref = v_ref_raw if b is None else v_ref_seq
    v64 = to_f64(np.asarray(ref)[..., :n, :], dtype)
    assert_close(got.cpu().numpy(), np.sqrt((v64 * v64).sum(axis=-1)), f"{what} norms", rel=1e-5)
