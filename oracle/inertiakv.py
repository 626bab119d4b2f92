"""Plain, slow, float64 CPU oracle of the InertiaKV / InertiaKV-Lazy decode-step eviction path.

THIS IS TEST INFRASTRUCTURE. Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import it. The product (the HIP library and its Python binding) never calls it and shares no code with it.

Paper: "What Matters for Aggressive Decoding-Time KV Eviction? Temporal Aggregation and Ranking Preservation".
Each function names the passage it follows:

* Sec. 3 (problem statement): budget B = floor((1 - rho) L0); eviction is irreversible; whenever the cache
  holds more than B tokens the lowest-utility tokens are evicted.
* Eq. 1: s_t(i) = (1/H) sum_h a_t^(h)(i), the last-query attention of every head, mean-pooled over the H
  query heads.  Appendix "Implementation Details / Per-step scoring": under GQA each KV head's attention is
  shared by its query-head group before pooling.
* Eq. 2 / 3 / 4: single-step, cumulative and EMA aggregation rules.
* The step's decode attention (the softmax Eq. 1 pools, applied to V), for the fused attention + score path.
* Appendix "Mechanistic Diagnostics": rank-trace set sizes (raw / EMA top-k churn, raw-EMA Jaccard,
  raw-top evicted rate).
* Sec. 5.1 / appendix "Per-step scoring": VNorm (attention times the mean-normalised l2 norm of the value
  row) and entropy weighting (the layer's score times the normalised entropy of its attention).
* Appendix "Implementation Details / Layer scoring": the EMA state is updated after every eligible layer,
  m_{t,l} = alpha m_{t,l-1} + (1 - alpha) s_{t,l}, l = 1..K, m_{t,0} = m_{t-1,K}.
* Appendix "Implementation Details / Momentum initialization": m_0 = 0 for every prefill position.
* Eq. 5 and Sec. 3.2 "Lazy refresh": refresh set R_r = {t >= 1 : (t - 1) mod r = 0}; off the refresh set the
  utility is carried unchanged and eviction still runs on the stale ranking (Appendix "Eviction on
  non-refresh steps").
* Appendix "New token insertion during non-refresh steps": the new token starts at the mean utility of the
  L_t - 1 existing tokens and may be evicted on the same step.
* Sec. 3.2 "Score-Free decoding" box: score once at decode step 1, freeze, new tokens take the current mean
  momentum, evict whenever the cache exceeds B.

Readings where the paper is silent (the same list is kept in the design notes):
* H in Eq. 1 is the number of query heads; every query head gets its own softmax over its KV head's keys.
* The logit is the scaled dot product q.k / sqrt(d), with an optional additive recency bias on the
  `window` most recent absolute positions (a workload knob, 0 = off).
* One retention set per sequence per step, taken after the last layer's fold and applied to every layer
  and KV head.
* A new token's prior at a refresh step is 0, like m_0 (the paper only fixes the non-refresh case).
* Ties in utility are broken by keeping the lower absolute position.
* Compaction is "hole-fill": with k = min(B, n), kept rows in slots >= k move, in ascending order, into the
  evicted slots < k, in ascending order.  Attention is invariant to row order, so any layout is faithful;
  this one moves the fewest rows.
* Non-refresh initialisation policy "min" (lowest existing utility) is offered beside the paper's "mean".
* VNorm's mean runs over the cached tokens of the same layer and KV head at scoring time; entropy weighting
  uses the entropy of the layer's pooled attention (before VNorm) divided by ln(n), per sequence; with both
  enabled the entropy factor multiplies the VNorm-weighted score.
* Rank trace: the "raw" score of a step is the mean over layers of the plain per-layer score (Eq. 1); both
  top-k sets are taken over the n tokens cached before that step's eviction, identified by position.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

F32 = "f32"
BF16 = "bf16"


# ----------------------------------------------------------------------------------------------------------
# element handling
# ----------------------------------------------------------------------------------------------------------
def to_f64(raw: np.ndarray, dtype: str) -> np.ndarray:
    """Exact up-conversion of stored elements to float64.

    bf16 elements are carried as their uint16 bit patterns; a bf16 value is the float32 whose upper 16 bits
    are those bits, so the conversion is exact.
    """
    if dtype == F32:
        return np.asarray(raw, dtype=np.float32).astype(np.float64)
    if dtype == BF16:
        bits = np.asarray(raw, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


# ----------------------------------------------------------------------------------------------------------
# Sec. 3: budget, Eq. 5: refresh schedule
# ----------------------------------------------------------------------------------------------------------
def budget_from_ratio(prefill_len: int, compression_ratio: float) -> int:
    """Sec. 3: B = floor((1 - rho) * L0)."""
    return int(math.floor((1.0 - compression_ratio) * prefill_len + 1e-9))


def refresh_due(t: int, period: int, score_free: bool) -> bool:
    """Eq. 5: t is in R_r = {t >= 1 : (t-1) mod r == 0}.  Score-Free refreshes only at t = 1 (Sec. 3.2 box)."""
    if t < 1:
        raise ValueError("decode steps are numbered from 1")
    if score_free:
        return t == 1
    return (t - 1) % period == 0


# ----------------------------------------------------------------------------------------------------------
# Eq. 1: last-query attention, mean-pooled over query heads (GQA-shared)
# ----------------------------------------------------------------------------------------------------------
def head_attention(q_h: np.ndarray, keys_g: np.ndarray, pos: np.ndarray | None = None, cur_pos: int = 0,
                   recency_bias: float = 0.0, recency_window: int = 0) -> np.ndarray:
    """a^(h)(i) = softmax_i(q_h . k_i / sqrt(d) [+ bias if pos_i is among the `window` newest positions])."""
    d = q_h.shape[-1]
    z = keys_g @ q_h / math.sqrt(d)
    if recency_bias != 0.0 and recency_window > 0:
        recent = np.asarray(pos) >= (cur_pos - (recency_window - 1))
        z = z + recency_bias * recent
    z = z - z.max()
    e = np.exp(z)
    return e / e.sum()


def layer_scores(q_l: np.ndarray, keys_l: np.ndarray, pos: np.ndarray | None = None, cur_pos: int = 0,
                 recency_bias: float = 0.0, recency_window: int = 0) -> np.ndarray:
    """Eq. 1 for one layer and one sequence.

    q_l:    [H_q, d]       float64, the current (last) query of every query head
    keys_l: [H_kv, n, d]   float64, the cached keys of every KV head
    returns s: [n] = (1/H_q) sum_h a^(h), query head h reading KV head h // (H_q / H_kv).
    """
    hq, hkv = q_l.shape[0], keys_l.shape[0]
    if hq % hkv:
        raise ValueError("query heads must be a multiple of KV heads")
    group = hq // hkv
    s = np.zeros(keys_l.shape[1], dtype=np.float64)
    for h in range(hq):
        s += head_attention(q_l[h], keys_l[h // group], pos, cur_pos, recency_bias, recency_window)
    return s / hq


# ----------------------------------------------------------------------------------------------------------
# Sec. 5.1 and appendix "Per-step scoring": the two order-preserving scorer perturbations
# ----------------------------------------------------------------------------------------------------------
def value_norm_weights(values_g: np.ndarray) -> np.ndarray:
    """VNorm factor of every cached token of one KV head: the l2 norm of its value row divided by the mean
    of those norms over the cached tokens (so the factors average to 1).  All-zero values: factor 1."""
    norms = np.sqrt(np.sum(values_g * values_g, axis=-1))
    mean = norms.mean()
    return norms / mean if mean > 0 else np.ones_like(norms)


def normalized_entropy(s: np.ndarray) -> float:
    """Entropy of the distribution s (normalised to sum 1) divided by its maximum ln(n); 1 when n = 1."""
    n = len(s)
    if n <= 1:
        return 1.0
    p = s / s.sum()
    nz = p > 0
    return float(-np.sum(p[nz] * np.log(p[nz])) / math.log(n))


def layer_scores_variant(q_l: np.ndarray, keys_l: np.ndarray, values_l: np.ndarray, pos: np.ndarray | None,
                         cur_pos: int, recency_bias: float, recency_window: int, vnorm: bool,
                         entropy: bool) -> np.ndarray:
    """Eq. 1 with the optional perturbations, both applied to the step's score before the fold:
    VNorm multiplies each head's attention a^(h)(i) by the VNorm factor of token i under that head's KV
    head before pooling; entropy weighting multiplies the layer's pooled score by the normalised entropy
    of the layer's pooled attention distribution (a per-layer, per-sequence scalar)."""
    hq, hkv = q_l.shape[0], keys_l.shape[0]
    if hq % hkv:
        raise ValueError("query heads must be a multiple of KV heads")
    group = hq // hkv
    nu = [value_norm_weights(values_l[g]) for g in range(hkv)] if vnorm else None
    s = np.zeros(keys_l.shape[1], dtype=np.float64)
    s_attn = np.zeros_like(s)
    for h in range(hq):
        a = head_attention(q_l[h], keys_l[h // group], pos, cur_pos, recency_bias, recency_window)
        s_attn += a
        s += a * nu[h // group] if vnorm else a
    s /= hq
    s_attn /= hq
    if entropy:
        s = s * normalized_entropy(s_attn)
    return s


# ----------------------------------------------------------------------------------------------------------
# The step's own decode attention: the same softmax of the last query that Eq. 1 pools, applied to V
# (scaled dot-product attention, Sec. 3 cites it for a_t)
# ----------------------------------------------------------------------------------------------------------
def attention_output(q_l: np.ndarray, keys_l: np.ndarray, values_l: np.ndarray, pos: np.ndarray | None = None,
                     cur_pos: int = 0, recency_bias: float = 0.0, recency_window: int = 0):
    """Last-query attention of one layer and one sequence.

    q_l: [H_q, d]; keys_l, values_l: [H_kv, n, d] float64.  Returns (o, scale), both [H_q, d]:
    o_h = sum_i a^(h)(i) v_{h // G}(i) with a^(h) the softmax of `head_attention`, and
    scale_h = sum_i a^(h)(i) |v_{h // G}(i)|, the magnitude that bounds rounding in the weighted sum.
    """
    hq, hkv = q_l.shape[0], keys_l.shape[0]
    if hq % hkv:
        raise ValueError("query heads must be a multiple of KV heads")
    group = hq // hkv
    o = np.zeros((hq, values_l.shape[-1]), dtype=np.float64)
    scale = np.zeros_like(o)
    for h in range(hq):
        a = head_attention(q_l[h], keys_l[h // group], pos, cur_pos, recency_bias, recency_window)
        o[h] = a @ values_l[h // group]
        scale[h] = a @ np.abs(values_l[h // group])
    return o, scale


# ----------------------------------------------------------------------------------------------------------
# Eq. 2-4 + Appendix "Layer scoring": per-layer sequential aggregation
# ----------------------------------------------------------------------------------------------------------
EMA, SINGLE_STEP, CUMULATIVE = "ema", "single", "cumulative"


def fold_layers(u: np.ndarray, s_layers, alpha: float, rule: str = EMA) -> np.ndarray:
    """Fold the layer scores s_1..s_K (in ascending layer order) into the running utility.

    EMA (Eq. 4, Appendix "Layer scoring"):  u <- alpha u + (1 - alpha) s_l for l = 1..K.
    Single-step (Eq. 2):                    u <- s_l (only the last processed layer survives).
    Cumulative (Eq. 3):                     u <- u + s_l.
    """
    u = np.array(u, dtype=np.float64, copy=True)
    for s in s_layers:
        if rule == EMA:
            u = alpha * u + (1.0 - alpha) * np.asarray(s, dtype=np.float64)
        elif rule == SINGLE_STEP:
            u = np.array(s, dtype=np.float64, copy=True)
        elif rule == CUMULATIVE:
            u = u + np.asarray(s, dtype=np.float64)
        else:
            raise ValueError(f"unknown aggregation rule {rule!r}")
    return u


# ----------------------------------------------------------------------------------------------------------
# Sec. 3 eviction rule: keep the B highest utilities (ties: lower position kept)
# ----------------------------------------------------------------------------------------------------------
def select_keep(u: np.ndarray, pos: np.ndarray, budget: int) -> np.ndarray:
    """Boolean mask over the n cached tokens: the first min(B, n) under (u descending, position ascending)."""
    n = len(u)
    keep = np.zeros(n, dtype=bool)
    if n <= budget:
        keep[:] = True
        return keep
    order = np.lexsort((np.asarray(pos), -np.asarray(u, dtype=np.float64)))
    keep[order[:budget]] = True
    return keep


def holefill_moves(keep: np.ndarray, budget: int):
    """Hole-fill compaction plan.  k = min(B, n); holes = ascending evicted slots < k; tails = ascending kept
    slots >= k; row tails[j] moves to holes[j].  Returns (dst, src) index arrays of equal length."""
    n = len(keep)
    k = min(budget, n)
    holes = np.nonzero(~keep[:k])[0]
    tails = np.nonzero(keep[k:])[0] + k
    if len(holes) != len(tails):
        raise ValueError("keep mask must retain exactly min(B, n) tokens")
    return holes, tails


# ----------------------------------------------------------------------------------------------------------
# cache state and one decode step
# ----------------------------------------------------------------------------------------------------------
@dataclass
class Params:
    alpha: float
    budget: int
    refresh_period: int = 1
    score_free: bool = False
    nonrefresh_init: str = "mean"      # "mean" (Appendix, new-token insertion) or "min"
    recency_bias: float = 0.0
    recency_window: int = 0
    rule: str = EMA
    vnorm: bool = False                # Sec. 5.1 scorer perturbations
    entropy: bool = False


@dataclass
class Cache:
    """One batch of sequences.  k, v: [K, b, H_kv, cap, d] raw elements (uint16 bf16 bits or float32);
    u: [b, cap] float64 utility; pos: [b, cap] int64 absolute positions; n: rows in use (same for all b)."""
    k: np.ndarray
    v: np.ndarray
    u: np.ndarray
    pos: np.ndarray
    n: int
    dtype: str

    def copy(self) -> "Cache":
        return Cache(self.k.copy(), self.v.copy(), self.u.copy(), self.pos.copy(), self.n, self.dtype)


@dataclass
class StepResult:
    refreshed: bool
    n_scored: int                              # tokens in the cache after the append
    keep: np.ndarray                           # [b, n_scored] bool, the retention decision
    u_pre: np.ndarray                          # [b, n_scored] utility on which the decision was taken
    s_layers: np.ndarray | None = None         # [K, b, n_scored] per-layer scores (refresh steps)
    moves: list = field(default_factory=list)  # per sequence (dst, src)
    n_out: int = 0
    raw: np.ndarray | None = None              # [b, n_scored] raw step score: mean over layers of Eq. 1
    pos_pre: np.ndarray | None = None          # [b, n_scored] positions before compaction
    o: np.ndarray | None = None                # [K, b, H_q, d] decode attention output (when asked for)
    o_scale: np.ndarray | None = None          # [K, b, H_q, d] sum_i a |v|, the output's rounding scale


def new_token_prior(u_existing: np.ndarray, refresh: bool, policy: str) -> float:
    """Prior utility of the token appended at this step.

    Refresh steps: 0, like m_0 (reading; the paper fixes only the non-refresh case).
    Non-refresh steps: mean of the existing utilities (Appendix, new-token insertion; Score-Free box:
    'current mean momentum'), or their minimum under the "min" policy.
    """
    if refresh or len(u_existing) == 0:
        return 0.0
    if policy == "mean":
        return float(np.mean(u_existing))
    if policy == "min":
        return float(np.min(u_existing))
    raise ValueError(f"unknown init policy {policy!r}")


def evict_step(cache: Cache, q: np.ndarray, k_new: np.ndarray, v_new: np.ndarray, t: int, new_pos: int,
               params: Params, keep_override: np.ndarray | None = None, attention: bool = False) -> StepResult:
    """One decode step, mutating `cache` in place.

    q: [K, b, H_q, d] raw; k_new, v_new: [K, b, H_kv, d] raw.
    1. append the new token (K/V row at slot n, its position and prior utility);
    2. on refresh steps, score every cached token layer by layer (Eq. 1) and fold (Eq. 4, layer-sequential);
    3. if more than B tokens are cached, keep the top B (ties: lower position);
    4. hole-fill compaction of K, V, u and pos.
    `attention`: also return the step's decode attention output of every layer over the n + 1 cached tokens
    (after the append, before eviction; computed on every step, refresh or not).
    `keep_override` lets a caller replace the selection by an equally valid one (used only to keep two
    implementations in lockstep after a tie inside the rounding band): either a [b, >= n] mask, or a callable
    receiving (the oracle's own [b, n] decision, the [b, n] utilities it was taken on) and returning the mask
    to apply.  The applied mask must keep exactly min(B, n) tokens per sequence.
    """
    nl, nb, hkv, cap, d = cache.k.shape
    n = cache.n
    if n + 1 > cap:
        raise ValueError("cache capacity exceeded")
    refresh = refresh_due(t, params.refresh_period, params.score_free)

    # 1. append
    for b in range(nb):
        cache.u[b, n] = new_token_prior(cache.u[b, :n], refresh, params.nonrefresh_init)
        cache.pos[b, n] = new_pos
    cache.k[:, :, :, n, :] = k_new
    cache.v[:, :, :, n, :] = v_new
    n += 1
    cache.n = n

    # decode attention of the step (the decoder runs it whether or not the step refreshes the scores)
    o_all = o_scale = None
    if attention:
        o_all = np.zeros((nl, nb, q.shape[2], d), dtype=np.float64)
        o_scale = np.zeros_like(o_all)
        for b in range(nb):
            for l in range(nl):
                o_all[l, b], o_scale[l, b] = attention_output(
                    to_f64(q[l, b], cache.dtype), to_f64(cache.k[l, b, :, :n, :], cache.dtype),
                    to_f64(cache.v[l, b, :, :n, :], cache.dtype), cache.pos[b, :n], new_pos,
                    params.recency_bias, params.recency_window)

    # 2. score + fold
    s_all = raw = None
    if refresh:
        s_all = np.zeros((nl, nb, n), dtype=np.float64)
        raw = np.zeros((nb, n), dtype=np.float64)
        for b in range(nb):
            for l in range(nl):
                keys = to_f64(cache.k[l, b, :, :n, :], cache.dtype)
                ql = to_f64(q[l, b], cache.dtype)
                plain = layer_scores(ql, keys, cache.pos[b, :n], new_pos, params.recency_bias,
                                     params.recency_window)
                raw[b] += plain / nl
                if params.vnorm or params.entropy:
                    s_all[l, b] = layer_scores_variant(ql, keys, to_f64(cache.v[l, b, :, :n, :], cache.dtype),
                                                       cache.pos[b, :n], new_pos, params.recency_bias,
                                                       params.recency_window, params.vnorm, params.entropy)
                else:
                    s_all[l, b] = plain
            cache.u[b, :n] = fold_layers(cache.u[b, :n], s_all[:, b], params.alpha, params.rule)
    u_pre = cache.u[:, :n].copy()
    pos_pre = cache.pos[:, :n].copy()

    # 3. select
    keep = np.zeros((nb, n), dtype=bool)
    for b in range(nb):
        keep[b] = select_keep(cache.u[b, :n], cache.pos[b, :n], params.budget)
    if keep_override is not None:
        if callable(keep_override):
            keep_override = keep_override(keep.copy(), u_pre.copy())
        keep_override = np.asarray(keep_override, dtype=bool)[:, :n]
        if not np.all(keep_override.sum(axis=1) == min(params.budget, n)):
            raise ValueError("override must keep exactly min(B, n) tokens per sequence")
        keep = keep_override

    # 4. compact
    moves = []
    for b in range(nb):
        dst, src = holefill_moves(keep[b], params.budget)
        cache.k[:, b, :, dst, :] = cache.k[:, b, :, src, :]
        cache.v[:, b, :, dst, :] = cache.v[:, b, :, src, :]
        cache.u[b, dst] = cache.u[b, src]
        cache.pos[b, dst] = cache.pos[b, src]
        moves.append((dst, src))
    cache.n = min(params.budget, n)
    return StepResult(refresh, n, keep, u_pre, s_all, moves, cache.n, raw, pos_pre, o_all, o_scale)


# ----------------------------------------------------------------------------------------------------------
# Appendix "Mechanistic Diagnostics": rank-trace observables of the stabilisation claim (Sec. 4, Prop. 1)
# ----------------------------------------------------------------------------------------------------------
@dataclass
class RankTraceState:
    """Previous traced step's top-k position sets of one sequence (None before the first traced step)."""
    raw: set | None = None
    ema: set | None = None


def rank_trace_counts(state: RankTraceState, raw: np.ndarray, u: np.ndarray, pos: np.ndarray, keep: np.ndarray,
                      k: int, raw_keep: np.ndarray | None = None, ema_keep: np.ndarray | None = None) -> dict:
    """Set sizes of one refresh step of one sequence, over the n tokens cached before eviction.

    R_t = top-k of the raw step score (mean over layers of the per-layer attention score, no temporal
    memory), E_t = top-k of the folded utility u, both under (value descending, position ascending) and
    identified by absolute position; `keep` is the step's retention decision.  Returns the sizes of R_t,
    E_t, R_t & R_(t-1), E_t & E_(t-1), R_t & E_t, R_t & evicted_t, R_(t-1), E_(t-1), from which
    churn = 1 - |A & A'| / |A | A'| (Jaccard) and the raw-top evicted rate = |R & evicted| / |R|.
    `raw_keep` / `ema_keep` may replace the two top-k decisions by equally valid ones (lockstep use).
    Updates `state` to this step's sets."""
    rk = select_keep(raw, pos, k) if raw_keep is None else np.asarray(raw_keep, dtype=bool)
    ek = select_keep(u, pos, k) if ema_keep is None else np.asarray(ema_keep, dtype=bool)
    R = set(int(p) for p in pos[rk])
    E = set(int(p) for p in pos[ek])
    ev = set(int(p) for p in pos[~np.asarray(keep, dtype=bool)])
    has_prev = state.raw is not None
    out = dict(r=len(R), e=len(E), has_prev=int(has_prev),
               rr=len(R & state.raw) if has_prev else 0, ee=len(E & state.ema) if has_prev else 0,
               re=len(R & E), rev=len(R & ev),
               rp=len(state.raw) if has_prev else 0, ep=len(state.ema) if has_prev else 0)
    state.raw, state.ema = R, E
    return out


def trace_metrics(c: dict) -> dict:
    """Churn, Jaccard and evicted rate from rank_trace_counts (NaN where undefined)."""
    def jac(inter, a, b):
        union = a + b - inter
        return inter / union if union else float("nan")
    nan = float("nan")
    return dict(raw_churn=1 - jac(c["rr"], c["r"], c["rp"]) if c["has_prev"] else nan,
                ema_churn=1 - jac(c["ee"], c["e"], c["ep"]) if c["has_prev"] else nan,
                raw_ema_jaccard=jac(c["re"], c["r"], c["e"]),
                raw_top_evicted=c["rev"] / c["r"] if c["r"] else nan)


def compact_rows(rows: np.ndarray, keep: np.ndarray, budget: int) -> np.ndarray:
    """Hole-fill applied to one [n_slots, ...] array (e.g. a K slab); returns a new array."""
    out = np.array(rows, copy=True)
    dst, src = holefill_moves(keep, budget)
    out[dst] = rows[src]
    return out
