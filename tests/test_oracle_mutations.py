"""Mutation check of the oracle's pins: each plausible mistake below, planted in the float64 oracle on the CPU,
must make at least one pin of tests/test_oracle_*.py fail.  A mistake that no pin catches would mean the
oracle could carry it into every parity verdict unnoticed.

Each mutant replaces one oracle function (in the oracle's module and wherever a pin module imported it by
name) for the duration of one run of every pin; the real functions are restored afterwards.  Pins are called
directly: parametrized ones over all their parameter sets, property-based ones with a reduced number of
examples, no shrinking and no example database (a failure only has to be found, not minimised)."""
import importlib
import math

import numpy as np
import pytest
from hypothesis import Phase, settings

import oracle
import oracle.inertiakv as O

PIN_MODULES = ("test_oracle_score", "test_oracle_fold", "test_oracle_select", "test_oracle_step",
               "test_oracle_attention", "test_oracle_variants", "test_oracle_trace")


# ---- the planted mistakes ----------------------------------------------------------------------------------
def gqa_interleaved(q_l, keys_l, pos=None, cur_pos=0, recency_bias=0.0, recency_window=0):
    """Query head h reads KV head h mod H_kv instead of h // G."""
    hq, hkv = q_l.shape[0], keys_l.shape[0]
    s = np.zeros(keys_l.shape[1])
    for h in range(hq):
        s += O.head_attention(q_l[h], keys_l[h % hkv], pos, cur_pos, recency_bias, recency_window)
    return s / hq


def mean_over_kv_heads(q_l, keys_l, pos=None, cur_pos=0, recency_bias=0.0, recency_window=0):
    """Eq. 1's 1/H taken as one over the KV heads."""
    hq, hkv = q_l.shape[0], keys_l.shape[0]
    group = hq // hkv
    s = np.zeros(keys_l.shape[1])
    for h in range(hq):
        s += O.head_attention(q_l[h], keys_l[h // group], pos, cur_pos, recency_bias, recency_window)
    return s / hkv


def _attention(q_h, keys_g, pos, cur_pos, bias, window, scale=True, window_extra=0, sign=1.0):
    d = q_h.shape[-1]
    z = sign * (keys_g @ q_h) / (math.sqrt(d) if scale else 1.0)
    if bias != 0.0 and window > 0:
        z = z + bias * (np.asarray(pos) >= (cur_pos - (window - 1) - window_extra))
    e = np.exp(z - z.max())
    return e / e.sum()


def unscaled_logits(q_h, keys_g, pos=None, cur_pos=0, recency_bias=0.0, recency_window=0):
    """The 1/sqrt(d) of scaled dot-product attention dropped."""
    return _attention(q_h, keys_g, pos, cur_pos, recency_bias, recency_window, scale=False)


def window_off_by_one(q_h, keys_g, pos=None, cur_pos=0, recency_bias=0.0, recency_window=0):
    """The recency bias reaches one position too far back (window + 1 positions)."""
    return _attention(q_h, keys_g, pos, cur_pos, recency_bias, recency_window, window_extra=1)


def softmax_of_negated_logits(q_h, keys_g, pos=None, cur_pos=0, recency_bias=0.0, recency_window=0):
    """The dot product's sign flipped."""
    return _attention(q_h, keys_g, pos, cur_pos, recency_bias, recency_window, sign=-1.0)


def _fold(u, s_layers, alpha, rule, swap=False, reverse=False, cum_scale=1.0, single_first=False):
    u = np.array(u, dtype=np.float64, copy=True)
    layers = list(s_layers)[::-1] if reverse else list(s_layers)
    for i, s in enumerate(layers):
        s = np.asarray(s, dtype=np.float64)
        if rule == O.EMA:
            u = (1.0 - alpha) * u + alpha * s if swap else alpha * u + (1.0 - alpha) * s
        elif rule == O.SINGLE_STEP:
            if not single_first or i == 0:
                u = np.array(s, copy=True)
        elif rule == O.CUMULATIVE:
            u = u + cum_scale * s
        else:
            raise ValueError(rule)
    return u


def alpha_swapped(u, s_layers, alpha, rule=O.EMA):
    """Eq. 4 with alpha and 1 - alpha exchanged."""
    return _fold(u, s_layers, alpha, rule, swap=True)


def layers_reversed(u, s_layers, alpha, rule=O.EMA):
    """Layers folded from the last to the first."""
    return _fold(u, s_layers, alpha, rule, reverse=True)


def cumulative_weighted(u, s_layers, alpha, rule=O.EMA):
    """Eq. 3 with each layer weighted by alpha."""
    return _fold(u, s_layers, alpha, rule, cum_scale=alpha)


def single_step_first_layer(u, s_layers, alpha, rule=O.EMA):
    """Eq. 2 keeping the first layer's score instead of the last one's."""
    return _fold(u, s_layers, alpha, rule, single_first=True)


def ties_to_higher_position(u, pos, budget):
    """Equal utilities keep the higher position."""
    n = len(u)
    keep = np.zeros(n, dtype=bool)
    if n <= budget:
        keep[:] = True
        return keep
    keep[np.lexsort((-np.asarray(pos), -np.asarray(u, dtype=np.float64)))[:budget]] = True
    return keep


def holefill_descending(keep, budget):
    """Tails paired with holes in descending order."""
    dst, src = _ORIG["holefill_moves"](keep, budget)
    return dst, src[::-1]


def refresh_index_shifted(t, period, score_free):
    """Eq. 5 read as t mod r == 0."""
    if score_free:
        return t == 1
    return t % period == 0


def refresh_every_step(t, period, score_free):
    """Lazy and Score-Free schedules ignored: every step rescored."""
    return True


def prior_on_refresh_steps(u_existing, refresh, policy):
    """The non-refresh prior also given to the token appended on refresh steps."""
    return _ORIG["new_token_prior"](u_existing, False, policy)


def priors_swapped(u_existing, refresh, policy):
    """Mean and minimum policies exchanged."""
    return _ORIG["new_token_prior"](u_existing, refresh, {"mean": "min", "min": "mean"}[policy])


def budget_rounded_up(prefill_len, compression_ratio):
    """B = ceil((1 - rho) L0)."""
    return int(math.ceil((1.0 - compression_ratio) * prefill_len - 1e-9))


def bf16_read_as_f16(raw, dtype):
    """bf16 bit patterns decoded as IEEE half precision."""
    if dtype == O.BF16:
        return np.asarray(raw, dtype=np.uint16).view(np.float16).astype(np.float64)
    return _ORIG["to_f64"](raw, dtype)


def vnorm_unnormalised(values_g):
    """VNorm factor = the raw value norm, not divided by the mean norm."""
    return np.sqrt(np.sum(values_g * values_g, axis=-1))


def entropy_wrong_maximum(s):
    """Normalised entropy divided by ln(n + 1) instead of ln(n)."""
    n = len(s)
    if n <= 1:
        return 1.0
    p = s / s.sum()
    nz = p > 0
    return float(-np.sum(p[nz] * np.log(p[nz])) / math.log(n + 1))


def attention_values_interleaved(q_l, keys_l, values_l, pos=None, cur_pos=0, recency_bias=0.0, recency_window=0):
    """The output of head h reads the value rows of KV head h mod H_kv."""
    hq, hkv = q_l.shape[0], keys_l.shape[0]
    group = hq // hkv
    o = np.zeros((hq, values_l.shape[-1]))
    scale = np.zeros_like(o)
    for h in range(hq):
        a = O.head_attention(q_l[h], keys_l[h // group], pos, cur_pos, recency_bias, recency_window)
        o[h] = a @ values_l[h % hkv]
        scale[h] = a @ np.abs(values_l[h % hkv])
    return o, scale


def trace_union_for_intersection(state, raw, u, pos, keep, k, raw_keep=None, ema_keep=None):
    """|R & E| counted as |R | E|."""
    out = _ORIG["rank_trace_counts"](state, raw, u, pos, keep, k, raw_keep, ema_keep)
    out["re"] = out["r"] + out["e"] - out["re"]
    return out


MUTANTS = [
    ("layer_scores", gqa_interleaved),
    ("layer_scores", mean_over_kv_heads),
    ("head_attention", unscaled_logits),
    ("head_attention", window_off_by_one),
    ("head_attention", softmax_of_negated_logits),
    ("fold_layers", alpha_swapped),
    ("fold_layers", layers_reversed),
    ("fold_layers", cumulative_weighted),
    ("fold_layers", single_step_first_layer),
    ("select_keep", ties_to_higher_position),
    ("holefill_moves", holefill_descending),
    ("refresh_due", refresh_index_shifted),
    ("refresh_due", refresh_every_step),
    ("new_token_prior", prior_on_refresh_steps),
    ("new_token_prior", priors_swapped),
    ("budget_from_ratio", budget_rounded_up),
    ("to_f64", bf16_read_as_f16),
    ("value_norm_weights", vnorm_unnormalised),
    ("normalized_entropy", entropy_wrong_maximum),
    ("attention_output", attention_values_interleaved),
    ("rank_trace_counts", trace_union_for_intersection),
]
_ORIG = {name: getattr(O, name) for name, _ in MUTANTS}


# ---- running the pins ----------------------------------------------------------------------------------------
def _run_fast(fn):
    """A property-based pin with fewer examples, no shrinking and no example database (its own settings are
    put back afterwards)."""
    own = fn._hypothesis_internal_use_settings
    fn._hypothesis_internal_use_settings = settings(own, max_examples=60, database=None, deadline=None,
                                                    phases=[Phase.explicit, Phase.generate])
    try:
        fn()
    finally:
        fn._hypothesis_internal_use_settings = own


def _pin_calls():
    """(name, zero-argument callable) for every pin function of the oracle's test modules."""
    calls = []
    for modname in PIN_MODULES:
        mod = importlib.import_module(modname)
        for name, fn in sorted(vars(mod).items()):
            if not name.startswith("test_") or not callable(fn):
                continue
            if getattr(fn, "is_hypothesis_test", False):
                calls.append((f"{modname}.{name}", lambda fn=fn: _run_fast(fn)))
                continue
            marks = [m for m in getattr(fn, "pytestmark", []) if m.name == "parametrize"]
            if not marks:
                calls.append((f"{modname}.{name}", fn))
                continue
            argnames, values = marks[0].args[0], marks[0].args[1]
            names = [a.strip() for a in argnames.split(",")] if isinstance(argnames, str) else list(argnames)
            for v in values:
                v = v if len(names) > 1 else (v,)
                calls.append((f"{modname}.{name}{list(v)}", lambda fn=fn, v=v, names=names: fn(**dict(zip(names, v)))))
    return calls


class _Planted:
    """Replaces oracle function `name` by `fn` in the oracle and in every pin module that imported it."""

    def __init__(self, name, fn):
        self.name, self.fn = name, fn
        self.mods = [O, oracle] + [importlib.import_module(m) for m in PIN_MODULES]

    def __enter__(self):
        self.undo = [(m, getattr(m, self.name)) for m in self.mods if getattr(m, self.name, None) is _ORIG[self.name]]
        for m, _ in self.undo:
            setattr(m, self.name, self.fn)

    def __exit__(self, *exc):
        for m, orig in self.undo:
            setattr(m, self.name, orig)
        return False


def _failing_pins(calls):
    failed = []
    for name, call in calls:
        try:
            with np.errstate(all="ignore"):
                call()
        except Exception:  # noqa: BLE001 - any failure (assertion or error) counts as caught
            failed.append(name)
    return failed


def test_pins_pass_on_the_real_oracle():
    """The harness itself: every pin passes when nothing is planted."""
    assert _failing_pins(_pin_calls()) == []


@pytest.mark.parametrize("target,mutant", MUTANTS, ids=[m.__name__ for _, m in MUTANTS])
def test_planted_mistake_is_caught(target, mutant):
    calls = _pin_calls()
    with _Planted(target, mutant):
        failed = _failing_pins(calls)
    assert failed, f"no pin catches the planted mistake {mutant.__name__} in {target}: {mutant.__doc__}"
    print(f"{mutant.__name__}: caught by {len(failed)} pins, e.g. {failed[:3]}")
