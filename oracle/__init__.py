"""Float64 CPU oracle of the InertiaKV decode-step eviction path.

Test infrastructure only: the test-suite, the smoke check and the benchmark's CPU-baseline leg import it;
the HIP library and its binding never do, and the two share no code.
"""
from .inertiakv import (  # noqa: F401
    BF16, CUMULATIVE, EMA, F32, SINGLE_STEP, Cache, Params, StepResult, attention_output, budget_from_ratio,
    compact_rows, layer_scores_variant, normalized_entropy, value_norm_weights, RankTraceState, rank_trace_counts,
    trace_metrics,
    evict_step, fold_layers, head_attention, holefill_moves, layer_scores, new_token_prior, refresh_due,
    select_keep, to_f64,
)
