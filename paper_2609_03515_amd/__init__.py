"""InertiaKV / InertiaKV-Lazy decode-step KV eviction on MI355X (gfx950): HIP kernels behind a C ABI.

`binding` wraps the C entry points of libinertiakv.so (kv_score_ema, kv_topk_select, kv_compact,
kv_evict_step, kv_append, kv_attend_score, kv_evict_finish, kv_rank_trace_state_bytes) and a cache-level
`evict_step(cache, q, k_new, v_new, t, params, new_pos)` over a `KvCache`; `build` compiles the
library with hipcc.  The library is loaded on first use and its absence
is an error.
"""
