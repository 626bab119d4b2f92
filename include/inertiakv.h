/*
 * inertiakv.h - C ABI of the InertiaKV / InertiaKV-Lazy decode-step KV-eviction path on one MI355X (gfx950).
 *
 * Method: "What Matters for Aggressive Decoding-Time KV Eviction? Temporal Aggregation and Ranking
 * Preservation".  Every decode step appends one token to a KV cache; on refresh steps every cached token is
 * scored by the last query's softmax attention, mean-pooled over query heads (Eq. 1; GQA groups share their KV
 * head, implementation appendix "Per-step scoring"), and the scores of layers 1..K are folded in order into one
 * utility per token, u <- alpha u + (1 - alpha) s_l (Eq. 4 and appendix "Layer scoring").  Whenever the cache
 * holds more than B tokens the lowest utilities are evicted (Sec. 3), ties going to the higher position, and the
 * retained K/V rows are compacted.  Lazy refresh (Eq. 5) scores only on steps t with (t - 1) mod R == 0;
 * Score-Free (Sec. 3.2) scores only at t = 1.  Off the refresh set the new token starts at the mean (or, as an
 * option, the minimum) of the existing utilities (appendix "New token insertion") and eviction uses the stale
 * ranking (appendix "Eviction on non-refresh steps").
 *
 * Conventions for every call
 *  - Buffer pointers are DEVICE pointers owned by the caller; the library never allocates, frees or
 *    synchronises device memory and never reads them on the host.  Scratch comes from a caller workspace of
 *    at least kv_workspace_bytes() bytes, 256-byte aligned; calls that share a workspace must not overlap in
 *    time.  The workspace's first 4 bytes are its sticky fault word (kv_fault bits, set by the device when a
 *    call could not produce valid results): zero it once after allocating the workspace (kv_fault_status with
 *    clear, or any zero fill) and read it with kv_fault_status.  The rest needs no initialisation.
 *  - Work is queued asynchronously on `stream` (a hipStream_t; NULL = the default stream) in stream order.
 *  - Arguments are validated on the host before anything is queued; an invalid call returns a negative
 *    kv_status and queues nothing.  KV_ERR_HIP reports a failed launch (hipGetLastError).
 *  - Layouts (row-major, innermost last; d = head_dim, cap = capacity):
 *      K, V cache  [layers][batch][n_kv_heads][cap][d]   dtype (f32 or bf16), rows [0, n) in use
 *      q           [layers][batch][n_q_heads][d]         dtype, the current query of every head and layer
 *      k_new,v_new [layers][batch][n_kv_heads][d]        dtype, the token appended at this step
 *      u           [batch][cap] float                    utility per cached token
 *      pos         [batch][cap] int32                    absolute position per cached token (unique, >= 0)
 *      keep        [batch][cap] uint8                    1 = retained (first n entries written)
 *      s_out       [layers][batch][n] float              per-layer pooled score s_l (optional, may be NULL)
 *      v_norms     [layers][batch][n_kv_heads][cap] float  optional value-norm cache (see kv_value_norms)
 *    Query head h reads KV head h / (n_q_heads / n_kv_heads).  Every sequence holds the same n tokens.
 *  - Preconditions not checked on the device: keys, queries and utilities are finite; utilities are >= 0
 *    when produced by this library; positions are unique within a sequence.
 *  - The calls keep no state between calls (apart from per-device caches of kernel attributes and occupancy,
 *    filled on first use under atomics, and the exchange wait limit below) and may run concurrently, from
 *    several host threads, on different streams with disjoint buffers and workspaces, with one exception: a
 *    refresh step whose slabs are too long for one workgroup's LDS (kv_score_plan reports path
 *    KV_PATH_EXCHANGE, e.g. the first decode step over a 32k-token prefill) scores them with chunks that wait
 *    for one another's softmax statistics, on a grid sized to the workgroups the device holds at once.  Such a
 *    call needs the device to itself while it runs: when other work (another stream or process) holds CUs,
 *    a slab's later chunks may not start while its earlier ones wait.  Every wait is bounded; a chunk that
 *    gives up sets its scores to NaN and raises KV_FAULT_EXCHANGE_TIMEOUT in the workspace's fault word.
 */
#ifndef INERTIAKV_H
#define INERTIAKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    KV_OK = 0,
    KV_ERR_INVALID_ARG = -1, /* null pointer, bad size, n out of range, alpha outside [0, 1), ...        */
    KV_ERR_UNSUPPORTED = -2, /* head_dim not 64/128, group size > 16, dtype not f32/bf16, misalignment   */
    KV_ERR_WORKSPACE = -3,   /* workspace missing or smaller than kv_workspace_bytes()                   */
    KV_ERR_HIP = -4          /* a kernel launch failed                                                    */
} kv_status;

typedef enum { KV_F32 = 0, KV_BF16 = 1 } kv_dtype;

/* Bits of the workspace's fault word.  KV_FAULT_EXCHANGE_TIMEOUT: a chunk of a long-slab scorer (path
 * KV_PATH_EXCHANGE) did not receive its peers' softmax statistics within the wait limit; its scores, and
 * everything computed from them by that call (utilities, retention decision, compaction), are invalid. */
typedef enum { KV_FAULT_EXCHANGE_TIMEOUT = 1 } kv_fault;

/* Prior utility of the token appended on a NON-refresh step (appendix "New token insertion": MEAN). */
typedef enum { KV_INIT_MEAN = 0, KV_INIT_MIN = 1 } kv_init;

/* Aggregation rule (Eq. 2-4), applied layer by layer: EMA u <- alpha u + (1-alpha) s_l; single-step u <- s_l;
 * cumulative u <- u + s_l. */
typedef enum { KV_RULE_EMA = 0, KV_RULE_SINGLE_STEP = 1, KV_RULE_CUMULATIVE = 2 } kv_rule;

/* Scorer perturbations of Sec. 5.1 (implementation appendix "Per-step scoring"), a bit mask applied to the
 * score of every refresh step before the fold (kv_evict_step, kv_evict_finish; kv_score_ema is plain Eq. 1):
 *  KV_SCORE_VNORM:   head h's attention to token i is multiplied by |v_i| / mean_j |v_j|, the l2 norm of
 *                    token i's value row under h's KV head over the mean of those norms over the n cached
 *                    tokens of that layer and KV head (factor 1 if all those norms are zero);
 *  KV_SCORE_ENTROPY: the layer's pooled score is multiplied by the entropy of the layer's pooled attention
 *                    distribution (before VNorm) divided by ln n, one factor per layer and sequence (1 if
 *                    n = 1).  s_out then holds the perturbed scores that were folded. */
typedef enum {
    KV_SCORE_ATTENTION = 0,
    KV_SCORE_VNORM = 1,
    KV_SCORE_ENTROPY = 2,
    /* kv_evict_finish only, with KV_SCORE_VNORM: the step's attention calls emitted the value norms
     * (KV_EMIT_VNORMS), so V is not read again */
    KV_SCORE_NORMS_EMITTED = 4
} kv_score_variant;

typedef struct {
    int32_t batch;      /* sequences                                   >= 1              */
    int32_t layers;     /* eligible layers K, folded in ascending order 1..256           */
    int32_t n_q_heads;  /* query heads H (Eq. 1)                       multiple of n_kv  */
    int32_t n_kv_heads; /* KV heads; group size n_q/n_kv <= 16                           */
    int32_t head_dim;   /* 64 or 128                                                     */
    int32_t capacity;   /* rows per (layer, sequence, KV head) slab                      */
    int32_t dtype;      /* kv_dtype of q, K, V, k_new, v_new                              */
} kv_shape;

typedef struct {
    float alpha;            /* EMA coefficient, 0 <= alpha < 1 (alpha = 0: last layer only)        */
    int32_t budget;         /* B >= 1: tokens kept whenever more are cached                         */
    int32_t refresh_period; /* R >= 1: refresh iff (t - 1) mod R == 0 (Eq. 5); 1 = full refresh     */
    int32_t score_free;     /* nonzero: refresh only at t = 1 (Score-Free)                          */
    int32_t nonrefresh_init;/* kv_init                                                             */
    float recency_bias;     /* added to logits of the `recency_window` newest positions; 0 = off    */
    int32_t recency_window; /* positions p >= new_pos - (window - 1) get the bias                   */
    int32_t rule;           /* kv_rule                                                             */
    int32_t score_variant;  /* kv_score_variant bits (0 = the attention score of Eq. 1)             */
    int32_t score_merge;    /* performance only (the same sums added in another order: results agree
                               to rounding): KV heads of one (layer, sequence) whose group sums one
                               scoring workgroup, or one team of chunks exchanging their statistics,
                               adds before writing them.  0 = chosen from the shape and the device;
                               else a divisor of n_kv_heads, at most 8, and 1 with VNorm.  Long slabs
                               scored by chunks that write logits keep 1.  kv_evict_finish must be
                               given the value the separate step would use.                        */
} kv_params;

/* Optional timing hooks: when an entry is non-NULL, kv_evict_step records that hipEvent_t on its stream
 * immediately before (begin) / after (end) the kernels of the phase.  Phases: 0 append, 1 score, 2 fold,
 * 3 select, 4 compact.  On a refresh step over a cache of at most B tokens (without a rank trace, and with
 * the value-norm cache when VNorm is on) the newcomer is scored from k_new and written once, into the slot it
 * takes: phase 3 then times the selection with that placement, and phases 0 and 4 record their events back
 * to back. */
#define KV_PHASES 5
typedef struct {
    void* begin[KV_PHASES];
    void* end[KV_PHASES];
} kv_trace;

/* Rank trace (appendix "Mechanistic Diagnostics"): observables of how stable the ranking is, taken on every
 * refresh step over the n tokens cached before that step's eviction.  R_t = top-k of the raw step score
 * (the plain per-layer score of Eq. 1 averaged over layers: no memory), E_t = top-k of the folded utility,
 * both ordered by (value descending, position ascending) and identified by absolute position.  counts[b]
 * receives, per sequence:
 *   [0] 1 = traced, 0 = not a refresh step (nothing else written, state unchanged), -2 = a position outside
 *       [0, max_pos) was in a set (not recorded);
 *   [1] |R_t|  [2] |E_t|  [3] 1 if a previous traced step exists  [4] |R_t & R_t-1|  [5] |E_t & E_t-1|
 *   [6] |R_t & E_t|  [7] |R_t & evicted_t|  [8] |R_t-1|  [9] |E_t-1|
 * so that churn = 1 - |A & A'| / (|A| + |A'| - |A & A'|), raw/EMA Jaccard = [6] / ([1] + [2] - [6]) and the
 * raw-top evicted rate = [7] / [1].  `state` carries the previous sets (position bitmaps) between steps; it
 * must be zero-filled before a sequence's first traced step. */
#define KV_TRACE_COUNTS 10
typedef struct {
    int32_t k;          /* size of the traced top-k sets, >= 1 (e.g. the budget B)                  */
    int32_t max_pos;    /* every traced position must be < max_pos                                   */
    uint32_t* state;    /* DEVICE, kv_rank_trace_state_bytes() bytes                                 */
    int32_t* counts;    /* DEVICE [batch][KV_TRACE_COUNTS]                                           */
    uint8_t* raw_keep;  /* nullable DEVICE [batch][cap]: R_t as a mask over the pre-eviction slots    */
    uint8_t* ema_keep;  /* nullable DEVICE [batch][cap]: E_t as a mask over the pre-eviction slots    */
} kv_rank_trace;

/* Bytes of rank-trace state for `batch` sequences and positions < max_pos (host only). */
kv_status kv_rank_trace_state_bytes(int32_t batch, int32_t max_pos, size_t* bytes);

/* Bytes of workspace needed by every call below for any n <= n_max cached tokens (host only). */
kv_status kv_workspace_bytes(const kv_shape* shape, int32_t n_max, size_t* bytes);

/* The params->score_merge that kv_evict_step resolves for a refresh step over n cached tokens (after the
 * append) on the current device: KV heads whose group sums one scoring workgroup (or one team of chunks that
 * exchange their statistics, path KV_PATH_EXCHANGE below) adds, in KV-head order (1 for VNorm and for slabs
 * scored by chunks that write logits; a positive params->score_merge is returned as given when it applies).
 * Exception: a steady VNorm step given the value-norm cache, without entropy weighting and without a forced
 * merge, weights the sums inside the scorer and keeps a planned merge where its shape allows (vector-form
 * logits, LDS room); this call reports 1 for it.  Host only; the automatic choice reads the device's CU count.
 * KV_ERR_INVALID_ARG as kv_evict_step for bad params. */
kv_status kv_score_merge(const kv_shape* shape, int32_t n, const kv_params* params, int32_t* merge);

/* How a refresh step over n cached tokens (after the append) scores them on the current device (host only):
 * merge as kv_score_merge; path KV_PATH_LDS (one workgroup per slab, logits in LDS), KV_PATH_EXCHANGE (slabs
 * too long for that, cut into `chunks` chunks that exchange their softmax statistics: see the concurrency
 * note above) or KV_PATH_LOGITS (chunks that write their logits to the workspace for a finish pass: slabs with
 * more statistics than one exchange grid handles); chunks = workgroups per slab. */
typedef enum { KV_PATH_LDS = 0, KV_PATH_EXCHANGE = 1, KV_PATH_LOGITS = 2 } kv_score_path;
typedef struct {
    int32_t merge;
    int32_t path;
    int32_t chunks;
} kv_score_info;
kv_status kv_score_plan(const kv_shape* shape, int32_t n, const kv_params* params, kv_score_info* info);

/* Fault word of a workspace (see the conventions above), in stream order: *out (DEVICE, nullable) receives
 * the kv_fault bits set since the word was last cleared; clear != 0 then zeroes the word.  Asynchronous like
 * every call: read *out after synchronising the stream.  KV_ERR_INVALID_ARG when out is NULL and clear is 0. */
kv_status kv_fault_status(void* ws, size_t ws_bytes, uint32_t* out, int32_t clear, void* stream);

/* Polls a waiting chunk of the exchange path makes before it gives up (process-wide; default, or polls < 0:
 * about 0.1 s of sleeps, far beyond any chunk's streaming time; 0: give up without waiting, every chunk then
 * reports KV_FAULT_EXCHANGE_TIMEOUT).  For tests of the fault report.  Returns the previous limit. */
int32_t kv_set_exchange_wait_limit(int32_t polls);

/* Scoring + fold (Eq. 1 and Eq. 4, layer-sequential).  For every layer l = 1..K, query head h and cached
 * token i < n: z_h(i) = q_h . k_i / sqrt(d) (+ recency_bias if pos[i] >= cur_pos - (recency_window - 1)),
 * a_h = softmax over the n tokens, s_l(i) = (1/H) sum_h a_h(i); then u <- alpha u + (1 - alpha) s_l for
 * l = 1..K in order (u updated in place for i < n; entries >= n untouched).  s_out (nullable) receives s_l. */
kv_status kv_score_ema(const kv_shape* shape, int32_t n, const void* q, const void* k, const int32_t* pos,
                       int32_t cur_pos, float alpha, float recency_bias, int32_t recency_window, float* u,
                       float* s_out, void* ws, size_t ws_bytes, void* stream);

/* Top-B selection (Sec. 3): keep[b][i] = 1 for the min(B, n) tokens first under (u descending, position
 * ascending), 0 for the others, for i < n. */
kv_status kv_topk_select(const kv_shape* shape, int32_t n, int32_t budget, const float* u, const int32_t* pos,
                         uint8_t* keep, void* ws, size_t ws_bytes, void* stream);

/* Value-norm cache for VNorm (Sec. 5.1; implementation appendix "Per-step scoring": VNorm weights a token's
 * attention by the l2 norm of its value row over the mean norm of the cached tokens of that layer and KV head).
 * A value row never changes once cached, it only moves, so its norm can be computed once: kv_value_norms
 * fills v_norms[l][b][g][i] = |V[l][b][g][i]| for the rows i < n of every slab (once, after the prefill).
 * Every call below that takes a non-NULL v_norms keeps it in step with V: the appended token's norm is written
 * where its V row goes, and the compaction moves norms with their rows.  VNorm refresh steps given v_norms read
 * the cached norms (4 bytes per row) instead of V (d elements per row), and the steady refresh step then keeps
 * its three-kernel form.  Rows of v_norms at and beyond the cache's n are unspecified, like those of V. */
kv_status kv_value_norms(const kv_shape* shape, int32_t n, const void* v, float* v_norms, void* stream);

/* Hole-fill compaction of a retention decision (which must keep exactly min(B, n) tokens per sequence).
 * Sec. 3: eviction is irreversible, the evicted tokens' K/V pairs leave the cache and the retained ones stay;
 * the paper leaves the row layout open (attention does not depend on row order), and this call reads it as
 * the layout that moves the fewest rows: with k = min(B, n), the kept rows in slots >= k move, in ascending
 * order, into the dropped slots < k, in ascending order, for every layer and KV head of K and V, and for u
 * and pos.  Rows [0, k) then hold exactly the retained tokens; rows >= k are left as they were.  A mask that
 * keeps a different count is rejected on the device by moving nothing beyond the smaller of the two lists. */
kv_status kv_compact(const kv_shape* shape, int32_t n, int32_t budget, const uint8_t* keep, void* k, void* v,
                     float* u, int32_t* pos, float* v_norms, void* ws, size_t ws_bytes, void* stream);

/* One decode step t >= 1 on a cache of n_in tokens (n_in + 1 <= capacity):
 *  1. append k_new/v_new at slot n_in, pos = new_pos, u = 0 on refresh steps, else the mean (or min) of the
 *     n_in existing utilities;
 *  2. refresh steps only: kv_score_ema over the n_in + 1 tokens with q, cur_pos = new_pos;
 *  3. if n_in + 1 > B: select the top B (stale utilities on non-refresh steps) and compact as kv_compact.
 * *n_out (HOST pointer) receives min(B, n_in + 1); cache rows at and beyond *n_out are unspecified
 * afterwards.  v_norms (nullable) is the value-norm cache, kept in step and read by VNorm; keep_out (nullable)
 * receives the decision over the n_in + 1 slots before compaction; s_out (nullable) the per-layer scores of a
 * refresh step; trace (nullable) timing events; rank_trace (nullable) the diagnostics above. */
kv_status kv_evict_step(const kv_shape* shape, const kv_params* params, int32_t t, int32_t n_in,
                        int32_t new_pos, const void* q, const void* k_new, const void* v_new, void* k, void* v,
                        float* u, int32_t* pos, float* v_norms, int32_t* n_out, uint8_t* keep_out, float* s_out,
                        const kv_trace* trace, const kv_rank_trace* rank_trace, void* ws, size_t ws_bytes,
                        void* stream);

/* ---- Allocation-free decode step: for callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops that forbid allocation) ----
 * kv_evict_step without the workspace: its scratch is a static device array inside the library of
 * KV_STATIC_SCRATCH_BYTES per device (one copy on each GPU the library runs on, held until the process ends;
 * no call allocates or frees anything).  Supported steps: those whose slabs are scored in one workgroup each
 * (kv_score_plan path KV_PATH_LDS on refresh steps; any non-refresh step) and whose scratch fits (the
 * workspace of kv_evict_step without the regions of chunked scoring and of the attention calls: e.g. every
 * steady step of a batch-8, 32-layer, 8-KV-head cache of ~3,300 tokens).  Otherwise, before anything is
 * queued: KV_ERR_UNSUPPORTED (chunked scoring, e.g. a first step over a long prefill: use kv_evict_step) or
 * KV_ERR_WORKSPACE (scratch too small).  Every call on one device shares that device's scratch, which keeps
 * the last call's contents: calls that overlap in time on one GPU (several streams or host threads) race, and
 * the caller must serialise them.  Arguments and results are kv_evict_step's. */
#define KV_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
kv_status kv_evict_step_static(const kv_shape* shape, const kv_params* params, int32_t t, int32_t n_in,
                               int32_t new_pos, const void* q, const void* k_new, const void* v_new, void* k,
                               void* v, float* u, int32_t* pos, float* v_norms, int32_t* n_out, uint8_t* keep_out,
                               float* s_out, const kv_trace* trace, const kv_rank_trace* rank_trace, void* stream);

/* ---- Decode step around the model's own attention (fused decode attention + score) ----
 * A decoder that attends the cache anyway can take the step's score from its attention (Eq. 1 is the softmax
 * of the last query, the one that produces the attention output): K is then read once for both, instead of
 * once by attention and again by a separate scoring pass (the paper profiles that reconstruction as the
 * dominant per-step cost, appendix "Hook-level profiling").  A step t is
 *     kv_append(t) ; kv_attend_score(layers ...) over every layer, emit_scores = refresh step ;
 *     kv_evict_finish(t)
 * and leaves the cache, u and pos as kv_evict_step would: bit for bit when each slab of an attention call is
 * one workgroup (the scorer's arithmetic in its order, e.g. all layers of a steady step in one call), else with
 * scores that agree to rounding (a slab cut into row chunks whose statistics a second kernel combines).
 * All three calls of a step use the same workspace (the group sums of each layer live in it between the
 * attention calls and the finish), sized by kv_workspace_bytes for at least n_in + 1 tokens.
 *
 * kv_append: step 1 of kv_evict_step alone (appendix "New token insertion"; the refresh decision of Eq. 5
 * picks the prior: 0 on refresh steps, else the mean or min of the existing utilities); v_norms (nullable)
 * receives the new row's value norm. */
kv_status kv_append(const kv_shape* shape, const kv_params* params, int32_t t, int32_t n_in, int32_t new_pos,
                    const void* k_new, const void* v_new, void* k, void* v, float* u, int32_t* pos, float* v_norms,
                    void* stream);

/* What kv_attend_score records in the workspace besides the output (bit mask): the layers' pooled scores
 * (Eq. 1), and the value-row norms that VNorm weights them by (read from V while the attention streams it). */
typedef enum { KV_EMIT_SCORES = 1, KV_EMIT_VNORMS = 2 } kv_emit;

/* Decode attention of layers [layer0, layer0 + layer_count) over the n cached tokens, for every sequence and
 * query head: a_h = softmax_i(z_h(i)) with z_h(i) = q_h . k_i / sqrt(d) (+ recency_bias if
 * pos[i] >= cur_pos - (recency_window - 1)), o_h = sum_i a_h(i) v_i.  q and o are [layer_count][batch]
 * [n_q_heads][d] in the cache dtype (o rounded to nearest); k, v are the whole caches (layer 0 at the
 * pointer).  emit_scores (kv_emit bits) additionally records these layers' pooled scores (Eq. 1) and/or value
 * norms in the workspace for kv_evict_finish; layers whose scores are not emitted keep whatever the workspace
 * held.  Layers may be attended in any number of calls (one per layer in a decoder). */
kv_status kv_attend_score(const kv_shape* shape, int32_t layer0, int32_t layer_count, int32_t n, const void* q,
                          const void* k, const void* v, const int32_t* pos, int32_t cur_pos, float recency_bias,
                          int32_t recency_window, int32_t emit_scores, void* o, void* ws, size_t ws_bytes,
                          void* stream);

/* Steps 2-3 of kv_evict_step after the attention calls: on refresh steps (Eq. 5) the layer fold of the
 * emitted scores of ALL layers (Eq. 4 by params->rule), then the top-B selection and compaction over the n
 * cached tokens (n = n_in + 1 of the step).  *n_out (HOST) = min(B, n); v_norms / keep_out / s_out / rank_trace
 * as kv_evict_step (VNorm takes the norms the attention emitted when KV_SCORE_NORMS_EMITTED is set, else those
 * of v_norms, else reads V). */
kv_status kv_evict_finish(const kv_shape* shape, const kv_params* params, int32_t t, int32_t n, void* k, void* v,
                          float* u, int32_t* pos, float* v_norms, int32_t* n_out, uint8_t* keep_out, float* s_out,
                          const kv_rank_trace* rank_trace, void* ws, size_t ws_bytes, void* stream);

/* Static description of a status code. */
const char* kv_status_string(kv_status status);

#ifdef __cplusplus
}
#endif

#endif /* INERTIAKV_H */
