// C ABI of the eviction path: argument validation, workspace layout and the launch sequence of a decode
// step.  Everything is queued on the caller's stream; nothing is allocated, synchronised or read back.
#include <math.h>
#include <string.h>

#include "../../include/inertiakv.h"
#include "kernels.h"
#include "kv_common.h"

namespace ikv {
namespace {

struct Layout {
    int n_stride;
    int max_pairs;
    ScorePlan plan;
    size_t r_off, z_off, part_off, pdst_off, psrc_off, np_off, total;
};

int esize(const kv_shape& s) { return s.dtype == KV_F32 ? 4 : 2; }

kv_status check_shape(const kv_shape* s) {
    if (!s) return KV_ERR_INVALID_ARG;
    if (s->batch < 1 || s->layers < 1 || s->n_q_heads < 1 || s->n_kv_heads < 1 || s->capacity < 1)
        return KV_ERR_INVALID_ARG;
    if (s->layers > kMaxLayers) return KV_ERR_UNSUPPORTED;
    if (s->n_q_heads % s->n_kv_heads) return KV_ERR_INVALID_ARG;
    if (s->dtype != KV_F32 && s->dtype != KV_BF16) return KV_ERR_UNSUPPORTED;
    if (s->head_dim != 64 && s->head_dim != 128) return KV_ERR_UNSUPPORTED;
    const int group = s->n_q_heads / s->n_kv_heads;
    ScorePlan p;
    if (!score_plan(s->dtype, s->head_dim, group, 1, &p)) return KV_ERR_UNSUPPORTED;
    // every index fits the kernels' arithmetic: slab offsets are 64-bit, row counts 32-bit
    const double elems = (double)s->layers * s->batch * s->n_kv_heads * s->capacity * s->head_dim;
    if (elems > 9.0e15 || (double)s->batch * s->capacity > 2.0e9) return KV_ERR_UNSUPPORTED;
    return KV_OK;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

Layout layout_for(const kv_shape& s, int n) {
    Layout L{};
    L.n_stride = (n + 63) / 64 * 64;
    L.max_pairs = n;
    score_plan(s.dtype, s.head_dim, s.n_q_heads / s.n_kv_heads, n, &L.plan);
    size_t off = 0;
    L.r_off = off;
    off = align256(off + (size_t)s.layers * s.batch * s.n_kv_heads * L.n_stride * sizeof(float));
    L.z_off = off;
    if (L.plan.split) {
        off = align256(off + (size_t)s.layers * s.batch * s.n_q_heads * L.n_stride * sizeof(float));
        L.part_off = off;
        off = align256(off + (size_t)s.layers * s.batch * s.n_q_heads * L.plan.nchunk * sizeof(float2));
    } else {
        L.part_off = off;
    }
    L.pdst_off = off;
    off = align256(off + (size_t)s.batch * L.max_pairs * sizeof(int32_t));
    L.psrc_off = off;
    off = align256(off + (size_t)s.batch * L.max_pairs * sizeof(int32_t));
    L.np_off = off;
    off = align256(off + (size_t)s.batch * sizeof(int32_t));
    L.total = off;
    return L;
}

template <typename T>
T* at(void* ws, size_t off) {
    return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

kv_status check_ws(const Layout& L, void* ws, size_t ws_bytes) {
    if (!ws || ws_bytes < L.total) return KV_ERR_WORKSPACE;
    if (!aligned(ws, 256)) return KV_ERR_INVALID_ARG;
    return KV_OK;
}

kv_status hip_status(hipError_t e) { return e == hipSuccess ? KV_OK : KV_ERR_HIP; }

void record(const kv_trace* tr, int phase, bool begin, hipStream_t s) {
    if (!tr) return;
    void* ev = begin ? tr->begin[phase] : tr->end[phase];
    if (ev) (void)hipEventRecord(static_cast<hipEvent_t>(ev), s);
}

// Scoring (Eq. 1) of rows [0, n) into the workspace r, then the layer fold into u.
kv_status run_score_fold(const kv_shape& s, const Layout& L, int n, const void* q, const void* k,
                         const int32_t* pos, int cur_pos, float recency_bias, int recency_window, float* u,
                         float* s_out, int rule, float alpha, void* ws, hipStream_t st, const kv_trace* tr) {
    ScoreArgs a{};
    a.q = q;
    a.k = k;
    a.pos = pos;
    a.r = at<float>(ws, L.r_off);
    a.z = at<float>(ws, L.z_off);
    a.part = at<float2>(ws, L.part_off);
    a.batch = s.batch;
    a.layers = s.layers;
    a.hq = s.n_q_heads;
    a.hkv = s.n_kv_heads;
    a.group = s.n_q_heads / s.n_kv_heads;
    a.cap = s.capacity;
    a.n = n;
    a.n_stride = L.n_stride;
    a.recent_from = cur_pos - (recency_window - 1);
    a.bias = recency_window > 0 ? recency_bias : 0.0f;
    a.scale = (float)(1.0 / sqrt((double)s.head_dim));
    a.chunk_rows = L.plan.chunk_rows;
    a.nchunk = L.plan.nchunk;
    ScorePlan plan = L.plan;
    plan.grid = s.layers * s.batch * s.n_kv_heads * plan.nchunk;

    record(tr, 1, true, st);
    kv_status rc = hip_status(launch_score(s.dtype, s.head_dim, plan, a, st));
    if (rc == KV_OK && plan.split) rc = hip_status(launch_split_finish(a, st));
    record(tr, 1, false, st);
    if (rc != KV_OK) return rc;

    FoldArgs f{};
    f.r = a.r;
    f.u = u;
    f.s_out = s_out;
    f.batch = s.batch;
    f.layers = s.layers;
    f.hkv = s.n_kv_heads;
    f.n = n;
    f.n_stride = L.n_stride;
    f.cap = s.capacity;
    f.inv_hq = 1.0f / (float)s.n_q_heads;
    // Weights of the layer-sequential rule: EMA gives alpha^K to the prior and (1-alpha) alpha^(K-l) to
    // layer l; single-step keeps only the last layer; cumulative adds every layer to the prior.
    const int K = s.layers;
    if (rule == KV_RULE_EMA) {
        double w = 1.0;
        for (int l = K - 1; l >= 0; --l) {
            f.w[l] = (float)((1.0 - alpha) * w);
            w *= alpha;
        }
        f.prior_w = (float)w;
    } else if (rule == KV_RULE_SINGLE_STEP) {
        for (int l = 0; l < K; ++l) f.w[l] = l == K - 1 ? 1.0f : 0.0f;
        f.prior_w = 0.0f;
    } else {
        for (int l = 0; l < K; ++l) f.w[l] = 1.0f;
        f.prior_w = 1.0f;
    }
    record(tr, 2, true, st);
    rc = hip_status(launch_fold(f, st));
    record(tr, 2, false, st);
    return rc;
}

SelectArgs select_args(const kv_shape& s, const Layout& L, int n, int budget, const float* u,
                       const int32_t* pos, void* ws) {
    SelectArgs a{};
    a.u = u;
    a.pos = pos;
    a.pair_dst = at<int32_t>(ws, L.pdst_off);
    a.pair_src = at<int32_t>(ws, L.psrc_off);
    a.npairs = at<int32_t>(ws, L.np_off);
    a.batch = s.batch;
    a.cap = s.capacity;
    a.n = n;
    a.budget = budget;
    a.max_pairs = L.max_pairs;
    return a;
}

MoveArgs move_args(const kv_shape& s, const Layout& L, int n, int budget, void* k, void* v, float* u,
                   int32_t* pos, void* ws) {
    MoveArgs m{};
    m.k = k;
    m.v = v;
    m.u = u;
    m.pos = pos;
    m.pair_dst = at<int32_t>(ws, L.pdst_off);
    m.pair_src = at<int32_t>(ws, L.psrc_off);
    m.npairs = at<int32_t>(ws, L.np_off);
    m.batch = s.batch;
    m.layers = s.layers;
    m.hkv = s.n_kv_heads;
    m.cap = s.capacity;
    m.row_bytes = s.head_dim * esize(s);
    const int kk = budget < n ? budget : n;
    const int bound = n - kk < kk ? n - kk : kk;  // pairs <= min(#slots >= k, #slots < k)
    m.max_pairs = bound < L.max_pairs ? bound : L.max_pairs;
    m.pair_stride = L.max_pairs;
    return m;
}

}  // namespace
}  // namespace ikv

using namespace ikv;

extern "C" {

kv_status kv_workspace_bytes(const kv_shape* shape, int32_t n_max, size_t* bytes) {
    kv_status rc = check_shape(shape);
    if (rc != KV_OK) return rc;
    if (!bytes || n_max < 1 || n_max > shape->capacity) return KV_ERR_INVALID_ARG;
    *bytes = layout_for(*shape, n_max).total;
    return KV_OK;
}

kv_status kv_score_ema(const kv_shape* shape, int32_t n, const void* q, const void* k, const int32_t* pos,
                       int32_t cur_pos, float alpha, float recency_bias, int32_t recency_window, float* u,
                       float* s_out, void* ws, size_t ws_bytes, void* stream) {
    kv_status rc = check_shape(shape);
    if (rc != KV_OK) return rc;
    const kv_shape& s = *shape;
    if (n < 1 || n > s.capacity) return KV_ERR_INVALID_ARG;
    if (!(alpha >= 0.0f && alpha < 1.0f) || recency_window < 0 || !isfinite(recency_bias))
        return KV_ERR_INVALID_ARG;
    if (!q || !k || !pos || !u) return KV_ERR_INVALID_ARG;
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(pos, 4) || !aligned(u, 4) || !aligned(s_out, 4))
        return KV_ERR_UNSUPPORTED;
    const Layout L = layout_for(s, n);
    if ((rc = check_ws(L, ws, ws_bytes)) != KV_OK) return rc;
    return run_score_fold(s, L, n, q, k, pos, cur_pos, recency_bias, recency_window, u, s_out, KV_RULE_EMA,
                          alpha, ws, static_cast<hipStream_t>(stream), nullptr);
}

kv_status kv_topk_select(const kv_shape* shape, int32_t n, int32_t budget, const float* u, const int32_t* pos,
                         uint8_t* keep, void* ws, size_t ws_bytes, void* stream) {
    kv_status rc = check_shape(shape);
    if (rc != KV_OK) return rc;
    const kv_shape& s = *shape;
    if (n < 1 || n > s.capacity || budget < 1) return KV_ERR_INVALID_ARG;
    if (!u || !pos || !keep) return KV_ERR_INVALID_ARG;
    if (!aligned(u, 4) || !aligned(pos, 4)) return KV_ERR_UNSUPPORTED;
    const Layout L = layout_for(s, n);
    if ((rc = check_ws(L, ws, ws_bytes)) != KV_OK) return rc;
    SelectArgs a = select_args(s, L, n, budget, u, pos, ws);
    a.keep_out = keep;
    return hip_status(launch_select(a, false, static_cast<hipStream_t>(stream)));
}

kv_status kv_compact(const kv_shape* shape, int32_t n, int32_t budget, const uint8_t* keep, void* k, void* v,
                     float* u, int32_t* pos, void* ws, size_t ws_bytes, void* stream) {
    kv_status rc = check_shape(shape);
    if (rc != KV_OK) return rc;
    const kv_shape& s = *shape;
    if (n < 1 || n > s.capacity || budget < 1) return KV_ERR_INVALID_ARG;
    if (!keep || !k || !v || !u || !pos) return KV_ERR_INVALID_ARG;
    if (!aligned(k, 16) || !aligned(v, 16) || !aligned(u, 4) || !aligned(pos, 4)) return KV_ERR_UNSUPPORTED;
    const Layout L = layout_for(s, n);
    if ((rc = check_ws(L, ws, ws_bytes)) != KV_OK) return rc;
    if (n <= budget) return KV_OK;  // nothing is dropped, nothing moves
    hipStream_t st = static_cast<hipStream_t>(stream);
    SelectArgs a = select_args(s, L, n, budget, u, pos, ws);
    a.keep_in = keep;
    if ((rc = hip_status(launch_select(a, true, st))) != KV_OK) return rc;
    return hip_status(launch_move(move_args(s, L, n, budget, k, v, u, pos, ws), st));
}

kv_status kv_evict_step(const kv_shape* shape, const kv_params* params, int32_t t, int32_t n_in,
                        int32_t new_pos, const void* q, const void* k_new, const void* v_new, void* k, void* v,
                        float* u, int32_t* pos, int32_t* n_out, uint8_t* keep_out, float* s_out,
                        const kv_trace* trace, void* ws, size_t ws_bytes, void* stream) {
    kv_status rc = check_shape(shape);
    if (rc != KV_OK) return rc;
    const kv_shape& s = *shape;
    if (!params || !n_out) return KV_ERR_INVALID_ARG;
    const kv_params& p = *params;
    if (t < 1 || n_in < 0 || n_in + 1 > s.capacity || new_pos < 0) return KV_ERR_INVALID_ARG;
    if (!(p.alpha >= 0.0f && p.alpha < 1.0f) || p.budget < 1 || p.refresh_period < 1) return KV_ERR_INVALID_ARG;
    if (p.nonrefresh_init != KV_INIT_MEAN && p.nonrefresh_init != KV_INIT_MIN) return KV_ERR_INVALID_ARG;
    if (p.rule < KV_RULE_EMA || p.rule > KV_RULE_CUMULATIVE) return KV_ERR_INVALID_ARG;
    if (p.recency_window < 0 || !isfinite(p.recency_bias)) return KV_ERR_INVALID_ARG;
    if (!q || !k_new || !v_new || !k || !v || !u || !pos) return KV_ERR_INVALID_ARG;
    if (!aligned(q, 16) || !aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k, 16) || !aligned(v, 16) ||
        !aligned(u, 4) || !aligned(pos, 4) || !aligned(s_out, 4))
        return KV_ERR_UNSUPPORTED;
    const int n = n_in + 1;
    const Layout L = layout_for(s, n);
    if ((rc = check_ws(L, ws, ws_bytes)) != KV_OK) return rc;
    hipStream_t st = static_cast<hipStream_t>(stream);

    const bool refresh = p.score_free ? (t == 1) : ((t - 1) % p.refresh_period == 0);

    AppendArgs ap{};
    ap.k = k;
    ap.v = v;
    ap.k_new = k_new;
    ap.v_new = v_new;
    ap.u = u;
    ap.pos = pos;
    ap.batch = s.batch;
    ap.layers = s.layers;
    ap.hkv = s.n_kv_heads;
    ap.cap = s.capacity;
    ap.row_bytes = s.head_dim * esize(s);
    ap.n_in = n_in;
    ap.new_pos = new_pos;
    ap.init_mode = refresh ? 0 : (p.nonrefresh_init == KV_INIT_MEAN ? 1 : 2);

    record(trace, 0, true, st);
    rc = hip_status(launch_append(ap, st));
    record(trace, 0, false, st);
    if (rc != KV_OK) return rc;

    if (refresh) {
        rc = run_score_fold(s, L, n, q, k, pos, new_pos, p.recency_bias, p.recency_window, u, s_out, p.rule,
                            p.alpha, ws, st, trace);
        if (rc != KV_OK) return rc;
    }

    if (n > p.budget || keep_out) {
        SelectArgs a = select_args(s, L, n, p.budget, u, pos, ws);
        a.keep_out = keep_out;
        record(trace, 3, true, st);
        rc = hip_status(launch_select(a, false, st));
        record(trace, 3, false, st);
        if (rc != KV_OK) return rc;
        if (n > p.budget) {
            record(trace, 4, true, st);
            rc = hip_status(launch_move(move_args(s, L, n, p.budget, k, v, u, pos, ws), st));
            record(trace, 4, false, st);
            if (rc != KV_OK) return rc;
        }
    }
    *n_out = n < p.budget ? n : p.budget;
    return KV_OK;
}

const char* kv_status_string(kv_status status) {
    switch (status) {
        case KV_OK: return "ok";
        case KV_ERR_INVALID_ARG: return "invalid argument";
        case KV_ERR_UNSUPPORTED: return "unsupported shape, dtype or alignment";
        case KV_ERR_WORKSPACE: return "workspace missing or too small";
        case KV_ERR_HIP: return "HIP launch failed";
        default: return "unknown status";
    }
}

}  // extern "C"
