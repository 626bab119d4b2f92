// C ABI of the eviction path: argument validation, workspace layout and the launch sequence of a decode
// step.  Everything is queued on the caller's stream; nothing is allocated, synchronised or read back.
#include <math.h>
#include <string.h>

#include <atomic>

#include "../../include/inertiakv.h"
#include "kernels.h"
#include "kv_common.h"

// Scratch of kv_evict_step_static, the variant for callers that cannot allocate: one copy per device, held
// until the process ends.  On the host this name is only a stand-in for the symbol, never a device address:
// host code takes the device's copy from hipGetSymbolAddress (static_scratch below) and passes that pointer.
static __device__ __align__(256) unsigned char scratch[KV_STATIC_SCRATCH_BYTES];

namespace ikv {
namespace {

constexpr size_t kStaticScratchBytes = KV_STATIC_SCRATCH_BYTES;

// Device address of this device's scratch copy, looked up once per device with that device current.
kv_status static_scratch(void** out) {
    constexpr int kDevices = 64;
    static std::atomic<void*> addr[kDevices];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kDevices) return KV_ERR_HIP;
    void* p = addr[dev].load(std::memory_order_acquire);
    if (!p) {
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return KV_ERR_HIP;
        addr[dev].store(p, std::memory_order_release);
    }
    *out = p;
    return KV_OK;
}

// Long slabs (first steps) are scored in groups of layers whose logits stay within this many bytes, so that
// the finish kernel reads them back while the 256 MiB last-level cache may still hold them: measured with 1,
// 2, 4, 8, 16 and all 32 layers per group, 4 layers (~130 MB of logits) was fastest on every first step (8B
// 5.09 -> 4.85 ms, Score-Free 128k 5.34 -> 5.14 ms, Qwen-shaped 3.27 -> 3.11 ms).
#ifndef IKV_SPLIT_LOGIT_MIB
#define IKV_SPLIT_LOGIT_MIB 160
#endif
constexpr size_t kSplitLogitBytes = (size_t)IKV_SPLIT_LOGIT_MIB << 20;
#ifndef IKV_COOP_SPLIT
#define IKV_COOP_SPLIT 1
#endif
constexpr bool kCoopSplit = IKV_COOP_SPLIT != 0;
// KV heads whose group sums a team of exchanging chunks adds by default (the largest divisor of n_kv up to
// this): fewer rows of r written while K streams, and fewer for the fold to read.
#ifndef IKV_COOP_MERGE
#define IKV_COOP_MERGE 4
#endif
constexpr int kCoopMerge = IKV_COOP_MERGE;

// The workspace's first 256 bytes hold the sticky fault word (kv_fault bits), at the same place for every n.
constexpr size_t kFaultBytes = 256;
static_assert(kFaultExchangeTimeout == (uint32_t)KV_FAULT_EXCHANGE_TIMEOUT, "fault bits of the kernels and the ABI");

struct Layout {
    int n;  // cached tokens the layout serves
    int n_stride;
    int max_pairs;
    ScorePlan plan;
    size_t r_off, z_off, part_off, opart_off, npart_off, vn_off, vinv_off, eta_off, pdst_off, psrc_off, np_off;
    size_t raw_off, rmask_off, emask_off, kmask_off, tdst_off, tsrc_off, tnp_off, cand_off, wide_off, total;
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

// One layout serves every entry point for a given n, so that the group sums r written by the attention
// calls of a step are where kv_evict_finish folds them.  The logits / partial regions are shared by the
// scorer's split path and the attention's chunked path (never live at the same time).
// step_lds_only: the regions of a kv_evict_step whose slabs are scored in one workgroup each (no logits,
// chunk partials or attention partials), for the allocation-free variant.
Layout layout_for(const kv_shape& s, int n, bool step_lds_only = false) {
    Layout L{};
    L.n = n;
    L.n_stride = (n + 63) / 64 * 64;
    L.max_pairs = n;
    const int group = s.n_q_heads / s.n_kv_heads;
    score_plan(s.dtype, s.head_dim, group, n, &L.plan);
    AttendBound ab = attend_bound(s.dtype, s.head_dim, group, n, s.batch * s.n_kv_heads, s.layers);
    if (step_lds_only) ab = AttendBound{0, false};
    const size_t heads = (size_t)s.layers * s.batch * s.n_q_heads;
    const size_t logits = heads * L.n_stride * sizeof(float);
    const size_t z_bytes = ((L.plan.split && !step_lds_only) || ab.may_split) ? logits : 0;
    // chunk partials of long slabs (scorer) and of the attention
    size_t part_bytes = (size_t)ab.chunk_layers * s.batch * s.n_q_heads * sizeof(float2);
    if (L.plan.split && !step_lds_only) {
        // the logits path's (max, sum) pairs and the exchange path's words (8 bytes each per query head and
        // chunk); merged teams cut slabs into more chunks (their LDS also holds the item sums)
        const int slabs = s.layers * s.batch * s.n_kv_heads;
        ScorePlan cp;
        int chunks = 0;
        if (attend_plan(s.dtype, s.head_dim, group, n, slabs, &cp, kScoreChunkLds)) chunks = cp.nchunk;
        for (int m = 1; m <= 2; ++m)
            if (coop_plan(s.dtype, s.head_dim, group, n, slabs, m, &cp) && cp.nchunk > chunks) chunks = cp.nchunk;
        const size_t sp = heads * chunks * sizeof(uint64_t);
        if (sp > part_bytes) part_bytes = sp;
    }
    size_t off = kFaultBytes;
    L.r_off = off;
    off = align256(off + (size_t)s.layers * s.batch * s.n_kv_heads * L.n_stride * sizeof(float));
    L.z_off = off;
    off = align256(off + z_bytes);
    L.part_off = off;
    off = align256(off + part_bytes);
    L.opart_off = off;
    off = align256(off + (size_t)ab.chunk_layers * s.batch * s.n_q_heads * s.head_dim * sizeof(float));
    L.npart_off = off;
    off = align256(off + (size_t)ab.chunk_layers * s.batch * s.n_kv_heads * sizeof(float));
    L.vn_off = off;
    off = align256(off + (size_t)s.layers * s.batch * s.n_kv_heads * L.n_stride * sizeof(float));
    L.vinv_off = off;
    off = align256(off + (size_t)s.layers * s.batch * s.n_kv_heads * sizeof(float));
    L.eta_off = off;
    off = align256(off + (size_t)s.layers * s.batch * sizeof(float));
    L.pdst_off = off;
    off = align256(off + (size_t)s.batch * L.max_pairs * sizeof(int32_t));
    L.psrc_off = off;
    off = align256(off + (size_t)s.batch * L.max_pairs * sizeof(int32_t));
    L.np_off = off;
    off = align256(off + (size_t)s.batch * sizeof(int32_t));
    // rank trace: raw score, the three decisions, and a private selection plan (the eviction's stays intact)
    const size_t slots = (size_t)s.batch * s.capacity;
    L.raw_off = off;
    off = align256(off + slots * sizeof(float));
    L.rmask_off = off;
    off = align256(off + slots);
    L.emask_off = off;
    off = align256(off + slots);
    L.kmask_off = off;
    off = align256(off + slots);
    L.tdst_off = off;
    off = align256(off + (size_t)s.batch * L.max_pairs * sizeof(int32_t));
    L.tsrc_off = off;
    off = align256(off + (size_t)s.batch * L.max_pairs * sizeof(int32_t));
    L.tnp_off = off;
    off = align256(off + (size_t)s.batch * sizeof(int32_t));
    // the fold's per-workgroup eviction candidates of a single-eviction refresh step
    L.cand_off = off;
    off = align256(off + (size_t)s.batch * fold_groups(n) * sizeof(EvictCand));
    // the multi-workgroup selection's histograms, counts and state (long sequences in a small batch)
    L.wide_off = off;
    off = align256(off + select_wide_words(s.batch) * sizeof(uint32_t));
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

ScoreArgs score_args(const kv_shape& s, const Layout& L, int n, const void* q, const void* k, const int32_t* pos,
                     int cur_pos, float recency_bias, int recency_window, void* ws) {
    ScoreArgs a{};
    a.q = q;
    a.k = k;
    a.pos = pos;
    a.r = at<float>(ws, L.r_off);
    a.z = at<float>(ws, L.z_off);
    a.part = at<float2>(ws, L.part_off);
    a.opart = at<float>(ws, L.opart_off);
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
    a.merge = 1;
    return a;
}

// How a refresh step's scorer runs over n rows: one workgroup per slab with its logits in LDS; or, for slabs
// too long for that, chunks that exchange their softmax statistics and write the group sums directly (on a
// grid the device holds at once); or chunks that write logits for a finish kernel (slabs with more exchange
// words than one chunk grid handles).
struct ScoreRoute {
    enum Kind { kLds = 0, kExchange = 1, kLogits = 2 } kind;
    ScorePlan xp;  // kExchange: the chunk plan
    long grid;     // kExchange: workgroups of the persistent grid
};

// Layers per launch of the logits path: groups whose logits fit kSplitLogitBytes (read back by the finish
// kernel while they may still be cached).
int logit_layer_group(const kv_shape& s, const Layout& L) {
    const size_t layer_logits = (size_t)s.batch * s.n_q_heads * L.n_stride * sizeof(float);
    const size_t fit = kSplitLogitBytes / layer_logits;
    return fit < 1 ? 1 : (fit > (size_t)s.layers ? s.layers : (int)fit);
}

static_assert((int)ScoreRoute::kLds == KV_PATH_LDS && (int)ScoreRoute::kExchange == KV_PATH_EXCHANGE &&
                  (int)ScoreRoute::kLogits == KV_PATH_LOGITS,
              "scorer paths of the planner and the ABI");

// plan.merge > 1 (split plans): the exchange route with teams that add that many KV heads' sums, else the
// logits route (whose finish writes one row per KV head, so a plan only carries such a merge when the
// exchange route takes it: scorer_plan).
ScoreRoute score_route(const kv_shape& s, const Layout& L, int n, const ScorePlan& plan) {
    ScoreRoute r{ScoreRoute::kLds, plan, 0};
    if (!plan.split) return r;
    r.kind = ScoreRoute::kLogits;
    const int group = s.n_q_heads / s.n_kv_heads;
    const long slabs = (long)s.layers * s.batch * s.n_kv_heads;
    ScorePlan xp;
    if (kCoopSplit && coop_plan(s.dtype, s.head_dim, group, n, (int)slabs, plan.merge, &xp) && xp.split &&
        xp.nchunk * xp.group_pad <= kCoopMaxWords) {
        const long items = slabs / xp.merge;
        long grid = coop_workgroups(s.dtype, s.head_dim, xp) / xp.nchunk * xp.nchunk;
        if (grid > items * xp.nchunk) grid = items * xp.nchunk;
        if (grid >= xp.nchunk &&
            (size_t)s.layers * s.batch * s.n_q_heads * xp.nchunk * sizeof(uint64_t) <= L.opart_off - L.part_off) {
            r.kind = ScoreRoute::kExchange;
            r.xp = xp;
            r.grid = grid;
        }
    }
    return r;
}

// The scorer's plan for a refresh step with these scorer variants: KV heads of one (layer, sequence) share a
// workgroup (or, for slabs scored in exchanging chunks, a team of chunks) and add their group sums (`merge`
// of them: 0 = planned) unless VNorm needs each KV head's sums apart (it weights them per head).  Slabs scored
// by the logits route keep one row per KV head.
ScorePlan scorer_plan(const kv_shape& s, const Layout& L, int variant, int merge) {
    ScorePlan plan = L.plan;
    const bool vnorm = (variant & KV_SCORE_VNORM) != 0;
    score_merge(&plan, s.dtype, s.head_dim, s.n_kv_heads, s.layers * s.batch, vnorm ? 1 : merge);
    if (plan.split && !vnorm) {
        int m = merge;
        if (m <= 0) {
            m = kCoopMerge < kMaxMerge ? kCoopMerge : kMaxMerge;
            while (m > 1 && s.n_kv_heads % m) --m;
        }
        if (m > 1) {
            ScorePlan t = plan;
            t.merge = m;
            if (score_route(s, L, L.n, t).kind == ScoreRoute::kExchange) plan.merge = m;
        }
    }
    return plan;
}

// Scoring (Eq. 1) of rows [0, n) of every layer into the workspace r: [layers][batch][n_kv / merge] rows.
// k_new (one workgroup per slab only): row n - 1 is the step's newcomer, read from k_new instead of the cache,
// with position cur_pos.  vn_cache (a plan from vnorm_fused_plan only): VNorm applied by the scorer, with the
// newcomer's V row from v_new.
kv_status run_score(const kv_shape& s, const Layout& L, int n, const void* q, const void* k, const int32_t* pos,
                    int cur_pos, float recency_bias, int recency_window, const ScorePlan& splan, void* ws,
                    hipStream_t st, const void* k_new = nullptr, const float* vn_cache = nullptr,
                    const void* v_new = nullptr) {
    ScoreArgs a = score_args(s, L, n, q, k, pos, cur_pos, recency_bias, recency_window, ws);
    ScorePlan plan = splan;
    if (plan.split) {
        const int group = s.n_q_heads / s.n_kv_heads;
        const ScoreRoute route = score_route(s, L, n, plan);
        if (route.kind == ScoreRoute::kExchange) {
            a.v = k;
            a.chunk_rows = route.xp.chunk_rows;
            a.nchunk = route.xp.nchunk;
            a.merge = route.xp.merge;
            a.emit = 1;
            return hip_status(launch_score_coop(s.dtype, s.head_dim, route.xp, a, at<uint64_t>(ws, L.part_off),
                                                (int)route.grid, at<uint32_t>(ws, 0), st));
        }
        // LDS-resident chunks of the attention kernel's K pass that write logits, then the finish kernel, per
        // group of layers (one row of r per KV head: scorer_plan merges only for the exchange route)
        if (plan.merge != 1) return KV_ERR_UNSUPPORTED;
        const int lg = logit_layer_group(s, L);
        const size_t e = (size_t)esize(s);
        for (int l0 = 0; l0 < s.layers; l0 += lg) {
            const int lc = s.layers - l0 < lg ? s.layers - l0 : lg;
            ScorePlan cp;
            if (!attend_plan(s.dtype, s.head_dim, group, n, lc * s.batch * s.n_kv_heads, &cp, kScoreChunkLds) ||
                !cp.split)
                return KV_ERR_UNSUPPORTED;  // (a slab too long for one workgroup's LDS always splits)
            if ((size_t)lc * s.batch * s.n_q_heads * cp.nchunk * sizeof(float2) > L.opart_off - L.part_off)
                return KV_ERR_UNSUPPORTED;
            ScoreArgs g = a;
            g.layers = lc;
            g.q = static_cast<const char*>(q) + (size_t)l0 * s.batch * s.n_q_heads * s.head_dim * e;
            g.k = static_cast<const char*>(k) + (size_t)l0 * s.batch * s.n_kv_heads * s.capacity * s.head_dim * e;
            g.v = g.k;  // not read: the kernel's V stream is compiled out
            g.r = a.r + (size_t)l0 * s.batch * s.n_kv_heads * L.n_stride;
            g.chunk_rows = cp.chunk_rows;
            g.nchunk = cp.nchunk;
            g.emit = 1;
            kv_status rc = hip_status(launch_score_chunks(s.dtype, s.head_dim, cp, g, st));
            if (rc == KV_OK) rc = hip_status(launch_split_finish(g, st));
            if (rc != KV_OK) return rc;
        }
        return KV_OK;
    }
    a.chunk_rows = plan.chunk_rows;
    a.nchunk = plan.nchunk;
    a.merge = plan.merge;
    a.k_new = k_new;
    a.new_pos = cur_pos;
    a.vn_cache = vn_cache;
    a.v_new = v_new;
    return hip_status(launch_score(s.dtype, s.head_dim, plan, a, st));
}

// VNorm from the value-norm cache on a steady refresh step is applied by the multi-slab scorer (each KV head's
// group sums weighted by norm / mean before the item adds them), so the step keeps a merged schedule and needs
// neither the norms' mean kernel nor the fold's factors: when the logits are the vector form, entropy weighting
// is off (it is taken over the plain scores), no merge is forced, and the item's norms fit in LDS beside its
// sums with a merge above one.  8B steady step with VNorm, alternating builds in one process: 308.1 -> 282.0 us
// (the plain step 263 us).
bool vnorm_fused_plan(const kv_shape& s, const Layout& L, const kv_params& p, ScorePlan* out) {
    if (!(p.score_variant & KV_SCORE_VNORM) || (p.score_variant & KV_SCORE_ENTROPY) || p.score_merge != 0)
        return false;
    ScorePlan plan = L.plan;
    if (plan.split || !score_vnorm_fusable(s.dtype, s.head_dim, plan.group_pad)) return false;
    score_merge(&plan, s.dtype, s.head_dim, s.n_kv_heads, s.layers * s.batch, 0, true);
    if (plan.merge < 2) return false;
    *out = plan;
    return true;
}

// Scorer perturbations (Sec. 5.1) of a refresh step: value-row norms and entropy factors for the fold.  With
// the caller's norm cache (norms, [layers][batch][n_kv][cap]) VNorm reads the cached norms instead of V; v_new
// set: row n - 1 is the step's newcomer, whose norm is computed from v_new and cached first.
kv_status run_variants(const kv_shape& s, const Layout& L, int n, const void* v, int variant, int r_groups,
                       int rblock, void* ws, hipStream_t st, float* norms = nullptr, const void* v_new = nullptr) {
    if (!variant) return KV_OK;
    VariantArgs a{};
    a.v = v;
    a.r = at<float>(ws, L.r_off);
    a.vnorm = norms ? norms : at<float>(ws, L.vn_off);
    a.vnorm_stride = norms ? s.capacity : L.n_stride;
    a.v_new = v_new;
    a.vnorm_inv_mean = at<float>(ws, L.vinv_off);
    a.entropy = at<float>(ws, L.eta_off);
    a.batch = s.batch;
    a.layers = s.layers;
    a.hkv = s.n_kv_heads;
    a.cap = s.capacity;
    a.n = n;
    a.n_stride = L.n_stride;
    a.r_groups = r_groups;
    a.rblock = rblock;
    a.inv_hq = 1.0f / (float)s.n_q_heads;
    kv_status rc = KV_OK;
    if (variant & KV_SCORE_ENTROPY) rc = hip_status(launch_entropy(a, st));
    if (rc == KV_OK && (variant & KV_SCORE_VNORM))
        rc = hip_status(norms ? launch_vnorm_mean(s.dtype, s.head_dim, a, st) : launch_vnorm(s.dtype, s.head_dim, a, st));
    return rc;
}

// Layer fold of the workspace r into u (Eq. 2-4 by `rule`): r_groups rows per (layer, sequence), added in
// blocks of rblock.  Options for single-eviction steps: candidates (each fold workgroup's first token to
// leave, for launch_place) and new_pos >= 0 (token n - 1 is the newcomer, not yet in u / pos).
struct FoldExtra {
    int32_t* pos = nullptr;
    int new_pos = -1;
    bool candidates = false;
    const float* norms = nullptr;  // VNorm's norms from the caller's cache (stride cap) instead of the workspace
};
kv_status run_fold(const kv_shape& s, const Layout& L, int n, float* u, float* s_out, int rule, float alpha,
                   int variant, int r_groups, int rblock, bool raw_out, void* ws, hipStream_t st,
                   const kv_trace* tr, const FoldExtra& ex = FoldExtra{}) {
    FoldArgs f{};
    f.pos = ex.pos;
    f.new_pos = ex.new_pos;
    f.cand = ex.candidates ? at<EvictCand>(ws, L.cand_off) : nullptr;
    f.raw = raw_out ? at<float>(ws, L.raw_off) : nullptr;
    f.raw_scale = (float)(1.0 / ((double)s.layers * s.n_q_heads));
    f.r = at<float>(ws, L.r_off);
    f.vnorm = (variant & KV_SCORE_VNORM) ? (ex.norms ? ex.norms : at<float>(ws, L.vn_off)) : nullptr;
    f.vnorm_stride = ex.norms ? s.capacity : L.n_stride;
    f.vnorm_inv_mean = at<float>(ws, L.vinv_off);
    f.entropy = (variant & KV_SCORE_ENTROPY) ? at<float>(ws, L.eta_off) : nullptr;
    f.u = u;
    f.s_out = s_out;
    f.batch = s.batch;
    f.layers = s.layers;
    f.hkv = s.n_kv_heads;
    f.n = n;
    f.n_stride = L.n_stride;
    f.cap = s.capacity;
    f.r_groups = r_groups;
    f.rblock = rblock;
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
    kv_status rc = hip_status(launch_fold(f, st));
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
    a.wide = select_wide_words(s.batch) ? at<uint32_t>(ws, L.wide_off) : nullptr;
    return a;
}

MoveArgs move_args(const kv_shape& s, const Layout& L, int n, int budget, void* k, void* v, float* u,
                   int32_t* pos, float* norms, void* ws) {
    MoveArgs m{};
    m.norms = norms;
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

kv_status check_params(const kv_params* params) {
    if (!params) return KV_ERR_INVALID_ARG;
    const kv_params& p = *params;
    if (!(p.alpha >= 0.0f && p.alpha < 1.0f) || p.budget < 1 || p.refresh_period < 1) return KV_ERR_INVALID_ARG;
    if (p.nonrefresh_init != KV_INIT_MEAN && p.nonrefresh_init != KV_INIT_MIN) return KV_ERR_INVALID_ARG;
    if (p.rule < KV_RULE_EMA || p.rule > KV_RULE_CUMULATIVE) return KV_ERR_INVALID_ARG;
    if (p.recency_window < 0 || !isfinite(p.recency_bias)) return KV_ERR_INVALID_ARG;
    if (p.score_variant & ~(KV_SCORE_VNORM | KV_SCORE_ENTROPY | KV_SCORE_NORMS_EMITTED)) return KV_ERR_INVALID_ARG;
    if (p.score_merge < 0 || p.score_merge > kMaxMerge) return KV_ERR_INVALID_ARG;
    if ((p.score_variant & KV_SCORE_VNORM) && p.score_merge > 1) return KV_ERR_INVALID_ARG;
    return KV_OK;
}

kv_status check_merge(const kv_shape& s, const kv_params& p) {
    return (p.score_merge > 0 && s.n_kv_heads % p.score_merge) ? KV_ERR_INVALID_ARG : KV_OK;
}

// Refresh set (Eq. 5); Score-Free refreshes only at the first decode step.
bool is_refresh(const kv_params& p, int t) { return p.score_free ? (t == 1) : ((t - 1) % p.refresh_period == 0); }

AppendArgs append_args(const kv_shape& s, const kv_params& p, int t, int n_in, int new_pos, const void* k_new,
                       const void* v_new, void* k, void* v, float* u, int32_t* pos, float* norms) {
    AppendArgs ap{};
    ap.norms = norms;
    ap.bf16 = s.dtype == KV_BF16;
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
    ap.init_mode = is_refresh(p, t) ? 0 : (p.nonrefresh_init == KV_INIT_MEAN ? 1 : 2);
    return ap;
}

kv_status run_append(const kv_shape& s, const kv_params& p, int t, int n_in, int new_pos, const void* k_new,
                     const void* v_new, void* k, void* v, float* u, int32_t* pos, float* norms, hipStream_t st,
                     const kv_trace* tr) {
    AppendArgs ap = append_args(s, p, t, n_in, new_pos, k_new, v_new, k, v, u, pos, norms);
    record(tr, 0, true, st);
    kv_status rc = hip_status(launch_append(ap, st));
    record(tr, 0, false, st);
    return rc;
}

size_t trace_words(int max_pos) { return ((size_t)max_pos + 31) / 32; }

kv_status check_rank_trace(const kv_rank_trace* rt) {
    if (!rt) return KV_OK;
    if (rt->k < 1 || rt->max_pos < 1 || !rt->state || !rt->counts) return KV_ERR_INVALID_ARG;
    if (!aligned(rt->state, 4) || !aligned(rt->counts, 4)) return KV_ERR_UNSUPPORTED;
    return KV_OK;
}

// A step that is not traced (not a refresh step) still writes its counts: row 0 of each sequence = 0.
kv_status mark_untraced(const kv_shape& s, const kv_rank_trace* rt, hipStream_t st) {
    TraceArgs ta{};
    ta.counts = rt->counts;
    ta.batch = s.batch;
    return hip_status(launch_trace_stats(ta, true, st));
}

// Top-B selection over the n cached tokens and, when tokens are dropped, the compaction.  With a rank trace
// on a refresh step, the traced top-k decisions (raw score from the fold; the EMA set is the retention
// decision itself when k = B) and their statistics are taken before the compaction, on the same slots.
kv_status run_select_compact(const kv_shape& s, const Layout& L, int n, int budget, void* k, void* v, float* u,
                             int32_t* pos, float* norms, uint8_t* keep_out, const kv_rank_trace* rt, bool refresh,
                             void* ws, hipStream_t st, const kv_trace* tr) {
    TraceArgs ta{};
    kv_status rc = KV_OK;
    const bool traced = rt && refresh;
    if (rt) {
        ta.pos = pos;
        ta.state = rt->state;
        ta.counts = rt->counts;
        ta.batch = s.batch;
        ta.cap = s.capacity;
        ta.n = n;
        ta.max_pos = rt->max_pos;
        ta.words = (int)trace_words(rt->max_pos);
        if (!traced) {
            if ((rc = mark_untraced(s, rt, st)) != KV_OK) return rc;
        } else if (!keep_out) {
            keep_out = at<uint8_t>(ws, L.kmask_off);  // the statistics need the decision
        }
    }
    if (n <= budget && !keep_out) return KV_OK;
    SelectArgs a = select_args(s, L, n, budget, u, pos, ws);
    a.keep_out = keep_out;
    record(tr, 3, true, st);
    rc = hip_status(launch_select(a, false, st));
    if (rc == KV_OK && traced) {
        ta.keep = keep_out;
        ta.raw_keep = rt->raw_keep ? rt->raw_keep : at<uint8_t>(ws, L.rmask_off);
        const bool ema_is_keep = rt->k == budget && !rt->ema_keep;
        ta.ema_keep = ema_is_keep ? keep_out : (rt->ema_keep ? rt->ema_keep : at<uint8_t>(ws, L.emask_off));
        for (int which = 0; which < (ema_is_keep ? 1 : 2) && rc == KV_OK; ++which) {
            SelectArgs t = select_args(s, L, n, rt->k, which == 0 ? at<float>(ws, L.raw_off) : u, pos, ws);
            t.pair_dst = at<int32_t>(ws, L.tdst_off);
            t.pair_src = at<int32_t>(ws, L.tsrc_off);
            t.npairs = at<int32_t>(ws, L.tnp_off);
            t.keep_out = const_cast<uint8_t*>(which == 0 ? ta.raw_keep : ta.ema_keep);
            rc = hip_status(launch_select(t, false, st));
        }
        if (rc == KV_OK) rc = hip_status(launch_trace_stats(ta, false, st));
    }
    record(tr, 3, false, st);
    if (rc != KV_OK || n <= budget) return rc;
    record(tr, 4, true, st);
    rc = hip_status(launch_move(move_args(s, L, n, budget, k, v, u, pos, norms, ws), st));
    record(tr, 4, false, st);
    return rc;
}

// Placement of the newcomer of a single-eviction refresh step (n <= budget + 1) after a fold with
// candidates: its K/V rows come from k_new / v_new, or from row n - 1 of the cache when those are null.
kv_status run_place(const kv_shape& s, const Layout& L, int n, int budget, const void* k_new, const void* v_new,
                    void* k, void* v, float* u, int32_t* pos, float* norms, uint8_t* keep_out, void* ws,
                    hipStream_t st) {
    PlaceArgs a{};
    a.norms = norms;
    a.bf16 = s.dtype == KV_BF16;
    a.k = k;
    a.v = v;
    a.u = u;
    a.pos = pos;
    if (k_new) {
        a.src_k = k_new;
        a.src_v = v_new;
        a.src_slab_rows = 1;
        a.src_row0 = 0;
    } else {
        a.src_k = k;
        a.src_v = v;
        a.src_slab_rows = (size_t)s.capacity;
        a.src_row0 = (size_t)(n - 1);
    }
    a.cand = at<EvictCand>(ws, L.cand_off);
    a.ncand = fold_groups(n);
    a.keep_out = keep_out;
    a.batch = s.batch;
    a.layers = s.layers;
    a.hkv = s.n_kv_heads;
    a.cap = s.capacity;
    a.row_bytes = s.head_dim * esize(s);
    a.n = n;
    a.budget = budget;
    return hip_status(launch_place(a, st));
}

kv_status check_step(const kv_shape* shape, const kv_params* params, int t, int n_in, int new_pos, const void* q,
                     const void* k_new, const void* v_new, const void* k, const void* v, const float* u,
                     const int32_t* pos, const float* v_norms, const int32_t* n_out, const float* s_out,
                     const kv_rank_trace* rank_trace) {
    kv_status rc = check_shape(shape);
    if (rc != KV_OK) return rc;
    const kv_shape& s = *shape;
    if ((rc = check_params(params)) != KV_OK) return rc;
    if ((rc = check_rank_trace(rank_trace)) != KV_OK) return rc;
    if ((rc = check_merge(s, *params)) != KV_OK) return rc;
    if (!n_out) return KV_ERR_INVALID_ARG;
    if (t < 1 || n_in < 0 || n_in + 1 > s.capacity || new_pos < 0) return KV_ERR_INVALID_ARG;
    if (!q || !k_new || !v_new || !k || !v || !u || !pos) return KV_ERR_INVALID_ARG;
    if (!aligned(q, 16) || !aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k, 16) || !aligned(v, 16) ||
        !aligned(u, 4) || !aligned(pos, 4) || !aligned(s_out, 4) || !aligned(v_norms, 4))
        return KV_ERR_UNSUPPORTED;
    return KV_OK;
}

// One decode step (a0 ... a5) on validated arguments, with the workspace ws laid out as L.  v_norms (nullable):
// the caller's value-norm cache, kept in step with V by every row write and move; VNorm reads it.
kv_status evict_step(const kv_shape& s, const kv_params& p, int t, int n_in, int new_pos, const void* q,
                     const void* k_new, const void* v_new, void* k, void* v, float* u, int32_t* pos,
                     float* v_norms, int32_t* n_out, uint8_t* keep_out, float* s_out, const kv_trace* trace,
                     const kv_rank_trace* rank_trace, const Layout& L, void* ws, hipStream_t st) {
    kv_status rc = KV_OK;
    const int n = n_in + 1;
    const bool refresh = is_refresh(p, t);
    if (!refresh && n_in <= p.budget) {
        // every Lazy / Score-Free step after the first: one kernel per sequence
        AppendArgs ap = append_args(s, p, t, n_in, new_pos, k_new, v_new, k, v, u, pos, v_norms);
        if (rank_trace && (rc = mark_untraced(s, rank_trace, st)) != KV_OK) return rc;
        record(trace, 0, true, st);
        // the per-sequence pair counts of the workspace are free on this path: they carry the newcomer's slot
        rc = hip_status(launch_nonrefresh(ap, keep_out, p.budget, at<int32_t>(ws, L.np_off), st));
        record(trace, 0, false, st);
        if (rc != KV_OK) return rc;
        *n_out = n < p.budget ? n : p.budget;
        return KV_OK;
    }
    const bool vnorm = (p.score_variant & KV_SCORE_VNORM) != 0;
    if (refresh && n_in <= p.budget && !rank_trace && (!vnorm || v_norms)) {
        ScorePlan plan = scorer_plan(s, L, p.score_variant, p.score_merge);
        const bool vn_fused = vnorm && vnorm_fused_plan(s, L, p, &plan);
        const int variant = vn_fused ? (p.score_variant & ~KV_SCORE_VNORM) : p.score_variant;
        if (!plan.split) {
            // A steady refresh step (one eviction, or none while under budget) in three kernels: the scorer
            // takes the newcomer from k_new as row n - 1, the fold gives it the refresh prior and reports each
            // workgroup's first token to leave, and the placement writes the newcomer's rows once, into the
            // slot it takes (the append's and the compaction's row copies in one).  VNorm (with the norm cache
            // only: V's row n - 1 is not written yet) adds the norms' mean, the newcomer's norm from v_new.
            const int r_groups = s.n_kv_heads / plan.merge;
            record(trace, 0, true, st);
            record(trace, 0, false, st);
            record(trace, 1, true, st);
            rc = run_score(s, L, n, q, k, pos, new_pos, p.recency_bias, p.recency_window, plan, ws, st, k_new,
                           vn_fused ? v_norms : nullptr, vn_fused ? v_new : nullptr);
            if (rc == KV_OK) rc = run_variants(s, L, n, v, variant, r_groups, 1, ws, st, v_norms, v_new);
            record(trace, 1, false, st);
            FoldExtra ex;
            ex.pos = pos;
            ex.new_pos = new_pos;
            ex.candidates = n > p.budget;
            ex.norms = v_norms;
            if (rc == KV_OK)
                rc = run_fold(s, L, n, u, s_out, p.rule, p.alpha, variant, r_groups, 1, false, ws, st, trace, ex);
            record(trace, 3, true, st);
            if (rc == KV_OK)
                rc = run_place(s, L, n, p.budget, k_new, v_new, k, v, u, pos, v_norms, keep_out, ws, st);
            record(trace, 3, false, st);
            record(trace, 4, true, st);
            record(trace, 4, false, st);
            if (rc != KV_OK) return rc;
            *n_out = n < p.budget ? n : p.budget;
            return KV_OK;
        }
    }
    if ((rc = run_append(s, p, t, n_in, new_pos, k_new, v_new, k, v, u, pos, v_norms, st, trace)) != KV_OK)
        return rc;
    if (refresh) {
        const ScorePlan plan = scorer_plan(s, L, p.score_variant, p.score_merge);
        const int r_groups = s.n_kv_heads / plan.merge;
        record(trace, 1, true, st);
        rc = run_score(s, L, n, q, k, pos, new_pos, p.recency_bias, p.recency_window, plan, ws, st);
        if (rc == KV_OK) rc = run_variants(s, L, n, v, p.score_variant, r_groups, 1, ws, st, v_norms);
        record(trace, 1, false, st);
        FoldExtra ex;
        ex.norms = v_norms;
        if (rc == KV_OK)
            rc = run_fold(s, L, n, u, s_out, p.rule, p.alpha, p.score_variant, r_groups, 1, rank_trace != nullptr,
                          ws, st, trace, ex);
        if (rc != KV_OK) return rc;
    }
    rc = run_select_compact(s, L, n, p.budget, k, v, u, pos, v_norms, keep_out, rank_trace, refresh, ws, st, trace);
    if (rc != KV_OK) return rc;
    *n_out = n < p.budget ? n : p.budget;
    return KV_OK;
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

kv_status kv_score_merge(const kv_shape* shape, int32_t n, const kv_params* params, int32_t* merge) {
    kv_status rc = check_shape(shape);
    if (rc != KV_OK) return rc;
    if ((rc = check_params(params)) != KV_OK) return rc;
    const kv_shape& s = *shape;
    if ((rc = check_merge(s, *params)) != KV_OK) return rc;
    if (!merge || n < 1 || n > s.capacity) return KV_ERR_INVALID_ARG;
    *merge = scorer_plan(s, layout_for(s, n), params->score_variant, params->score_merge).merge;
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
    hipStream_t st = static_cast<hipStream_t>(stream);
    const ScorePlan plan = scorer_plan(s, L, 0, 0);
    if ((rc = run_score(s, L, n, q, k, pos, cur_pos, recency_bias, recency_window, plan, ws, st)) != KV_OK)
        return rc;
    return run_fold(s, L, n, u, s_out, KV_RULE_EMA, alpha, 0, s.n_kv_heads / plan.merge, 1, false, ws, st,
                    nullptr);
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
                     float* u, int32_t* pos, float* v_norms, void* ws, size_t ws_bytes, void* stream) {
    kv_status rc = check_shape(shape);
    if (rc != KV_OK) return rc;
    const kv_shape& s = *shape;
    if (n < 1 || n > s.capacity || budget < 1) return KV_ERR_INVALID_ARG;
    if (!keep || !k || !v || !u || !pos) return KV_ERR_INVALID_ARG;
    if (!aligned(k, 16) || !aligned(v, 16) || !aligned(u, 4) || !aligned(pos, 4) || !aligned(v_norms, 4))
        return KV_ERR_UNSUPPORTED;
    const Layout L = layout_for(s, n);
    if ((rc = check_ws(L, ws, ws_bytes)) != KV_OK) return rc;
    if (n <= budget) return KV_OK;  // nothing is dropped, nothing moves
    hipStream_t st = static_cast<hipStream_t>(stream);
    SelectArgs a = select_args(s, L, n, budget, u, pos, ws);
    a.keep_in = keep;
    if ((rc = hip_status(launch_select(a, true, st))) != KV_OK) return rc;
    return hip_status(launch_move(move_args(s, L, n, budget, k, v, u, pos, v_norms, ws), st));
}

kv_status kv_evict_step(const kv_shape* shape, const kv_params* params, int32_t t, int32_t n_in,
                        int32_t new_pos, const void* q, const void* k_new, const void* v_new, void* k, void* v,
                        float* u, int32_t* pos, float* v_norms, int32_t* n_out, uint8_t* keep_out, float* s_out,
                        const kv_trace* trace, const kv_rank_trace* rank_trace, void* ws, size_t ws_bytes,
                        void* stream) {
    kv_status rc = check_step(shape, params, t, n_in, new_pos, q, k_new, v_new, k, v, u, pos, v_norms, n_out,
                              s_out, rank_trace);
    if (rc != KV_OK) return rc;
    const Layout L = layout_for(*shape, n_in + 1);
    if ((rc = check_ws(L, ws, ws_bytes)) != KV_OK) return rc;
    return evict_step(*shape, *params, t, n_in, new_pos, q, k_new, v_new, k, v, u, pos, v_norms, n_out, keep_out,
                      s_out, trace, rank_trace, L, ws, static_cast<hipStream_t>(stream));
}

kv_status kv_evict_step_static(const kv_shape* shape, const kv_params* params, int32_t t, int32_t n_in,
                               int32_t new_pos, const void* q, const void* k_new, const void* v_new, void* k,
                               void* v, float* u, int32_t* pos, float* v_norms, int32_t* n_out, uint8_t* keep_out,
                               float* s_out, const kv_trace* trace, const kv_rank_trace* rank_trace, void* stream) {
    kv_status rc = check_step(shape, params, t, n_in, new_pos, q, k_new, v_new, k, v, u, pos, v_norms, n_out,
                              s_out, rank_trace);
    if (rc != KV_OK) return rc;
    const kv_shape& s = *shape;
    const kv_params& p = *params;
    const int n = n_in + 1;
    const Layout L = layout_for(s, n, true);
    // slabs too long for one workgroup (the chunked scorers) need the workspace variant
    if (is_refresh(p, t) && scorer_plan(s, L, p.score_variant, p.score_merge).split) return KV_ERR_UNSUPPORTED;
    if (L.total > kStaticScratchBytes) return KV_ERR_WORKSPACE;
    void* ws = nullptr;
    if ((rc = static_scratch(&ws)) != KV_OK) return rc;
    return evict_step(s, p, t, n_in, new_pos, q, k_new, v_new, k, v, u, pos, v_norms, n_out, keep_out, s_out,
                      trace, rank_trace, L, ws, static_cast<hipStream_t>(stream));
}

kv_status kv_append(const kv_shape* shape, const kv_params* params, int32_t t, int32_t n_in, int32_t new_pos,
                    const void* k_new, const void* v_new, void* k, void* v, float* u, int32_t* pos, float* v_norms,
                    void* stream) {
    kv_status rc = check_shape(shape);
    if (rc != KV_OK) return rc;
    const kv_shape& s = *shape;
    if ((rc = check_params(params)) != KV_OK) return rc;
    if (t < 1 || n_in < 0 || n_in + 1 > s.capacity || new_pos < 0) return KV_ERR_INVALID_ARG;
    if (!k_new || !v_new || !k || !v || !u || !pos) return KV_ERR_INVALID_ARG;
    if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(u, 4) ||
        !aligned(pos, 4) || !aligned(v_norms, 4))
        return KV_ERR_UNSUPPORTED;
    return run_append(s, *params, t, n_in, new_pos, k_new, v_new, k, v, u, pos, v_norms,
                      static_cast<hipStream_t>(stream), nullptr);
}

kv_status kv_attend_score(const kv_shape* shape, int32_t layer0, int32_t layer_count, int32_t n, const void* q,
                          const void* k, const void* v, const int32_t* pos, int32_t cur_pos, float recency_bias,
                          int32_t recency_window, int32_t emit_scores, void* o, void* ws, size_t ws_bytes,
                          void* stream) {
    kv_status rc = check_shape(shape);
    if (rc != KV_OK) return rc;
    const kv_shape& s = *shape;
    if (layer0 < 0 || layer_count < 1 || layer0 + layer_count > s.layers) return KV_ERR_INVALID_ARG;
    if (n < 1 || n > s.capacity || recency_window < 0 || !isfinite(recency_bias)) return KV_ERR_INVALID_ARG;
    if (!q || !k || !v || !pos || !o) return KV_ERR_INVALID_ARG;
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(pos, 4) || !aligned(o, esize(s)))
        return KV_ERR_UNSUPPORTED;
    const Layout L = layout_for(s, n);
    if ((rc = check_ws(L, ws, ws_bytes)) != KV_OK) return rc;
    const int group = s.n_q_heads / s.n_kv_heads;
    ScorePlan plan;
    if (!attend_plan(s.dtype, s.head_dim, group, n, layer_count * s.batch * s.n_kv_heads, &plan))
        return KV_ERR_UNSUPPORTED;
    // the call's layers are its own index space: K/V and r advance to layer0, q and o are per call
    const size_t slab_elems = (size_t)s.batch * s.n_kv_heads * s.capacity * s.head_dim;
    const char* kb = static_cast<const char*>(k) + (size_t)layer0 * slab_elems * esize(s);
    const char* vb = static_cast<const char*>(v) + (size_t)layer0 * slab_elems * esize(s);
    ScoreArgs a = score_args(s, L, n, q, kb, pos, cur_pos, recency_bias, recency_window, ws);
    a.v = vb;
    a.o = o;
    a.r += (size_t)layer0 * s.batch * s.n_kv_heads * L.n_stride;
    a.layers = layer_count;
    a.chunk_rows = plan.chunk_rows;
    a.nchunk = plan.nchunk;
    if (emit_scores & ~(KV_EMIT_SCORES | KV_EMIT_VNORMS)) return KV_ERR_INVALID_ARG;
    a.emit = (emit_scores & KV_EMIT_SCORES) != 0;
    const size_t slab0 = (size_t)layer0 * s.batch * s.n_kv_heads;
    a.vn = at<float>(ws, L.vn_off) + slab0 * L.n_stride;
    a.vinv = at<float>(ws, L.vinv_off) + slab0;
    a.npart = at<float>(ws, L.npart_off);
    a.emit_norms = (emit_scores & KV_EMIT_VNORMS) != 0;
    return hip_status(launch_attend(s.dtype, s.head_dim, plan, a, static_cast<hipStream_t>(stream)));
}

kv_status kv_evict_finish(const kv_shape* shape, const kv_params* params, int32_t t, int32_t n, void* k, void* v,
                          float* u, int32_t* pos, float* v_norms, int32_t* n_out, uint8_t* keep_out, float* s_out,
                          const kv_rank_trace* rank_trace, void* ws, size_t ws_bytes, void* stream) {
    kv_status rc = check_shape(shape);
    if (rc != KV_OK) return rc;
    const kv_shape& s = *shape;
    if ((rc = check_params(params)) != KV_OK) return rc;
    if ((rc = check_rank_trace(rank_trace)) != KV_OK) return rc;
    const kv_params& p = *params;
    if ((rc = check_merge(s, p)) != KV_OK) return rc;
    if (!n_out || t < 1 || n < 1 || n > s.capacity) return KV_ERR_INVALID_ARG;
    if (!k || !v || !u || !pos) return KV_ERR_INVALID_ARG;
    if (!aligned(k, 16) || !aligned(v, 16) || !aligned(u, 4) || !aligned(pos, 4) || !aligned(s_out, 4) ||
        !aligned(v_norms, 4))
        return KV_ERR_UNSUPPORTED;
    const Layout L = layout_for(s, n);
    if ((rc = check_ws(L, ws, ws_bytes)) != KV_OK) return rc;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const bool refresh = is_refresh(p, t);
    // a refresh step with at most one eviction: the fold reports candidates and one placement kernel takes the
    // eviction and moves the newcomer (row n - 1, appended by kv_append) into its slot
    const bool single = refresh && n <= p.budget + 1 && !rank_trace;
    if (refresh) {
        // value norms already written by the step's attention calls: only the entropy factors remain; else the
        // norms come from the caller's norm cache (kv_append cached the newcomer's) or from V
        const bool emitted = (p.score_variant & KV_SCORE_NORMS_EMITTED) != 0;
        const int computed = emitted ? (p.score_variant & ~KV_SCORE_VNORM) : p.score_variant;
        float* cache_norms = emitted ? nullptr : v_norms;
        // the attention wrote one row of r per KV head; they are added in the blocks the scorer would merge,
        // so the fused and the separate step give identical utilities
        const int rblock = scorer_plan(s, L, p.score_variant, p.score_merge).merge;
        if ((rc = run_variants(s, L, n, v, computed & (KV_SCORE_VNORM | KV_SCORE_ENTROPY), s.n_kv_heads, rblock,
                               ws, st, cache_norms)) != KV_OK)
            return rc;
        FoldExtra ex;
        ex.pos = pos;
        ex.candidates = single && n > p.budget;
        ex.norms = cache_norms;
        rc = run_fold(s, L, n, u, s_out, p.rule, p.alpha, p.score_variant, s.n_kv_heads, rblock,
                      rank_trace != nullptr, ws, st, nullptr, ex);
        if (rc != KV_OK) return rc;
    }
    if (single) {
        if (n > p.budget || keep_out)
            rc = run_place(s, L, n, p.budget, nullptr, nullptr, k, v, u, pos, v_norms, keep_out, ws, st);
        if (rc != KV_OK) return rc;
        *n_out = n < p.budget ? n : p.budget;
        return KV_OK;
    }
    rc = run_select_compact(s, L, n, p.budget, k, v, u, pos, v_norms, keep_out, rank_trace, refresh, ws, st,
                            nullptr);
    if (rc != KV_OK) return rc;
    *n_out = n < p.budget ? n : p.budget;
    return KV_OK;
}

kv_status kv_score_plan(const kv_shape* shape, int32_t n, const kv_params* params, kv_score_info* info) {
    kv_status rc = check_shape(shape);
    if (rc != KV_OK) return rc;
    if ((rc = check_params(params)) != KV_OK) return rc;
    const kv_shape& s = *shape;
    if ((rc = check_merge(s, *params)) != KV_OK) return rc;
    if (!info || n < 1 || n > s.capacity) return KV_ERR_INVALID_ARG;
    const Layout L = layout_for(s, n);
    const ScorePlan plan = scorer_plan(s, L, params->score_variant, params->score_merge);
    const ScoreRoute route = score_route(s, L, n, plan);
    info->merge = plan.merge;
    info->path = (int32_t)route.kind;
    info->chunks = 1;
    if (route.kind == ScoreRoute::kExchange) {
        info->chunks = route.xp.nchunk;
    } else if (route.kind == ScoreRoute::kLogits) {
        ScorePlan cp;
        const int group = s.n_q_heads / s.n_kv_heads;
        const int lc = logit_layer_group(s, L);
        if (!attend_plan(s.dtype, s.head_dim, group, n, lc * s.batch * s.n_kv_heads, &cp, kScoreChunkLds))
            return KV_ERR_UNSUPPORTED;
        info->chunks = cp.nchunk;
    }
    return KV_OK;
}

kv_status kv_value_norms(const kv_shape* shape, int32_t n, const void* v, float* v_norms, void* stream) {
    kv_status rc = check_shape(shape);
    if (rc != KV_OK) return rc;
    const kv_shape& s = *shape;
    if (n < 1 || n > s.capacity || !v || !v_norms) return KV_ERR_INVALID_ARG;
    if (!aligned(v, 16) || !aligned(v_norms, 4)) return KV_ERR_UNSUPPORTED;
    VariantArgs a{};
    a.v = v;
    a.vnorm = v_norms;
    a.vnorm_stride = s.capacity;
    a.batch = s.batch;
    a.layers = s.layers;
    a.hkv = s.n_kv_heads;
    a.cap = s.capacity;
    a.n = n;
    a.n_stride = (n + 63) / 64 * 64;
    a.norms_direct = 1;  // the cache is not padded: one store per live row
    return hip_status(launch_vnorm(s.dtype, s.head_dim, a, static_cast<hipStream_t>(stream)));
}

kv_status kv_fault_status(void* ws, size_t ws_bytes, uint32_t* out, int32_t clear, void* stream) {
    if (!ws || ws_bytes < kFaultBytes) return KV_ERR_WORKSPACE;
    if (!aligned(ws, 256) || !aligned(out, 4)) return KV_ERR_INVALID_ARG;
    if (!out && !clear) return KV_ERR_INVALID_ARG;
    return hip_status(launch_fault_word(static_cast<uint32_t*>(ws), out, clear != 0, static_cast<hipStream_t>(stream)));
}

int32_t kv_set_exchange_wait_limit(int32_t polls) { return set_exchange_wait_limit(polls); }

kv_status kv_rank_trace_state_bytes(int32_t batch, int32_t max_pos, size_t* bytes) {
    if (batch < 1 || max_pos < 1 || !bytes) return KV_ERR_INVALID_ARG;
    *bytes = (size_t)batch * (4 + 2 * trace_words(max_pos)) * sizeof(uint32_t);
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
