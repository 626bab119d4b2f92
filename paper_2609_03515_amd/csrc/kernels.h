// Host-side launchers of the eviction-path kernels (implemented in the .hip files beside this header).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ikv {

constexpr int kMaxLayers = 256;
constexpr int kMaxGroup = 16;
constexpr int kMaxMerge = 8;   // KV heads one scoring workgroup may add up
constexpr size_t kLdsPerCu = 160 * 1024;  // gfx950

// Bits of the workspace's sticky fault word (the ABI's kv_fault values).
constexpr uint32_t kFaultExchangeTimeout = 1u;  // a first-step scoring chunk gave up waiting for its peers

// Compute units of the current device (cached per device; 0 when the query fails).
int device_cus();

// Scoring of one step (Eq. 1).  One workgroup streams a whole (layer, sequence, KV head) slab and keeps its
// logits in LDS, writing the group probability sums r.  Slabs too long for that are cut into chunks: the chunks
// of a slab exchange their per-head (max, sum) pairs and write r themselves (launch_score_coop), or, when the
// exchange words would not fit, write logits z and partial (max, sum) pairs (launch_score_chunks) that a finish
// kernel turns into r.
struct ScoreArgs {
    const void* q;
    const void* k;
    const int32_t* pos;
    float* r;       // [layers][batch][n_kv][n_stride]
    float* z;       // split: [layers][batch][n_q][n_stride] logits (score-only chunks) or exponentials relative
                    // to the chunk's maximum (attention chunks)
    float2* part;   // split: [layers][batch][n_q][nchunk] (max, sum)
    int batch, layers, hq, hkv, group, cap, n, n_stride;
    int recent_from;  // positions >= recent_from receive `bias`
    float bias;
    float scale;      // 1 / sqrt(d)
    int chunk_rows, nchunk;
    // fused decode attention only
    const void* v;  // V cache, same layout as k
    void* o;        // [layers][batch][n_q][d] attention output (dtype of q)
    float* opart;   // split: [layers][batch][n_q][nchunk][d] unnormalised partial outputs
    int emit;       // nonzero: also produce the eviction score (r)
    // fused attention, VNorm (Sec. 5.1) norms from the V pass: value-row l2 norms [layers][batch][n_kv]
    // [n_stride], the slab's 1 / mean norm, and per-chunk norm sums when chunked (emit_norms nonzero)
    float* vn;
    float* vinv;
    float* npart;   // [layers][batch][n_kv][nchunk]
    int emit_norms;
    int merge;      // scorer: KV heads per workgroup whose group sums are added (r: [layers][batch][n_kv / merge])
    // scorer (one workgroup per slab): when non-null, row n - 1 of every slab is the step's newcomer, read from
    // here ([layers][batch][n_kv][d]) instead of the cache (that row of K and of pos is not read), with
    // position new_pos
    const void* k_new;
    int new_pos;
    // multi-slab scorer with VNorm (Sec. 5.1) applied to the group sums: the caller's value-norm cache
    // ([layers][batch][n_kv][cap]), read with the K rows, and with k_new the newcomer's V rows
    // ([layers][batch][n_kv][d]); null: plain attention scores
    const float* vn_cache;
    const void* v_new;
};

struct ScorePlan {
    bool split;        // the slab is cut into chunks (planned by attend_plan)
    int group_pad;     // group size rounded up to a power of two
    int waves;         // waves per workgroup
    int rows_per_iter; // rows one workgroup covers per loop iteration
    int chunk_rows;    // rows per workgroup
    int nchunk;        // workgroups per slab
    int merge;         // KV heads whose group sums one workgroup adds (score_merge; coop_plan for chunks)
    size_t lds_bytes;  // dynamic LDS per workgroup (fast path)
    int grid;
};

bool score_plan(int dtype, int head_dim, int group, int n, ScorePlan* plan);
// Picks how many KV heads of a (layer, sequence) one LDS-resident scoring workgroup handles (lb_count =
// layers * batch; `forced` > 0: that many, a divisor of hkv) and grows the plan's LDS by their merged sums;
// 1 for split plans or when the sums do not fit.  The automatic choice queries the device (CU count, and the
// merged kernel's occupancy on first use per kernel instance).
// vnorm: the item also keeps its slabs' value norms in LDS (the scorer with VNorm fused)
int score_merge(ScorePlan* plan, int dtype, int head_dim, int hkv, int lb_count, int forced, bool vnorm = false);
// the VNorm-fused scorer exists for this shape (vector-form logits)
bool score_vnorm_fusable(int dtype, int head_dim, int group_pad);
hipError_t launch_score(int dtype, int head_dim, const ScorePlan& plan, const ScoreArgs& a, hipStream_t s);
hipError_t launch_split_finish(const ScoreArgs& a, hipStream_t s);

// Decode attention fused with the score: o_h = sum_i a_h(i) v_i for every query head, and (when emit) the
// same r as the scorer.  The plan cuts each slab into nchunk row ranges so that `slabs` slabs fill the chip;
// with nchunk > 1 the chunks write partial outputs / logits and a combine kernel (one workgroup per slab)
// produces the outputs and scores.
// max_lds caps the logits one chunk keeps in LDS (0: the largest a workgroup may use).
bool attend_plan(int dtype, int head_dim, int group, int n, int slabs, ScorePlan* plan, size_t max_lds = 0);
// LDS cap of the scorer's chunks: 52 KiB, three workgroups per CU (measured on the 32k and 128k first steps
// against 20, 40 and 80 KiB; the attention's chunks are planned for one workgroup per CU instead)
#ifndef IKV_SCORE_CHUNK_LDS
#define IKV_SCORE_CHUNK_LDS (52 * 1024)
#endif
constexpr size_t kScoreChunkLds = IKV_SCORE_CHUNK_LDS;
// LDS of one chunk of the chunk-exchange scorer: padded groups of 8 and 16 (matrix-core logits) hold two
// workgroups per CU by their registers anyway, so their chunks take the fast-path maximum of 80 KiB (fewer,
// longer chunks: fewer exchange rounds; Qwen-shaped step 1 2.47 -> 2.45 ms).  Smaller groups: 52 KiB of
// logits, three workgroups per CU; with merged teams 42.5 KiB of logits and item sums.  Step 1 with teams of
// 4 KV heads, builds alternating in one process (8B 32k / Score-Free 128k / Qwen-shaped, ms): one KV head
// per row at 52 KiB 3.996 / 4.185 / 2.412; merged at 40 KiB 3.798 / 4.156 (65 chunks of the 128k slab: too
// many words to exchange, so unmerged) / 2.356; 42.5 KiB 3.828 / 3.801 / 2.347; 46 KiB 3.748 / 3.962 / 2.355.
// Another run (unmerged at 52 KiB 4.007 / 4.181): merged at 52 KiB 4.006 / 4.007, 64 KiB (two per CU) 3.802 /
// 3.938, 80 KiB 3.784 / 4.165.
#ifndef IKV_COOP_MERGED_LDS
#define IKV_COOP_MERGED_LDS (42 * 1024 + 512)
#endif
constexpr size_t coop_chunk_lds(int group_pad, bool merged) {
    return group_pad >= 8 ? 80 * 1024 : merged ? (size_t)IKV_COOP_MERGED_LDS : kScoreChunkLds;
}
// Workspace bound over every call of 1..layers layers on n rows: the largest (layers of the call) x nchunk,
// and whether any such call splits.
struct AttendBound {
    long chunk_layers;
    bool may_split;
};
AttendBound attend_bound(int dtype, int head_dim, int group, int n, int slabs_per_layer, int layers);
hipError_t launch_attend(int dtype, int head_dim, const ScorePlan& plan, const ScoreArgs& a, hipStream_t s);
// Scoring of long slabs in LDS-resident chunks (the attention kernel without its V pass): logits and per-chunk
// (max, sum) for launch_split_finish; plan from attend_plan.
hipError_t launch_score_chunks(int dtype, int head_dim, const ScorePlan& plan, const ScoreArgs& a, hipStream_t s);
// Scoring of long slabs in chunks that exchange their softmax statistics instead of writing logits: plan
// (chunk_rows, nchunk, lds_bytes) from attend_plan with at most kCoopMaxWords / group_pad chunks; grid = a
// multiple of nchunk no larger than coop_workgroups() (the workgroups the device holds at once).  xchg: zeroed
// here, then one 64-bit word per (layer, sequence, query head, chunk).  A chunk whose peers' words do not all
// arrive within the wait limit sets its group sums to NaN and ORs kFaultExchangeTimeout into *faults.
// With merge > 1 (a divisor of n_kv) the chunks of one team score the merge KV heads of a (layer, sequence)
// in consecutive rounds and add their group sums in LDS (a.merge; r: [layers][batch][n_kv / merge] rows).
constexpr int kCoopMaxWords = 4 * 64;
// The chunk plan of the exchange scorer for `merge`: attend_plan's chunks under the LDS cap coop_chunk_lds(),
// which with merge > 1 also holds the item sums (4 bytes per row); lds_bytes is the kernel's whole dynamic LDS.
bool coop_plan(int dtype, int head_dim, int group, int n, int slabs, int merge, ScorePlan* plan);
int coop_workgroups(int dtype, int head_dim, const ScorePlan& plan);
hipError_t launch_score_coop(int dtype, int head_dim, const ScorePlan& plan, const ScoreArgs& a, uint64_t* xchg,
                             int grid, uint32_t* faults, hipStream_t s);
// Polls of the exchange wait (< 0: the default, about 0.1 s of sleeps; 0: give up at once); returns the
// previous limit.  Process-wide.
int set_exchange_wait_limit(int polls);
// Fault word: zeroes it, or copies it to `out` (device) and optionally zeroes it, in stream order.
hipError_t launch_fault_word(uint32_t* word, uint32_t* out, bool clear, hipStream_t s);

// Eviction candidate of a range of tokens: the token that leaves first under (u ascending, position
// descending), as the order-preserving key of its utility, its position and its slot (-1: none).
struct EvictCand {
    uint32_t key;
    int pos, idx;
};

// Layer fold (Eq. 2-4): u <- prior_w * u + sum_l w_l s_l with s_l = (1/H) sum_g r_{l,g}.
struct FoldArgs {
    const float* r;
    const float* vnorm;           // nullable: [layers][batch][n_kv][n_stride] value-row l2 norms
    const float* vnorm_inv_mean;  // [layers][batch][n_kv] 1 / mean norm (0: all norms zero, factor 1)
    const float* entropy;         // nullable: [layers][batch] normalised entropy of the layer's attention
    int vnorm_stride;             // row stride of vnorm: n_stride (workspace) or cap (the caller's norm cache)
    float* raw;                   // nullable: [batch][cap] rank trace's raw score (plain scores, layer mean)
    float raw_scale;              // 1 / (layers * n_q)
    float* u;
    float* s_out;  // nullable [layers][batch][n]
    int batch, layers, hkv, n, n_stride, cap;
    // rows of r per (layer, sequence), added in blocks of rblock consecutive rows (block sums first, then the
    // blocks in order: the order a scorer merging rblock KV heads per workgroup adds them in)
    int r_groups, rblock;
    float inv_hq;
    float prior_w;
    // new_pos >= 0: token n - 1 is the step's newcomer, not yet in u / pos: its previous utility is taken as
    // 0 (the refresh prior) and pos[n - 1] = new_pos is written with its folded utility
    int new_pos;
    int32_t* pos;     // positions (read for the candidates, written for the newcomer)
    EvictCand* cand;  // nullable: [batch][fold_groups(n)] eviction candidate of each workgroup's tokens
    float w[kMaxLayers];
};
hipError_t launch_fold(const FoldArgs& a, hipStream_t s);
// Workgroups of the fold per sequence (each covers a fixed range of tokens and writes one candidate).
int fold_groups(int n);

// Scorer perturbations (Sec. 5.1): value-row norms with their per-slab mean, and the normalised entropy of
// each layer's pooled attention, computed from the group sums r.
struct VariantArgs {
    const void* v;
    const float* r;
    float* vnorm;           // [layers][batch][n_kv][vnorm_stride]
    float* vnorm_inv_mean;  // [layers][batch][n_kv] (nullable for launch_vnorm: norms only)
    float* entropy;         // [layers][batch]
    int batch, layers, hkv, cap, n, n_stride;
    int vnorm_stride;       // n_stride (workspace norms) or cap (the caller's norm cache)
    int norms_direct;       // launch_vnorm: one 4-byte store per live row (unpadded rows, e.g. the norm cache)
    int r_groups, rblock;  // as in FoldArgs
    float inv_hq;
    // launch_vnorm_mean: when non-null, row n - 1 is the step's newcomer, not yet cached: its norm is taken
    // from v_new ([layers][batch][n_kv][d]) and written to the cache before the mean
    const void* v_new;
};
// Norms of rows [0, n) read from V into vnorm, and (when vnorm_inv_mean is set) each slab's n / sum of norms.
hipError_t launch_vnorm(int dtype, int head_dim, const VariantArgs& a, hipStream_t s);
// Each slab's n / sum of norms from the norm cache (vnorm, stride cap), with the newcomer's norm from v_new.
hipError_t launch_vnorm_mean(int dtype, int head_dim, const VariantArgs& a, hipStream_t s);
hipError_t launch_entropy(const VariantArgs& a, hipStream_t s);

// Rank trace (appendix "Mechanistic Diagnostics"): per-sequence set statistics (the raw step score comes from
// the fold).
constexpr int kTraceCounts = 10;
struct TraceArgs {
    const int32_t* pos;      // positions before compaction
    const uint8_t* raw_keep; // [batch][cap] top-k of raw
    const uint8_t* ema_keep; // [batch][cap] top-k of u
    const uint8_t* keep;     // [batch][cap] the step's retention decision
    uint32_t* state;         // per sequence: header (4 words) + raw bitmap + ema bitmap
    int32_t* counts;         // [batch][kTraceCounts]
    int batch, cap, n, max_pos, words;  // words: bitmap words per set
};
hipError_t launch_trace_stats(const TraceArgs& a, bool skip, hipStream_t s);

// Selection + compaction plan, one workgroup per sequence.
struct SelectArgs {
    const float* u;
    const int32_t* pos;
    const uint8_t* keep_in;  // plan-only mode: the retention decision to compact
    uint8_t* keep_out;       // nullable: decision written here ([batch][cap])
    int32_t* pair_dst;       // [batch][max_pairs]
    int32_t* pair_src;
    int32_t* npairs;         // [batch]
    int batch, cap, n, budget, max_pairs;
    uint32_t* wide;          // scratch of the multi-workgroup selection (select_wide_words words)
};
hipError_t launch_select(const SelectArgs& a, bool plan_only, hipStream_t s);
// Scratch words of the multi-workgroup selection for a batch (0: that path is never taken for it).
size_t select_wide_words(int batch);

// Row moves of the compaction plan for K, V, u and pos.
struct MoveArgs {
    void* k;
    void* v;
    float* u;
    int32_t* pos;
    const int32_t* pair_dst;
    const int32_t* pair_src;
    const int32_t* npairs;
    int batch, layers, hkv, cap, row_bytes;
    int max_pairs;    // loop bound on pairs per sequence
    int pair_stride;  // row stride of pair_dst / pair_src
    float* norms;     // nullable: value-norm cache [layers][batch][n_kv][cap], moved with V
};
hipError_t launch_move(const MoveArgs& a, hipStream_t s);

// Append of the new token's K/V rows, position and prior utility.
struct AppendArgs {
    void* k;
    void* v;
    const void* k_new;
    const void* v_new;
    float* u;
    int32_t* pos;
    int batch, layers, hkv, cap, row_bytes, n_in, new_pos;
    int init_mode;  // 0: zero (refresh step), 1: mean, 2: min of u[0, n_in)
    float* norms;   // nullable: value-norm cache [layers][batch][n_kv][cap]: the newcomer's norms are written
                    // where its V rows go
    int bf16;       // element type of the rows (for the norms)
};
hipError_t launch_append(const AppendArgs& a, hipStream_t s);
// A non-refresh step on a cache of n_in <= budget tokens (init_mode 1 or 2): the newcomer's prior, the single
// eviction and the newcomer's slot (one workgroup per sequence; slot[batch] in device memory), then its rows
// copied into that slot by a kernel over every (layer, KV head) row.
hipError_t launch_nonrefresh(const AppendArgs& a, uint8_t* keep_out, int budget, int* slot, hipStream_t s);

// A refresh step on a cache of n - 1 <= budget tokens after the fold: the newcomer (slot n - 1, already folded
// into u[n - 1] / pos[n - 1]) takes the slot of the single evicted token, the least of the fold's candidates
// (n = budget + 1), or slot n - 1 when nothing is evicted; it is dropped when it is itself the least.  Its K/V
// rows are read from src (row src_row0 of slab s at src + (s * src_slab_rows + src_row0) * row_bytes: the
// step's k_new / v_new, or row n - 1 of the cache) and written into that slot, with its utility and position.
// One workgroup per (layer, sequence).
struct PlaceArgs {
    void* k;
    void* v;
    float* u;
    int32_t* pos;
    const void* src_k;
    const void* src_v;
    size_t src_slab_rows, src_row0;
    const EvictCand* cand;  // [batch][ncand]
    uint8_t* keep_out;      // nullable: the decision over the n slots
    int ncand;
    int batch, layers, hkv, cap, row_bytes, n, budget;
    float* norms;           // nullable: value-norm cache, the newcomer's norms written into its slot
    int bf16;
};
hipError_t launch_place(const PlaceArgs& a, hipStream_t s);

}  // namespace ikv
