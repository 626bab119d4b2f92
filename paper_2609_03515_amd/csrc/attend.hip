// Decode attention fused with the eviction score (Eq. 1) for gfx950.
//
// At every layer a decoder attends its last query over the cached rows; the method's per-step score is the
// same softmax, mean-pooled over query heads.  Computing both in one kernel lets a single pass over K serve
// the attention output and the score (the separate score pass is the dominant per-step cost of the method in
// the paper's profiling), and V is read once for the output.
//
// One workgroup per (layer, sequence, KV head, row chunk):
//   1. K pass: logits of the chunk's rows for the group's heads into LDS (the scorer's lane machinery and
//      dynamic unit claiming), running per-head max;
//   2. e = exp(z - max) in place with per-head sums (with the score: a pass of its own; without: by the wave
//      that claims a block in the V pass), then the V pass: every lane accumulates e_h(row) * v(row) for the
//      GP heads over its 16-byte V chunks, the probabilities of a row being GP consecutive LDS words;
//   3. cross-lane / cross-wave reduction in a fixed order, then either the normalised output (one chunk per
//      slab) or the chunk's unnormalised partial output with its per-head (max, sum);
//   4. when the score is wanted: the group probability sums r of the rows (one chunk), or the chunk's
//      exponentials (several chunks), which a combine kernel turns into outputs and scores.
// Chunks exist so that one layer's slabs (batch x KV heads, e.g. 64) still occupy all 256 CUs.
#include "stream_lane.h"

namespace ikv {
namespace {

#ifndef IKV_ATTN_TARGET
#define IKV_ATTN_TARGET 256
#endif
#ifndef IKV_ATTN_NBUF
#define IKV_ATTN_NBUF 0
#endif
#ifndef IKV_ATTN_MIN_ROWS
#define IKV_ATTN_MIN_ROWS 256
#endif
// workgroups per launch wanted: one per CU.  Measured for one decoder layer at batch 8 (64 slabs): 256 chunks
// beat 512 by 8%; counts that are not a multiple of the CU count (320, 384) leave CUs unevenly loaded.
constexpr int kAttnTargetWgs = IKV_ATTN_TARGET;
constexpr int kAttnMinRows = IKV_ATTN_MIN_ROWS;   // smallest chunk: below it a chunk's fixed costs dominate

template <int GP>
__device__ __forceinline__ void read_probs(const float* src, float (&e)[GP]) {
    if constexpr (GP >= 4) {
#pragma unroll
        for (int i = 0; i < GP; i += 4) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(src + i);
            e[i] = v.x;
            e[i + 1] = v.y;
            e[i + 2] = v.z;
            e[i + 3] = v.w;
        }
    } else {
#pragma unroll
        for (int i = 0; i < GP; ++i) e[i] = src[i];
    }
}

// Several chunks per slab: a combine kernel after the chunks' launch, combine_parts(n) workgroups per slab:
//   o_h = sum_c exp(m_c - M_h) o_c / sum_c exp(m_c - M_h) S_c,  M_h = max_c m_c   (part 0);
//   r(row) = sum_{h in group} exp(z_h(row) - M_h) / S_h = sum_h e_h(row) exp(m_c - M_h) / S_h from the
//   exponentials e_h = exp(z_h - m_c) the chunks wrote (c: the row's chunk), when emitting (part p: rows
//   [p kCombineRows, (p + 1) kCombineRows)).
// The rows are spread over several workgroups because one per slab left the score's rows (52 KB of logits per
// slab at the 8B shape) to 64 workgroups at one decoder layer's batch.
// Electing the last chunk of a slab inside the attention kernel instead was measured twice at the 8B shape:
// with a device-scope release/acquire fence in every chunk (a full L2 write-back and invalidate) 5x slower per
// layer; with the partials written and read back by device-scope (write-through) accesses and a completion
// wait before the arrival count, no faster without the score (the chunk's store, count and reload round trips
// cost what the kernel boundary does) and 9% slower with it (one workgroup per slab takes the score's rows).
constexpr int kCombineRows = 1024;
__host__ __device__ constexpr int combine_parts(int n, bool emit) { return emit ? (n + kCombineRows - 1) / kCombineRows : 1; }

template <typename T, int D, int GP>
__global__ __launch_bounds__(kThreads) void attend_combine_kernel(ScoreArgs a) {
    __shared__ float cm[GP], ci[GP];
    const int parts = combine_parts(a.n, a.emit);
    const int s = blockIdx.x / parts;  // slab: (l * batch + b) * hkv + g, l relative to the call
    const int part = blockIdx.x % parts;
    const size_t head0 = (size_t)(s / a.hkv) * a.hq + (size_t)(s % a.hkv) * a.group;
    // The loops over chunks load four chunks' values before using them (the loads are independent; the
    // arithmetic keeps the sequential order, so the result does not depend on the unrolling).
    constexpr int kU = 4;
    if (threadIdx.x < a.group) {
        const float2* pp = a.part + (head0 + threadIdx.x) * a.nchunk;
        float mx = -INFINITY;
        int c = 0;
        for (; c + kU <= a.nchunk; c += kU) {
            float2 p[kU];
#pragma unroll
            for (int j = 0; j < kU; ++j) p[j] = pp[c + j];
#pragma unroll
            for (int j = 0; j < kU; ++j) mx = fmaxf(mx, p[j].x);
        }
        for (; c < a.nchunk; ++c) mx = fmaxf(mx, pp[c].x);
        float tot = 0.0f;
        for (c = 0; c + kU <= a.nchunk; c += kU) {
            float2 p[kU];
#pragma unroll
            for (int j = 0; j < kU; ++j) p[j] = pp[c + j];
#pragma unroll
            for (int j = 0; j < kU; ++j) tot = fmaf(__expf(p[j].x - mx), p[j].y, tot);
        }
        for (; c < a.nchunk; ++c) tot = fmaf(__expf(pp[c].x - mx), pp[c].y, tot);
        cm[threadIdx.x] = mx;
        ci[threadIdx.x] = tot > 0.0f ? 1.0f / tot : 0.0f;
    }
    if (a.emit_norms && part == 0 && threadIdx.x == kWave) {  // (another wave than the one filling cm / ci)
        float tot = 0.0f;
        for (int c = 0; c < a.nchunk; ++c) tot += a.npart[(size_t)s * a.nchunk + c];
        a.vinv[s] = tot > 0.0f ? (float)a.n / tot : 0.0f;
    }
    __syncthreads();
    T* ob = static_cast<T*>(a.o) + head0 * D;
    for (int idx = threadIdx.x; part == 0 && idx < a.group * D; idx += kThreads) {
        const int h = idx / D;
        const float2* pp = a.part + (head0 + h) * a.nchunk;
        const float* op = a.opart + (head0 + h) * a.nchunk * D + idx % D;
        float acc = 0.0f;
        int c = 0;
        for (; c + kU <= a.nchunk; c += kU) {
            float m[kU], x[kU];
#pragma unroll
            for (int j = 0; j < kU; ++j) {
                m[j] = pp[c + j].x;
                x[j] = op[(size_t)(c + j) * D];
            }
#pragma unroll
            for (int j = 0; j < kU; ++j) acc = fmaf(__expf(m[j] - cm[h]), x[j], acc);
        }
        for (; c < a.nchunk; ++c) acc = fmaf(__expf(pp[c].x - cm[h]), op[(size_t)c * D], acc);
        Elem<T>::store(ob + idx, acc * ci[h]);
    }
    if (a.emit) {
        // the rows hold e_h(row) = exp(z - m_c) of their chunk c (4 rows per thread and pass lie in one chunk: chunks
        // are a multiple of 4 rows; rows are padded to a multiple of 64, rows >= n are scratch):
        // r(row) = sum_h e_h(row) exp(m_c - M_h) / S_h
        const float* zb = a.z + head0 * a.n_stride;
        float* rb = a.r + (size_t)s * a.n_stride;
        const int row_end = min(a.n, (part + 1) * kCombineRows);
        for (int row = part * kCombineRows + threadIdx.x * 4; row < row_end; row += kThreads * 4) {
            const int c = row / a.chunk_rows;
            f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
            for (int h = 0; h < a.group; ++h) {
                const f32x4 e = *reinterpret_cast<const f32x4*>(zb + (size_t)h * a.n_stride + row);
                const float f = __expf(a.part[(head0 + h) * a.nchunk + c].x - cm[h]) * ci[h];
                acc.x += e.x * f;
                acc.y += e.y * f;
                acc.z += e.z * f;
                acc.w += e.w * f;
            }
            *reinterpret_cast<f32x4*>(rb + row) = acc;
        }
    }
}

// Waves per SIMD the compiler must leave room for: bf16 rows of d = 128 with groups of 4 (the 8B shape) are held
// to 128 registers, i.e. two workgroups per CU, which the all-layer call (2,048 workgroups) uses: uncapped the
// kernel takes 129 and that call with the score measured 1% slower.  Other instances keep what they need.
template <typename T, int D, int GP, bool kV>
constexpr int attend_waves_per_eu() {
    return (kV && GP == 4 && D == 128 && std::is_same<T, bf16_t>::value) ? 4 : 1;
}

// kV = false: score only (no V pass, no output), for scoring long slabs in chunks: the chunks write their
// logits and per-head (max, sum) for the scorer's finish kernel.
template <typename T, int D, int GP, bool kV>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(attend_waves_per_eu<T, D, GP, kV>())))
void attend_kernel(ScoreArgs a) {
    using L = Lane<T, D, GP>;
    using E = Elem<T>;
    using chunk_t = typename L::chunk_t;
    constexpr int RPG = L::RPG, CPL = L::CPL, RPW = L::RPW, LPR = L::LPR, EPC = L::EPC;
    // K/V loads of two units in flight, one when a lane's share of a unit is already large (a single head
    // per KV head: 16 rows per lane), which would otherwise spill
    constexpr int kNbuf = IKV_ATTN_NBUF > 0 ? IKV_ATTN_NBUF : (RPG * CPL > 8 ? 1 : 2);
    using KP = KUnit<T, D, GP>;
    constexpr int kNbufK = use_mfma<T, D, GP>() ? 2 : kNbuf;  // K units in flight (16 rows each on MFMA)

    // the waves' partial outputs are added in one step when every wave's slice fits 16 KiB of LDS (GP * D <= 512
    // floats: groups up to 4 at d = 128), else wave by wave (one barrier each); the sums are the same
    constexpr bool kWaveSlices = kWaves * GP * D <= 4096;
    extern __shared__ float zs[];
    __shared__ float red_m[kWaves][GP], red_s[kWaves][GP], red_n[kWaves];
    __shared__ float obuf[kV ? (kWaveSlices ? kWaves : 1) * GP * D : 1];
    __shared__ int next_unit[2];

    const L ln;
    const KP kp;
    const int chunk = blockIdx.x % a.nchunk;
    const int s = blockIdx.x / a.nchunk;  // slab: (l * batch + b) * hkv + g, l relative to the call
    const int g = s % a.hkv;
    const int lb = s / a.hkv;
    const int b = lb % a.batch;
    const int row0 = chunk * a.chunk_rows;
    const int nrows = min(a.n - row0, a.chunk_rows);  // >= 1: the plan leaves no empty chunk
    const int nunits = (nrows + RPW - 1) / RPW;          // LDS blocks of logits (and V units)
    const int nku = (nrows + KP::kRows - 1) / KP::kRows;  // claimed units of the K pass
    const size_t base = ((size_t)s * a.cap + row0) * D;
    const __amdgpu_buffer_rsrc_t krs = raw_rsrc(static_cast<const T*>(a.k) + base, nrows * L::kRowBytes);
    const __amdgpu_buffer_rsrc_t vrs = raw_rsrc(static_cast<const T*>(a.v) + base, nrows * L::kRowBytes);
    const __amdgpu_buffer_rsrc_t prs = raw_rsrc(a.pos + (size_t)b * a.cap + row0, nrows * 4);

    if (threadIdx.x == 0) {
        next_unit[0] = 0;
        next_unit[1] = 0;
    }
    typename KP::q_t qv;
    kp.load_q(a, (size_t)lb, g, qv);
    __syncthreads();
    auto claim = [&](int which) -> int {
        int u = 0;
        if (ln.lane == 0) u = atomicAdd(&next_unit[which], 1);
        return __builtin_amdgcn_readfirstlane(u);
    };

    // 1. K pass
    typename KP::max_t mk = kp.max_init();
    {
        typename KP::buf_t kbuf[kNbufK];
        int pbuf[kNbufK];
        claimed_units<kNbufK>(
            nku, -1, [&]() __attribute__((always_inline)) { return claim(0); },
            [&](auto slot, int u) __attribute__((always_inline)) { kp.load(krs, prs, u, kbuf[slot], pbuf[slot]); },
            [&](auto slot, int u) __attribute__((always_inline)) { kp.logits(a, kbuf[slot], qv, pbuf[slot], u, nrows, zs, mk); });
    }

    // the V stream's first loads are issued now, so their latency overlaps the K pass's epilogue (barriers
    // wait for LDS only, not for these loads)
    chunk_t vbuf[kNbuf][RPG][CPL];
    int vfirst = -1;
    if constexpr (kV && kNbuf == 2) {
        vfirst = claim(1);
        ln.load_rows(vrs, vfirst, vbuf[0]);
    }

    // per-head max, then the exponentials in place with their per-head sums: in a pass of their own when a score
    // is produced (several chunks: the logits go to HBM on the way, for the finish or combine kernel), else
    // inside the V pass (below)
    kp.publish_max(mk, red_m[ln.wave]);
    __syncthreads();
    float m = red_m[0][ln.hh];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) m = fmaxf(m, red_m[w][ln.hh]);

    float* zl = zs + ln.wave * kWave + ln.lane;
    constexpr int kStep = kWaves * kWave;
    const int mine = nunits > ln.wave ? (nunits - ln.wave + kWaves - 1) / kWaves : 0;
    const bool write_z = !kV && a.emit && a.nchunk > 1;  // (with V, a chunk's exponentials are stored later)
    // this lane's head's logit row (lanes of one wave hold different heads: stored by address)
    float* zrow = a.z + ((size_t)lb * a.hq + (size_t)g * a.group + ln.hh) * a.n_stride + row0;
    float ssum = 0.0f;
    auto expo = [&](float z, int unit) {
        // -inf: padded head or row past the end
        if (write_z && z != -INFINITY) store_stream_at(zrow + ln.unit_row(unit), z);
        return z == -INFINITY ? 0.0f : __expf(z - m);
    };
    // Measured for one decoder layer per call (8B shape): exponentials inside the V pass save the pass and its
    // barrier (32 calls 790 -> 769 us without the score).  With the score, a slab cut in chunks then stores its
    // exponentials after the streams (stored during the V pass, with the logits, they had cost 842 -> 867 us);
    // one chunk per slab keeps the pass, whose sums are the scorer's bit for bit.
    const bool exp_apart = !kV || (a.emit && a.nchunk == 1);
    if (exp_apart) {
        int i = 0;
        for (; i + kEpi <= mine; i += kEpi) {
            float e[kEpi];
#pragma unroll
            for (int v = 0; v < kEpi; ++v) e[v] = zl[(i + v) * kStep];
#pragma unroll
            for (int v = 0; v < kEpi; ++v) {
                e[v] = expo(e[v], ln.wave + (i + v) * kWaves);
                ssum += e[v];
                if (kV) zl[(i + v) * kStep] = e[v];
            }
        }
        for (; i < mine; ++i) {
            const float e = expo(zl[i * kStep], ln.wave + i * kWaves);
            ssum += e;
            if (kV) zl[i * kStep] = e;
        }
#pragma unroll
        for (int o = GP; o < kWave; o <<= 1) ssum += __shfl_xor(ssum, o, kWave);
        if (ln.lane < GP) red_s[ln.wave][ln.lane] = ssum;
        __syncthreads();  // also publishes every exponential to the V pass
    }
    if constexpr (!kV) {
        if (threadIdx.x < a.group) {
            const size_t h = (size_t)lb * a.hq + (size_t)g * a.group + threadIdx.x;
            float mx = red_m[0][threadIdx.x], tot = red_s[0][threadIdx.x];
#pragma unroll
            for (int w = 1; w < kWaves; ++w) {
                mx = fmaxf(mx, red_m[w][threadIdx.x]);
                tot += red_s[w][threadIdx.x];
            }
            a.part[h * a.nchunk + chunk] = make_float2(mx, tot);
        }
        return;
    } else {

    // 2. V pass: acc[h][c][x] = sum over this lane's rows of e_h(row) * v(row)[(p + c LPR) EPC + x]; with
    //    emit_norms also the rows' value norms (VNorm), written out and summed.  Without the score the wave
    //    that claims a block first turns its logits into exponentials in place (each lane the word it owns) and
    //    adds them to its sums; the block's probabilities are then read by the wave's own lanes, so no
    //    workgroup barrier separates the exponentials from the V stream.
    const __amdgpu_buffer_rsrc_t vns =
        raw_rsrc(a.vn + (size_t)s * a.n_stride + row0, a.emit_norms ? nrows * 4 : 0);
    float nsum = 0.0f;
    float acc[GP][CPL][EPC];
#pragma unroll
    for (int h = 0; h < GP; ++h)
#pragma unroll
        for (int c = 0; c < CPL; ++c)
#pragma unroll
            for (int x = 0; x < EPC; ++x) acc[h][c][x] = 0.0f;
    {
        int ubuf[kNbuf];
        if constexpr (kNbuf == 2) ubuf[0] = vfirst;
        bool more = true;
        while (more) {
#pragma unroll
            for (int j = 0; j < kNbuf; ++j) {
                const int slot = (j + kNbuf - 1) % kNbuf;
                ubuf[slot] = claim(1);
                ln.load_rows(vrs, ubuf[slot], vbuf[slot]);
                if (more && ubuf[j] < nunits) {
                    float* eb = zs + ubuf[j] * kWave;
                    if (!exp_apart) {
                        const float e = expo(eb[ln.lane], ubuf[j]);
                        ssum += e;
                        eb[ln.lane] = e;
                        __builtin_amdgcn_wave_barrier();  // (the reads below are of words other lanes just wrote)
                    }
                    // row k * NG + grp of the unit: its GP probabilities are words grp * LPR + k * GP + [0, GP)
                    const float* eu = eb + ln.grp * LPR;
#pragma unroll
                    for (int k = 0; k < RPG; ++k) {
                        float e[GP];
                        read_probs<GP>(eu + k * GP, e);
                        float ss = 0.0f;
#pragma unroll
                        for (int c = 0; c < CPL; ++c) {
                            float f[EPC];
                            E::unpack(vbuf[j][k][c], f);
#pragma unroll
                            for (int h = 0; h < GP; ++h)
#pragma unroll
                                for (int x = 0; x < EPC; ++x) acc[h][c][x] = fmaf(e[h], f[x], acc[h][c][x]);
#pragma unroll
                            for (int x = 0; x < EPC; ++x) ss = fmaf(f[x], f[x], ss);
                        }
                        if (a.emit_norms) {  // VNorm: the row's l2 norm, summed over its lane group
                            ss = group_allsum<LPR>(ss);
                            const int row = ubuf[j] * RPW + k * L::NG + ln.grp;
                            if (ln.p == 0 && row < nrows) {
                                const float nrm = sqrtf(ss);
                                store_stream(vns, row * 4, nrm);
                                nsum += nrm;
                            }
                        }
                    }
                } else {
                    more = false;
                }
            }
        }
    }

    if (a.emit_norms) {
#pragma unroll
        for (int o = kWave / 2; o >= 1; o >>= 1) nsum += __shfl_xor(nsum, o, kWave);
        if (ln.lane == 0) red_n[ln.wave] = nsum;  // read after the barriers below
    }
    if (!exp_apart) {  // the sums the waves took over the blocks they claimed
#pragma unroll
        for (int o = GP; o < 16; o <<= 1) ssum += __shfl_xor(ssum, o, kWave);
        ssum = rows_allsum(ssum);
        if (ln.lane < GP) red_s[ln.wave][ln.lane] = ssum;  // read after the barriers below
    }

    // 3. lanes holding the same chunk of different rows (stride LPR), then the waves in order.  With 16 lanes
    //    per row the four rows hold the same chunks: four accumulators at a time are reduced over the rows with
    //    row swaps, leaving accumulator 4i + r in row r (in the butterfly's order, so the sums are unchanged),
    //    and every lane stores its share of the wave's slice.  Measured at the 8B shape, one decoder layer per
    //    call: 24.6 -> 23.4 us; the 64 cross-row shuffles of the butterfly had kept the LDS crossbar busy for
    //    ~1 us after the V pass.
    constexpr int kAcc = GP * CPL * EPC;
    constexpr bool kRowSwaps = kWaveSlices && LPR == 16 && kAcc % 4 == 0;
    if constexpr (!kRowSwaps) {
#pragma unroll
        for (int o = LPR; o < kWave; o <<= 1)
#pragma unroll
            for (int h = 0; h < GP; ++h)
#pragma unroll
                for (int c = 0; c < CPL; ++c)
#pragma unroll
                    for (int x = 0; x < EPC; ++x) acc[h][c][x] += __shfl_xor(acc[h][c][x], o, kWave);
    }
    if constexpr (kWaveSlices) {
        // each wave's partial in its own slice; then output idx = ((w0 + w1) + w2) + ... by the thread that later
        // stores it (the same thread-to-output mapping as the stores below, so no barrier between)
        float* slice = obuf + ln.wave * GP * D;
        if constexpr (kRowSwaps) {
            const float* flat = &acc[0][0][0];  // index (h CPL + c) EPC + x
            const int r = ln.lane / 16;
#pragma unroll
            for (int i = 0; i < kAcc / 4; ++i) {
                const float t = rows_sum4(flat[4 * i], flat[4 * i + 1], flat[4 * i + 2], flat[4 * i + 3]);
                const int ai = 4 * i + r;
                const int h = ai / (CPL * EPC), c = ai / EPC % CPL, x = ai % EPC;
                slice[h * D + (ln.p + c * LPR) * EPC + x] = t;
            }
        } else if (ln.lane < LPR) {
#pragma unroll
            for (int h = 0; h < GP; ++h)
#pragma unroll
                for (int c = 0; c < CPL; ++c)
#pragma unroll
                    for (int x = 0; x < EPC; ++x) slice[h * D + (ln.p + c * LPR) * EPC + x] = acc[h][c][x];
        }
        __syncthreads();
        for (int idx = threadIdx.x; idx < a.group * D; idx += kThreads) {
            float t = obuf[idx];
#pragma unroll
            for (int w = 1; w < kWaves; ++w) t += obuf[w * GP * D + idx];
            obuf[idx] = t;
        }
    } else {
        for (int w = 0; w < kWaves; ++w) {
            if (ln.wave == w && ln.lane < LPR) {
#pragma unroll
                for (int h = 0; h < GP; ++h)
#pragma unroll
                    for (int c = 0; c < CPL; ++c)
#pragma unroll
                        for (int x = 0; x < EPC; ++x) {
                            const int idx = h * D + (ln.p + c * LPR) * EPC + x;
                            obuf[idx] = w == 0 ? acc[h][c][x] : obuf[idx] + acc[h][c][x];
                        }
            }
            __syncthreads();
        }
    }
    if (a.emit && a.nchunk > 1) {
        // the chunk's exponentials e_h(row) = exp(z - m_h) (m_h: this chunk's maximum), every block's already in
        // LDS (the barriers above follow the V pass), to the logit rows for the combine: 4 rows of one head per
        // thread and 16-byte store; rows past the chunk give 0 (rows are padded to a multiple of 64)
        float* zc = a.z + ((size_t)lb * a.hq + (size_t)g * a.group) * a.n_stride + row0;
        const int quads = (nrows + 3) / 4;
        for (int t = threadIdx.x; t < a.group * quads; t += kThreads) {
            const int h = t / quads, r0 = t % quads * 4;
            f32x4 e;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int row = r0 + j, rib = row % RPW;
                e[j] = row < nrows ? zs[row / RPW * kWave + rib % L::NG * LPR + rib / L::NG * GP + h] : 0.0f;
            }
            *reinterpret_cast<f32x4*>(zc + (size_t)h * a.n_stride + r0) = e;
        }
    }
    auto head_sum = [&](int h) {
        float t = red_s[0][h];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) t += red_s[w][h];
        return t;
    };
    auto head_max = [&](int h) {
        float t = red_m[0][h];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) t = fmaxf(t, red_m[w][h]);
        return t;
    };
    const size_t head0 = (size_t)lb * a.hq + (size_t)g * a.group;
    if (a.emit_norms && threadIdx.x == 0) {
        float tot = 0.0f;
        for (int w = 0; w < kWaves; ++w) tot += red_n[w];
        if (a.nchunk == 1)
            a.vinv[s] = tot > 0.0f ? (float)a.n / tot : 0.0f;
        else
            a.npart[(size_t)s * a.nchunk + chunk] = tot;
    }
    if (a.nchunk == 1) {
        T* ob = static_cast<T*>(a.o) + head0 * D;
        for (int idx = threadIdx.x; idx < a.group * D; idx += kThreads) {
            const float tot = head_sum(idx / D);
            E::store(ob + idx, tot > 0.0f ? obuf[idx] / tot : 0.0f);
        }
    } else {
        for (int idx = threadIdx.x; idx < a.group * D; idx += kThreads) {
            const int h = idx / D;
            a.opart[((head0 + h) * a.nchunk + chunk) * D + idx % D] = obuf[idx];
        }
        if (threadIdx.x < a.group)
            a.part[(head0 + threadIdx.x) * a.nchunk + chunk] =
                make_float2(head_max(threadIdx.x), head_sum(threadIdx.x));
        return;
    }

    // 4. one chunk: the score's group probability sums, staged in each unit's first RPW words (only this
    //    wave reads its units, and the V pass is over) and written with 16-byte stores
    if (a.emit && a.nchunk == 1) {
        static_assert(RPW % 4 == 0, "the coalesced store moves 4 rows at a time");
        const float tot = head_sum(ln.hh);
        const float inv = tot > 0.0f ? 1.0f / tot : 0.0f;
        const int row_in = ln.kk * L::NG + ln.grp;  // this lane's row inside a unit
        int i = 0;
        for (; i + kEpi <= mine; i += kEpi) {  // kEpi units' reads in flight at a time
            float e[kEpi];
#pragma unroll
            for (int v = 0; v < kEpi; ++v) e[v] = zl[(i + v) * kStep];
#pragma unroll
            for (int v = 0; v < kEpi; ++v) e[v] = group_allsum<GP>(e[v] * inv);
            if (ln.hh == 0)
#pragma unroll
                for (int v = 0; v < kEpi; ++v) zs[(ln.wave + (i + v) * kWaves) * kWave + row_in] = e[v];
        }
        for (; i < mine; ++i) {
            const float sum = group_allsum<GP>(zl[i * kStep] * inv);
            if (ln.hh == 0) zs[(ln.wave + i * kWaves) * kWave + row_in] = sum;
        }
        __syncthreads();
        const __amdgpu_buffer_rsrc_t rrs = raw_rsrc(a.r + (size_t)s * a.n_stride, a.n_stride * 4);
        for (int j = threadIdx.x; j * 4 < nrows; j += kThreads) {
            const int row = j * 4;
            store_stream(rrs, row * 4, *reinterpret_cast<const f32x4*>(&zs[(row / RPW) * kWave + row % RPW]));
        }
    }
    }  // kV
}

template <typename T, int D, int GP>
hipError_t launch_attend_gp(const ScorePlan& plan, const ScoreArgs& a, hipStream_t s) {
    if constexpr (Geometry<T, D, 1>::kChunks < GP) {
        return hipErrorInvalidValue;
    } else {
        auto kern = attend_kernel<T, D, GP, true>;
        if (plan.lds_bytes > 64 * 1024) {
            static std::atomic<bool> raised[kMaxDevices];
            const hipError_t e = raise_lds_limit(reinterpret_cast<const void*>(kern), raised);
            if (e != hipSuccess) return e;
        }
        hipLaunchKernelGGL(kern, dim3(plan.grid), dim3(kThreads), plan.lds_bytes, s, a);
        if (plan.split) {
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
            hipLaunchKernelGGL((attend_combine_kernel<T, D, GP>),
                               dim3(plan.grid / plan.nchunk * combine_parts(a.n, a.emit)), dim3(kThreads), 0, s, a);
        }
        return hipGetLastError();
    }
}

template <typename T, int D, int GP>
hipError_t launch_chunks_gp(const ScorePlan& plan, const ScoreArgs& a, hipStream_t s) {
    if constexpr (Geometry<T, D, 1>::kChunks < GP) {
        return hipErrorInvalidValue;
    } else {
        auto kern = attend_kernel<T, D, GP, false>;
        if (plan.lds_bytes > 64 * 1024) {
            static std::atomic<bool> raised[kMaxDevices];
            const hipError_t e = raise_lds_limit(reinterpret_cast<const void*>(kern), raised);
            if (e != hipSuccess) return e;
        }
        hipLaunchKernelGGL(kern, dim3(plan.grid), dim3(kThreads), plan.lds_bytes, s, a);
        return hipGetLastError();
    }
}

template <typename T, int D>
hipError_t launch_chunks_d(const ScorePlan& plan, const ScoreArgs& a, hipStream_t s) {
    switch (plan.group_pad) {
        case 1: return launch_chunks_gp<T, D, 1>(plan, a, s);
        case 2: return launch_chunks_gp<T, D, 2>(plan, a, s);
        case 4: return launch_chunks_gp<T, D, 4>(plan, a, s);
        case 8: return launch_chunks_gp<T, D, 8>(plan, a, s);
        case 16: return launch_chunks_gp<T, D, 16>(plan, a, s);
        default: return hipErrorInvalidValue;
    }
}

template <typename T, int D>
hipError_t launch_attend_d(const ScorePlan& plan, const ScoreArgs& a, hipStream_t s) {
    switch (plan.group_pad) {
        case 1: return launch_attend_gp<T, D, 1>(plan, a, s);
        case 2: return launch_attend_gp<T, D, 2>(plan, a, s);
        case 4: return launch_attend_gp<T, D, 4>(plan, a, s);
        case 8: return launch_attend_gp<T, D, 8>(plan, a, s);
        case 16: return launch_attend_gp<T, D, 16>(plan, a, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool attend_plan(int dtype, int head_dim, int group, int n, int slabs, ScorePlan* plan, size_t max_lds) {
    if (slabs < 1 || !score_plan(dtype, head_dim, group, 1, plan)) return false;
    const int rpw = kWave / plan->group_pad;  // rows per unit
    if (max_lds == 0 || max_lds > kFastLdsMax) max_lds = kFastLdsMax;
    const int lds_rows = (int)(max_lds / (kWave * sizeof(float))) * rpw;
    const int want = (kAttnTargetWgs + slabs - 1) / slabs;
    const int by_rows = (n + kAttnMinRows - 1) / kAttnMinRows;
    int nchunk = (n + lds_rows - 1) / lds_rows;
    nchunk = max(nchunk, min(want, by_rows));
    int rows = (n + nchunk - 1) / nchunk;
    rows = (rows + rpw - 1) / rpw * rpw;  // <= lds_rows, a multiple of rpw
    plan->chunk_rows = rows;
    plan->nchunk = (n + rows - 1) / rows;
    plan->split = plan->nchunk > 1;
    plan->lds_bytes = (size_t)(rows / rpw) * kWave * sizeof(float);
    plan->grid = slabs * plan->nchunk;
    return true;
}

AttendBound attend_bound(int dtype, int head_dim, int group, int n, int slabs_per_layer, int layers) {
    AttendBound r{0, false};
    ScorePlan p;
    if (slabs_per_layer < 1 || layers < 1 || !score_plan(dtype, head_dim, group, 1, &p)) return r;
    const int rpw = kWave / p.group_pad;
    const long lds_rows = (long)(kFastLdsMax / (kWave * sizeof(float))) * rpw;
    const long c0 = (n + lds_rows - 1) / lds_rows;
    const long by_rows = (n + kAttnMinRows - 1) / kAttnMinRows;
    const long want1 = (kAttnTargetWgs + slabs_per_layer - 1) / slabs_per_layer;
    // a call over lc layers makes lc * nchunk(lc) chunks per slab column, nchunk = max(c0, min(want, by_rows))
    // with want = ceil(target / (lc * slabs_per_layer)); lc * want <= target / slabs_per_layer + lc
    const long by_target = layers * c0 > want1 + layers ? layers * c0 : want1 + layers;
    const long by_size = layers * (c0 > by_rows ? c0 : by_rows);
    r.chunk_layers = by_target < by_size ? by_target : by_size;
    r.may_split = c0 > 1 || (by_rows > 1 && want1 > 1);
    return r;
}

hipError_t launch_score_chunks(int dtype, int head_dim, const ScorePlan& plan, const ScoreArgs& a, hipStream_t s) {
    if (dtype == 0) {
        if (head_dim == 64) return launch_chunks_d<float, 64>(plan, a, s);
        if (head_dim == 128) return launch_chunks_d<float, 128>(plan, a, s);
    } else {
        if (head_dim == 64) return launch_chunks_d<bf16_t, 64>(plan, a, s);
        if (head_dim == 128) return launch_chunks_d<bf16_t, 128>(plan, a, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_attend(int dtype, int head_dim, const ScorePlan& plan, const ScoreArgs& a, hipStream_t s) {
    if (dtype == 0) {
        if (head_dim == 64) return launch_attend_d<float, 64>(plan, a, s);
        if (head_dim == 128) return launch_attend_d<float, 128>(plan, a, s);
    } else {
        if (head_dim == 64) return launch_attend_d<bf16_t, 64>(plan, a, s);
        if (head_dim == 128) return launch_attend_d<bf16_t, 128>(plan, a, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace ikv
