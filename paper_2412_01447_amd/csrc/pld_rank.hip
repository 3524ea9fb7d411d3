// pld_rank.hip -- ranking of the occurrences by model artifacts and the
// argmax selection (arXiv 2412.01447):
//   hidden states, Eq. 2 (Sec. 4.2.2):  s_j = cos(H[j-1], H[T-2])
//   attention,     Eq. 3 (Sec. 4.2.1) and the head-aggregation ablation
//                  (Sec. 7.1):           s_j = sum_r or max_r A[r][j-1]
//   j* = argmax_j (s_j, j): the highest score, then the most recent occurrence.
//
// The candidate lists of all sequences are treated as one flattened list.
// Every block computes the prefix sums of the (clamped) candidate counts in
// LDS, so the host never learns the counts and never synchronises.  A fixed
// grid of blocks splits the flattened list into equal contiguous ranges:
// perfect balance whatever the per-sequence counts are.
//
// Hidden ranking: a range crosses few sequences; for each sequence piece the
// block stages the query row H[T-2] in LDS (bf16), and each wave takes whole
// candidate rows: 16-byte loads of the bf16 row, fp32 FMAs of the dot product
// and the squared norm with eight per-lane accumulators, a butterfly wave sum.
// The reduction order depends only on d, never on the slot, so equal rows give
// bit-identical scores, and a row equal to the query gives exactly 1.
//
// Attention ranking: one lane per candidate gathers A[b][r][j-1] for r < R in
// r order (the candidates are ascending, so neighbouring lanes read
// neighbouring keys).
//
// Selection: a candidate with s > threshold contributes the 64-bit key
// (orderable(s) << 32 | j); waves reduce keys and atomically max them into the
// per-sequence workspace slot.  A small finishing kernel, launched right
// after on the same stream, turns the keys into best_pos / best_score and
// zeroes the slots (the kernel boundary orders the two; no block of the
// ranking kernel ever waits for, or fences against, another).
#include <math.h>

#include "pld.h"
#include "pld_device.h"

namespace pld {

constexpr int kRankThreads = 256;
constexpr int kRankWaves = kRankThreads / kWave;

struct RankCommon {
    const int32_t *lens;
    const int32_t *cand_pos;
    int64_t cap;
    const int32_t *cand_count;
    int B;
    float threshold;
    float *scores;
    int32_t *best_pos;
    float *best_score;
    uint64_t *keys;     // [B], zero on entry
};

struct RankHiddenArgs {
    RankCommon c;
    const uint16_t *hidden;
    int64_t hs, hr, n_rows;
    int d;
};

struct RankAttnArgs {
    RankCommon c;
    const float *attn;
    int64_t as, ar, n_keys;
    int R;
    int agg;
};

// pre[b] = number of candidates before sequence b; pre[B] = total.  Counts
// outside [0, cap] count as 0.  Block-wide: each thread sums a contiguous run
// of sequences; the thread sums are scanned with wave shuffles and one LDS
// exchange of the wave totals.
__device__ __forceinline__ uint32_t clamped_count(const RankCommon &c, int b) {
    const int32_t n = c.cand_count[b];
    return (n >= 0 && (int64_t)n <= c.cap) ? (uint32_t)n : 0u;
}

__device__ void candidate_prefix(const RankCommon &c, uint32_t *pre) {
    __shared__ uint32_t s_wave[kRankWaves];
    const int per = (c.B + kRankThreads - 1) / kRankThreads;
    const int b0 = threadIdx.x * per;
    const int b1 = min(b0 + per, c.B);
    uint32_t sum = 0;
    for (int b = b0; b < b1; ++b) sum += clamped_count(c, b);
    // inclusive scan across the wave
    uint32_t inc = sum;
    const int lane = lane_id();
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const uint32_t v = (uint32_t)__shfl_up((int)inc, off);
        if (lane >= off) inc += v;
    }
    const int w = threadIdx.x / kWave;
    if (lane == kWave - 1) s_wave[w] = inc;
    __syncthreads();
    uint32_t run = inc - sum;
    for (int i = 0; i < w; ++i) run += s_wave[i];
    for (int b = b0; b < b1; ++b) {
        pre[b] = run;
        run += clamped_count(c, b);
    }
    if (threadIdx.x == 0) {
        uint32_t t = 0;
        for (int i = 0; i < kRankWaves; ++i) t += s_wave[i];
        pre[c.B] = t;
    }
    __syncthreads();
}

// Largest b with pre[b] <= i (i < pre[B]); lands on a non-empty sequence.
__device__ __forceinline__ int seq_of(const uint32_t *pre, int B, uint32_t i) {
    int lo = 0, hi = B;   // invariant: pre[lo] <= i < pre[hi]
    while (hi - lo > 1) {
        int mid = (lo + hi) >> 1;
        if (pre[mid] <= i) lo = mid; else hi = mid;
    }
    return lo;
}

// best_pos / best_score from the keys, which are returned to zero.
__global__ __launch_bounds__(256) void rank_finish_kernel(RankCommon c) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= c.B) return;
    const uint64_t k = c.keys[b];
    c.keys[b] = 0;
    if (k == 0) {
        c.best_pos[b] = -1;
        c.best_score[b] = -INFINITY;
    } else {
        c.best_pos[b] = (int32_t)(uint32_t)(k & 0xffffffffu);
        c.best_score[b] = unord_f32((uint32_t)(k >> 32));
    }
}

// ---------------------------------------------------------------- hidden
// Dot product and squared norm of one bf16 row against the bf16 query in LDS.
// Lane l owns the 8-element chunks l, l+64, l+128, ...; element t of a chunk
// accumulates into acc[t]; the eight accumulators are added in a fixed tree,
// then summed across the wave.  `row` may point to LDS (query norm) or HBM.
__device__ __forceinline__ void row_dot(const uint4 *row, const uint4 *q, int nch, float &dot,
                                        float &nrm) {
    constexpr int U = 16;   // every 16-byte load of a row up to d = 8192 in flight at once
    const int lane = lane_id();
    float ad[8], an[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) ad[t] = an[t] = 0.f;
    for (int c0 = lane; c0 < nch; c0 += kWave * U) {
        uint4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            int ch = c0 + u * kWave;
            v[u] = ch < nch ? row[ch] : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            int ch = c0 + u * kWave;
            if (ch < nch) {
                uint4 qq = q[ch];
                const uint32_t hw[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
                const uint32_t qw[4] = {qq.x, qq.y, qq.z, qq.w};
#pragma unroll
                for (int p = 0; p < 4; ++p) {
                    float h0 = bf16_lo(hw[p]), h1 = bf16_hi(hw[p]);
                    float q0 = bf16_lo(qw[p]), q1 = bf16_hi(qw[p]);
                    ad[2 * p] = __builtin_fmaf(h0, q0, ad[2 * p]);
                    ad[2 * p + 1] = __builtin_fmaf(h1, q1, ad[2 * p + 1]);
                    an[2 * p] = __builtin_fmaf(h0, h0, an[2 * p]);
                    an[2 * p + 1] = __builtin_fmaf(h1, h1, an[2 * p + 1]);
                }
            }
        }
    }
    float d = ((ad[0] + ad[1]) + (ad[2] + ad[3])) + ((ad[4] + ad[5]) + (ad[6] + ad[7]));
    float n = ((an[0] + an[1]) + (an[2] + an[3])) + ((an[4] + an[5]) + (an[6] + an[7]));
    dot = wave_sum_f32(d);
    nrm = wave_sum_f32(n);
}

__global__ __launch_bounds__(kRankThreads) void rank_hidden_kernel(RankHiddenArgs a) {
    extern __shared__ uint4 smem[];
    const RankCommon &c = a.c;
    const int nch = a.d / 8;
    uint4 *q_s = smem;                                     // nch chunks of 8 bf16
    uint32_t *pre = reinterpret_cast<uint32_t *>(smem + nch);  // B + 1
    candidate_prefix(c, pre);
    const uint32_t total = pre[c.B];
    const uint32_t lo0 = (uint32_t)(((uint64_t)blockIdx.x * total) / gridDim.x);
    const uint32_t hi = (uint32_t)(((uint64_t)(blockIdx.x + 1) * total) / gridDim.x);
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    if (lo0 < hi) {
        int b = seq_of(pre, c.B, lo0);
        uint32_t lo = lo0;
        while (lo < hi) {
            while (pre[b + 1] <= lo) ++b;                  // skip empty sequences
            const uint32_t seg_hi = min(hi, pre[b + 1]);
            const int64_t T = c.lens[b];
            const bool seq_ok = (T >= 2 && T - 2 < a.n_rows);
            const uint16_t *Hb = a.hidden + (int64_t)b * a.hs;
            if (seq_ok) {
                const uint4 *qg = reinterpret_cast<const uint4 *>(Hb + (T - 2) * a.hr);
                for (int i = threadIdx.x; i < nch; i += kRankThreads) q_s[i] = qg[i];
            }
            __syncthreads();
            float qdot = 0.f, qq = 0.f;
            if (seq_ok) row_dot(q_s, q_s, nch, qdot, qq);
            uint64_t best = 0;
            for (uint32_t i = lo + w; i < seg_hi; i += kRankWaves) {
                const int64_t slot = (int64_t)(i - pre[b]);
                const int32_t j = c.cand_pos[(int64_t)b * c.cap + slot];
                float s = __builtin_nanf("");
                const bool ok = seq_ok && j >= 1 && (int64_t)j <= T - 2;
                if (ok) {
                    const uint4 *row = reinterpret_cast<const uint4 *>(Hb + (int64_t)(j - 1) * a.hr);
                    float dot, hh;
                    row_dot(row, q_s, nch, dot, hh);
                    s = dot / sqrtf(fmaxf(hh * qq, 1e-16f));
                    if (s > c.threshold) {
                        uint64_t k = rank_key(s, j);
                        best = k > best ? k : best;
                    }
                }
                if (c.scores && lane == 0) c.scores[(int64_t)b * c.cap + slot] = s;
            }
            if (best && lane == 0) atomicMax((unsigned long long *)&c.keys[b], (unsigned long long)best);
            __syncthreads();                               // q_s is restaged next
            lo = seg_hi;
        }
    }
}

// ------------------------------------------------------------------ attn
__global__ __launch_bounds__(kRankThreads) void rank_attn_kernel(RankAttnArgs a) {
    __shared__ uint32_t pre[PLD_MAX_BATCH + 1];
    const RankCommon &c = a.c;
    candidate_prefix(c, pre);
    const uint32_t total = pre[c.B];
    const uint32_t lo = (uint32_t)(((uint64_t)blockIdx.x * total) / gridDim.x);
    const uint32_t hi = (uint32_t)(((uint64_t)(blockIdx.x + 1) * total) / gridDim.x);
    for (uint32_t base = lo; base < hi; base += kRankThreads) {
        const uint32_t i = base + threadIdx.x;
        const bool active = i < hi;
        int b = active ? seq_of(pre, c.B, i) : 0;
        uint64_t key = 0;
        if (active) {
            const int64_t slot = (int64_t)(i - pre[b]);
            const int32_t j = c.cand_pos[(int64_t)b * c.cap + slot];
            const int64_t T = c.lens[b];
            float s = __builtin_nanf("");
            if (T >= 2 && j >= 1 && (int64_t)j <= T - 2 && (int64_t)(j - 1) < a.n_keys) {
                const float *col = a.attn + (int64_t)b * a.as + (j - 1);
                if (a.agg == PLD_AGG_SUM) {
                    float acc = 0.f;
                    int r = 0;
                    for (; r + 8 <= a.R; r += 8) {
                        float v[8];
#pragma unroll
                        for (int u = 0; u < 8; ++u) v[u] = col[(int64_t)(r + u) * a.ar];
#pragma unroll
                        for (int u = 0; u < 8; ++u) acc += v[u];
                    }
                    for (; r < a.R; ++r) acc += col[(int64_t)r * a.ar];
                    s = acc;
                } else {
                    float acc = -INFINITY;
                    int r = 0;
                    for (; r + 8 <= a.R; r += 8) {
                        float v[8];
#pragma unroll
                        for (int u = 0; u < 8; ++u) v[u] = col[(int64_t)(r + u) * a.ar];
#pragma unroll
                        for (int u = 0; u < 8; ++u) acc = fmaxf(acc, v[u]);
                    }
                    for (; r < a.R; ++r) acc = fmaxf(acc, col[(int64_t)r * a.ar]);
                    s = acc;
                }
                if (s > c.threshold) key = rank_key(s, j);
            }
            if (c.scores) c.scores[(int64_t)b * c.cap + slot] = s;
        }
        // one atomic per wave when all its lanes share a sequence
        const int b0 = __shfl(b, 0);
        const bool same = __ballot(active && b != b0) == 0ull;
        if (same) {
            uint64_t m = wave_max_u64(key);
            if (lane_id() == 0 && m) atomicMax((unsigned long long *)&c.keys[b0], (unsigned long long)m);
        } else if (key) {
            atomicMax((unsigned long long *)&c.keys[b], (unsigned long long)key);
        }
    }
}

// Blocks of the persistent ranking grids: a few per CU keeps enough rows in
// flight; the ranges are equal, so the grid size does not affect balance.
constexpr int kRankBlocks = 1024;

static int check_common(const int32_t *lens, const int32_t *cand_pos, int64_t cap,
                        const int32_t *cand_count, int B, float threshold, int32_t *best_pos,
                        float *best_score, void *workspace, size_t workspace_bytes) {
    if (!lens || !cand_pos || !cand_count || !best_pos || !best_score) return PLD_ERR_INVALID;
    if (B < 1 || B > PLD_MAX_BATCH || cap < 1 || isnan(threshold)) return PLD_ERR_INVALID;
    if ((uint64_t)B * (uint64_t)cap >= (1ull << 32)) return PLD_ERR_INVALID;
    if (!workspace || workspace_bytes < rank_ws_bytes(B)) return PLD_ERR_WORKSPACE;
    return PLD_OK;
}

static RankCommon make_common(const int32_t *lens, const int32_t *cand_pos, int64_t cap,
                              const int32_t *cand_count, int B, float threshold, float *scores,
                              int32_t *best_pos, float *best_score, void *workspace) {
    RankCommon c;
    c.lens = lens;
    c.cand_pos = cand_pos;
    c.cap = cap;
    c.cand_count = cand_count;
    c.B = B;
    c.threshold = threshold;
    c.scores = scores;
    c.best_pos = best_pos;
    c.best_score = best_score;
    c.keys = (uint64_t *)workspace;
    return c;
}

}  // namespace pld

using namespace pld;

extern "C" int pld_rank_hidden(const uint16_t *hidden, int64_t h_seq_stride, int64_t h_row_stride,
                               int64_t n_rows, int d, const int32_t *lens, const int32_t *cand_pos,
                               int64_t cap, const int32_t *cand_count, int B, float threshold,
                               float *scores, int32_t *best_pos, float *best_score,
                               void *workspace, size_t workspace_bytes, void *stream) {
    if (!hidden) return PLD_ERR_INVALID;
    int rc = check_common(lens, cand_pos, cap, cand_count, B, threshold, best_pos, best_score,
                          workspace, workspace_bytes);
    if (rc != PLD_OK) return rc;
    if (d < 8 || d > PLD_MAX_HIDDEN || d % 8 != 0 || n_rows < 1) return PLD_ERR_INVALID;
    if (h_row_stride < d || h_seq_stride < 0) return PLD_ERR_INVALID;
    if (((uintptr_t)hidden & 15) || (h_row_stride % 8) || (h_seq_stride % 8)) return PLD_ERR_ALIGN;
    RankHiddenArgs a;
    a.c = make_common(lens, cand_pos, cap, cand_count, B, threshold, scores, best_pos, best_score,
                      workspace);
    a.hidden = hidden;
    a.hs = h_seq_stride;
    a.hr = h_row_stride;
    a.n_rows = n_rows;
    a.d = d;
    size_t lds = (size_t)(d / 8) * sizeof(uint4) + (size_t)(B + 1) * sizeof(uint32_t);
    hipLaunchKernelGGL(rank_hidden_kernel, dim3(kRankBlocks), dim3(kRankThreads), lds,
                       (hipStream_t)stream, a);
    hipLaunchKernelGGL(rank_finish_kernel, dim3((B + 255) / 256), dim3(256), 0, (hipStream_t)stream,
                       a.c);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}

extern "C" int pld_rank_attn(const float *attn, int64_t a_seq_stride, int64_t a_row_stride,
                             int64_t n_keys, int R, int agg, const int32_t *lens,
                             const int32_t *cand_pos, int64_t cap, const int32_t *cand_count, int B,
                             float threshold, float *scores, int32_t *best_pos, float *best_score,
                             void *workspace, size_t workspace_bytes, void *stream) {
    if (!attn) return PLD_ERR_INVALID;
    int rc = check_common(lens, cand_pos, cap, cand_count, B, threshold, best_pos, best_score,
                          workspace, workspace_bytes);
    if (rc != PLD_OK) return rc;
    if (R < 1 || n_keys < 1 || (agg != PLD_AGG_SUM && agg != PLD_AGG_MAX)) return PLD_ERR_INVALID;
    if (a_row_stride < 0 || a_seq_stride < 0) return PLD_ERR_INVALID;
    if ((uintptr_t)attn & 3) return PLD_ERR_ALIGN;
    RankAttnArgs a;
    a.c = make_common(lens, cand_pos, cap, cand_count, B, threshold, scores, best_pos, best_score,
                      workspace);
    a.attn = attn;
    a.as = a_seq_stride;
    a.ar = a_row_stride;
    a.n_keys = n_keys;
    a.R = R;
    a.agg = agg;
    hipLaunchKernelGGL(rank_attn_kernel, dim3(kRankBlocks), dim3(kRankThreads), 0,
                       (hipStream_t)stream, a);
    hipLaunchKernelGGL(rank_finish_kernel, dim3((B + 255) / 256), dim3(256), 0, (hipStream_t)stream,
                       a.c);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}
