// pld_draft.hip -- the whole drafting half of a PLD+ step in one kernel
// (arXiv 2412.01447, Sec. 4): occurrence search (Eq. 1, n-grams longest
// first), ranking by hidden-state cosine (Eq. 2) or aggregated attention
// (Eq. 3, Sec. 7.1), selection of the best occurrence, and the draft span
// (Sec. 4.3).
//
// One 1024-thread block owns one sequence (tok_stride <= 8192), so nothing
// crosses blocks: the tokens are staged in LDS once, the occurrence list is
// built in LDS (and written out), the query row is staged in LDS, the
// candidates are scored by the same per-wave row routine as the multi-block
// ranking (bit-identical scores), the argmax is a block reduction of packed
// keys, and the draft is copied from the staged tokens.  A step therefore
// costs one launch and three dependent trips to memory (lengths, tokens,
// artifact rows) instead of four kernels.  The block's work grows with its
// own candidate count, so this path is for short candidate lists (small
// batches, the latency regime); the separate calls balance long lists across
// the whole GPU.
#include <math.h>

#include "pld.h"
#include "pld_device.h"
#include "pld_match.h"

namespace pld {

constexpr int kDraftWaves = kFindWavesFused;
constexpr int kDraftThreads = kDraftWaves * kWave;

struct DraftArgs {
    const int32_t *tokens;
    int64_t tok_stride;
    const int32_t *lens;
    int B;
    int nmin, nmax;
    int32_t *cand_pos;
    int64_t cap;
    int32_t *cand_count;
    int32_t *ngram_used;
    const uint16_t *hidden;
    int64_t hs, hr, n_rows;
    int d;
    const float *attn;
    int64_t as, ar, n_keys;
    int R, agg;
    float threshold;
    float *scores;
    int32_t *best_pos;
    float *best_score;
    int K;
    int32_t *draft;
    int32_t *draft_len;
};

// Scores this wave's candidates c = w, w + 16, ... of the block's list, G
// rows at a time (the same per-row arithmetic as the multi-block ranking).
template <int G>
__device__ void draft_score_rows(const DraftArgs &a, int b, int64_t T, bool seq_ok,
                                 const uint16_t *Hb, const uint4 *q_s, float qq,
                                 const int32_t *s_cand, int total, uint64_t &best) {
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    const int nch = a.d / 8;
    const int n = total > w ? (total - w + kDraftWaves - 1) / kDraftWaves : 0;
    for (int k = 0; k < n; k += G) {
        const uint4 *rows[G];
        int32_t js[G];
#pragma unroll
        for (int g = 0; g < G; ++g) {
            js[g] = (k + g < n) ? s_cand[w + (k + g) * kDraftWaves] : 0;
            const bool ok = (k + g < n) && seq_ok && js[g] >= 1 && (int64_t)js[g] <= T - 2;
            rows[g] = ok ? reinterpret_cast<const uint4 *>(Hb + (int64_t)(js[g] - 1) * a.hr)
                         : nullptr;
        }
        float dot[G], nrm[G];
        if (G == 1 && nch > 16 * kWave) {
            if (rows[0]) row_dot<true>(rows[0], q_s, nch, dot[0], nrm[0]);
        } else {
            rows_dot<G>(rows, q_s, nch, dot, nrm);
        }
#pragma unroll
        for (int g = 0; g < G; ++g) {
            if (k + g >= n) break;
            float s = __builtin_nanf("");
            if (rows[g]) {
                s = cosine(dot[g], nrm[g], qq);
                if (s > a.threshold) {
                    const uint64_t key = rank_key(s, js[g]);
                    best = key > best ? key : best;
                }
            }
            if (a.scores && lane == 0) a.scores[(int64_t)b * a.cap + w + (k + g) * kDraftWaves] = s;
        }
    }
}

template <bool kHidden>
__global__ __launch_bounds__(kDraftThreads) void draft_kernel(DraftArgs a) {
    __shared__ int32_t s_x[kFindFusedMax];                       // tokens of the sequence
    __shared__ int32_t s_cand[kFindFusedMax];                    // occurrence positions
    __shared__ uint4 s_q[kHidden ? PLD_MAX_HIDDEN / 8 : 1];      // query row H[T-2], bf16
    __shared__ int s_lvl[kDraftWaves][kMaxNgram];
    __shared__ int s_wc[kDraftWaves];
    __shared__ uint64_t s_key[kDraftWaves];
    const int b = blockIdx.x;
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    const int32_t *x = a.tokens + (int64_t)b * a.tok_stride;
    const int64_t T = a.lens[b];
    const bool tok_ok = (T >= 1 && T <= a.tok_stride);   // block-uniform

    // ---- occurrences (Eq. 1), longest n first
    int n_used = -1, total = 0;
    const bool seq_ok = kHidden ? (T >= 2 && T - 2 < a.n_rows) : (T >= 2);
    const uint16_t *Hb = kHidden ? a.hidden + (int64_t)b * a.hs : nullptr;
    const int nch = kHidden ? a.d / 8 : 0;
    if (tok_ok) {
        stage_tokens(x, 0, T, s_x);
        if (kHidden && seq_ok) {
            // the query row depends only on T: fetch it together with the tokens
            const uint4 *qg = reinterpret_cast<const uint4 *>(Hb + (T - 2) * a.hr);
            for (int i = threadIdx.x; i < nch; i += kDraftThreads) s_q[i] = qg[i];
        }
        __syncthreads();
        Query q;
#pragma unroll
        for (int k = 0; k < kMaxNgram; ++k)
            q.v[k] = (k < a.nmax && T - 1 - k >= 0) ? s_x[T - 1 - k] : 0;
        const int64_t base = (int64_t)w * 512;
        int m[8];
        wave_match(s_x, 0, T, base, q, a.nmax, m);
        int cnt[8];
        wave_level_counts(m, a.nmax, cnt);
        if (lane == 0) {
#pragma unroll
            for (int k = 0; k < kMaxNgram; ++k) s_lvl[w][k] = cnt[k];
        }
        __syncthreads();
        n_used = 0;
        for (int n = a.nmax; n >= a.nmin; --n) {
            int t = 0;
            for (int i = 0; i < kDraftWaves; ++i) t += s_lvl[i][n - 1];
            if (t > 0) {
                n_used = n;
                total = t;
                break;
            }
        }
        if (n_used > 0) {
            const int wc = wave_hits(m, n_used);
            if (lane == 0) s_wc[w] = wc;
            __syncthreads();
            int start = 0;
            for (int i = 0; i < w; ++i) start += s_wc[i];
            int32_t *out = a.cand_pos + (int64_t)b * a.cap;
            const uint64_t lt = lanemask_lt();
#pragma unroll
            for (int it = 0; it < 8; ++it) {
                const uint64_t mk = __ballot(m[it] >= n_used);
                if ((mk >> lane) & 1ull) {
                    const int slot = start + __popcll(mk & lt);
                    const int32_t p = (int32_t)(base + it * kWave + lane);
                    out[slot] = p;
                    s_cand[slot] = p;
                }
                start += __popcll(mk);
            }
            __syncthreads();
        }
    }

    // ---- ranking and selection (Eq. 2 / Eq. 3): highest score, then latest j
    uint64_t best = 0;
    if (total > 0) {   // block-uniform
        if constexpr (kHidden) {
            float qdot = 0.f, qq = 0.f;
            if (seq_ok) row_dot<false>(s_q, s_q, nch, qdot, qq);
            if (nch <= 4 * kWave)
                draft_score_rows<4>(a, b, T, seq_ok, Hb, s_q, qq, s_cand, total, best);
            else if (nch <= 8 * kWave)
                draft_score_rows<2>(a, b, T, seq_ok, Hb, s_q, qq, s_cand, total, best);
            else
                draft_score_rows<1>(a, b, T, seq_ok, Hb, s_q, qq, s_cand, total, best);
        } else {
            const float *Ab = a.attn + (int64_t)b * a.as;
            for (int c = threadIdx.x; c < total; c += kDraftThreads) {
                const int32_t j = s_cand[c];
                float s = __builtin_nanf("");
                if (seq_ok && j >= 1 && (int64_t)j <= T - 2 && (int64_t)(j - 1) < a.n_keys) {
                    s = attn_gather(Ab + (j - 1), a.ar, a.R, a.agg == PLD_AGG_SUM);
                    if (s > a.threshold) {
                        const uint64_t k = rank_key(s, j);
                        best = k > best ? k : best;
                    }
                }
                if (a.scores) a.scores[(int64_t)b * a.cap + c] = s;
            }
            best = wave_max_u64(best);
        }
        // (hidden: every lane of a wave already holds the wave's best)
        if (lane == 0) s_key[w] = best;
        __syncthreads();
        best = 0;
        for (int i = 0; i < kDraftWaves; ++i) best = s_key[i] > best ? s_key[i] : best;
    }

    // ---- outputs and the draft (Sec. 4.3)
    const int32_t bp = best ? (int32_t)(uint32_t)(best & 0xffffffffu) : -1;
    if (threadIdx.x == 0) {
        a.cand_count[b] = total;
        a.ngram_used[b] = n_used;
        a.best_pos[b] = bp;
        a.best_score[b] = best ? unord_f32((uint32_t)(best >> 32)) : -INFINITY;
    }
    int64_t L = 0;
    if (tok_ok && bp >= 0 && (int64_t)bp <= T - 2) L = min((int64_t)a.K, T - 1 - bp);
    for (int i = threadIdx.x; i < a.K; i += kDraftThreads)
        a.draft[(int64_t)b * a.K + i] = (i < L) ? s_x[bp + 1 + i] : -1;
    if (threadIdx.x == 0) a.draft_len[b] = (int32_t)L;
}

static int check_draft(const int32_t *tokens, int64_t tok_stride, const int32_t *lens, int B,
                       int ngram_min, int ngram_max, float threshold, int K,
                       const int32_t *cand_pos, int64_t cap, const int32_t *cand_count,
                       const int32_t *ngram_used, const int32_t *best_pos,
                       const float *best_score, const int32_t *draft, const int32_t *draft_len) {
    if (!tokens || !lens || !cand_pos || !cand_count || !ngram_used || !best_pos || !best_score ||
        !draft || !draft_len)
        return PLD_ERR_INVALID;
    if (B < 1 || B > 65535 || tok_stride < 1 || tok_stride > kFindFusedMax) return PLD_ERR_INVALID;
    if (ngram_min < 1 || ngram_max < ngram_min || ngram_max > PLD_MAX_NGRAM) return PLD_ERR_INVALID;
    if (cap < tok_stride || K < 1 || isnan(threshold)) return PLD_ERR_INVALID;
    return PLD_OK;
}

static DraftArgs make_draft(const int32_t *tokens, int64_t tok_stride, const int32_t *lens, int B,
                            int ngram_min, int ngram_max, float threshold, int K,
                            int32_t *cand_pos, int64_t cap, int32_t *cand_count,
                            int32_t *ngram_used, float *scores, int32_t *best_pos,
                            float *best_score, int32_t *draft, int32_t *draft_len) {
    DraftArgs a{};
    a.tokens = tokens;
    a.tok_stride = tok_stride;
    a.lens = lens;
    a.B = B;
    a.nmin = ngram_min;
    a.nmax = ngram_max;
    a.cand_pos = cand_pos;
    a.cap = cap;
    a.cand_count = cand_count;
    a.ngram_used = ngram_used;
    a.threshold = threshold;
    a.scores = scores;
    a.best_pos = best_pos;
    a.best_score = best_score;
    a.K = K;
    a.draft = draft;
    a.draft_len = draft_len;
    return a;
}

}  // namespace pld

using namespace pld;

extern "C" int pld_draft_hidden(const int32_t *tokens, int64_t tok_stride, const int32_t *lens,
                                int B, int ngram_min, int ngram_max, const uint16_t *hidden,
                                int64_t h_seq_stride, int64_t h_row_stride, int64_t n_rows, int d,
                                float threshold, int K, int32_t *cand_pos, int64_t cap,
                                int32_t *cand_count, int32_t *ngram_used, float *scores,
                                int32_t *best_pos, float *best_score, int32_t *draft,
                                int32_t *draft_len, void *stream) {
    int rc = check_draft(tokens, tok_stride, lens, B, ngram_min, ngram_max, threshold, K, cand_pos,
                         cap, cand_count, ngram_used, best_pos, best_score, draft, draft_len);
    if (rc != PLD_OK) return rc;
    if (!hidden || d < 8 || d > PLD_MAX_HIDDEN || d % 8 != 0 || n_rows < 1) return PLD_ERR_INVALID;
    if (h_row_stride < d || h_seq_stride < 0) return PLD_ERR_INVALID;
    if (((uintptr_t)hidden & 15) || (h_row_stride % 8) || (h_seq_stride % 8)) return PLD_ERR_ALIGN;
    DraftArgs a = make_draft(tokens, tok_stride, lens, B, ngram_min, ngram_max, threshold, K,
                             cand_pos, cap, cand_count, ngram_used, scores, best_pos, best_score,
                             draft, draft_len);
    a.hidden = hidden;
    a.hs = h_seq_stride;
    a.hr = h_row_stride;
    a.n_rows = n_rows;
    a.d = d;
    hipLaunchKernelGGL(draft_kernel<true>, dim3(B), dim3(kDraftThreads), 0, (hipStream_t)stream, a);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}

extern "C" int pld_draft_attn(const int32_t *tokens, int64_t tok_stride, const int32_t *lens, int B,
                              int ngram_min, int ngram_max, const float *attn, int64_t a_seq_stride,
                              int64_t a_row_stride, int64_t n_keys, int R, int agg,
                              float threshold, int K, int32_t *cand_pos, int64_t cap,
                              int32_t *cand_count, int32_t *ngram_used, float *scores,
                              int32_t *best_pos, float *best_score, int32_t *draft,
                              int32_t *draft_len, void *stream) {
    int rc = check_draft(tokens, tok_stride, lens, B, ngram_min, ngram_max, threshold, K, cand_pos,
                         cap, cand_count, ngram_used, best_pos, best_score, draft, draft_len);
    if (rc != PLD_OK) return rc;
    if (!attn || R < 1 || n_keys < 1 || (agg != PLD_AGG_SUM && agg != PLD_AGG_MAX))
        return PLD_ERR_INVALID;
    if (a_row_stride < 0 || a_seq_stride < 0) return PLD_ERR_INVALID;
    if ((uintptr_t)attn & 3) return PLD_ERR_ALIGN;
    DraftArgs a = make_draft(tokens, tok_stride, lens, B, ngram_min, ngram_max, threshold, K,
                             cand_pos, cap, cand_count, ngram_used, scores, best_pos, best_score,
                             draft, draft_len);
    a.attn = attn;
    a.as = a_seq_stride;
    a.ar = a_row_stride;
    a.n_keys = n_keys;
    a.R = R;
    a.agg = agg;
    hipLaunchKernelGGL(draft_kernel<false>, dim3(B), dim3(kDraftThreads), 0, (hipStream_t)stream, a);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}
