// pld_draft.hip -- the drafting half of a PLD+ step (arXiv 2412.01447, Sec. 4)
// in one call: occurrence search (Eq. 1, n-grams longest first), ranking by
// hidden-state cosine (Eq. 2) or aggregated attention (Eq. 3, Sec. 7.1),
// selection of the best occurrence, and the draft span (Sec. 4.3).
//
// S blocks share one sequence (grid S x B).  Every block stages the whole
// token row in LDS -- the load does not wait for the length -- finds the
// occurrences itself (the search is a few microseconds of LDS work, so
// repeating it costs less than a launch), builds the ordered occurrence list
// in LDS, and scores the occurrences c = s, s+S, s+2S, ... with the same
// per-row routines as the separate ranking calls (bit-identical scores).
//   S == 1: one block owns the sequence; it selects the best occurrence and
//           writes the draft itself -- one launch, three dependent trips to
//           memory (length and tokens, query row, candidate rows).
//   S  > 1: each block folds its best key into the sequence's spread key
//           slots in the workspace, and a small finishing kernel selects and
//           writes the draft -- long candidate lists are spread over S CUs.
#include <math.h>

#include "pld.h"
#include "pld_device.h"
#include "pld_match.h"

namespace pld {

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
    uint64_t *keys;   // [B][kKeySlots] when S > 1, zero on entry
};

// Scores this wave's share of the candidates: list slots c = first, first +
// step, ... < total, G rows at a time (the same per-row arithmetic as the
// multi-block ranking kernel).
template <int G>
__device__ void draft_score_rows(const DraftArgs &a, int b, int64_t T, bool seq_ok,
                                 const uint16_t *Hb, const uint4 *q_s, float qq,
                                 const int32_t *s_cand, int first, int step, int total,
                                 uint64_t &best) {
    const int lane = lane_id();
    const int nch = a.d / 8;
    const int n = total > first ? (total - first + step - 1) / step : 0;
    for (int k = 0; k < n; k += G) {
        const uint4 *rows[G];
        int32_t js[G];
#pragma unroll
        for (int g = 0; g < G; ++g) {
            js[g] = (k + g < n) ? s_cand[first + (k + g) * step] : 0;
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
            if (a.scores && lane == 0) a.scores[(int64_t)b * a.cap + first + (k + g) * step] = s;
        }
    }
}

// The draft of sequence b from its best key (Sec. 4.3), written by one wave;
// `x` is the sequence's token row (global memory or its LDS copy).
__device__ void write_draft(const DraftArgs &a, int b, int64_t T, bool tok_ok, uint64_t best,
                            const int32_t *x) {
    const int lane = lane_id();
    const int32_t bp = best ? (int32_t)(uint32_t)(best & 0xffffffffu) : -1;
    if (lane == 0) {
        a.best_pos[b] = bp;
        a.best_score[b] = best ? unord_f32((uint32_t)(best >> 32)) : -INFINITY;
    }
    int64_t L = 0;
    if (tok_ok && bp >= 0 && (int64_t)bp <= T - 2) L = min((int64_t)a.K, T - 1 - bp);
    for (int i = lane; i < a.K; i += kWave)
        a.draft[(int64_t)b * a.K + i] = (i < L) ? x[bp + 1 + i] : -1;
    if (lane == 0) a.draft_len[b] = (int32_t)L;
}

template <bool kHidden, int kWaves>
__global__ __launch_bounds__(kWaves * kWave) void draft_kernel(DraftArgs a) {
    constexpr int kThreads = kWaves * kWave;
    constexpr int kSteps = kFindFusedMax / (kWaves * kWave * kLanePos);   // passes per wave
    static_assert(kSteps * kWaves * kWave * kLanePos == kFindFusedMax, "whole passes");
    // One block per sequence (16 waves) keeps the tokens for the draft and puts
    // the occurrence list in an array of its own; with several blocks per
    // sequence the list overwrites the tokens (more blocks fit on a CU).
    constexpr bool kKeep = kWaves == 16;
    __shared__ __align__(16) int32_t s_buf[kFindFusedMax];   // the tokens
    __shared__ int32_t s_own[kKeep ? kFindFusedMax : 1];
    int32_t *s_list = kKeep ? s_own : s_buf;                 // the occurrence list
    extern __shared__ uint4 s_q[];             // query row H[T-2], bf16 (hidden only)
    __shared__ int s_lvl[kWaves][kMaxNgram];
    __shared__ uint64_t s_key[kWaves];
    const int split = blockIdx.x, S = gridDim.x, b = blockIdx.y;
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    const int32_t *x = a.tokens + (int64_t)b * a.tok_stride;

    // the query row, the token row and the length are all requested before
    // the first wait
    const int64_t T = a.lens[b];
    const bool tok_ok = (T >= 1 && T <= a.tok_stride);   // block-uniform
    const bool seq_ok = kHidden ? (T >= 2 && T - 2 < a.n_rows) : (T >= 2);
    const uint16_t *Hb = kHidden ? a.hidden + (int64_t)b * a.hs : nullptr;
    const int nch = kHidden ? a.d / 8 : 0;
    // the token row straight into LDS when it is 16-byte aligned (it does not
    // wait for the length), then the query row
    if (((uintptr_t)x & 15) == 0 && (a.tok_stride & 3) == 0)
        copy_to_lds(reinterpret_cast<const uint4 *>(x), reinterpret_cast<uint4 *>(s_buf),
                    (int)(a.tok_stride / 4));
    else
        stage_tokens(x, 0, a.tok_stride, s_buf);
    if (kHidden && tok_ok && seq_ok)
        copy_to_lds(reinterpret_cast<const uint4 *>(Hb + (T - 2) * a.hr), s_q, nch);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    // ---- occurrences (Eq. 1), longest n first
    int n_used = -1, total = 0;
    if (tok_ok) {
        const Query q = load_query(s_buf, T, a.nmax);
        // wave w covers [w, w+1) * kSteps * 512; pass st, lane l: 8 positions from base[st]
        const int64_t base0 = ((int64_t)w * kSteps * kWave + lane) * kLanePos;
        uint64_t hits[kSteps];
        int cnt[kMaxNgram];
#pragma unroll
        for (int k = 0; k < kMaxNgram; ++k) cnt[k] = 0;
#pragma unroll
        for (int st = 0; st < kSteps; ++st) {
            hits[st] = lane_hits(s_buf, 0, T, base0 + st * kWave * kLanePos, q, a.nmax);
            count_levels(hits[st], a.nmax, cnt);
        }
#pragma unroll
        for (int k = 0; k < kMaxNgram; ++k) {
            if (k < a.nmax) {   // uniform
                const int t = wave_sum_i32(cnt[k]);
                if (lane == 0) s_lvl[w][k] = t;
            }
        }
        __syncthreads();   // every token read of the search is done
        n_used = 0;
        for (int n = a.nmax; n >= a.nmin; --n) {
            int t = 0;
            for (int i = 0; i < kWaves; ++i) t += s_lvl[i][n - 1];
            if (t > 0) {
                n_used = n;
                total = t;
                break;
            }
        }
        if (n_used > 0) {   // block-uniform; the ascending list
            int64_t run = 0;
            for (int i = 0; i < w; ++i) run += s_lvl[i][n_used - 1];
            int32_t *out = split == 0 ? a.cand_pos + (int64_t)b * a.cap : nullptr;
#pragma unroll
            for (int st = 0; st < kSteps; ++st)
                run = emit_bits(level_bits(hits[st], n_used), base0 + st * kWave * kLanePos,
                                s_list, out, run);
            __syncthreads();
        }
    }
    if (split == 0 && threadIdx.x == 0) {
        a.cand_count[b] = total;
        a.ngram_used[b] = n_used;
    }

    // ---- this block's share of the ranking (Eq. 2 / Eq. 3)
    uint64_t best = 0;
    if (total > 0) {   // block-uniform
        if constexpr (kHidden) {
            float qdot = 0.f, qq = 0.f;
            if (seq_ok) row_dot<false>(s_q, s_q, nch, qdot, qq);
            const int first = split + S * w, step = S * kWaves;
            if (nch <= 4 * kWave)
                draft_score_rows<4>(a, b, T, seq_ok, Hb, s_q, qq, s_list, first, step, total, best);
            else if (nch <= 8 * kWave)
                draft_score_rows<2>(a, b, T, seq_ok, Hb, s_q, qq, s_list, first, step, total, best);
            else
                draft_score_rows<1>(a, b, T, seq_ok, Hb, s_q, qq, s_list, first, step, total, best);
        } else {
            const float *Ab = a.attn + (int64_t)b * a.as;
            for (int c = split + S * (int)threadIdx.x; c < total; c += S * kThreads) {
                const int32_t j = s_list[c];
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
        for (int i = 0; i < kWaves; ++i) best = s_key[i] > best ? s_key[i] : best;
    }

    // ---- selection and the draft (Sec. 4.3)
    if (S == 1) {
        if (w == 0) write_draft(a, b, T, tok_ok, best, kKeep ? s_buf : x);
    } else if (threadIdx.x == 0 && best) {
        atomicMax((unsigned long long *)&a.keys[(int64_t)b * kKeySlots + (split % kKeySlots)],
                  (unsigned long long)best);
    }
}

// S > 1: one wave per sequence folds the key slots (returning them to zero)
// and writes best_pos, best_score and the draft.
__global__ __launch_bounds__(256) void draft_finish_kernel(DraftArgs a) {
    const int b = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / kWave);
    if (b >= a.B) return;   // wave-uniform
    const int lane = lane_id();
    uint64_t k = 0;
    if (lane < kKeySlots) {
        k = a.keys[(int64_t)b * kKeySlots + lane];
        a.keys[(int64_t)b * kKeySlots + lane] = 0;
    }
    k = wave_max_u64(k);
    const int64_t T = a.lens[b];
    write_draft(a, b, T, T >= 1 && T <= a.tok_stride, k, a.tokens + (int64_t)b * a.tok_stride);
}

static int check_draft(const int32_t *tokens, int64_t tok_stride, const int32_t *lens, int B,
                       int ngram_min, int ngram_max, float threshold, int K,
                       const int32_t *cand_pos, int64_t cap, const int32_t *cand_count,
                       const int32_t *ngram_used, const int32_t *best_pos,
                       const float *best_score, const int32_t *draft, const int32_t *draft_len,
                       int S, void *workspace, size_t workspace_bytes) {
    if (!tokens || !lens || !cand_pos || !cand_count || !ngram_used || !best_pos || !best_score ||
        !draft || !draft_len)
        return PLD_ERR_INVALID;
    if (B < 1 || B > 65535 || tok_stride < 1 || tok_stride > kFindFusedMax) return PLD_ERR_INVALID;
    if (ngram_min < 1 || ngram_max < ngram_min || ngram_max > PLD_MAX_NGRAM) return PLD_ERR_INVALID;
    if (cap < tok_stride || K < 1 || isnan(threshold)) return PLD_ERR_INVALID;
    if (S < 1 || S > PLD_MAX_DRAFT_SPLIT) return PLD_ERR_INVALID;
    if (S > 1 && (!workspace || workspace_bytes < rank_ws_bytes(B))) return PLD_ERR_WORKSPACE;
    return PLD_OK;
}

static DraftArgs make_draft(const int32_t *tokens, int64_t tok_stride, const int32_t *lens, int B,
                            int ngram_min, int ngram_max, float threshold, int K,
                            int32_t *cand_pos, int64_t cap, int32_t *cand_count,
                            int32_t *ngram_used, float *scores, int32_t *best_pos,
                            float *best_score, int32_t *draft, int32_t *draft_len,
                            void *workspace) {
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
    a.keys = (uint64_t *)workspace;
    return a;
}

// One block of 16 waves when it owns its sequence; 4 waves when S blocks share
// it (more blocks fit on a CU, and each scores a fraction of the list).
template <bool kHidden>
static void launch_draft(const DraftArgs &a, int S, hipStream_t s) {
    const size_t lds = kHidden ? (size_t)(a.d / 8) * sizeof(uint4) : 0;
    if (S == 1) {
        hipLaunchKernelGGL((draft_kernel<kHidden, 16>), dim3(1, a.B), dim3(16 * kWave), lds, s, a);
    } else {
        hipLaunchKernelGGL((draft_kernel<kHidden, 4>), dim3(S, a.B), dim3(4 * kWave), lds, s, a);
        hipLaunchKernelGGL(draft_finish_kernel, dim3((a.B + 3) / 4), dim3(256), 0, s, a);
    }
}

}  // namespace pld

using namespace pld;

extern "C" int pld_draft_hidden(const int32_t *tokens, int64_t tok_stride, const int32_t *lens,
                                int B, int ngram_min, int ngram_max, const uint16_t *hidden,
                                int64_t h_seq_stride, int64_t h_row_stride, int64_t n_rows, int d,
                                float threshold, int K, int32_t *cand_pos, int64_t cap,
                                int32_t *cand_count, int32_t *ngram_used, float *scores,
                                int32_t *best_pos, float *best_score, int32_t *draft,
                                int32_t *draft_len, int blocks_per_seq, void *workspace,
                                size_t workspace_bytes, void *stream) {
    int rc = check_draft(tokens, tok_stride, lens, B, ngram_min, ngram_max, threshold, K, cand_pos,
                         cap, cand_count, ngram_used, best_pos, best_score, draft, draft_len,
                         blocks_per_seq, workspace, workspace_bytes);
    if (rc != PLD_OK) return rc;
    if (!hidden || d < 8 || d > PLD_MAX_HIDDEN || d % 8 != 0 || n_rows < 1) return PLD_ERR_INVALID;
    if (h_row_stride < d || h_seq_stride < 0) return PLD_ERR_INVALID;
    if (((uintptr_t)hidden & 15) || (h_row_stride % 8) || (h_seq_stride % 8)) return PLD_ERR_ALIGN;
    DraftArgs a = make_draft(tokens, tok_stride, lens, B, ngram_min, ngram_max, threshold, K,
                             cand_pos, cap, cand_count, ngram_used, scores, best_pos, best_score,
                             draft, draft_len, workspace);
    a.hidden = hidden;
    a.hs = h_seq_stride;
    a.hr = h_row_stride;
    a.n_rows = n_rows;
    a.d = d;
    launch_draft<true>(a, blocks_per_seq, (hipStream_t)stream);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}

extern "C" int pld_draft_attn(const int32_t *tokens, int64_t tok_stride, const int32_t *lens, int B,
                              int ngram_min, int ngram_max, const float *attn, int64_t a_seq_stride,
                              int64_t a_row_stride, int64_t n_keys, int R, int agg,
                              float threshold, int K, int32_t *cand_pos, int64_t cap,
                              int32_t *cand_count, int32_t *ngram_used, float *scores,
                              int32_t *best_pos, float *best_score, int32_t *draft,
                              int32_t *draft_len, int blocks_per_seq, void *workspace,
                              size_t workspace_bytes, void *stream) {
    int rc = check_draft(tokens, tok_stride, lens, B, ngram_min, ngram_max, threshold, K, cand_pos,
                         cap, cand_count, ngram_used, best_pos, best_score, draft, draft_len,
                         blocks_per_seq, workspace, workspace_bytes);
    if (rc != PLD_OK) return rc;
    if (!attn || R < 1 || n_keys < 1 || (agg != PLD_AGG_SUM && agg != PLD_AGG_MAX))
        return PLD_ERR_INVALID;
    if (a_row_stride < 0 || a_seq_stride < 0) return PLD_ERR_INVALID;
    if ((uintptr_t)attn & 3) return PLD_ERR_ALIGN;
    DraftArgs a = make_draft(tokens, tok_stride, lens, B, ngram_min, ngram_max, threshold, K,
                             cand_pos, cap, cand_count, ngram_used, scores, best_pos, best_score,
                             draft, draft_len, workspace);
    a.attn = attn;
    a.as = a_seq_stride;
    a.ar = a_row_stride;
    a.n_keys = n_keys;
    a.R = R;
    a.agg = agg;
    launch_draft<false>(a, blocks_per_seq, (hipStream_t)stream);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}
