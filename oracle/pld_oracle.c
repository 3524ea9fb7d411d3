/*
 * pld_oracle.c -- plain, slow CPU oracle for the PLD+ drafting step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header, table or helper with
 * the HIP library and is compiled by gcc, not hipcc.
 *
 * Every function states the definition it writes out, citing the paper
 * (Somasundaram, Phukan, Saxena, "PLD+: Accelerating LLM inference by
 * leveraging Language Model Artifacts", arXiv 2412.01447).  Floating point
 * is done in IEEE double from exactly widened bf16 / fp32 inputs.  The
 * method's results are plainly defined objects (a set, an argmax, a slice,
 * a prefix compare), so the oracle is the definition itself, one scalar
 * loop per quantifier, with no blocking, fusion or reordering.
 *
 * Indexing is 0-based.  Sequence b has length T = lens[b]; its last token
 * x[T-1] is the paper's x_t (Sec. 4.2) and the artifact query position is
 * T-2, the paper's t-1 (Sec. 4.2.2; the Fig. 1 caption calls the same two
 * positions "t-1" and "t-2").
 *
 * Readings taken where the paper is silent (each is also listed in the
 * design notes of the repository):
 *   - candidate j is the last index of an occurrence of the query n-gram, and
 *     1 <= j <= T-2 (Eq. 1 "j < t"; j = 0 has no row j-1 for Eq. 2);
 *   - n > 1 is tried longest-first, as prompt lookup decoding does (Sec. 2,
 *     Fig. 3 caption); only the winning n's occurrences are ranked;
 *   - the attention score of candidate j reads key j-1 of the query row
 *     (Eq. 3 leaves the key index out);
 *   - argmax ties go to the highest score, then the most recent position;
 *   - the draft is truncated at the end of the context (Sec. 4.3);
 *   - greedy verification takes the lowest vocabulary id among equal
 *     maxima (Sec. 3 "greedy acceptance", Sec. 4.4).
 *
 * Parity status: every function here is pinned by the CPU tests (brute
 * force on tiny inputs, library reductions, closed forms and invariants).
 */
#include <math.h>
#include <stdlib.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>

#define REF_OK 0
#define REF_ERR (-1)

/* bf16 bit pattern -> double, exact: a bf16 value is the upper half of an
 * IEEE binary32 value. */
static double bf16_to_double(uint16_t bits) {
    uint32_t u = ((uint32_t)bits) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* ------------------------------------------------------------------ find */
/*
 * Occurrence set, Eq. 1 (Sec. 4.2.1):  P = { j | x_j = x_t, j < t },
 * generalised to an n-gram query as prompt lookup decoding does (Sec. 2):
 *   P_n = { j : max(n-1,1) <= j <= T-2  and  x[j-n+1+i] == x[T-n+i], i < n }
 * For n = ngram_max down to ngram_min the first non-empty P_n is the result
 * (ngram_used = n); if none is non-empty P = {} and ngram_used = 0.  A
 * length outside [1, tok_stride] is reported as ngram_used = -1, count 0.
 * cand_pos[b][0..count) is written in ascending order; later slots are not
 * touched.
 */
int pld_ref_find(const int32_t *tokens, int64_t tok_stride, const int32_t *lens, int B,
                 int ngram_min, int ngram_max, int32_t *cand_pos, int64_t cap,
                 int32_t *cand_count, int32_t *ngram_used) {
    if (!tokens || !lens || !cand_pos || !cand_count || !ngram_used) return REF_ERR;
    if (B < 0 || ngram_min < 1 || ngram_max < ngram_min || cap < tok_stride) return REF_ERR;
    for (int b = 0; b < B; ++b) {
        const int32_t *x = tokens + (int64_t)b * tok_stride;
        int32_t *out = cand_pos + (int64_t)b * cap;
        int64_t T = lens[b];
        cand_count[b] = 0;
        ngram_used[b] = 0;
        if (T < 1 || T > tok_stride) {
            ngram_used[b] = -1;
            continue;
        }
        for (int n = ngram_max; n >= ngram_min; --n) {
            int64_t count = 0;
            if (T >= n + 1) {
                int64_t lo = (n - 1 > 1) ? (int64_t)(n - 1) : 1;
                for (int64_t j = lo; j <= T - 2; ++j) {
                    int match = 1;
                    for (int i = 0; i < n; ++i) {
                        if (x[j - n + 1 + i] != x[T - n + i]) {
                            match = 0;
                            break;
                        }
                    }
                    if (match) out[count++] = (int32_t)j;
                }
            }
            if (count > 0) {
                cand_count[b] = (int32_t)count;
                ngram_used[b] = n;
                break;
            }
        }
    }
    return REF_OK;
}

/* ------------------------------------------------------------ selection */
/*
 * argmax over the occurrence set (Eq. 2 / Eq. 3) with the tie rule "highest
 * score, then most recent position".  An occurrence is eligible only when
 * its score is greater than the threshold theta (App. B, "greater than the
 * threshold"); theta = -inf keeps every finite score.  NaN scores mark
 * candidates that are out of range and are never eligible.
 */
static void select_best(const double *s, const int32_t *pos, int64_t C, double threshold,
                        int32_t *best_pos, double *best_score) {
    int32_t bj = -1;
    double bs = -INFINITY;
    for (int64_t c = 0; c < C; ++c) {
        double v = s[c];
        if (isnan(v) || !(v > threshold)) continue;
        if (bj < 0 || v > bs || (v == bs && pos[c] > bj)) {
            bs = v;
            bj = pos[c];
        }
    }
    *best_pos = bj;
    *best_score = bs;
}

/* ---------------------------------------------------------- rank hidden */
/*
 * Hidden-state ranking, Eq. 2 (Sec. 4.2.2):
 *   s_j = cos_sim(H_{j-1}, H_{t-1}),  j* = argmax_{j in P} s_j,
 * with q = H[T-2] and h = H[j-1] of one layer, in double from exactly
 * widened bf16:  s = (h.q) / sqrt(max(|h|^2 |q|^2, 1e-16)).  The clamp is
 * the usual eps = 1e-8 guard for zero rows.
 * A sequence is usable when 2 <= T and row T-2 < n_rows; a candidate when
 * 1 <= j <= T-2.  Unusable candidates get score NaN; an unusable sequence
 * gets best_pos = -1, best_score = -inf and NaN scores.
 * `scores` (may be NULL) has layout [B][cap].  `work` must hold cap doubles.
 */
int pld_ref_rank_hidden(const uint16_t *hidden, int64_t h_seq_stride, int64_t h_row_stride,
                        int d, int64_t n_rows, const int32_t *lens, const int32_t *cand_pos,
                        int64_t cap, const int32_t *cand_count, int B, double threshold,
                        double *scores, int32_t *best_pos, double *best_score, double *work) {
    if (!hidden || !lens || !cand_pos || !cand_count || !best_pos || !best_score || !work)
        return REF_ERR;
    if (B < 0 || d < 1 || cap < 0) return REF_ERR;
    for (int b = 0; b < B; ++b) {
        const uint16_t *Hb = hidden + (int64_t)b * h_seq_stride;
        const int32_t *pos = cand_pos + (int64_t)b * cap;
        int64_t T = lens[b];
        int64_t C = cand_count[b];
        if (C < 0 || C > cap) C = 0;
        int seq_ok = (T >= 2 && T - 2 < n_rows);
        double qq = 0.0;
        const uint16_t *q = seq_ok ? Hb + (T - 2) * h_row_stride : Hb;
        if (seq_ok)
            for (int k = 0; k < d; ++k) qq += bf16_to_double(q[k]) * bf16_to_double(q[k]);
        for (int64_t c = 0; c < C; ++c) {
            int64_t j = pos[c];
            if (!seq_ok || j < 1 || j > T - 2) {
                work[c] = NAN;
                continue;
            }
            const uint16_t *h = Hb + (j - 1) * h_row_stride;
            double dot = 0.0, hh = 0.0;
            for (int k = 0; k < d; ++k) {
                double hv = bf16_to_double(h[k]);
                dot += hv * bf16_to_double(q[k]);
                hh += hv * hv;
            }
            double den2 = hh * qq;
            if (den2 < 1e-16) den2 = 1e-16;
            work[c] = dot / sqrt(den2);
        }
        if (scores)
            for (int64_t c = 0; c < C; ++c) scores[(int64_t)b * cap + c] = work[c];
        if (seq_ok) {
            select_best(work, pos, C, threshold, &best_pos[b], &best_score[b]);
        } else {
            best_pos[b] = -1;
            best_score[b] = -INFINITY;
        }
    }
    return REF_OK;
}

/* ------------------------------------------------------------ rank attn */
/*
 * Attention ranking, Eq. 3 (Sec. 4.2.1) and the all-heads aggregation
 * ablation (Sec. 7.1):  the caller passes R rows, each the attention of
 * query position T-2 over keys 0..n_keys-1 for one selected (layer, head).
 *   agg = 0 (sum):  s_j = sum_{r<R} A[r][j-1], added in r order in double
 *   agg = 1 (max):  s_j = max_{r<R} A[r][j-1]
 * j* = argmax_{j in P} s_j.  A sequence is usable when T >= 2; a candidate
 * when 1 <= j <= T-2 and j-1 < n_keys.  Outputs as for the hidden ranking.
 */
int pld_ref_rank_attn(const float *attn, int64_t a_seq_stride, int64_t a_row_stride, int R,
                      int64_t n_keys, int agg, const int32_t *lens, const int32_t *cand_pos,
                      int64_t cap, const int32_t *cand_count, int B, double threshold,
                      double *scores, int32_t *best_pos, double *best_score, double *work) {
    if (!attn || !lens || !cand_pos || !cand_count || !best_pos || !best_score || !work)
        return REF_ERR;
    if (B < 0 || R < 1 || (agg != 0 && agg != 1) || cap < 0) return REF_ERR;
    for (int b = 0; b < B; ++b) {
        const float *Ab = attn + (int64_t)b * a_seq_stride;
        const int32_t *pos = cand_pos + (int64_t)b * cap;
        int64_t T = lens[b];
        int64_t C = cand_count[b];
        if (C < 0 || C > cap) C = 0;
        int seq_ok = (T >= 2);
        for (int64_t c = 0; c < C; ++c) {
            int64_t j = pos[c];
            if (!seq_ok || j < 1 || j > T - 2 || j - 1 >= n_keys) {
                work[c] = NAN;
                continue;
            }
            double s = (agg == 0) ? 0.0 : -INFINITY;
            for (int r = 0; r < R; ++r) {
                double a = (double)Ab[(int64_t)r * a_row_stride + (j - 1)];
                if (agg == 0)
                    s += a;
                else if (a > s)
                    s = a;
            }
            work[c] = s;
        }
        if (scores)
            for (int64_t c = 0; c < C; ++c) scores[(int64_t)b * cap + c] = work[c];
        if (seq_ok) {
            select_best(work, pos, C, threshold, &best_pos[b], &best_score[b]);
        } else {
            best_pos[b] = -1;
            best_score[b] = -INFINITY;
        }
    }
    return REF_OK;
}

/* ----------------------------------------------------------------- emit */
/*
 * Draft prediction (Sec. 4.3):  xhat_i = x_{j*+i}, i = 1..K, truncated at
 * the end of the context:  L = min(K, T-1-j*) when 0 <= j* <= T-2, else
 * L = 0 (no occurrence).  draft[b][i] = x[j*+1+i] for i < L, -1 after.
 */
int pld_ref_emit(const int32_t *tokens, int64_t tok_stride, const int32_t *lens,
                 const int32_t *best_pos, int B, int K, int32_t *draft, int32_t *draft_len) {
    if (!tokens || !lens || !best_pos || !draft || !draft_len) return REF_ERR;
    if (B < 0 || K < 1) return REF_ERR;
    for (int b = 0; b < B; ++b) {
        const int32_t *x = tokens + (int64_t)b * tok_stride;
        int64_t T = lens[b];
        int64_t j = best_pos[b];
        int64_t L = 0;
        if (T >= 1 && T <= tok_stride && j >= 0 && j <= T - 2) {
            L = T - 1 - j;
            if (L > K) L = K;
        }
        for (int i = 0; i < K; ++i) draft[(int64_t)b * K + i] = (i < L) ? x[j + 1 + i] : -1;
        draft_len[b] = (int32_t)L;
    }
    return REF_OK;
}

/* --------------------------------------------------------------- verify */
/* The acceptance rule shared by both verifications (Sec. 4.4): a = the first
 * i < L whose model token y[i] differs from draft[i], else L; the step emits
 * draft[0..a-1] followed by y[a] (count a + 1). */
static void accept_prefix(const int *y, const int32_t *draft, int L, int32_t *out,
                          int32_t *accept_len, int32_t *out_count) {
    int a = L;
    for (int i = 0; i < L; ++i) {
        if (y[i] != draft[i]) {
            a = i;
            break;
        }
    }
    for (int i = 0; i < a; ++i) out[i] = draft[i];
    out[a] = y[a];
    *accept_len = a;
    *out_count = a + 1;
}

/*
 * Greedy verification (Sec. 3 "greedy acceptance"; Sec. 4.4): one forward
 * pass gives K+1 distributions; at temperature 0 the model's token at
 * future position i is y_i = argmax_v Z[i][v] (lowest v among equal maxima,
 * values compared as IEEE numbers so -0 == +0).  The accepted length is
 * a = the first i < L with y_i != draft[i], else L; after the first
 * mismatch the rest of the draft is discarded.  The step emits
 * draft[0..a-1] followed by y_a:  out_count = a+1, out_tokens padded with -1.
 * Rows i > L are never read.  A draft length outside [0, K] is reported as
 * accept_len = -1, out_count = 0.
 * logits: dtype 0 = fp32, 1 = bf16 bits; element (b, i, v) sits at
 * b*l_seq_stride + i*l_row_stride + v.  row_argmax ([B][K+1], may be NULL)
 * receives y_i for i <= L and -1 elsewhere.
 */
int pld_ref_verify(const void *logits, int dtype, int64_t l_seq_stride, int64_t l_row_stride,
                   int V, int K, const int32_t *draft, const int32_t *draft_len, int B,
                   int32_t *accept_len, int32_t *out_tokens, int32_t *out_count,
                   int32_t *row_argmax) {
    if (!logits || !draft || !draft_len || !accept_len || !out_tokens || !out_count)
        return REF_ERR;
    if (B < 0 || K < 1 || V < 1 || (dtype != 0 && dtype != 1)) return REF_ERR;
    for (int b = 0; b < B; ++b) {
        int L = draft_len[b];
        int32_t *out = out_tokens + (int64_t)b * (K + 1);
        for (int i = 0; i <= K; ++i) {
            out[i] = -1;
            if (row_argmax) row_argmax[(int64_t)b * (K + 1) + i] = -1;
        }
        if (L < 0 || L > K) {
            accept_len[b] = -1;
            out_count[b] = 0;
            continue;
        }
        int y[K + 1];
        for (int i = 0; i <= L; ++i) {
            int64_t base = (int64_t)b * l_seq_stride + (int64_t)i * l_row_stride;
            double best = 0.0;
            int arg = 0;
            for (int v = 0; v < V; ++v) {
                double z = (dtype == 0) ? (double)((const float *)logits)[base + v]
                                        : bf16_to_double(((const uint16_t *)logits)[base + v]);
                if (v == 0 || z > best) {
                    best = z;
                    arg = v;
                }
            }
            y[i] = arg;
            if (row_argmax) row_argmax[(int64_t)b * (K + 1) + i] = arg;
        }
        accept_prefix(y, draft + (int64_t)b * K, L, out, &accept_len[b], &out_count[b]);
    }
    return REF_OK;
}

/* Sampling verification (Sec. 4.4: sample a token at every draft position
 * from the target model's distribution and keep the draft up to the first
 * mismatch; Sec. 5 runs it at temperature 1).  For the rows i = 0..L of
 * sequence b, with z = Z[b][i] and tau = temperature:
 *     p_v = exp((z_v - max_w z_w) / tau),  S = sum_v p_v,  t = u[b][i] * S,
 *     y_i = the smallest v with p_0 + ... + p_v > t
 * (the inverse CDF of softmax(z / tau) at the caller's uniform draw u; if
 * rounding leaves no such v, the last v with p_v > 0).  A row whose entries
 * are all -inf has no mass: y_i = 0.  u outside [0, 1) is clamped to it.
 * Acceptance is the greedy rule on these samples: a = the first i < L with
 * y_i != draft[i], else L; the step emits draft[0..a-1] followed by y_a.  */
int pld_ref_verify_sample(const void *logits, int dtype, int64_t l_seq_stride,
                          int64_t l_row_stride, int V, int K, const int32_t *draft,
                          const int32_t *draft_len, int B, double temperature,
                          const float *uniforms, int64_t u_stride, int32_t *accept_len,
                          int32_t *out_tokens, int32_t *out_count, int32_t *row_sample) {
    if (!logits || !draft || !draft_len || !uniforms || !accept_len || !out_tokens || !out_count)
        return REF_ERR;
    if (B < 0 || K < 1 || V < 1 || (dtype != 0 && dtype != 1)) return REF_ERR;
    if (!(temperature > 0.0) || isinf(temperature) || u_stride < K + 1) return REF_ERR;
    double *p = (double *)malloc(sizeof(double) * (size_t)V);
    if (!p) return REF_ERR;
    for (int b = 0; b < B; ++b) {
        int L = draft_len[b];
        int32_t *out = out_tokens + (int64_t)b * (K + 1);
        for (int i = 0; i <= K; ++i) {
            out[i] = -1;
            if (row_sample) row_sample[(int64_t)b * (K + 1) + i] = -1;
        }
        if (L < 0 || L > K) {
            accept_len[b] = -1;
            out_count[b] = 0;
            continue;
        }
        int y[K + 1];
        for (int i = 0; i <= L; ++i) {
            int64_t base = (int64_t)b * l_seq_stride + (int64_t)i * l_row_stride;
            double m = -INFINITY;
            for (int v = 0; v < V; ++v) {
                double z = (dtype == 0) ? (double)((const float *)logits)[base + v]
                                        : bf16_to_double(((const uint16_t *)logits)[base + v]);
                p[v] = z;
                if (z > m) m = z;
            }
            int pick = 0;
            if (m > -INFINITY) {
                double S = 0.0;
                for (int v = 0; v < V; ++v) {
                    p[v] = exp((p[v] - m) / temperature);
                    S += p[v];
                }
                double u = (double)uniforms[(int64_t)b * u_stride + i];
                if (!(u >= 0.0)) u = 0.0;
                if (u >= 1.0) u = (double)nextafterf(1.0f, 0.0f);   /* the draws are fp32 */
                double t = u * S, c = 0.0;
                int last = 0, found = 0;
                for (int v = 0; v < V; ++v) {
                    if (p[v] > 0.0) last = v;
                    c += p[v];
                    if (c > t) {
                        pick = v;
                        found = 1;
                        break;
                    }
                }
                if (!found) pick = last;
            }
            y[i] = pick;
            if (row_sample) row_sample[(int64_t)b * (K + 1) + i] = pick;
        }
        accept_prefix(y, draft + (int64_t)b * K, L, out, &accept_len[b], &out_count[b]);
    }
    free(p);
    return REF_OK;
}

/* ------------------------------------------------------- prefix selection */
/*
 * Prompt lookup decoding's selection, the baseline PLD+ improves on (Sec. 2;
 * the Fig. 3 caption: PLD proposes the candidate span with the longest
 * matching prefix).  For a candidate j, 0 <= j <= T-2, its match length is
 *   m_j = the largest m <= max_match with x[j-k] = x[T-1-k] for every k < m
 *         (only indices j-k >= 0 exist),
 * and j* = the candidate with the largest m_j, the earliest among equal
 * lengths (prompt lookup scans the context from the start and keeps the first
 * match).  best_score = m_j.  Out-of-range candidates get score NaN and are
 * never chosen; a sequence with T < 2 or T > tok_stride gets best_pos = -1,
 * best_score = -inf.  `scores` (may be NULL) has layout [B][cap].
 */
int pld_ref_select_prefix(const int32_t *tokens, int64_t tok_stride, const int32_t *lens,
                          const int32_t *cand_pos, int64_t cap, const int32_t *cand_count, int B,
                          int max_match, double *scores, int32_t *best_pos, double *best_score) {
    if (!tokens || !lens || !cand_pos || !cand_count || !best_pos || !best_score) return REF_ERR;
    if (B < 0 || cap < 0 || max_match < 1) return REF_ERR;
    for (int b = 0; b < B; ++b) {
        const int32_t *x = tokens + (int64_t)b * tok_stride;
        const int32_t *pos = cand_pos + (int64_t)b * cap;
        int64_t T = lens[b];
        int64_t C = cand_count[b];
        if (C < 0 || C > cap) C = 0;
        int seq_ok = (T >= 2 && T <= tok_stride);
        int32_t bj = -1;
        double bs = -INFINITY;
        for (int64_t c = 0; c < C; ++c) {
            int64_t j = pos[c];
            double s = NAN;
            if (seq_ok && j >= 0 && j <= T - 2) {
                int64_t m = 0;
                while (m < max_match && j - m >= 0 && x[j - m] == x[T - 1 - m]) ++m;
                s = (double)m;
                if (bj < 0 || s > bs || (s == bs && j < bj)) {
                    bs = s;
                    bj = (int32_t)j;
                }
            }
            if (scores) scores[(int64_t)b * cap + c] = s;
        }
        best_pos[b] = seq_ok ? bj : -1;
        best_score[b] = seq_ok ? bs : -INFINITY;
    }
    return REF_OK;
}

/* ----------------------------------------------------------------- commit */
/*
 * The step after verification in the generation loop (Sec. 3, Sec. 4.4: the
 * accepted draft tokens and the model's own token join the sequence):
 *   cap_b = min(limit[b], tok_stride)   (tok_stride when limit is NULL)
 *   m     = min(out_count[b], cap_b - T)
 *   x[T + i] = out_tokens[b][i] for i < m;  lens[b] = T + m
 *   stats[b] += (m, 1 if m > 0)          (emitted tokens, steps; may be NULL)
 * A sequence with T outside [0, cap_b] or out_count outside [0, K+1] is left
 * as it is.  The paper's average acceptance length (tokens per generation
 * step, Sec. 5.3) is stats[b][0] / stats[b][1].
 */
int pld_ref_commit(int32_t *tokens, int64_t tok_stride, int32_t *lens, const int32_t *limit,
                   const int32_t *out_tokens, const int32_t *out_count, int B, int K,
                   int64_t *stats) {
    if (!tokens || !lens || !out_tokens || !out_count) return REF_ERR;
    if (B < 0 || K < 1 || tok_stride < 1) return REF_ERR;
    for (int b = 0; b < B; ++b) {
        int64_t cap_b = tok_stride;
        if (limit && limit[b] < cap_b) cap_b = limit[b];
        int64_t T = lens[b];
        int64_t n = out_count[b];
        if (T < 0 || T > cap_b || n < 0 || n > K + 1) continue;
        int64_t m = n;
        if (m > cap_b - T) m = cap_b - T;
        for (int64_t i = 0; i < m; ++i)
            tokens[(int64_t)b * tok_stride + T + i] = out_tokens[(int64_t)b * (K + 1) + i];
        lens[b] = (int32_t)(T + m);
        if (stats) {
            stats[2 * b] += m;
            stats[2 * b + 1] += (m > 0) ? 1 : 0;
        }
    }
    return REF_OK;
}
