/*
 * pld.h -- C ABI of the PLD+ drafting step on AMD Instinct MI355X (gfx950).
 *
 * PLD+ (Somasundaram, Phukan, Saxena, "PLD+: Accelerating LLM inference by
 * leveraging Language Model Artifacts", arXiv 2412.01447) drafts K future
 * tokens by copying a span of the context: it finds the earlier occurrences
 * of the last token (Eq. 1), ranks them by model artifacts -- the cosine
 * similarity of hidden states (Eq. 2) or aggregated attention (Eq. 3) --
 * copies the K tokens after the best one (Sec. 4.3), and keeps the longest
 * prefix the model agrees with (greedy verification, Sec. 3 and 4.4).
 *
 * Conventions shared by every call
 * --------------------------------
 * - Indexing is 0-based.  Sequence b has T = lens[b] tokens; its last token
 *   x[T-1] is the paper's x_t and the artifact query position is T-2, the
 *   paper's t-1 (the Fig. 1 caption calls them "t-1" and "t-2").
 * - A candidate j is the last index of an occurrence of the query n-gram;
 *   1 <= j <= T-2.  Its artifact row / key is j-1, its draft starts at j+1.
 * - Every data pointer is a DEVICE pointer (memory of the GPU that `stream`
 *   belongs to).  The caller owns all memory; inputs are never modified.
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *   Calls validate their arguments on the host, enqueue kernels on the stream
 *   and return.  They never allocate, never synchronise and keep no pointer.
 * - Host-checkable faults return a non-zero pld_status and enqueue nothing.
 *   Faults only visible on the device (bad lengths, positions, counts) are
 *   reported through the outputs as documented per call.
 * - `workspace` (ranking and verification calls) is device memory of at
 *   least pld_workspace_bytes(B, K) bytes.  It must be zero-filled once after
 *   allocation; every call returns it to all-zero by the time its kernels
 *   complete, so one buffer serves every such call of a stream in turn.
 * - `scratch` (occurrence search) is device memory of at least
 *   pld_find_scratch_bytes(B, tok_stride) bytes with no requirement on its
 *   contents; it may be NULL when that size is 0.  It must not overlap a
 *   workspace.
 * - Two calls in flight at once (on different streams) must not share a
 *   workspace or a scratch buffer.
 * - Results are deterministic: the same inputs give bit-identical outputs.
 */
#ifndef PLD_H
#define PLD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes returned by every call. */
enum {
    PLD_OK = 0,
    PLD_ERR_INVALID = 1,   /* a NULL required pointer, a size or enum out of range   */
    PLD_ERR_ALIGN = 2,     /* a pointer or stride that breaks an alignment rule       */
    PLD_ERR_WORKSPACE = 3, /* workspace NULL or smaller than the call needs           */
    PLD_ERR_LAUNCH = 4,    /* the HIP runtime reported an error when launching        */
    PLD_ERR_SCRATCH = 5    /* sizes beyond the static scratch of pld_verify_greedy_noalloc */
};

/* Element types of the verification logits. */
enum { PLD_F32 = 0, PLD_BF16 = 1 };

/* Aggregations of the attention ranking. */
enum { PLD_AGG_SUM = 0, PLD_AGG_MAX = 1 };

/* Limits checked on the host. */
#define PLD_MAX_NGRAM 8         /* ngram_max <= 8                                    */
#define PLD_MAX_HIDDEN 16384    /* d <= 16384 (the query row is staged in LDS)       */
#define PLD_MAX_BATCH 4096      /* B <= 4096 for the ranking calls                   */

/* Version of this ABI (major * 10000 + minor * 100 + patch); pld_version()
 * returns the library's, which equals PLD_ABI_VERSION for a matching build. */
#define PLD_ABI_VERSION 200
int pld_version(void);

/* A static, human-readable name for a status code. */
const char *pld_status_string(int status);

/*
 * Bytes of workspace for the ranking and verification calls with batch B and
 * draft length K (size it for the largest B and K used on the buffer).
 * Returns 0 when an argument is out of range.
 */
size_t pld_workspace_bytes(int B, int K);

/*
 * Bytes of scratch pld_find_candidates needs for batch B and token stride
 * tok_stride: 0 up to tok_stride = 16384 (one block per sequence), else the
 * per-tile occurrence counts of every n (2048 positions per tile), and past
 * 256 tiles (524288 tokens) also each tile's output offset and each
 * sequence's chosen n and count.  Returns 0 when an argument is out of range.
 */
size_t pld_find_scratch_bytes(int B, int64_t tok_stride);

/*
 * pld_find_candidates -- the occurrence set P (Eq. 1, Sec. 4.2), with
 * n-gram queries tried longest first as prompt lookup decoding does (Sec. 2,
 * Fig. 3 caption):
 *   P_n = { j : max(n-1,1) <= j <= T-2, x[j-n+1+i] == x[T-n+i] for i < n }
 * for n = ngram_max down to ngram_min; the first non-empty P_n is the result.
 *
 *   tokens      int32 [B][tok_stride], token ids (any values; only equality matters)
 *   lens        int32 [B], sequence lengths
 *   ngram_min/max  1 <= ngram_min <= ngram_max <= PLD_MAX_NGRAM
 *   cand_pos    int32 [B][cap], cap >= tok_stride: P in ascending order in
 *               slots [0, cand_count[b]); later slots are not written
 *   cand_count  int32 [B], |P|
 *   ngram_used  int32 [B], the n that produced P; 0 when no n has an occurrence;
 *               -1 when lens[b] is outside [1, tok_stride] (then cand_count = 0)
 *   scratch     see the conventions above (pld_find_scratch_bytes)
 * Errors: PLD_ERR_INVALID for NULL pointers, B outside [1, 65535], tok_stride
 * outside [1, 2^30], a bad n range or cap < tok_stride; PLD_ERR_WORKSPACE when
 * the scratch is missing or too small; PLD_ERR_LAUNCH.
 */
int pld_find_candidates(const int32_t *tokens, int64_t tok_stride, const int32_t *lens, int B,
                        int ngram_min, int ngram_max, int32_t *cand_pos, int64_t cap,
                        int32_t *cand_count, int32_t *ngram_used, void *scratch,
                        size_t scratch_bytes, void *stream);

/*
 * pld_rank_hidden -- hidden-state ranking, Eq. 2 (Sec. 4.2.2):
 *   s_j = cos(H[j-1], H[T-2]) = (h.q) / sqrt(max(|h|^2 |q|^2, 1e-16)),
 *   best_pos[b] = argmax over eligible j of (s_j, j)
 * i.e. the highest score, ties to the most recent occurrence.  A candidate is
 * eligible when s_j > threshold (App. B; pass -INFINITY to keep all).  The
 * dot product and norms accumulate in fp32 from bf16 inputs.
 *
 *   hidden      bf16 bit patterns; row r of sequence b starts at element
 *               b*h_seq_stride + r*h_row_stride.  Base 16-byte aligned,
 *               both strides multiples of 8 elements.
 *   n_rows      rows available per sequence (row T-2 must be < n_rows)
 *   d           hidden width, 8 <= d <= PLD_MAX_HIDDEN, d % 8 == 0
 *   lens, cand_pos [B][cap], cand_count  as written by pld_find_candidates
 *   scores      fp32 [B][cap] or NULL: s_j per slot (NaN for an unusable candidate)
 *   best_pos    int32 [B]: j*, or -1 when no candidate is eligible
 *   best_score  fp32 [B]:  s_{j*}, or -INFINITY
 * Device-side rules: a count outside [0, cap] counts as 0; a sequence with
 * T < 2 or T-2 >= n_rows, and a slot with j outside [1, T-2], is unusable.
 * Errors: PLD_ERR_INVALID (NULL, B outside [1, PLD_MAX_BATCH], d out of range,
 * n_rows < 1, cap < 1, NaN threshold), PLD_ERR_ALIGN, PLD_ERR_WORKSPACE,
 * PLD_ERR_LAUNCH.
 */
int pld_rank_hidden(const uint16_t *hidden, int64_t h_seq_stride, int64_t h_row_stride,
                    int64_t n_rows, int d, const int32_t *lens, const int32_t *cand_pos,
                    int64_t cap, const int32_t *cand_count, int B, float threshold,
                    float *scores, int32_t *best_pos, float *best_score, void *workspace,
                    size_t workspace_bytes, void *stream);

/*
 * pld_rank_attn -- attention ranking, Eq. 3 (Sec. 4.2.1) and the all-heads
 * aggregation of the ablation (Sec. 7.1).  The caller passes, per sequence,
 * R rows: the attention of query position T-2 over keys 0..n_keys-1 for each
 * selected (layer, head).
 *   agg = PLD_AGG_SUM:  s_j = sum_{r<R} A[r][j-1], added in fp32 in a fixed
 *                       order: eight partial sums (rows t, t+8, ... in order,
 *                       t = 0..7), then combined pairwise (t^1, t^2, t^7)
 *   agg = PLD_AGG_MAX:  s_j = max_{r<R} A[r][j-1]
 * Selection, threshold and outputs as in pld_rank_hidden.
 *
 *   attn        fp32; element (b, r, k) at b*a_seq_stride + r*a_row_stride + k
 *   n_keys      keys per row; a slot with j-1 >= n_keys is unusable
 * Errors: as pld_rank_hidden (R < 1, n_keys < 1 or a bad agg are
 * PLD_ERR_INVALID; a base not 4-byte aligned is PLD_ERR_ALIGN).
 */
int pld_rank_attn(const float *attn, int64_t a_seq_stride, int64_t a_row_stride, int64_t n_keys,
                  int R, int agg, const int32_t *lens, const int32_t *cand_pos, int64_t cap,
                  const int32_t *cand_count, int B, float threshold, float *scores,
                  int32_t *best_pos, float *best_score, void *workspace,
                  size_t workspace_bytes, void *stream);

/*
 * pld_emit_draft -- draft prediction, Sec. 4.3: xhat_i = x[j*+i], i = 1..K,
 * cut at the end of the context:
 *   L = min(K, T-1-j*) when 0 <= j* <= T-2 and 1 <= T <= tok_stride, else 0
 *   draft[b][i] = x[j*+1+i] for i < L, -1 for L <= i < K;  draft_len[b] = L
 * Errors: PLD_ERR_INVALID (NULL, B < 1, K < 1, tok_stride < 1), PLD_ERR_LAUNCH.
 */
int pld_emit_draft(const int32_t *tokens, int64_t tok_stride, const int32_t *lens,
                   const int32_t *best_pos, int B, int K, int32_t *draft, int32_t *draft_len,
                   void *stream);

/*
 * pld_verify_greedy -- greedy verification (Sec. 3 "greedy acceptance",
 * Sec. 4.4).  One forward pass over the context plus the draft gives K+1
 * rows of logits per sequence.  With y_i = argmax_v Z[b][i][v] (lowest v
 * among equal maxima; -0 and +0 compare equal):
 *   accept_len[b] = the first i < L with y_i != draft[b][i], else L
 *   out_tokens[b] = draft[b][0..a-1], y_a, then -1 padding;  out_count[b] = a+1
 * where L = draft_len[b].  Rows i > L do not affect any output.  NaN
 * logits are outside the contract (a row holding one gets an unspecified
 * y_i).
 *
 *   logits      PLD_F32 or PLD_BF16 (bit patterns); element (b, i, v) at
 *               b*l_seq_stride + i*l_row_stride + v; element-aligned.  All
 *               K+1 rows of every sequence (the last one's included) must be
 *               readable device memory whatever draft_len holds: the argmax
 *               requests the first part of each row before the draft length
 *               arrives, so the rows past a short draft are read in part or
 *               in full (their values are never used).
 *   V           vocabulary size >= 1;  K >= 1 draft slots per sequence
 *   draft       int32 [B][K], draft_len int32 [B] (from pld_emit_draft)
 *   accept_len, out_count int32 [B];  out_tokens int32 [B][K+1]
 * Device-side rule: draft_len outside [0, K] gives accept_len = -1,
 * out_count = 0 and out_tokens all -1.
 * Errors: PLD_ERR_INVALID (NULL, B outside [1, 65535], K outside [1, 65534],
 * V < 1, bad dtype, strides smaller than a row / K+1 rows), PLD_ERR_ALIGN,
 * PLD_ERR_WORKSPACE, PLD_ERR_LAUNCH.
 */
int pld_verify_greedy(const void *logits, int dtype, int64_t l_seq_stride, int64_t l_row_stride,
                      int V, int K, const int32_t *draft, const int32_t *draft_len, int B,
                      int32_t *accept_len, int32_t *out_tokens, int32_t *out_count,
                      void *workspace, size_t workspace_bytes, void *stream);

/*
 * pld_verify_greedy_noalloc -- pld_verify_greedy for callers that cannot
 * allocate device memory or pass a workspace (code under stream capture,
 * tight serving loops, harnesses that forbid allocation).  Same arguments
 * minus the workspace, same outputs and device-side rules, bit for bit.
 *
 * The row maxima live in a static array of the library, 65536 64-bit keys
 * (512 KiB) per GPU, held from the first call on that GPU until the process
 * ends; the call clears the B*(K+1) keys it uses (a fill kernel, then the
 * argmax and acceptance kernels: three launches) and never allocates.  The
 * stream must belong to the current device.  Every call on one GPU shares
 * that GPU's array: calls that overlap in time on one GPU (different streams,
 * threads or processes' streams of one context) race and give undefined
 * results, so serialise them.
 * Errors: those of pld_verify_greedy (no workspace errors), and
 * PLD_ERR_SCRATCH when B*(K+1) > 65536; PLD_ERR_LAUNCH also when the array's
 * device address cannot be obtained.
 */
int pld_verify_greedy_noalloc(const void *logits, int dtype, int64_t l_seq_stride,
                              int64_t l_row_stride, int V, int K, const int32_t *draft,
                              const int32_t *draft_len, int B, int32_t *accept_len,
                              int32_t *out_tokens, int32_t *out_count, void *stream);

/*
 * pld_verify_sample -- sampling verification (Sec. 3 and Sec. 4.4 with a
 * temperature; the paper's sampling experiments use tau = 1).  Instead of the
 * argmax, y_i is drawn from softmax(Z[b][i] / tau) by inversion at the
 * caller's uniform u = uniforms[b][i]: with p_v = exp((Z[v] - max Z) / tau)
 * and S = sum_v p_v, y_i is the first v whose cumulative mass p_0 + ... + p_v
 * exceeds u * S.  Acceptance and outputs are then those of pld_verify_greedy
 * with these y_i; for a draft that puts all its mass on one token this is
 * the usual speculative rejection sampling.
 *
 *   temperature  tau > 0, finite, with log2(e) / tau representable in fp32
 *   uniforms     fp32 [B][u_stride] device memory, u_stride >= K+1, 4-byte
 *                aligned; u < 0 or NaN counts as 0, u >= 1 as the largest
 *                float below 1.  Entries i <= draft_len[b] are used (others
 *                of the first K+1 may be read ahead and are ignored).
 *   row_sample   int32 [B][K+1] or NULL: y_i for i <= L, -1 for the rows
 *                past the draft (all -1 when draft_len is out of range)
 *   workspace    at least pld_verify_sample_workspace_bytes(B, K, V, dtype)
 *                bytes, zero-filled once like every workspace; its first
 *                pld_workspace_bytes(B, K) bytes are left zero by the call,
 *                then come per-call statistics, B counters that every call
 *                leaves zero (K+1 > 16: the blocks that share a sequence's
 *                rows count themselves done there, the last one accepting)
 *                and the tokens those blocks hand over, rewritten each time.
 * Arithmetic: the masses are fp32 (2^((z - m) * log2(e)/tau)) and are summed
 * per 512-vector segment of the row, then over the segments; a row of -inf
 * gives y = 0, and where rounding leaves no element past the target the last
 * element with nonzero mass is taken.  +inf and NaN logits are outside the
 * contract.  Results are bit-identical from run to run.
 * Errors: as pld_verify_greedy, plus PLD_ERR_INVALID for a bad temperature,
 * K+1 > PLD_MAX_SAMPLE_ROWS, NULL uniforms or u_stride < K+1, and
 * PLD_ERR_ALIGN for misaligned uniforms.
 */
#define PLD_MAX_SAMPLE_ROWS 16384
int pld_verify_sample(const void *logits, int dtype, int64_t l_seq_stride, int64_t l_row_stride,
                      int V, int K, const int32_t *draft, const int32_t *draft_len, int B,
                      double temperature, const float *uniforms, int64_t u_stride,
                      int32_t *accept_len, int32_t *out_tokens, int32_t *out_count,
                      int32_t *row_sample, void *workspace, size_t workspace_bytes, void *stream);

/* Workspace bytes of pld_verify_sample (0 for arguments out of range); it is
 * at least pld_workspace_bytes(B, K), so one buffer serves every call. */
size_t pld_verify_sample_workspace_bytes(int B, int K, int V, int dtype);

/*
 * The two halves of the ranking calls and of verification, for callers that
 * schedule (or time) the phases separately.  Run in order on one stream with
 * the same workspace, they produce exactly what the combined call produces.
 *
 * pld_score_hidden / pld_score_attn -- the scoring half of pld_rank_hidden /
 *   pld_rank_attn (Eq. 2 / Eq. 3): writes `scores` (may be NULL) and folds
 *   every eligible candidate into per-sequence keys held in the workspace.
 * pld_select_best -- the selection (argmax over the occurrences, highest
 *   score then most recent position): turns those keys into best_pos /
 *   best_score and returns the workspace to zero.
 * pld_verify_argmax -- y_i = argmax_v Z[b][i][v] for the rows i <= draft_len[b],
 *   kept in the workspace (rows past the draft may be read, as in
 *   pld_verify_greedy, and are never used).
 * pld_verify_accept -- the accepted length and emitted tokens from those
 *   row maxima (Sec. 4.4); returns the workspace to zero.
 * pld_verify_sample_stats -- the streaming pass of pld_verify_sample: per
 *   512-vector segment of each row i <= draft_len[b], the segment maximum and
 *   the mass relative to it, into the workspace's statistics region.
 * pld_verify_sample_finish -- the rest of pld_verify_sample from those
 *   statistics: the segment each target falls in, re-read to find y_i, then
 *   the acceptance and outputs; the same temperature as the statistics.
 * Arguments and errors as in the combined calls.
 */
int pld_score_hidden(const uint16_t *hidden, int64_t h_seq_stride, int64_t h_row_stride,
                     int64_t n_rows, int d, const int32_t *lens, const int32_t *cand_pos,
                     int64_t cap, const int32_t *cand_count, int B, float threshold,
                     float *scores, void *workspace, size_t workspace_bytes, void *stream);

int pld_score_attn(const float *attn, int64_t a_seq_stride, int64_t a_row_stride, int64_t n_keys,
                   int R, int agg, const int32_t *lens, const int32_t *cand_pos, int64_t cap,
                   const int32_t *cand_count, int B, float threshold, float *scores,
                   void *workspace, size_t workspace_bytes, void *stream);

/*
 * pld_score_both -- pld_score_hidden and pld_score_attn of the same occurrences
 * in one launch (Eq. 2 and Eq. 3 side by side, as when both artifacts rank one
 * candidate list): part of the grid gathers attention weights while the rest
 * streams hidden rows, so the gathers overlap the stream instead of following
 * it.  Scores and keys equal those of the two separate calls bit for bit.
 *
 *   hidden ... d       as pld_score_hidden
 *   attn ... agg       as pld_score_attn
 *   lens, cand_pos, cap, cand_count, B   the one candidate list both rank
 *   threshold_h, threshold_a   each ranking's threshold
 *   scores_h, scores_a         each ranking's scores, [B][cap] fp32 (may be NULL)
 *   workspace_h, workspace_a   each ranking's keys: two distinct workspaces
 *                   (the rules above); pld_select_draft with workspace_h and
 *                   aux_workspace = workspace_a resolves both
 * Errors: those of the two separate calls, checked in that order, and
 * PLD_ERR_WORKSPACE when the key regions of the two workspaces (the first
 * 128 * B bytes of each) overlap.
 */
int pld_score_both(const uint16_t *hidden, int64_t h_seq_stride, int64_t h_row_stride,
                   int64_t n_rows, int d, const float *attn, int64_t a_seq_stride,
                   int64_t a_row_stride, int64_t n_keys, int R, int agg, const int32_t *lens,
                   const int32_t *cand_pos, int64_t cap, const int32_t *cand_count, int B,
                   float threshold_h, float threshold_a, float *scores_h, float *scores_a,
                   void *workspace_h, size_t workspace_h_bytes, void *workspace_a,
                   size_t workspace_a_bytes, void *stream);

int pld_select_best(int B, int32_t *best_pos, float *best_score, void *workspace,
                    size_t workspace_bytes, void *stream);

/*
 * pld_select_draft -- pld_select_best followed by pld_emit_draft in one
 * launch (the argmax over the occurrences, then the draft of Sec. 4.3): from
 * the keys a scoring call left in `workspace`, best_pos / best_score, then
 * draft / draft_len exactly as pld_emit_draft writes them for that best_pos.
 * With aux_workspace non-NULL, the keys a second scoring call left there (a
 * second ranking of the same occurrences, e.g. attention beside hidden states)
 * are resolved as well, into aux_best_pos / aux_best_score only.  Both
 * workspaces are returned to zero.  One dependent launch fewer per step than
 * the separate calls, two fewer with a second ranking.
 *
 *   tokens, lens, K, draft, draft_len   as pld_emit_draft
 *   best_pos, best_score                as pld_select_best
 *   workspace       the first ranking's keys (pld_score_hidden / _attn)
 *   aux_workspace   NULL, or the second ranking's keys: a buffer of its own of
 *                   at least pld_workspace_bytes(B, K) bytes, zero-filled once
 *   aux_best_pos, aux_best_score   int32 [B], fp32 [B]; required with aux_workspace
 * Errors: PLD_ERR_INVALID (NULL required pointer, B outside [1, PLD_MAX_BATCH],
 * K < 1, tok_stride outside [1, 2^30], aux_workspace without its outputs),
 * PLD_ERR_WORKSPACE (a workspace NULL or too small, or the key regions of the
 * two, the first 128 * B bytes of each, overlapping), PLD_ERR_LAUNCH.
 */
int pld_select_draft(const int32_t *tokens, int64_t tok_stride, const int32_t *lens, int B, int K,
                     int32_t *best_pos, float *best_score, int32_t *draft, int32_t *draft_len,
                     void *workspace, size_t workspace_bytes, void *aux_workspace,
                     size_t aux_workspace_bytes, int32_t *aux_best_pos, float *aux_best_score,
                     void *stream);

int pld_verify_argmax(const void *logits, int dtype, int64_t l_seq_stride, int64_t l_row_stride,
                      int V, int K, const int32_t *draft_len, int B, void *workspace,
                      size_t workspace_bytes, void *stream);

int pld_verify_accept(const int32_t *draft, const int32_t *draft_len, int B, int K,
                      int32_t *accept_len, int32_t *out_tokens, int32_t *out_count,
                      void *workspace, size_t workspace_bytes, void *stream);

int pld_verify_sample_stats(const void *logits, int dtype, int64_t l_seq_stride,
                            int64_t l_row_stride, int V, int K, const int32_t *draft_len, int B,
                            double temperature, void *workspace, size_t workspace_bytes,
                            void *stream);

int pld_verify_sample_finish(const void *logits, int dtype, int64_t l_seq_stride,
                             int64_t l_row_stride, int V, int K, const int32_t *draft,
                             const int32_t *draft_len, int B, double temperature,
                             const float *uniforms, int64_t u_stride, int32_t *accept_len,
                             int32_t *out_tokens, int32_t *out_count, int32_t *row_sample,
                             void *workspace, size_t workspace_bytes, void *stream);

/*
 * pld_select_prefix -- prompt lookup's selection, the baseline PLD+ replaces
 * (Sec. 2; the Fig. 3 caption: the candidate span with the longest matching
 * prefix), for comparisons on the same occurrence lists.  For a candidate j,
 * 0 <= j <= T-2:
 *   m_j = the largest m <= max_match with x[j-k] = x[T-1-k] for all k < m
 *         (indices j-k >= 0 only);
 * j* = the largest m_j, the earliest j among equal lengths (prompt lookup
 * keeps the first match of a left-to-right scan).  best_score = m_j.  With
 * max_match equal to the n-gram length used by pld_find_candidates every
 * candidate ties, and j* is the first occurrence.
 *
 *   tokens, lens  as pld_find_candidates;  cand_pos [B][cap], cand_count [B]
 *   max_match     in [1, PLD_MAX_MATCH]
 *   scores        float [B][cap] or NULL: m_j, NaN for candidates outside
 *                 [0, T-2]; entries past cand_count are not written
 * Device-side rules: a count outside [0, cap] counts as 0; a sequence with
 * T < 2 or T > tok_stride gets best_pos = -1, best_score = -inf.
 * Cost: one 256-thread block per sequence, one trip to memory per 16 matched
 * tokens of a candidate, so a sequence takes about cand_count / 256 rounds
 * of ceil(m / 16) trips: made for the lists of a decoding step (thousands of
 * candidates), not for lists of millions.
 * Errors: PLD_ERR_INVALID (NULL, B outside [1, 65535], tok_stride or cap out
 * of range, bad max_match), PLD_ERR_LAUNCH.
 */
#define PLD_MAX_MATCH 1024
int pld_select_prefix(const int32_t *tokens, int64_t tok_stride, const int32_t *lens,
                      const int32_t *cand_pos, int64_t cap, const int32_t *cand_count, int B,
                      int max_match, float *scores, int32_t *best_pos, float *best_score,
                      void *stream);

/*
 * pld_commit -- the step after verification in the generation loop: the
 * accepted draft tokens and the model's own token join the sequence (Sec. 3,
 * Sec. 4.4).  Per sequence, with cap = min(limit[b], tok_stride) (tok_stride
 * when limit is NULL) and T = lens[b]:
 *   m = min(out_count[b], cap - T);  tokens[b][T + i] = out_tokens[b][i], i < m;
 *   lens[b] = T + m;  stats[b] += (m, 1 if m > 0)   (stats may be NULL)
 * stats[b] = (emitted tokens, steps) gives the paper's average acceptance
 * length, tokens per generation step (Sec. 5.3), as their ratio.
 *
 *   tokens     int32 [B][tok_stride], lens int32 [B] (both updated in place)
 *   limit      int32 [B] or NULL: a per-sequence length limit
 *   out_tokens int32 [B][K+1], out_count int32 [B] (from a verification call)
 *   stats      int64 [B][2] or NULL, accumulated
 * Device-side rule: a sequence with T outside [0, cap] or out_count outside
 * [0, K+1] is left unchanged.
 * Errors: PLD_ERR_INVALID (NULL, B outside [1, 65535], K outside [1, 65534]
 * (the verification calls' limits), tok_stride out of range), PLD_ERR_LAUNCH.
 */
int pld_commit(int32_t *tokens, int64_t tok_stride, int32_t *lens, const int32_t *limit,
               const int32_t *out_tokens, const int32_t *out_count, int B, int K,
               int64_t *stats, void *stream);

/*
 * pld_accept_commit -- pld_verify_accept followed by pld_commit in one launch,
 * for the generation loop after pld_verify_argmax (Sec. 3, Sec. 4.4): the
 * accepted length and emitted tokens from the row maxima in the workspace
 * (which is returned to zero), then those tokens appended to the sequence,
 * the length advanced and the counters added to.  Every output (accept_len,
 * out_tokens, out_count, tokens, lens, stats) is the same as the two calls
 * give; one dependent launch fewer per step.
 *
 *   draft ... workspace   as pld_verify_accept
 *   tokens ... stats      as pld_commit (K is the same)
 * Device-side rules: those of the two calls.
 * Errors: the union of the two calls' errors.
 */
int pld_accept_commit(const int32_t *draft, const int32_t *draft_len, int B, int K,
                      int32_t *accept_len, int32_t *out_tokens, int32_t *out_count,
                      int32_t *tokens, int64_t tok_stride, int32_t *lens, const int32_t *limit,
                      int64_t *stats, void *workspace, size_t workspace_bytes, void *stream);

/*
 * pld_draft_hidden / pld_draft_attn -- the drafting half of a step in one
 * call: pld_find_candidates, then pld_rank_hidden (or pld_rank_attn), then
 * pld_emit_draft, with the same definitions, outputs and device-side rules
 * (Eq. 1, Eq. 2 / Eq. 3 and Sec. 4.3); scores, choices and drafts are
 * bit-identical to the separate calls.
 *
 *   blocks_per_seq  S in [1, PLD_MAX_DRAFT_SPLIT]:
 *                   S = 1: one block per sequence and one launch, no
 *                     workspace; needs tok_stride <= 8192.  The lowest
 *                     latency for short contexts and short candidate lists.
 *                   S > 1: the positions are split into S slices of
 *                     P = ceil(tok_stride / S) rounded up to a multiple of 8
 *                     (P <= 8192), one block each; a block finds, scores and
 *                     lists the occurrences in its slice, and a finishing
 *                     launch compacts the lists and writes the selection and
 *                     the draft (with ngram_min < ngram_max a counting launch
 *                     comes first).  Spreads long contexts and long lists
 *                     over S x B blocks.
 *   workspace       S > 1: at least pld_draft_workspace_bytes(B, S) bytes of
 *                   its own (not shared with the ranking or verification
 *                   calls), zero before the first call.  Its first B*128
 *                   bytes (the key slots) are left zero by every call; the
 *                   rest is per-block counts, rewritten by each call.  Calls
 *                   that share one workspace must not overlap in time.
 *   cand_pos, scores  entries past cand_count are unspecified on return.
 *   scores          may be NULL.
 * Errors: as the separate calls; S out of range, S = 1 with tok_stride > 8192
 * or S > 1 with P > 8192 is PLD_ERR_INVALID; S > 1 without a large enough
 * workspace is PLD_ERR_WORKSPACE.
 */
#define PLD_MAX_DRAFT_SPLIT 1024

/* Workspace bytes of the one-call drafting for B sequences and S blocks per
 * sequence (0 for S = 1, and for arguments out of range). */
size_t pld_draft_workspace_bytes(int B, int blocks_per_seq);

int pld_draft_hidden(const int32_t *tokens, int64_t tok_stride, const int32_t *lens, int B,
                     int ngram_min, int ngram_max, const uint16_t *hidden, int64_t h_seq_stride,
                     int64_t h_row_stride, int64_t n_rows, int d, float threshold, int K,
                     int32_t *cand_pos, int64_t cap, int32_t *cand_count, int32_t *ngram_used,
                     float *scores, int32_t *best_pos, float *best_score, int32_t *draft,
                     int32_t *draft_len, int blocks_per_seq, void *workspace,
                     size_t workspace_bytes, void *stream);

int pld_draft_attn(const int32_t *tokens, int64_t tok_stride, const int32_t *lens, int B,
                   int ngram_min, int ngram_max, const float *attn, int64_t a_seq_stride,
                   int64_t a_row_stride, int64_t n_keys, int R, int agg, float threshold, int K,
                   int32_t *cand_pos, int64_t cap, int32_t *cand_count, int32_t *ngram_used,
                   float *scores, int32_t *best_pos, float *best_score, int32_t *draft,
                   int32_t *draft_len, int blocks_per_seq, void *workspace,
                   size_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* PLD_H */
