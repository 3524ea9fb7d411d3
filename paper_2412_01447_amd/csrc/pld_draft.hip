// pld_draft.hip -- the drafting half of a PLD+ step (arXiv 2412.01447, Sec. 4)
// in one call: occurrence search (Eq. 1, n-grams longest first), ranking by
// hidden-state cosine (Eq. 2) or aggregated attention (Eq. 3, Sec. 7.1),
// selection of the best occurrence, and the draft span (Sec. 4.3).
//
// S == 1 (tok_stride <= 8192): one 1024-thread block owns a sequence.  It
//   copies the token row and the query row into LDS, finds the occurrences
//   (the one-block search of the find call, listing them in LDS as well),
//   scores them with the same per-row routines as the separate ranking calls
//   (bit-identical scores), selects, and writes the draft -- one launch.
// S  > 1: the positions are partitioned.  Block s of a sequence owns the
//   positions [s*P, (s+1)*P) (P <= 8192, a multiple of 8): it stages only
//   those tokens, finds its own occurrences, scores them, and folds its best
//   key into the sequence's key slots.  Its part of the occurrence list (and
//   of the scores) goes to offset s*P of the outputs -- a block never holds
//   more occurrences than positions, so this stays inside the row.  A
//   finishing kernel turns the per-block counts into offsets, compacts the
//   parts in order, and selects and writes the draft.  With a range of n-gram
//   lengths a counting pass first writes per-block occurrence counts of every
//   n, from which every block takes the same longest n.  Work per block is a
//   P-position slice, so long contexts and long candidate lists spread over
//   as many CUs as the caller asks for.
#include <math.h>

#include "pld.h"
#include "pld_device.h"
#include "pld_match.h"

namespace pld {

constexpr int kPartMax = 8192;                  // positions per block, S > 1
constexpr int kPartWaves = 4;                   // counting pass; ranking blocks of many
constexpr int kPartWavesFew = 8;                // ranking blocks when the grid is small
constexpr int kFewBlocks = 512;                 // B*S up to which the blocks get 8 waves
// Positions searched per pass and passes per block for a block of kWaves waves.
template <int kWaves>
struct PartShape {
    static constexpr int kPass = kWaves * kWave * kLanePos;
    static constexpr int kPasses = kPartMax / kPass;
};
constexpr int kWindow = 16384;                  // list entries per compaction pass
constexpr int kFinishThreads = 1024;
constexpr int kWindowPer = kWindow / kFinishThreads;   // entries per thread and pass
constexpr int kSpecPer = 16;     // parts per wave read ahead by the finishing kernel
constexpr int kSpecWaves = kFinishThreads / kWave - 1;   // all but the draft's wave
constexpr int kSpecParts = kSpecWaves * kSpecPer;        // S it covers (240)
static_assert(PLD_MAX_DRAFT_SPLIT <= kFinishThreads, "one block count per finishing thread");

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
    // S > 1 only (workspace)
    int S;
    int64_t P;
    uint64_t *keys;     // [B][kKeySlots], zero on entry and on exit
    int32_t *hcount;    // [B][S] occurrences found by each block
    int32_t *lvl;       // [B][S][kMaxNgram] per-n counts (ngram_min < ngram_max)
};

static size_t part_ws_bytes(int B, int S) {
    return align_up((size_t)B * kKeySlots * 8, 256) + align_up((size_t)B * S * 4, 256) +
           align_up((size_t)B * S * kMaxNgram * 4, 256);
}

static void part_ws_layout(DraftArgs &a, void *ws) {
    char *p = (char *)ws;
    a.keys = (uint64_t *)p;
    p += align_up((size_t)a.B * kKeySlots * 8, 256);
    a.hcount = (int32_t *)p;
    p += align_up((size_t)a.B * a.S * 4, 256);
    a.lvl = (int32_t *)p;
}

// Scores this wave's share of the candidates: list slots c = first, first +
// step, ... < total, G rows at a time (the same per-row arithmetic as the
// multi-block ranking kernel); score c goes to scores[b][out0 + c].
template <int G>
__device__ void draft_score_rows(const DraftArgs &a, int b, int64_t T, bool seq_ok,
                                 const uint16_t *Hb, const uint4 *q_s, float qq,
                                 const int32_t *s_cand, int first, int step, int total,
                                 int64_t out0, uint64_t &best) {
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
            if (a.scores && lane == 0)
                a.scores[(int64_t)b * a.cap + out0 + first + (k + g) * step] = s;
        }
    }
}

// The same for rows of d = 1024 * kU, streamed through stream_rows' two-deep
// pipeline, two pieces per row (the same bits as draft_score_rows).
template <int kU>
__device__ void draft_score_rows_stream(const DraftArgs &a, int b, int64_t T, bool seq_ok,
                                        const uint16_t *Hb, const uint4 *q_s, float qq,
                                        const int32_t *s_cand, int first, int step, int total,
                                        int64_t out0, uint64_t &best) {
    const int lane = lane_id();
    const int n = total > first ? (total - first + step - 1) / step : 0;
    auto row = [&](int k) -> const uint4 * {
        const int32_t j = s_cand[first + k * step];
        const bool ok = seq_ok && j >= 1 && (int64_t)j <= T - 2;
        return ok ? reinterpret_cast<const uint4 *>(Hb + (int64_t)(j - 1) * a.hr) : nullptr;
    };
    stream_rows<2, kU>(n, row, q_s, [&](int k, bool ok, float dot, float nrm) {
        float s = __builtin_nanf("");
        if (ok) {
            s = cosine(dot, nrm, qq);
            if (s > a.threshold) {
                const uint64_t key = rank_key(s, s_cand[first + k * step]);
                best = key > best ? key : best;
            }
        }
        if (a.scores && lane == 0) a.scores[(int64_t)b * a.cap + out0 + first + k * step] = s;
    });
}

// The block's share of the ranking (Eq. 2 / Eq. 3) over the list s_cand of
// `total` candidates: list slots w, w + kWaves, ... per wave (hidden), or one
// slot per group of kGatherLanes lanes (attention).  Returns the block's best key in every thread;
// `s_q` holds the query row (hidden), `s_key` is kWaves words of LDS.
template <bool kHidden, int kWaves, int kU>
__device__ uint64_t rank_candidates(const DraftArgs &a, int b, int64_t T, bool seq_ok,
                                    const int32_t *s_cand, int total, int64_t out0,
                                    const uint4 *s_q, uint64_t *s_key) {
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    uint64_t best = 0;
    if constexpr (kHidden) {
        const uint16_t *Hb = a.hidden + (int64_t)b * a.hs;
        const int nch = a.d / 8;
        const float qq = seq_ok ? query_norm(s_q, nch) : 0.f;
        if constexpr (kU > 0)
            draft_score_rows_stream<kU>(a, b, T, seq_ok, Hb, s_q, qq, s_cand, w, kWaves,
                                             total, out0, best);
        else if (nch <= 4 * kWave)
            draft_score_rows<4>(a, b, T, seq_ok, Hb, s_q, qq, s_cand, w, kWaves, total, out0, best);
        else if (nch <= 8 * kWave)
            draft_score_rows<2>(a, b, T, seq_ok, Hb, s_q, qq, s_cand, w, kWaves, total, out0, best);
        else
            draft_score_rows<1>(a, b, T, seq_ok, Hb, s_q, qq, s_cand, w, kWaves, total, out0, best);
        // (every lane of a wave holds the wave's best)
    } else {
        const float *Ab = a.attn + (int64_t)b * a.as;
        constexpr int kPerPass = kWaves * kWave / kGatherLanes;   // a lane group per candidate
        for (int c0 = 0; c0 < total; c0 += kPerPass) {
            const int c = c0 + (int)threadIdx.x / kGatherLanes;
            const int32_t j = c < total ? s_cand[c] : 0;
            const bool ok = c < total && seq_ok && j >= 1 && (int64_t)j <= T - 2 &&
                            (int64_t)(j - 1) < a.n_keys;
            const float g = attn_gather_group(Ab + (ok ? j - 1 : 0), a.ar, a.R,
                                              a.agg == PLD_AGG_SUM, ok);
            const float s = ok ? g : __builtin_nanf("");
            if (ok && s > a.threshold) {
                const uint64_t k = rank_key(s, j);
                best = k > best ? k : best;
            }
            if (c < total && a.scores && (threadIdx.x & (kGatherLanes - 1)) == 0)
                a.scores[(int64_t)b * a.cap + out0 + c] = s;
        }
        best = wave_max_u64(best);
    }
    if (lane == 0) s_key[w] = best;
    __syncthreads();
    best = 0;
    for (int i = 0; i < kWaves; ++i) best = s_key[i] > best ? s_key[i] : best;
    return best;
}

// The choice and the draft of sequence b from its best key (Sec. 4.3),
// written by one wave; `x` is the sequence's token row (global memory or its
// LDS copy).
__device__ void write_draft(const DraftArgs &a, int b, int64_t T, bool tok_ok, uint64_t best,
                            const int32_t *x) {
    write_choice_draft(best, T, tok_ok, x, a.K, a.best_pos + b, a.best_score + b,
                       a.draft + (int64_t)b * a.K, a.draft_len + b);
}

// ------------------------------------------------------------------- S == 1
template <bool kHidden, int kU>
__global__ __launch_bounds__(kFindWavesFused * kWave) void draft_kernel(DraftArgs a) {
    constexpr int kWaves = kFindWavesFused;
    __shared__ __align__(16) int32_t s_buf[kFindFusedMax];   // the tokens
    __shared__ int32_t s_list[kFindFusedMax];                // the occurrence list
    extern __shared__ uint4 s_q[];                           // query row H[T-2] (hidden)
    __shared__ int s_lvl[kWaves][kMaxNgram];
    __shared__ uint64_t s_key[kWaves];
    const int b = blockIdx.y;
    const int w = threadIdx.x / kWave;
    const int32_t *x = a.tokens + (int64_t)b * a.tok_stride;

    // the token row straight into LDS when it is 16-byte aligned (it does not
    // wait for the length), then the query row
    const int64_t T = a.lens[b];
    const bool tok_ok = (T >= 1 && T <= a.tok_stride);   // block-uniform
    const bool seq_ok = kHidden ? (T >= 2 && T - 2 < a.n_rows) : (T >= 2);
    if (((uintptr_t)x & 15) == 0 && (a.tok_stride & 3) == 0)
        copy_to_lds(reinterpret_cast<const uint4 *>(x), reinterpret_cast<uint4 *>(s_buf),
                    (int)(a.tok_stride / 4));
    else
        stage_tokens(x, 0, a.tok_stride, s_buf);
    if (kHidden && tok_ok && seq_ok)
        copy_to_lds(reinterpret_cast<const uint4 *>(a.hidden + (int64_t)b * a.hs + (T - 2) * a.hr),
                    s_q, a.d / 8);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    // ---- occurrences (Eq. 1), longest n first, listed in LDS and in cand_pos
    int n_used = -1, total = 0;
    if (tok_ok) {   // block-uniform
        n_used = block_search<kWaves, kFindFusedMax / (kWaves * kWave)>(
            s_buf, T, a.nmin, a.nmax, s_lvl, a.cand_pos + (int64_t)b * a.cap, s_list, total);
        if (n_used > 0) __syncthreads();   // the list in LDS is complete
    }
    if (threadIdx.x == 0) {
        a.cand_count[b] = total;
        a.ngram_used[b] = n_used;
    }
    uint64_t best = 0;
    if (total > 0)   // block-uniform
        best = rank_candidates<kHidden, kWaves, kU>(a, b, T, seq_ok, s_list, total, 0, s_q,
                                                         s_key);
    if (w == 0) write_draft(a, b, T, tok_ok, best, s_buf);
}

// ------------------------------------------------------------------- S  > 1
// Block s of sequence b: positions [lo, lo + P) with lo = s*P; the tokens
// x[s0, s1) with s0 = lo - 8 (0 when lo == 0) and s1 = min(lo + P,
// tok_stride) are staged, asynchronously when the copy is 16-byte aligned.
__device__ __forceinline__ void stage_part(const int32_t *x, int64_t s0, int64_t s1, int32_t *s) {
    if ((((uintptr_t)(x + s0)) & 15) == 0 && ((s1 - s0) & 3) == 0)
        copy_to_lds(reinterpret_cast<const uint4 *>(x + s0), reinterpret_cast<uint4 *>(s),
                    (int)((s1 - s0) / 4));
    else
        stage_tokens(x, s0, s1, s);
}

// Hit words of this thread, pass by pass (pass t: the 8 positions from
// lo + t*2048 + 8*threadIdx.x); zero from lo + P on.
template <int kWaves>
__device__ __forceinline__ void part_hits(const int32_t *s_x, int64_t s0, int64_t T, int64_t lo,
                                          int64_t P, const Query &q, int nmax,
                                          uint64_t (&hits)[PartShape<kWaves>::kPasses]) {
    constexpr int kPasses = PartShape<kWaves>::kPasses, kPass = PartShape<kWaves>::kPass;
#pragma unroll
    for (int t = 0; t < kPasses; ++t) {
        const int64_t base = lo + (int64_t)t * kPass + (int64_t)threadIdx.x * kLanePos;
        hits[t] = (base < lo + P) ? lane_hits(s_x, s0, T, base, q, nmax) : 0ull;
    }
}

// Counting pass (ngram_min < ngram_max): per-block occurrence counts of every n.
__global__ __launch_bounds__(kPartWaves * kWave) void draft_count_kernel(DraftArgs a) {
    __shared__ __align__(16) int32_t s_x[kPartMax + 8];
    __shared__ int s_cnt[kMaxNgram];
    const int s = blockIdx.x, b = blockIdx.y;
    const int lane = lane_id();
    const int32_t *x = a.tokens + (int64_t)b * a.tok_stride;
    const int64_t T = a.lens[b];
    const int64_t lo = (int64_t)s * a.P;
    int32_t *out = a.lvl + ((int64_t)b * a.S + s) * kMaxNgram;
    if (!(T >= 1 && T <= a.tok_stride) || lo > T - 2) {   // block-uniform
        if (threadIdx.x < kMaxNgram) out[threadIdx.x] = 0;
        return;
    }
    if (threadIdx.x < kMaxNgram) s_cnt[threadIdx.x] = 0;
    const int64_t s0 = lo >= 8 ? lo - 8 : 0;
    const int64_t s1 = (lo + a.P < a.tok_stride) ? lo + a.P : a.tok_stride;
    stage_part(x, s0, s1, s_x);
    const Query q = load_query(x, T, a.nmax);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    uint64_t hits[PartShape<kPartWaves>::kPasses];
    part_hits<kPartWaves>(s_x, s0, T, lo, a.P, q, a.nmax, hits);
    int cnt[kMaxNgram];
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) cnt[k] = 0;
#pragma unroll
    for (int t = 0; t < PartShape<kPartWaves>::kPasses; ++t) count_levels(hits[t], a.nmax, cnt);
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) {
        if (k < a.nmax) {   // uniform
            const int c = wave_sum_i32(cnt[k]);
            if (lane == 0 && c) atomicAdd(&s_cnt[k], c);
        }
    }
    __syncthreads();
    if (threadIdx.x < kMaxNgram) out[threadIdx.x] = s_cnt[threadIdx.x];
}

// The n every block and the finishing kernel use: ngram_max when it is the
// only length; otherwise the longest n whose occurrence count over all blocks
// of the sequence is non-zero (0 when there is none).  Block-wide; s_tot is
// kMaxNgram words of LDS.
__device__ int part_n(const DraftArgs &a, int b, int *s_tot) {
    if (a.nmin == a.nmax) return a.nmax;
    if (threadIdx.x < kMaxNgram) s_tot[threadIdx.x] = 0;
    __syncthreads();
    int t[kMaxNgram];
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) t[k] = 0;
    for (int s = threadIdx.x; s < a.S; s += blockDim.x) {
        const int32_t *c = a.lvl + ((int64_t)b * a.S + s) * kMaxNgram;
#pragma unroll
        for (int k = 0; k < kMaxNgram; ++k)
            if (k < a.nmax) t[k] += c[k];
    }
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) {
        if (k < a.nmax) {   // uniform
            const int v = wave_sum_i32(t[k]);
            if (lane_id() == 0 && v) atomicAdd(&s_tot[k], v);
        }
    }
    __syncthreads();
    for (int n = a.nmax; n >= a.nmin; --n)
        if (s_tot[n - 1] > 0) return n;
    return 0;
}

// Dynamic LDS of the partitioned kernel: the block's tokens (P + 8, then its
// list), 16-byte aligned, then the query row (hidden) -- sized to the slice so
// that small slices leave room for many blocks per CU.
static size_t part_tok_bytes(int64_t P) { return align_up((size_t)(P + 8) * 4, 16); }

template <bool kHidden, int kWaves, int kU>
__global__ __launch_bounds__(kWaves * kWave) void draft_part_kernel(DraftArgs a) {
    constexpr int kPasses = PartShape<kWaves>::kPasses, kPass = PartShape<kWaves>::kPass;
    extern __shared__ uint4 s_dyn[];
    int32_t *s_x = reinterpret_cast<int32_t *>(s_dyn);   // tokens, then the block's list
    const uint4 *s_q = s_dyn + ((a.P + 8) * 4 + 15) / 16;   // query row H[T-2] (hidden)
    __shared__ int s_tot[kMaxNgram];
    __shared__ int s_wc[kPasses][kWaves];
    __shared__ uint64_t s_key[kWaves];
    const int s = blockIdx.x, b = blockIdx.y;
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    const int32_t *x = a.tokens + (int64_t)b * a.tok_stride;
    const int64_t lo = (int64_t)s * a.P;
    // the slice's tokens are requested with the length, not after it (the
    // slice lies inside the token row whatever the length)
    const int64_t s0 = lo >= 8 ? lo - 8 : 0;
    const int64_t s1 = (lo + a.P < a.tok_stride) ? lo + a.P : a.tok_stride;
    stage_part(x, s0, s1, s_x);
    const int64_t T = a.lens[b];
    if (!(T >= 1 && T <= a.tok_stride) || lo > T - 2) {   // block-uniform
        __builtin_amdgcn_s_waitcnt(0);                   // the copy lands before the block ends
        // an invalid length is reported by the finishing kernel; otherwise no
        // position of this block can match
        if (T >= 1 && T <= a.tok_stride && threadIdx.x == 0) a.hcount[(int64_t)b * a.S + s] = 0;
        return;
    }
    const bool seq_ok = kHidden ? (T >= 2 && T - 2 < a.n_rows) : (T >= 2);
    if (kHidden && seq_ok)
        copy_to_lds(reinterpret_cast<const uint4 *>(a.hidden + (int64_t)b * a.hs + (T - 2) * a.hr),
                    const_cast<uint4 *>(s_q), a.d / 8);
    const Query q = load_query(x, T, a.nmax);
    __builtin_amdgcn_s_waitcnt(0);
    const int n = part_n(a, b, s_tot);   // block-uniform
    __syncthreads();                     // (also: the staged tokens are in place)
    if (n == 0) {
        if (threadIdx.x == 0) a.hcount[(int64_t)b * a.S + s] = 0;
        return;
    }
    uint64_t hits[kPasses];
    part_hits<kWaves>(s_x, s0, T, lo, a.P, q, a.nmax, hits);
    uint32_t bits[kPasses];
#pragma unroll
    for (int t = 0; t < kPasses; ++t) {
        bits[t] = level_bits(hits[t], n);
        const int c = wave_sum_i32(__popc(bits[t]));
        if (lane == 0) s_wc[t][w] = c;
    }
    __syncthreads();   // every token read is done: s_x becomes the block's list
    // list order is ascending position: pass, then wave, then lane
    int total = 0;
    int start[kPasses];
#pragma unroll
    for (int t = 0; t < kPasses; ++t) {
        start[t] = total;
        for (int i = 0; i < kWaves; ++i) {
            if (i < w) start[t] += s_wc[t][i];
            total += s_wc[t][i];
        }
    }
    if (threadIdx.x == 0) a.hcount[(int64_t)b * a.S + s] = total;
    if (total == 0) return;   // block-uniform
    int32_t *out = a.cand_pos + (int64_t)b * a.cap + lo;
#pragma unroll
    for (int t = 0; t < kPasses; ++t)
        emit_bits(bits[t], lo + (int64_t)t * kPass + (int64_t)threadIdx.x * kLanePos, s_x,
                  out, start[t]);
    __syncthreads();
    const uint64_t best =
        rank_candidates<kHidden, kWaves, kU>(a, b, T, seq_ok, s_x, total, lo, s_q, s_key);
    if (threadIdx.x == 0 && best)
        atomicMax((unsigned long long *)&a.keys[(int64_t)b * kKeySlots + (s % kKeySlots)],
                  (unsigned long long)best);
}

// One block per sequence: the selection from the key slots (returned to
// zero) and the draft; the offsets of the blocks' parts, in-order compaction
// of the list (and the scores), ngram_used and the count.
//
// Read ahead: with S <= kSpecParts, wave w < 15 reads the first 64 entries
// of parts w, w + 15, ... while the per-part counts are on their way (the
// last wave, which writes the draft, keeps its memory queue to itself); when no
// part holds more than 64 entries these are all of them, and they are written
// to their offsets once every thread's reads have returned -- one trip to
// memory for the whole list.  Otherwise the list is compacted in windows of
// kWindow entries: entry e of part p moves from p*P + e to off[p] + e; with
// D[p] = p*P - off[p], which never decreases with p, the entry at list
// position x comes from x + D of its part.  Per window, each non-empty part
// marks D at its first position in the window, and a running maximum gives
// every position its D.  Entries only move towards the start of the row, so
// a window's sources lie at or after the window and the writes of a window
// never reach a later window's sources; within a window every thread holds
// its entries in registers and every read of the window has completed before
// any of it is written.
__global__ __launch_bounds__(kFinishThreads) void draft_finish_part_kernel(DraftArgs a) {
    __shared__ int32_t s_off[PLD_MAX_DRAFT_SPLIT + 1];
    __shared__ __align__(16) int32_t s_d[kWindow];   // D of each window position
    __shared__ int s_wmax[kFinishThreads / kWave];
    __shared__ int s_tot[kMaxNgram];
    __shared__ int s_wsum[kFinishThreads / kWave];
    __shared__ int s_wcmax[kFinishThreads / kWave];
    const int b = blockIdx.x;
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    // every load that does not wait for another goes out first: the key slots
    // (last wave), the per-block counts, the read-ahead, then the length
    const bool last = (w == kFinishThreads / kWave - 1);
    uint64_t key = 0;
    if (last && lane < kKeySlots) key = a.keys[(int64_t)b * kKeySlots + lane];
    const int cnt = ((int)threadIdx.x < a.S) ? a.hcount[(int64_t)b * a.S + threadIdx.x] : 0;
    int32_t *pos = a.cand_pos + (int64_t)b * a.cap;
    float *sc = a.scores ? a.scores + (int64_t)b * a.cap : nullptr;
    // read ahead: entry `lane` of parts w + 15 j (in the row whatever the counts)
    const bool spec = a.S <= kSpecParts;   // uniform
    int32_t spv[kSpecPer];
    float ssv[kSpecPer];
    if (spec && !last) {
#pragma unroll
        for (int j = 0; j < kSpecPer; ++j) {
            const int q = w + j * kSpecWaves;
            const int64_t src = (int64_t)q * a.P + lane;
            if (q < a.S && lane < a.P && src < a.tok_stride) {
                spv[j] = pos[src];
                if (sc) ssv[j] = sc[src];
            }
        }
    }
    const int64_t T = a.lens[b];
    const bool tok_ok = (T >= 1 && T <= a.tok_stride);   // block-uniform
    // the selection does not depend on the list: the last wave writes it and
    // the draft first, while the others start on the offsets
    if (last) {
        if (lane < kKeySlots) a.keys[(int64_t)b * kKeySlots + lane] = 0;
        key = wave_max_u64(key);
        write_draft(a, b, T, tok_ok, key, a.tokens + (int64_t)b * a.tok_stride);
    }
    int n = -1, total = 0;
    if (tok_ok) {
        n = part_n(a, b, s_tot);
        // exclusive scan of the per-block counts, one per thread
        const int c = n > 0 ? cnt : 0;
        int wt;
        const int ex = wave_excl_scan(c, wt);
        const int cmax = wave_max_nonneg_i32(c);
        if (lane == 0) {
            s_wsum[w] = wt;
            s_wcmax[w] = cmax;
        }
        __syncthreads();
        int pre = 0, most = 0;
        for (int i = 0; i < kFinishThreads / kWave; ++i) {
            if (i < w) pre += s_wsum[i];
            total += s_wsum[i];
            most = max(most, s_wcmax[i]);
        }
        if ((int)threadIdx.x < a.S) s_off[threadIdx.x] = pre + ex;
        if (threadIdx.x == 0) s_off[a.S] = total;
        __builtin_amdgcn_s_waitcnt(0);   // the read-ahead has returned ...
        __syncthreads();                 // ... in every thread (and s_off is complete)
        if (spec && most <= kWave) {     // block-uniform: the read-ahead holds the list
#pragma unroll
            for (int j = 0; j < kSpecPer; ++j) {
                const int q = last ? a.S : w + j * kSpecWaves;
                if (q < a.S && lane < s_off[q + 1] - s_off[q]) {
                    pos[s_off[q] + lane] = spv[j];
                    if (sc) sc[s_off[q] + lane] = ssv[j];
                }
            }
        }
        for (int w0 = 0; !(spec && most <= kWave) && w0 < total; w0 += kWindow) {
            const int wn = min(kWindow, total - w0);
            const int nk = (wn + kFinishThreads - 1) / kFinishThreads;   // block-uniform
            for (int i = threadIdx.x; i < wn; i += kFinishThreads) s_d[i] = 0;
            __syncthreads();
            for (int q = threadIdx.x; q < a.S; q += kFinishThreads) {
                const int o = s_off[q], e = s_off[q + 1];
                if (e > o && e > w0 && o < w0 + wn)
                    s_d[o > w0 ? o - w0 : 0] = (int)((int64_t)q * a.P - o);
            }
            __syncthreads();
            // running maximum: kWindowPer consecutive positions per thread,
            // then across the lanes (DPP) and the waves
            {
                const int base = (int)threadIdx.x * kWindowPer;
                int v[kWindowPer];
#pragma unroll
                for (int c = 0; c < kWindowPer / 4; ++c) {
                    const int4 t = reinterpret_cast<const int4 *>(s_d + base)[c];
                    v[4 * c] = t.x;
                    v[4 * c + 1] = t.y;
                    v[4 * c + 2] = t.z;
                    v[4 * c + 3] = t.w;
                }
#pragma unroll
                for (int c = 0; c < kWindowPer; ++c) {
                    if (base + c >= wn) v[c] = 0;
                    if (c > 0) v[c] = max(v[c], v[c - 1]);
                }
                int inc = v[kWindowPer - 1];
                inc = max(inc, dpp_move<kDppShr1, 0xf>(inc));
                inc = max(inc, dpp_move<kDppShr1 + 1, 0xf>(inc));
                inc = max(inc, dpp_move<kDppShr1 + 3, 0xf>(inc));
                inc = max(inc, dpp_move<kDppShr1 + 7, 0xf>(inc));
                inc = max(inc, dpp_move<kDppBcast15, 0xa>(inc));
                inc = max(inc, dpp_move<kDppBcast31, 0xc>(inc));
                if (lane == kWave - 1) s_wmax[w] = inc;
                int carry = __shfl_up(inc, 1);
                if (lane == 0) carry = 0;
                __syncthreads();
                for (int i = 0; i < w; ++i) carry = max(carry, s_wmax[i]);
#pragma unroll
                for (int c = 0; c < kWindowPer / 4; ++c)
                    reinterpret_cast<int4 *>(s_d + base)[c] =
                        make_int4(max(v[4 * c], carry), max(v[4 * c + 1], carry),
                                  max(v[4 * c + 2], carry), max(v[4 * c + 3], carry));
                __syncthreads();
            }
            int32_t pv[kWindowPer];
            float sv[kWindowPer];
            // all of this thread's reads of the window are issued before any
            // is waited for: one trip to memory per window
#pragma unroll
            for (int k = 0; k < kWindowPer; ++k) {
                const int i = (int)threadIdx.x + k * kFinishThreads;
                if (k < nk && i < wn) {
                    const int64_t src = (int64_t)s_d[i] + w0 + i;
                    pv[k] = pos[src];
                    if (sc) sv[k] = sc[src];
                }
            }
            __builtin_amdgcn_s_waitcnt(0);   // the reads have returned ...
            __syncthreads();                 // ... in every thread of the block
#pragma unroll
            for (int k = 0; k < kWindowPer; ++k) {
                const int i = (int)threadIdx.x + k * kFinishThreads;
                if (k < nk && i < wn) {
                    pos[w0 + i] = pv[k];
                    if (sc) sc[w0 + i] = sv[k];
                }
            }
        }
    }
    if (threadIdx.x == 0) {
        a.cand_count[b] = total;
        a.ngram_used[b] = tok_ok ? (total > 0 ? n : 0) : -1;
    }
}

// ------------------------------------------------------------------- host
static int64_t part_width(int64_t tok_stride, int S) {
    const int64_t p = (tok_stride + S - 1) / S;
    return (p + kLanePos - 1) / kLanePos * kLanePos;
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
    if (B < 1 || B > 65535 || tok_stride < 1 || tok_stride > kMaxTokStride) return PLD_ERR_INVALID;
    if (ngram_min < 1 || ngram_max < ngram_min || ngram_max > PLD_MAX_NGRAM) return PLD_ERR_INVALID;
    if (cap < tok_stride || K < 1 || isnan(threshold)) return PLD_ERR_INVALID;
    if (S < 1 || S > PLD_MAX_DRAFT_SPLIT) return PLD_ERR_INVALID;
    if (S == 1 && tok_stride > kFindFusedMax) return PLD_ERR_INVALID;
    if (S > 1 && part_width(tok_stride, S) > kPartMax) return PLD_ERR_INVALID;
    if (S > 1 && (!workspace || workspace_bytes < part_ws_bytes(B, S))) return PLD_ERR_WORKSPACE;
    return PLD_OK;
}

static DraftArgs make_draft(const int32_t *tokens, int64_t tok_stride, const int32_t *lens, int B,
                            int ngram_min, int ngram_max, float threshold, int K,
                            int32_t *cand_pos, int64_t cap, int32_t *cand_count,
                            int32_t *ngram_used, float *scores, int32_t *best_pos,
                            float *best_score, int32_t *draft, int32_t *draft_len, int S,
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
    a.S = S;
    if (S > 1) {
        a.P = part_width(tok_stride, S);
        part_ws_layout(a, workspace);
    }
    return a;
}

template <bool kHidden, int kU>
static void launch_draft_as(const DraftArgs &a, hipStream_t s) {
    const size_t lds = kHidden ? (size_t)(a.d / 8) * sizeof(uint4) : 0;
    if (a.S == 1) {
        hipLaunchKernelGGL((draft_kernel<kHidden, kU>), dim3(1, a.B),
                           dim3(kFindWavesFused * kWave), lds, s, a);
        return;
    }
    if (a.nmin < a.nmax)
        hipLaunchKernelGGL(draft_count_kernel, dim3(a.S, a.B), dim3(kPartWaves * kWave), 0, s, a);
    // blocks of 8 waves when the grid is small (more rows in flight per block),
    // of 4 otherwise (more blocks resident per CU); the results are the same
    if ((int64_t)a.B * a.S <= kFewBlocks)
        hipLaunchKernelGGL((draft_part_kernel<kHidden, kPartWavesFew, kU>), dim3(a.S, a.B),
                           dim3(kPartWavesFew * kWave), part_tok_bytes(a.P) + lds, s, a);
    else
        hipLaunchKernelGGL((draft_part_kernel<kHidden, kPartWaves, kU>), dim3(a.S, a.B),
                           dim3(kPartWaves * kWave), part_tok_bytes(a.P) + lds, s, a);
    hipLaunchKernelGGL(draft_finish_part_kernel, dim3(a.B), dim3(kFinishThreads), 0, s, a);
}

// Hidden rows of d = 4096 or 8192 take the streaming pipeline (a kernel of
// their own, so each keeps only the registers its path needs).
template <bool kHidden>
static void launch_draft(const DraftArgs &a, hipStream_t s) {
    if constexpr (kHidden) {
        if (a.d == 4096) return launch_draft_as<true, 4>(a, s);
        if (a.d == 8192) return launch_draft_as<true, 8>(a, s);
    }
    launch_draft_as<kHidden, 0>(a, s);
}

}  // namespace pld

using namespace pld;

extern "C" size_t pld_draft_workspace_bytes(int B, int blocks_per_seq) {
    if (B < 1 || B > 65535 || blocks_per_seq < 1 || blocks_per_seq > PLD_MAX_DRAFT_SPLIT) return 0;
    return blocks_per_seq == 1 ? 0 : part_ws_bytes(B, blocks_per_seq);
}

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
                             draft, draft_len, blocks_per_seq, workspace);
    a.hidden = hidden;
    a.hs = h_seq_stride;
    a.hr = h_row_stride;
    a.n_rows = n_rows;
    a.d = d;
    launch_draft<true>(a, (hipStream_t)stream);
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
                             draft, draft_len, blocks_per_seq, workspace);
    a.attn = attn;
    a.as = a_seq_stride;
    a.ar = a_row_stride;
    a.n_keys = n_keys;
    a.R = R;
    a.agg = agg;
    launch_draft<false>(a, (hipStream_t)stream);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}
