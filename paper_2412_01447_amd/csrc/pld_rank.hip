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
// candidate rows: 16-byte nontemporal loads of the bf16 row, the dot product
// and the squared norm by the bf16 dot instruction (two products added into an
// fp32 accumulator, four accumulators per lane), then a DPP wave sum.  The
// reduction order depends only on d, never on the slot, so equal rows give
// bit-identical scores, and a row equal to the query gives exactly 1.
//
// Attention ranking: a group of eight lanes per candidate gathers
// A[b][r][j-1] for r < R (lane t of the group takes rows t, t+8, ...) and the
// group's partials are combined by DPP moves; the candidates are ascending, so
// neighbouring groups read neighbouring keys.
//
// Both rankings of one candidate list (pld_score_both) share one grid: a
// fifth of the resident blocks run the attention blocks' code over the
// attention shares while the rest run the hidden blocks' code over theirs, so
// the scattered attention gathers overlap the stream of hidden rows instead of
// following it in a launch of their own.
//
// Selection: a candidate with s > threshold contributes the 64-bit key
// (orderable(s) << 32 | j); a block reduces its keys per sequence and folds
// them with one 64-bit atomic max into one of kKeySlots workspace slots of the
// sequence (the slot is picked by block index, so an atomic never waits
// behind more than a handful of others on the same address).  A small
// finishing kernel, launched right after on the same stream, turns the keys
// into best_pos / best_score (and, in pld_select_draft, the draft as well) and
// zeroes the slots (the kernel boundary orders the two; no block of the
// ranking kernel ever waits for, or fences against, another).
#include <math.h>

#include "pld.h"
#include "pld_device.h"

namespace pld {

#ifndef PLD_RANK_OVERSUB
#define PLD_RANK_OVERSUB 1           // ranking grid = resident blocks x this (tuning builds)
#endif

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
    uint64_t *keys;     // [B][kKeySlots], zero on entry
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
// of sequences; the thread sums are scanned across the wave (DPP) and with one
// LDS exchange of the wave totals.  With s_lens, the lengths are copied to
// LDS in the same pass.
__device__ __forceinline__ uint32_t clamped_count(const RankCommon &c, int b) {
    const int32_t n = c.cand_count[b];
    return (n >= 0 && (int64_t)n <= c.cap) ? (uint32_t)n : 0u;
}

template <int kThreads = kRankThreads>
__device__ void candidate_prefix(const RankCommon &c, uint32_t *pre, int32_t *s_lens = nullptr) {
    constexpr int kWaves = kThreads / kWave;
    __shared__ uint32_t s_wave[kWaves];
    const int per = (c.B + kThreads - 1) / kThreads;
    const int b0 = threadIdx.x * per;
    const int b1 = min(b0 + per, c.B);
    uint32_t sum = 0;
    for (int b = b0; b < b1; ++b) {
        sum += clamped_count(c, b);
        if (s_lens) s_lens[b] = c.lens[b];   // (requested with the count)
    }
    // inclusive scan across the wave (two's-complement sums: same bits as unsigned)
    int wt;
    const uint32_t inc = (uint32_t)wave_excl_scan((int)sum, wt) + sum;
    const int lane = lane_id();
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
        for (int i = 0; i < kWaves; ++i) t += s_wave[i];
        pre[c.B] = t;
    }
    __syncthreads();
}

// Block k's share [lo, hi) of n items split evenly over g blocks (32-bit).
__device__ __forceinline__ void block_share(uint32_t n, uint32_t k, uint32_t &lo, uint32_t &hi,
                                            uint32_t g) {
    const uint32_t q = n / g, r = n % g;
    lo = k * q + min(k, r);
    hi = lo + q + (k < r ? 1u : 0u);
}

// Consecutive blocks go to the eight XCDs in turn, and each XCD has its own
// L2.  For the attention gathers, whose neighbouring shares read some of the
// same 128-byte lines, block k takes share index
//   (i / m) * 8m + x * m + i % m,   x = k % 8, i = k / 8, m = kXcdRun,
// so that each XCD works through runs of m consecutive shares (most shared
// lines stay in one L2) while the runs of all XCDs interleave along the list
// (every XCD sees the same mix of cheap and costly candidates; one contiguous
// eighth per XCD was measured slower).  Blocks past the last whole group of
// 8m of the first g blocks keep their own index.  A permutation of [0, g)
// (and of the blocks past it): the results do not depend on it.
constexpr uint32_t kXcds = 8, kXcdRun = 16;
__device__ __forceinline__ uint32_t xcd_run_index(uint32_t k, uint32_t g) {
    const uint32_t group = kXcds * kXcdRun;
    if (k >= g / group * group) return k;
    const uint32_t x = k % kXcds, i = k / kXcds;
    return (i / kXcdRun) * group + x * kXcdRun + i % kXcdRun;
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
    uint64_t k = 0;
    uint64_t *slots = c.keys + (int64_t)b * kKeySlots;
#pragma unroll
    for (int i = 0; i < kKeySlots; ++i) {
        const uint64_t v = slots[i];
        k = v > k ? v : k;
    }
#pragma unroll
    for (int i = 0; i < kKeySlots; ++i) slots[i] = 0;
    if (k == 0) {
        c.best_pos[b] = -1;
        c.best_score[b] = -INFINITY;
    } else {
        c.best_pos[b] = (int32_t)(uint32_t)(k & 0xffffffffu);
        c.best_score[b] = unord_f32((uint32_t)(k >> 32));
    }
}

// The selection and the draft in one launch (Sec. 4.3): one wave per
// sequence reads the ranking's key slots (lanes 0..15) and, when a second
// ranking's keys are given, those too (lanes 16..31) together with the length;
// it returns the slots to zero, writes the second ranking's choice, then the
// first one's choice and draft (one more trip to memory, for the tokens).
struct SelectDraftArgs {
    const int32_t *tokens;
    int64_t tok_stride;
    const int32_t *lens;
    int B, K;
    uint64_t *keys;          // [B][kKeySlots], zero on exit
    int32_t *best_pos;
    float *best_score;
    int32_t *draft;
    int32_t *draft_len;
    uint64_t *aux_keys;      // [B][kKeySlots] or null
    int32_t *aux_best_pos;
    float *aux_best_score;
};

__global__ __launch_bounds__(256) void select_draft_kernel(SelectDraftArgs a) {
    const int b = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / kWave);
    if (b >= a.B) return;   // wave-uniform
    const int lane = lane_id();
    const bool own = lane < kKeySlots;
    const bool aux = a.aux_keys && !own && lane < 2 * kKeySlots;
    uint64_t *slot = own ? a.keys + (int64_t)b * kKeySlots + lane
                         : (aux ? a.aux_keys + (int64_t)b * kKeySlots + (lane - kKeySlots)
                                : nullptr);
    const uint64_t k = slot ? *slot : 0ull;
    const int64_t T = a.lens[b];
    if (slot) *slot = 0;
    const uint64_t best = wave_max_u64(own ? k : 0ull);
    if (a.aux_keys) {   // wave-uniform
        const uint64_t ab = wave_max_u64(aux ? k : 0ull);
        if (lane == 0) {
            a.aux_best_pos[b] = ab ? (int32_t)(uint32_t)(ab & 0xffffffffu) : -1;
            a.aux_best_score[b] = ab ? unord_f32((uint32_t)(ab >> 32)) : -INFINITY;
        }
    }
    const bool tok_ok = (T >= 1 && T <= a.tok_stride);
    write_choice_draft(best, T, tok_ok, a.tokens + (int64_t)b * a.tok_stride, a.K,
                       a.best_pos + b, a.best_score + b, a.draft + (int64_t)b * a.K,
                       a.draft_len + b);
}

// ---------------------------------------------------------------- hidden
// Scores the rows i = first, first + kRankWaves, ... < end of sequence b (one
// wave's share of a segment).  The wave fetches the candidate positions of up
// to 64 rows with one load (the first batch, jv0, comes in prefetched), then
// scores G rows at a time with all their loads in flight.  `best` collects the
// wave's best key.
template <int G, int kW>
__device__ void score_rows(const RankHiddenArgs &a, int b, int64_t T, bool seq_ok,
                           const uint16_t *Hb, const uint4 *q_s, float qq, uint32_t first,
                           uint32_t end, uint32_t seq_start, int32_t jv0, uint64_t &best) {
    const RankCommon &c = a.c;
    const int lane = lane_id();
    const int nch = a.d / 8;
    const uint32_t n = end > first ? (end - first + kW - 1) / kW : 0;
    for (uint32_t base = 0; base < n; base += kWave) {
        const uint32_t nb = min((uint32_t)kWave, n - base);
        const uint32_t mine = base + lane;
        int32_t jv = jv0;   // the first batch was requested with the query row
        if (base > 0 && mine < n)
            jv = c.cand_pos[(int64_t)b * c.cap + (first + mine * kW - seq_start)];
        for (uint32_t r = 0; r < nb; r += G) {
            const uint4 *rows[G];
            int32_t js[G];
#pragma unroll
            for (int g = 0; g < G; ++g) {
                js[g] = (r + g < nb) ? __builtin_amdgcn_readlane(jv, r + g) : 0;
                const bool ok = (r + g < nb) && seq_ok && js[g] >= 1 && (int64_t)js[g] <= T - 2;
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
                if (r + g >= nb) break;
                float s = __builtin_nanf("");
                if (rows[g]) {
                    s = cosine(dot[g], nrm[g], qq);
                    if (s > c.threshold) {
                        const uint64_t k = rank_key(s, js[g]);
                        best = k > best ? k : best;
                    }
                }
                if (c.scores && lane == 0)
                    c.scores[(int64_t)b * c.cap +
                             (first + (base + r + g) * kW - seq_start)] = s;
            }
        }
    }
}

// The same for rows of d = 1024 * kU: the wave's rows stream through
// stream_rows' two-deep pipeline, two pieces per row (same bits as score_rows).
template <int kU, int kW>
__device__ void score_rows_stream(const RankHiddenArgs &a, int b, int64_t T, bool seq_ok,
                                  const uint16_t *Hb, const uint4 *q_s, float qq, uint32_t first,
                                  uint32_t end, uint32_t seq_start, int32_t jv0, uint64_t &best) {
    const RankCommon &c = a.c;
    const int lane = lane_id();
    const uint32_t n = end > first ? (end - first + kW - 1) / kW : 0;
    for (uint32_t base = 0; base < n; base += kWave) {
        const uint32_t nb = min((uint32_t)kWave, n - base);
        const uint32_t mine = base + lane;
        int32_t jv = jv0;   // the first batch was requested with the query row
        if (base > 0 && mine < n)
            jv = c.cand_pos[(int64_t)b * c.cap + (first + mine * kW - seq_start)];
        auto row = [&](int k) -> const uint4 * {
            const int32_t j = __builtin_amdgcn_readlane(jv, k);
            const bool ok = seq_ok && j >= 1 && (int64_t)j <= T - 2;
            return ok ? reinterpret_cast<const uint4 *>(Hb + (int64_t)(j - 1) * a.hr) : nullptr;
        };
        stream_rows<2, kU>((int)nb, row, q_s,
                                            [&](int k, bool ok, float dot, float nrm) {
            float s = __builtin_nanf("");
            if (ok) {
                s = cosine(dot, nrm, qq);
                if (s > c.threshold) {
                    const uint64_t key = rank_key(s, __builtin_amdgcn_readlane(jv, k));
                    best = key > best ? key : best;
                }
            }
            if (c.scores && lane == 0)
                c.scores[(int64_t)b * c.cap + (first + (base + k) * kW - seq_start)] = s;
        });
    }
}

// Block k of g of the hidden-state ranking (its share of the flattened
// list).  smem: the query row (d/8 chunks), then pre (B + 1) and the lengths
// (B); s_best: kW words.
template <int kU, int kW>
__device__ void hidden_block(const RankHiddenArgs &a, uint32_t k, uint32_t g, uint4 *smem,
                             uint64_t *s_best) {
    const RankCommon &c = a.c;
    const int nch = a.d / 8;
    uint4 *q_s = smem;                                         // nch chunks of 8 bf16
    uint32_t *pre = reinterpret_cast<uint32_t *>(smem + nch);  // B + 1
    int32_t *lens = reinterpret_cast<int32_t *>(pre + c.B + 1); // B
    candidate_prefix<kW * kWave>(c, pre, lens);
    uint32_t lo0, hi;
    block_share(pre[c.B], k, lo0, hi, g);
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    if (lo0 >= hi) return;   // block-uniform: nothing to score
    int b = seq_of(pre, c.B, lo0);
    uint32_t lo = lo0;
    while (lo < hi) {
        while (pre[b + 1] <= lo) ++b;                          // skip empty sequences
        const uint32_t seg_hi = min(hi, pre[b + 1]);
        const int64_t T = lens[b];
        const bool seq_ok = (T >= 2 && T - 2 < a.n_rows);
        const uint16_t *Hb = a.hidden + (int64_t)b * a.hs;
        // the wave's first 64 candidate positions and the query row travel together
        const uint32_t first = lo + w;
        const uint32_t nw = seg_hi > first ? (seg_hi - first + kW - 1) / kW : 0;
        const int32_t jv0 = (uint32_t)lane < nw
            ? c.cand_pos[(int64_t)b * c.cap + (first + (uint32_t)lane * kW - pre[b])] : 0;
        if (seq_ok) copy_to_lds(reinterpret_cast<const uint4 *>(Hb + (T - 2) * a.hr), q_s, nch);
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        const float qq = seq_ok ? query_norm(q_s, nch) : 0.f;
        uint64_t best = 0;
        if constexpr (kU > 0)
            score_rows_stream<kU, kW>(a, b, T, seq_ok, Hb, q_s, qq, first, seg_hi, pre[b], jv0,
                                       best);
        else if (nch <= 4 * kWave)
            score_rows<4, kW>(a, b, T, seq_ok, Hb, q_s, qq, first, seg_hi, pre[b], jv0, best);
        else if (nch <= 8 * kWave)
            score_rows<2, kW>(a, b, T, seq_ok, Hb, q_s, qq, first, seg_hi, pre[b], jv0, best);
        else
            score_rows<1, kW>(a, b, T, seq_ok, Hb, q_s, qq, first, seg_hi, pre[b], jv0, best);
        if (lane == 0) s_best[w] = best;
        __syncthreads();                                       // also: q_s is restaged next
        if (threadIdx.x == 0) {
            uint64_t m = s_best[0];
            for (int i = 1; i < kW; ++i) m = s_best[i] > m ? s_best[i] : m;
            if (m)
                atomicMax((unsigned long long *)&c.keys[(int64_t)b * kKeySlots + (k % kKeySlots)],
                          (unsigned long long)m);
        }
        lo = seg_hi;
    }
}

// kU > 0: rows of d = 1024 * kU through the streaming pipeline; 0: any d
// through score_rows (one instantiation per path keeps each kernel's register
// count to what its path needs).
template <int kU, int kW>
__global__ __launch_bounds__(kW * kWave) void rank_hidden_kernel(RankHiddenArgs a) {
    extern __shared__ uint4 smem[];
    __shared__ uint64_t s_best[kW];
    hidden_block<kU, kW>(a, blockIdx.x, gridDim.x, smem, s_best);
}

// ------------------------------------------------------------------ attn
#ifndef PLD_ATTN_MIN_SHARE
#define PLD_ATTN_MIN_SHARE 8         // candidates per active attention block (tuning builds)
#endif
constexpr uint32_t kAttnMinShare = PLD_ATTN_MIN_SHARE;
// Only as many blocks as give every block at least kAttnMinShare candidates
// (a wave's pass: one per lane group) take shares; the rest return after the
// prefix.  With few candidates in all, a share per resident block would leave
// most blocks with one or two candidates, each paying the whole prologue
// (measured: 9.5 -> 7.5 us on 32 x 8192 with 40 rows; 8 per block was faster
// than 16 or 32, and the 64 x 16384 workload, with more candidates than
// 8 per resident block, keeps every block).
// Block blk of g of the attention ranking; pre: B + 1 words of LDS.
__device__ void attn_block(const RankAttnArgs &a, uint32_t blk, uint32_t g, uint32_t *pre) {
    const RankCommon &c = a.c;
    candidate_prefix(c, pre);
    // a group of kGatherLanes lanes per candidate
    constexpr uint32_t kPerPass = kRankThreads / kGatherLanes;
    const uint32_t total = pre[c.B];
    const uint32_t active = min(g, (total + kAttnMinShare - 1) / kAttnMinShare);
    const uint32_t k = xcd_run_index(blk, active);
    if (k >= active) return;   // block-uniform
    uint32_t lo, hi;
    block_share(total, k, lo, hi, active);
    for (uint32_t base = lo; base < hi; base += kPerPass) {
        const uint32_t i = base + threadIdx.x / kGatherLanes;
        const bool active = i < hi;
        int b = active ? seq_of(pre, c.B, i) : 0;
        uint64_t key = 0;
        const int64_t cs = active ? (int64_t)(i - pre[b]) : 0;   // the candidate's list slot
        const int32_t j = active ? c.cand_pos[(int64_t)b * c.cap + cs] : 0;
        const int64_t T = active ? c.lens[b] : 0;
        const bool ok = active && T >= 2 && j >= 1 && (int64_t)j <= T - 2 &&
                        (int64_t)(j - 1) < a.n_keys;
        const float g = attn_gather_group(a.attn + (int64_t)b * a.as + (ok ? j - 1 : 0), a.ar,
                                          a.R, a.agg == PLD_AGG_SUM, ok);
        const float s = ok ? g : __builtin_nanf("");
        if (ok && s > c.threshold) key = rank_key(s, j);
        if (active && c.scores && (threadIdx.x & (kGatherLanes - 1)) == 0)
            c.scores[(int64_t)b * c.cap + cs] = s;
        // one atomic per wave when all its lanes share a sequence
        const int b0 = __shfl(b, 0);
        const bool same = __ballot(active && b != b0) == 0ull;
        const int slot = (int)((blk * kRankWaves + threadIdx.x / kWave) % kKeySlots);
        if (same) {
            uint64_t m = wave_max_u64(key);
            if (lane_id() == 0 && m)
                atomicMax((unsigned long long *)&c.keys[(int64_t)b0 * kKeySlots + slot],
                          (unsigned long long)m);
        } else if (key) {
            atomicMax((unsigned long long *)&c.keys[(int64_t)b * kKeySlots + slot],
                      (unsigned long long)key);
        }
    }
}

__global__ __launch_bounds__(kRankThreads) void rank_attn_kernel(RankAttnArgs a) {
    __shared__ uint32_t pre[PLD_MAX_BATCH + 1];
    attn_block(a, blockIdx.x, gridDim.x, pre);
}

// Both rankings of the same occurrences in one launch: blocks [0, ga) rank
// by attention, blocks [ga, grid) by hidden states, each group over its own
// shares as the separate kernels would (the same scores and keys, bit for
// bit).  The attention gathers then overlap the stream of hidden rows instead
// of following it in a launch of their own.  ga is a multiple of 8, so the
// attention blocks' XCD runs line up with the hardware's round-robin.
template <int kU>
__global__ __launch_bounds__(kRankThreads) void rank_both_kernel(RankHiddenArgs h, RankAttnArgs t,
                                                                 uint32_t ga) {
    extern __shared__ uint4 smem[];
    __shared__ uint64_t s_best[kRankWaves];
    if (blockIdx.x < ga)   // block-uniform
        attn_block(t, blockIdx.x, ga, reinterpret_cast<uint32_t *>(smem));
    else
        hidden_block<kU, kRankWaves>(h, blockIdx.x - ga, gridDim.x - ga, smem, s_best);
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

static int prep_hidden(const uint16_t *hidden, int64_t h_seq_stride, int64_t h_row_stride,
                       int64_t n_rows, int d, const int32_t *lens, const int32_t *cand_pos,
                       int64_t cap, const int32_t *cand_count, int B, float threshold,
                       float *scores, void *workspace, size_t workspace_bytes,
                       RankHiddenArgs &a) {
    if (!hidden || !lens || !cand_pos || !cand_count) return PLD_ERR_INVALID;
    if (B < 1 || B > PLD_MAX_BATCH || cap < 1 || isnan(threshold)) return PLD_ERR_INVALID;
    if ((uint64_t)B * (uint64_t)cap >= (1ull << 32)) return PLD_ERR_INVALID;
    if (d < 8 || d > PLD_MAX_HIDDEN || d % 8 != 0 || n_rows < 1) return PLD_ERR_INVALID;
    if (h_row_stride < d || h_seq_stride < 0) return PLD_ERR_INVALID;
    if (((uintptr_t)hidden & 15) || (h_row_stride % 8) || (h_seq_stride % 8)) return PLD_ERR_ALIGN;
    if (!workspace || workspace_bytes < rank_ws_bytes(B)) return PLD_ERR_WORKSPACE;
    a.c = make_common(lens, cand_pos, cap, cand_count, B, threshold, scores, nullptr, nullptr,
                      workspace);
    a.hidden = hidden;
    a.hs = h_seq_stride;
    a.hr = h_row_stride;
    a.n_rows = n_rows;
    a.d = d;
    return PLD_OK;
}

static int prep_attn(const float *attn, int64_t a_seq_stride, int64_t a_row_stride,
                     int64_t n_keys, int R, int agg, const int32_t *lens, const int32_t *cand_pos,
                     int64_t cap, const int32_t *cand_count, int B, float threshold, float *scores,
                     void *workspace, size_t workspace_bytes, RankAttnArgs &a) {
    if (!attn || !lens || !cand_pos || !cand_count) return PLD_ERR_INVALID;
    if (B < 1 || B > PLD_MAX_BATCH || cap < 1 || isnan(threshold)) return PLD_ERR_INVALID;
    if ((uint64_t)B * (uint64_t)cap >= (1ull << 32)) return PLD_ERR_INVALID;
    if (R < 1 || n_keys < 1 || (agg != PLD_AGG_SUM && agg != PLD_AGG_MAX)) return PLD_ERR_INVALID;
    if (a_row_stride < 0 || a_seq_stride < 0) return PLD_ERR_INVALID;
    if ((uintptr_t)attn & 3) return PLD_ERR_ALIGN;
    if (!workspace || workspace_bytes < rank_ws_bytes(B)) return PLD_ERR_WORKSPACE;
    a.c = make_common(lens, cand_pos, cap, cand_count, B, threshold, scores, nullptr, nullptr,
                      workspace);
    a.attn = attn;
    a.as = a_seq_stride;
    a.ar = a_row_stride;
    a.n_keys = n_keys;
    a.R = R;
    a.agg = agg;
    return PLD_OK;
}

// The ranking grids are persistent: as many blocks as fit on the device at
// once, each taking an equal contiguous share of the flattened candidates.
template <int kU, int kW>
static void launch_hidden_as(const RankHiddenArgs &a, size_t lds, hipStream_t s) {
    const void *k = reinterpret_cast<const void *>(&rank_hidden_kernel<kU, kW>);
    const int grid = resident_blocks(k, kW * kWave, lds) * PLD_RANK_OVERSUB;
    hipLaunchKernelGGL((rank_hidden_kernel<kU, kW>), dim3(grid), dim3(kW * kWave), lds, s, a);
}

static void launch_hidden(const RankHiddenArgs &a, hipStream_t s) {
    const size_t lds = (size_t)(a.d / 8) * sizeof(uint4) + (size_t)(2 * a.c.B + 1) * sizeof(uint32_t);
    if (a.d == 4096)
        launch_hidden_as<4, kRankWaves>(a, lds, s);
    else if (a.d == 8192)
        launch_hidden_as<8, kRankWaves>(a, lds, s);
    else
        launch_hidden_as<0, kRankWaves>(a, lds, s);
}

#ifndef PLD_BOTH_ATTN_PERMILLE
#define PLD_BOTH_ATTN_PERMILLE 205   // rank_both_kernel: the share of the grid ranking by attention
#endif

// The grid of the combined ranking is the resident blocks; about a fifth of
// them (a multiple of 8) rank by attention, the rest by hidden states.  On the
// 64 x 16384 workload (1024 resident blocks) 192 to 224 attention blocks
// were equally fast, 208 in the middle.
template <int kU>
static void launch_both_as(const RankHiddenArgs &h, const RankAttnArgs &t, size_t lds,
                           hipStream_t s) {
    const void *k = reinterpret_cast<const void *>(&rank_both_kernel<kU>);
    const int grid = resident_blocks(k, kRankThreads, lds);
    uint32_t ga = (uint32_t)((int64_t)grid * PLD_BOTH_ATTN_PERMILLE / 1000) / 8 * 8;
    if (ga < 8) ga = 8;
    const unsigned total = (unsigned)(grid > (int)ga ? grid : (int)ga + 8);
    hipLaunchKernelGGL((rank_both_kernel<kU>), dim3(total), dim3(kRankThreads), lds, s, h, t, ga);
}

static void launch_both(const RankHiddenArgs &h, const RankAttnArgs &t, hipStream_t s) {
    const size_t lds = (size_t)(h.d / 8) * sizeof(uint4) + (size_t)(2 * h.c.B + 1) * sizeof(uint32_t);
    if (h.d == 4096)
        launch_both_as<4>(h, t, lds, s);
    else if (h.d == 8192)
        launch_both_as<8>(h, t, lds, s);
    else
        launch_both_as<0>(h, t, lds, s);
}

static void launch_attn(const RankAttnArgs &a, hipStream_t s) {
    const int grid = resident_blocks(reinterpret_cast<const void *>(&rank_attn_kernel),
                                     kRankThreads, 0) * PLD_RANK_OVERSUB;
    hipLaunchKernelGGL(rank_attn_kernel, dim3(grid), dim3(kRankThreads), 0, s, a);
}

static int launch_select(RankCommon c, int32_t *best_pos, float *best_score, hipStream_t s) {
    if (!best_pos || !best_score) return PLD_ERR_INVALID;
    c.best_pos = best_pos;
    c.best_score = best_score;
    hipLaunchKernelGGL(rank_finish_kernel, dim3((c.B + 255) / 256), dim3(256), 0, s, c);
    return PLD_OK;
}

// The bytes of a workspace that hold the ranking keys of B sequences.
static size_t key_bytes(int B) { return (size_t)B * kKeySlots * sizeof(uint64_t); }

static int launched() { return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH; }

}  // namespace pld

using namespace pld;

extern "C" int pld_score_hidden(const uint16_t *hidden, int64_t h_seq_stride, int64_t h_row_stride,
                                int64_t n_rows, int d, const int32_t *lens,
                                const int32_t *cand_pos, int64_t cap, const int32_t *cand_count,
                                int B, float threshold, float *scores, void *workspace,
                                size_t workspace_bytes, void *stream) {
    RankHiddenArgs a;
    int rc = prep_hidden(hidden, h_seq_stride, h_row_stride, n_rows, d, lens, cand_pos, cap,
                         cand_count, B, threshold, scores, workspace, workspace_bytes, a);
    if (rc != PLD_OK) return rc;
    launch_hidden(a, (hipStream_t)stream);
    return launched();
}

extern "C" int pld_score_attn(const float *attn, int64_t a_seq_stride, int64_t a_row_stride,
                              int64_t n_keys, int R, int agg, const int32_t *lens,
                              const int32_t *cand_pos, int64_t cap, const int32_t *cand_count,
                              int B, float threshold, float *scores, void *workspace,
                              size_t workspace_bytes, void *stream) {
    RankAttnArgs a;
    int rc = prep_attn(attn, a_seq_stride, a_row_stride, n_keys, R, agg, lens, cand_pos, cap,
                       cand_count, B, threshold, scores, workspace, workspace_bytes, a);
    if (rc != PLD_OK) return rc;
    launch_attn(a, (hipStream_t)stream);
    return launched();
}

extern "C" int pld_score_both(const uint16_t *hidden, int64_t h_seq_stride, int64_t h_row_stride,
                              int64_t n_rows, int d, const float *attn, int64_t a_seq_stride,
                              int64_t a_row_stride, int64_t n_keys, int R, int agg,
                              const int32_t *lens, const int32_t *cand_pos, int64_t cap,
                              const int32_t *cand_count, int B, float threshold_h,
                              float threshold_a, float *scores_h, float *scores_a,
                              void *workspace_h, size_t workspace_h_bytes, void *workspace_a,
                              size_t workspace_a_bytes, void *stream) {
    RankHiddenArgs h;
    int rc = prep_hidden(hidden, h_seq_stride, h_row_stride, n_rows, d, lens, cand_pos, cap,
                         cand_count, B, threshold_h, scores_h, workspace_h, workspace_h_bytes, h);
    if (rc != PLD_OK) return rc;
    RankAttnArgs t;
    rc = prep_attn(attn, a_seq_stride, a_row_stride, n_keys, R, agg, lens, cand_pos, cap,
                   cand_count, B, threshold_a, scores_a, workspace_a, workspace_a_bytes, t);
    if (rc != PLD_OK) return rc;
    if (ranges_overlap(workspace_h, key_bytes(B), workspace_a, key_bytes(B)))
        return PLD_ERR_WORKSPACE;
    launch_both(h, t, (hipStream_t)stream);
    return launched();
}

extern "C" int pld_select_best(int B, int32_t *best_pos, float *best_score, void *workspace,
                               size_t workspace_bytes, void *stream) {
    if (B < 1 || B > PLD_MAX_BATCH || !best_pos || !best_score) return PLD_ERR_INVALID;
    if (!workspace || workspace_bytes < rank_ws_bytes(B)) return PLD_ERR_WORKSPACE;
    RankCommon c{};
    c.B = B;
    c.keys = (uint64_t *)workspace;
    int rc = launch_select(c, best_pos, best_score, (hipStream_t)stream);
    return rc != PLD_OK ? rc : launched();
}

extern "C" int pld_select_draft(const int32_t *tokens, int64_t tok_stride, const int32_t *lens,
                                int B, int K, int32_t *best_pos, float *best_score,
                                int32_t *draft, int32_t *draft_len, void *workspace,
                                size_t workspace_bytes, void *aux_workspace,
                                size_t aux_workspace_bytes, int32_t *aux_best_pos,
                                float *aux_best_score, void *stream) {
    if (!tokens || !lens || !best_pos || !best_score || !draft || !draft_len)
        return PLD_ERR_INVALID;
    if (B < 1 || B > PLD_MAX_BATCH || K < 1 || tok_stride < 1 || tok_stride > kMaxTokStride)
        return PLD_ERR_INVALID;
    if (aux_workspace && (!aux_best_pos || !aux_best_score)) return PLD_ERR_INVALID;
    if (!workspace || workspace_bytes < rank_ws_bytes(B)) return PLD_ERR_WORKSPACE;
    if (aux_workspace && (aux_workspace_bytes < rank_ws_bytes(B) ||
                          ranges_overlap(workspace, key_bytes(B), aux_workspace, key_bytes(B))))
        return PLD_ERR_WORKSPACE;
    SelectDraftArgs a{tokens, tok_stride, lens, B, K, (uint64_t *)workspace, best_pos, best_score,
                      draft, draft_len, (uint64_t *)aux_workspace, aux_best_pos, aux_best_score};
    hipLaunchKernelGGL(select_draft_kernel, dim3((unsigned)((B + 3) / 4)), dim3(256), 0,
                       (hipStream_t)stream, a);
    return launched();
}

extern "C" int pld_rank_hidden(const uint16_t *hidden, int64_t h_seq_stride, int64_t h_row_stride,
                               int64_t n_rows, int d, const int32_t *lens, const int32_t *cand_pos,
                               int64_t cap, const int32_t *cand_count, int B, float threshold,
                               float *scores, int32_t *best_pos, float *best_score,
                               void *workspace, size_t workspace_bytes, void *stream) {
    if (!best_pos || !best_score) return PLD_ERR_INVALID;
    RankHiddenArgs a;
    int rc = prep_hidden(hidden, h_seq_stride, h_row_stride, n_rows, d, lens, cand_pos, cap,
                         cand_count, B, threshold, scores, workspace, workspace_bytes, a);
    if (rc != PLD_OK) return rc;
    launch_hidden(a, (hipStream_t)stream);
    launch_select(a.c, best_pos, best_score, (hipStream_t)stream);
    return launched();
}

extern "C" int pld_rank_attn(const float *attn, int64_t a_seq_stride, int64_t a_row_stride,
                             int64_t n_keys, int R, int agg, const int32_t *lens,
                             const int32_t *cand_pos, int64_t cap, const int32_t *cand_count, int B,
                             float threshold, float *scores, int32_t *best_pos, float *best_score,
                             void *workspace, size_t workspace_bytes, void *stream) {
    if (!best_pos || !best_score) return PLD_ERR_INVALID;
    RankAttnArgs a;
    int rc = prep_attn(attn, a_seq_stride, a_row_stride, n_keys, R, agg, lens, cand_pos, cap,
                       cand_count, B, threshold, scores, workspace, workspace_bytes, a);
    if (rc != PLD_OK) return rc;
    launch_attn(a, (hipStream_t)stream);
    launch_select(a.c, best_pos, best_score, (hipStream_t)stream);
    return launched();
}
