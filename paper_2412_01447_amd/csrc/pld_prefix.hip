// pld_prefix.hip -- prompt lookup's selection, the baseline PLD+ replaces
// (arXiv 2412.01447, Sec. 2; the Fig. 3 caption: prompt lookup proposes the
// candidate span with the longest matching prefix).
//
// For a candidate j (0 <= j <= T-2) the match length is the largest
// m <= max_match with x[j-k] = x[T-1-k] for every k < m (indices j-k >= 0);
// the chosen j* has the largest m, the earliest among equal lengths (prompt
// lookup scans the context from the start and keeps the first match).
//
// One block per sequence.  The query suffix x[T-1], x[T-2], ... is staged in
// LDS; each lane takes a candidate and compares 16 tokens back at a time with
// independent loads (one trip to memory per 16 matched tokens, not one per
// token).  The choice is the maximum of the packed key (m << 32 | ~j) over the
// block, by DPP wave maxima.
#include "pld.h"
#include "pld_device.h"

namespace pld {

constexpr int kPrefixThreads = 256;
constexpr int kPrefixChunk = 16;   // tokens compared per trip to memory

struct PrefixArgs {
    const int32_t *tokens;
    int64_t tok_stride;
    const int32_t *lens;
    const int32_t *cand_pos;
    int64_t cap;
    const int32_t *cand_count;
    int B;
    int max_match;
    float *scores;   // [B][cap] or null
    int32_t *best_pos;
    float *best_score;
};

__global__ __launch_bounds__(kPrefixThreads) void select_prefix_kernel(PrefixArgs a) {
    __shared__ int32_t s_q[PLD_MAX_MATCH];   // x[T-1-k]
    __shared__ uint64_t s_key[kPrefixThreads / kWave];
    const int b = blockIdx.x;
    const int32_t *x = a.tokens + (int64_t)b * a.tok_stride;
    const int64_t T = a.lens[b];
    int64_t C = a.cand_count[b];
    if (C < 0 || C > a.cap) C = 0;
    const bool seq_ok = T >= 2 && T <= a.tok_stride;   // block-uniform
    const int qn = seq_ok ? (int)min((int64_t)a.max_match, T) : 0;
    for (int k = threadIdx.x; k < qn; k += kPrefixThreads) s_q[k] = x[T - 1 - k];
    __syncthreads();

    const int32_t *pos = a.cand_pos + (int64_t)b * a.cap;
    uint64_t best = 0;
    for (int64_t c = threadIdx.x; c < (seq_ok ? C : 0); c += kPrefixThreads) {
        const int64_t j = pos[c];
        float s = NAN;
        if (j >= 0 && j <= T - 2) {
            // the run can reach back to x[0] and no further than the query suffix
            const int lim = (int)min((int64_t)qn, j + 1);
            int m = 0;
            bool run = true;
            while (run && m < lim) {
                int32_t v[kPrefixChunk];
#pragma unroll
                for (int k = 0; k < kPrefixChunk; ++k) v[k] = x[max(j - m - k, (int64_t)0)];
#pragma unroll
                for (int k = 0; k < kPrefixChunk; ++k) {
                    if (run && m < lim && v[k] == s_q[m]) ++m;
                    else run = false;
                }
            }
            s = (float)m;
            const uint64_t key = ((uint64_t)(uint32_t)m << 32) | (uint64_t)(0xffffffffu - (uint32_t)j);
            best = key > best ? key : best;
        }
        if (a.scores) a.scores[(int64_t)b * a.cap + c] = s;
    }
    best = wave_max_u64(best);
    if (lane_id() == 0) s_key[threadIdx.x / kWave] = best;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t k = s_key[0];
#pragma unroll
        for (int w = 1; w < kPrefixThreads / kWave; ++w) k = s_key[w] > k ? s_key[w] : k;
        a.best_pos[b] = k ? (int32_t)(0xffffffffu - (uint32_t)k) : -1;
        a.best_score[b] = k ? (float)(uint32_t)(k >> 32) : -INFINITY;
    }
}

}  // namespace pld

using namespace pld;

extern "C" int pld_select_prefix(const int32_t *tokens, int64_t tok_stride, const int32_t *lens,
                                 const int32_t *cand_pos, int64_t cap, const int32_t *cand_count,
                                 int B, int max_match, float *scores, int32_t *best_pos,
                                 float *best_score, void *stream) {
    if (!tokens || !lens || !cand_pos || !cand_count || !best_pos || !best_score)
        return PLD_ERR_INVALID;
    if (B < 1 || B > 65535 || tok_stride < 1 || tok_stride > kMaxTokStride || cap < 1)
        return PLD_ERR_INVALID;
    if (max_match < 1 || max_match > PLD_MAX_MATCH) return PLD_ERR_INVALID;
    PrefixArgs a{tokens, tok_stride, lens, cand_pos, cap, cand_count, B, max_match,
                 scores,  best_pos,   best_score};
    hipLaunchKernelGGL(select_prefix_kernel, dim3((unsigned)B), dim3(kPrefixThreads), 0,
                       (hipStream_t)stream, a);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}
