// pld_find.hip -- occurrence retrieval (Eq. 1, Sec. 4.2 of arXiv 2412.01447)
// with n-gram queries tried longest first (Sec. 2, Fig. 3 caption).
//
// Every position p of a sequence gets a match length m(p): how many tokens,
// going backwards from p, agree with the query read backwards from the last
// token x[T-1] (capped at ngram_max).  Position p is an occurrence of the
// n-gram query iff 1 <= p <= T-2 and m(p) >= n, so one pass yields the
// occurrence counts of every n at once; the largest n in [ngram_min,
// ngram_max] with a non-zero count wins, and its occurrences are compacted in
// ascending order.
//
// Compaction is a wave ballot (one bit per lane, 64 positions per ballot), a
// popcount of the lower lanes' bits for the lane's slot, and an exclusive
// scan of per-wave and per-block counts.  Sequences up to kFindFusedMax
// tokens take one 1024-thread block each (count, pick n, compact, in one
// kernel); longer ones split into kFindTile-position blocks: a count kernel
// writes per-tile counts to the workspace, and the compaction kernel derives
// its tile's output offset from the counts of the tiles before it.  The last
// compaction block of a sequence returns its workspace slice to zero.
#include "pld.h"
#include "pld_device.h"

namespace pld {

struct FindArgs {
    const int32_t *tokens;
    int64_t tok_stride;
    const int32_t *lens;
    int B;
    int nmin, nmax;
    int32_t *cand_pos;
    int64_t cap;
    int32_t *cand_count;
    int32_t *ngram_used;
    int32_t *tile_counts;   // [B][ntiles][8]
    uint32_t *tickets;      // [B]
    int ntiles;
};

// The query read backwards: qry[k] = x[T-1-k] (only read where it exists).
struct Query {
    int32_t v[kMaxNgram];
};

__device__ __forceinline__ Query load_query(const int32_t *x, int64_t T, int nmax) {
    Query q;
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) q.v[k] = (k < nmax && T - 1 - k >= 0) ? x[T - 1 - k] : 0;
    return q;
}

// m(p) for an in-range position (1 <= p <= T-2): the loop stops at the first
// disagreement, at the start of the sequence, or at nmax.  p - k >= 0 with
// p <= T-2 implies T-1-k >= 1, so q.v[k] is always a real query token.
__device__ __forceinline__ int match_len(const int32_t *x, int64_t p, const Query &q, int nmax) {
    int m = 0;
    bool go = true;
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) {
        if (k < nmax && go) {
            int64_t s = p - k;
            go = (s >= 0) && (x[s] == q.v[k]);
            m += go ? 1 : 0;
        }
    }
    return m;
}

// Match lengths of the 512 positions of one wave: m[it] belongs to position
// base + it*64 + lane (0 when the position is not a possible occurrence).
__device__ __forceinline__ void wave_match(const int32_t *x, int64_t T, int64_t base,
                                           const Query &q, int nmax, int (&m)[8]) {
    const int lane = lane_id();
#pragma unroll
    for (int it = 0; it < 8; ++it) {
        int64_t p = base + it * kWave + lane;
        m[it] = (p >= 1 && p <= T - 2) ? match_len(x, p, q, nmax) : 0;
    }
}

// Number of occurrences of each n (index n-1) among one wave's positions.
__device__ __forceinline__ void wave_level_counts(const int (&m)[8], int nmax, int (&cnt)[8]) {
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) cnt[k] = 0;
#pragma unroll
    for (int it = 0; it < 8; ++it) {
#pragma unroll
        for (int k = 0; k < kMaxNgram; ++k) {
            if (k < nmax) cnt[k] += __popcll(__ballot(m[it] >= k + 1));
        }
    }
}

// Writes the occurrences (m >= n) of one wave's positions to out + start, in
// ascending order.
__device__ __forceinline__ void wave_emit(const int (&m)[8], int n, int64_t base, int32_t *out,
                                          int64_t start) {
    const int lane = lane_id();
    const uint64_t lt = lanemask_lt();
    int64_t run = start;
#pragma unroll
    for (int it = 0; it < 8; ++it) {
        uint64_t mk = __ballot(m[it] >= n);
        if ((mk >> lane) & 1ull) out[run + __popcll(mk & lt)] = (int32_t)(base + it * kWave + lane);
        run += __popcll(mk);
    }
}

__device__ __forceinline__ int wave_hits(const int (&m)[8], int n) {
    int c = 0;
#pragma unroll
    for (int it = 0; it < 8; ++it) c += __popcll(__ballot(m[it] >= n));
    return c;
}

// ---------------------------------------------------------------- fused
// One 1024-thread block per sequence, tok_stride <= kFindFusedMax.
__global__ __launch_bounds__(kFindWavesFused * kWave) void find_fused_kernel(FindArgs a) {
    __shared__ int s_lvl[kFindWavesFused][kMaxNgram];
    __shared__ int s_wc[kFindWavesFused];
    const int b = blockIdx.x;
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    const int32_t *x = a.tokens + (int64_t)b * a.tok_stride;
    const int64_t T = a.lens[b];
    if (T < 1 || T > a.tok_stride) {
        if (threadIdx.x == 0) {
            a.cand_count[b] = 0;
            a.ngram_used[b] = -1;
        }
        return;
    }
    const Query q = load_query(x, T, a.nmax);
    const int64_t base = (int64_t)w * 512;
    int m[8];
    wave_match(x, T, base, q, a.nmax, m);
    int cnt[8];
    wave_level_counts(m, a.nmax, cnt);
    if (lane == 0) {
#pragma unroll
        for (int k = 0; k < kMaxNgram; ++k) s_lvl[w][k] = cnt[k];
    }
    __syncthreads();
    // pick the longest n with an occurrence (every thread, same answer)
    int n_used = 0, total = 0;
    for (int n = a.nmax; n >= a.nmin; --n) {
        int t = 0;
        for (int i = 0; i < kFindWavesFused; ++i) t += s_lvl[i][n - 1];
        if (t > 0) {
            n_used = n;
            total = t;
            break;
        }
    }
    if (n_used > 0) {
        int wc = wave_hits(m, n_used);
        if (lane == 0) s_wc[w] = wc;
        __syncthreads();
        int64_t start = 0;
        for (int i = 0; i < w; ++i) start += s_wc[i];
        wave_emit(m, n_used, base, a.cand_pos + (int64_t)b * a.cap, start);
    }
    if (threadIdx.x == 0) {
        a.cand_count[b] = total;
        a.ngram_used[b] = n_used;
    }
}

// ---------------------------------------------------------------- tiled
__global__ __launch_bounds__(kFindWavesTiled * kWave) void find_count_kernel(FindArgs a) {
    __shared__ int s_lvl[kFindWavesTiled][kMaxNgram];
    const int tile = blockIdx.x, b = blockIdx.y;
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    const int32_t *x = a.tokens + (int64_t)b * a.tok_stride;
    const int64_t T = a.lens[b];
    const int64_t base = (int64_t)tile * kFindTile + (int64_t)w * 512;
    int cnt[8];
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) cnt[k] = 0;
    if (T >= 1 && T <= a.tok_stride && base <= T - 2) {
        const Query q = load_query(x, T, a.nmax);
        int m[8];
        wave_match(x, T, base, q, a.nmax, m);
        wave_level_counts(m, a.nmax, cnt);
    }
    if (lane == 0) {
#pragma unroll
        for (int k = 0; k < kMaxNgram; ++k) s_lvl[w][k] = cnt[k];
    }
    __syncthreads();
    if (threadIdx.x < kMaxNgram) {
        int t = 0;
        for (int i = 0; i < kFindWavesTiled; ++i) t += s_lvl[i][threadIdx.x];
        a.tile_counts[((int64_t)b * a.ntiles + tile) * kMaxNgram + threadIdx.x] = t;
    }
}

__global__ __launch_bounds__(kFindWavesTiled * kWave) void find_compact_kernel(FindArgs a) {
    __shared__ int s_tot[kMaxNgram];
    __shared__ int s_pre[kMaxNgram];
    __shared__ int s_wc[kFindWavesTiled];
    __shared__ int s_last;
    const int tile = blockIdx.x, b = blockIdx.y;
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    const int32_t *x = a.tokens + (int64_t)b * a.tok_stride;
    const int64_t T = a.lens[b];
    const int32_t *tc = a.tile_counts + (int64_t)b * a.ntiles * kMaxNgram;
    if (threadIdx.x < kMaxNgram) {
        s_tot[threadIdx.x] = 0;
        s_pre[threadIdx.x] = 0;
    }
    __syncthreads();
    const bool valid = (T >= 1 && T <= a.tok_stride);
    if (valid) {
        // totals over all tiles, and over the tiles before this one
        int tot[8], pre[8];
#pragma unroll
        for (int k = 0; k < kMaxNgram; ++k) tot[k] = pre[k] = 0;
        for (int t = threadIdx.x; t < a.ntiles; t += blockDim.x) {
#pragma unroll
            for (int k = 0; k < kMaxNgram; ++k) {
                int v = tc[(int64_t)t * kMaxNgram + k];
                tot[k] += v;
                if (t < tile) pre[k] += v;
            }
        }
#pragma unroll
        for (int k = 0; k < kMaxNgram; ++k) {
            int tk = tot[k], pk = pre[k];
#pragma unroll
            for (int s = 32; s >= 1; s >>= 1) {
                tk += __shfl_xor(tk, s);
                pk += __shfl_xor(pk, s);
            }
            if (lane == 0 && (tk | pk)) {
                atomicAdd(&s_tot[k], tk);
                atomicAdd(&s_pre[k], pk);
            }
        }
    }
    __syncthreads();
    if (valid) {
        int n_used = 0;
        for (int n = a.nmax; n >= a.nmin; --n) {
            if (s_tot[n - 1] > 0) {
                n_used = n;
                break;
            }
        }
        const int64_t base = (int64_t)tile * kFindTile + (int64_t)w * 512;
        int m[8];
        int wc = 0;
        if (n_used > 0 && (int64_t)tile * kFindTile <= T - 2) {
            const Query q = load_query(x, T, a.nmax);
            wave_match(x, T, base, q, a.nmax, m);
            wc = wave_hits(m, n_used);
        }
        if (lane == 0) s_wc[w] = wc;
        __syncthreads();
        if (wc > 0) {
            int64_t start = s_pre[n_used - 1];
            for (int i = 0; i < w; ++i) start += s_wc[i];
            wave_emit(m, n_used, base, a.cand_pos + (int64_t)b * a.cap, start);
        }
        if (tile == 0 && threadIdx.x == 0) {
            a.cand_count[b] = n_used > 0 ? s_tot[n_used - 1] : 0;
            a.ngram_used[b] = n_used;
        }
    } else if (tile == 0 && threadIdx.x == 0) {
        a.cand_count[b] = 0;
        a.ngram_used[b] = -1;
    }
    // The last block of this sequence to finish clears its workspace slice.
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = __hip_atomic_fetch_add(&a.tickets[b], 1u, __ATOMIC_ACQ_REL,
                                            __HIP_MEMORY_SCOPE_AGENT);
        s_last = (t == (uint32_t)a.ntiles - 1u);
    }
    __syncthreads();
    if (s_last) {
        int32_t *mine = a.tile_counts + (int64_t)b * a.ntiles * kMaxNgram;
        for (int i = threadIdx.x; i < a.ntiles * kMaxNgram; i += blockDim.x) mine[i] = 0;
        if (threadIdx.x == 0) a.tickets[b] = 0u;
    }
}

}  // namespace pld

using namespace pld;

extern "C" int pld_find_candidates(const int32_t *tokens, int64_t tok_stride, const int32_t *lens,
                                   int B, int ngram_min, int ngram_max, int32_t *cand_pos,
                                   int64_t cap, int32_t *cand_count, int32_t *ngram_used,
                                   void *workspace, size_t workspace_bytes, void *stream) {
    if (!tokens || !lens || !cand_pos || !cand_count || !ngram_used) return PLD_ERR_INVALID;
    if (B < 1 || tok_stride < 1 || tok_stride > kMaxTokStride) return PLD_ERR_INVALID;
    if (ngram_min < 1 || ngram_max < ngram_min || ngram_max > PLD_MAX_NGRAM) return PLD_ERR_INVALID;
    if (cap < tok_stride) return PLD_ERR_INVALID;
    FindArgs a;
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
    a.tile_counts = nullptr;
    a.tickets = nullptr;
    a.ntiles = (int)((tok_stride + kFindTile - 1) / kFindTile);
    hipStream_t s = (hipStream_t)stream;
    if (tok_stride <= kFindFusedMax) {
        hipLaunchKernelGGL(find_fused_kernel, dim3(B), dim3(kFindWavesFused * kWave), 0, s, a);
    } else {
        if (!workspace) return PLD_ERR_WORKSPACE;
        if (workspace_bytes < find_ws_bytes(B, tok_stride)) return PLD_ERR_WORKSPACE;
        a.tile_counts = (int32_t *)workspace;
        a.tickets = (uint32_t *)((char *)workspace +
                                 align_up((size_t)B * a.ntiles * kMaxNgram * sizeof(int32_t), 256));
        dim3 grid(a.ntiles, B);
        hipLaunchKernelGGL(find_count_kernel, grid, dim3(kFindWavesTiled * kWave), 0, s, a);
        hipLaunchKernelGGL(find_compact_kernel, grid, dim3(kFindWavesTiled * kWave), 0, s, a);
    }
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}
