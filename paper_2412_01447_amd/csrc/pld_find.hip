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
// The tokens a block needs are first copied to LDS with independent loads
// (straight into LDS, with the length, in the one-block form), so the
// backwards comparisons never wait on a chain of global loads.  Sequences up
// to 16384 tokens take one 1024-thread block each (count, pick n, compact, in
// one kernel): the block searches in groups of 64 positions, one per lane,
// each group's hits a 64-bit compare mask (block_search), because on the one
// CU that holds a sequence the number of instructions per position sets the
// time.  Longer ones split into kFindTile-position blocks in which each lane
// takes 8 consecutive positions, reads the 16 tokens around them with four
// aligned 16-byte LDS loads and builds, per n, an 8-bit hit mask from
// register compares; a count kernel writes per-tile counts to the scratch
// buffer, and the compaction kernel derives its tile's output offset from the
// counts of the tiles before it (an exclusive wave scan of the lanes' hit
// counts plus the per-wave and per-tile counts).  Up to kFindScanTiles tiles
// per sequence each compaction block sums those counts itself; past that a
// scan launch between the two writes every tile's offset once, so a row of
// 2^30 tokens (524288 tiles) costs reads in proportion to its tiles, not to
// their square.
#include "pld.h"
#include "pld_device.h"
#include "pld_match.h"

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
    int32_t *tile_counts;   // [B][ntiles][8], scratch
    int32_t *tile_off;      // [B][ntiles], scratch (ntiles > kFindScanTiles; else null)
    int32_t *seq_n;         // [B][2]: the chosen n and its count (likewise)
    int ntiles;
};

// ---------------------------------------------------------------- fused
// One 1024-thread block per sequence, tok_stride <= kPasses * kFindFusedMax:
// the whole row sits in LDS (64 KB for two passes' worth, 16384 tokens) and
// block_search takes it in groups of 64 positions, kPasses * 8 per wave.
template <int kPasses>
__global__ __launch_bounds__(kFindWavesFused * kWave) void find_fused_kernel(FindArgs a) {
    constexpr int G = kPasses * kFindFusedMax / (kFindWavesFused * kWave);
    __shared__ __align__(16) int32_t s_x[kPasses * kFindFusedMax];
    __shared__ int s_lvl[kFindWavesFused][kMaxNgram];
    const int b = blockIdx.x;
    const int32_t *x = a.tokens + (int64_t)b * a.tok_stride;
    // the whole token row (tok_stride fits the LDS copy) is requested with
    // the length instead of after it: positions past T - 2 are never
    // compared, so the tokens past the length do no harm
    const int64_t T = a.lens[b];
    if (((uintptr_t)x & 15) == 0 && (a.tok_stride & 3) == 0)
        copy_to_lds(reinterpret_cast<const uint4 *>(x), reinterpret_cast<uint4 *>(s_x),
                    (int)(a.tok_stride / 4));
    else
        stage_tokens(x, 0, a.tok_stride, s_x);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (T < 1 || T > a.tok_stride) {
        if (threadIdx.x == 0) {
            a.cand_count[b] = 0;
            a.ngram_used[b] = -1;
        }
        return;
    }
    int total;
    const int n_used = block_search<kFindWavesFused, G>(s_x, T, a.nmin, a.nmax, s_lvl,
                                                        a.cand_pos + (int64_t)b * a.cap, nullptr,
                                                        total);
    if (threadIdx.x == 0) {
        a.cand_count[b] = total;
        a.ngram_used[b] = n_used;
    }
}

// ---------------------------------------------------------------- tiled
// A tile covers positions [tile*kFindTile, (tile+1)*kFindTile), one pass of
// 8 positions per lane; its LDS copy starts kHalo >= kMaxNgram-1 tokens
// earlier so the backwards comparisons stay inside (8, not 7, keeps every
// lane's 16-byte window loads aligned).
constexpr int kHalo = 8;
static_assert(kHalo >= kMaxNgram - 1 && kFindTile == kFindWavesTiled * kWave * kLanePos,
              "one pass per tile");

__device__ __forceinline__ int64_t tile_lo(int tile) {
    int64_t lo = (int64_t)tile * kFindTile - kHalo;
    return lo < 0 ? 0 : lo;
}

__global__ __launch_bounds__(kFindWavesTiled * kWave) void find_count_kernel(FindArgs a) {
    __shared__ __align__(16) int32_t s_x[kFindTile + kHalo];
    __shared__ int s_lvl[kFindWavesTiled][kMaxNgram];
    const int tile = blockIdx.x, b = blockIdx.y;
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    const int32_t *x = a.tokens + (int64_t)b * a.tok_stride;
    const int64_t T = a.lens[b];
    const int64_t t0 = (int64_t)tile * kFindTile;
    const bool live = (T >= 1 && T <= a.tok_stride && t0 <= T - 2);
    int cnt[kMaxNgram];
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) cnt[k] = 0;
    if (live) {   // block-uniform
        const int64_t lo = tile_lo(tile);
        const int64_t hi = (t0 + kFindTile < T - 1) ? t0 + kFindTile : T - 1;
        stage_tokens(x, lo, hi, s_x);
        const Query q = load_query(x, T, a.nmax);
        __syncthreads();
        count_levels(lane_hits(s_x, lo, T, t0 + (int64_t)threadIdx.x * kLanePos, q, a.nmax),
                     a.nmax, cnt);
    }
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) {
        const int t = wave_sum_i32(cnt[k]);
        if (lane == 0) s_lvl[w][k] = t;
    }
    __syncthreads();
    if (threadIdx.x < kMaxNgram) {
        int t = 0;
        for (int i = 0; i < kFindWavesTiled; ++i) t += s_lvl[i][threadIdx.x];
        a.tile_counts[((int64_t)b * a.ntiles + tile) * kMaxNgram + threadIdx.x] = t;
    }
}

// Long rows (more than kFindScanTiles tiles): one 1024-thread block per
// sequence sums every level's per-tile counts, picks the longest n with an
// occurrence, and writes each tile's exclusive prefix of that level's counts
// (tiles in order, 1024 per round, a wave scan and the waves' totals) and the
// sequence's (n, count).  The compaction blocks then read their own offset.
__global__ __launch_bounds__(kFindWavesFused * kWave) void find_scan_kernel(FindArgs a) {
    __shared__ int s_tot[kMaxNgram];
    __shared__ int s_w[kFindWavesFused];
    const int b = blockIdx.x;
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    const int64_t T = a.lens[b];
    if (T < 1 || T > a.tok_stride) return;   // block-uniform; the compaction reports it
    const int32_t *tc = a.tile_counts + (int64_t)b * a.ntiles * kMaxNgram;
    if (threadIdx.x < kMaxNgram) s_tot[threadIdx.x] = 0;
    __syncthreads();
    {
        int tot[kMaxNgram];
#pragma unroll
        for (int k = 0; k < kMaxNgram; ++k) tot[k] = 0;
        for (int t = threadIdx.x; t < a.ntiles; t += blockDim.x) {
#pragma unroll
            for (int k = 0; k < kMaxNgram; ++k) tot[k] += tc[(int64_t)t * kMaxNgram + k];
        }
#pragma unroll
        for (int k = 0; k < kMaxNgram; ++k) {
            const int v = wave_sum_i32(tot[k]);
            if (lane == 0 && v) atomicAdd(&s_tot[k], v);
        }
    }
    __syncthreads();
    int n_used = 0;
    for (int n = a.nmax; n >= a.nmin; --n) {
        if (s_tot[n - 1] > 0) {
            n_used = n;
            break;
        }
    }
    int32_t *off = a.tile_off + (int64_t)b * a.ntiles;
    int carry = 0;
    for (int t0 = 0; n_used > 0 && t0 < a.ntiles; t0 += (int)blockDim.x) {   // block-uniform
        const int t = t0 + (int)threadIdx.x;
        const int c = t < a.ntiles ? tc[(int64_t)t * kMaxNgram + n_used - 1] : 0;
        int wt;
        const int ex = wave_excl_scan(c, wt);
        if (lane == 0) s_w[w] = wt;
        __syncthreads();
        int before = carry, all = 0;
        for (int i = 0; i < kFindWavesFused; ++i) {
            if (i < w) before += s_w[i];
            all += s_w[i];
        }
        if (t < a.ntiles) off[t] = before + ex;
        carry += all;
        __syncthreads();   // s_w is written again in the next round
    }
    if (threadIdx.x == 0) {
        a.seq_n[2 * b] = n_used;
        a.seq_n[2 * b + 1] = n_used > 0 ? s_tot[n_used - 1] : 0;
    }
}

__global__ __launch_bounds__(kFindWavesTiled * kWave) void find_compact_kernel(FindArgs a) {
    __shared__ __align__(16) int32_t s_x[kFindTile + kHalo];
    __shared__ int s_tot[kMaxNgram];
    __shared__ int s_pre[kMaxNgram];
    __shared__ int s_wc[kFindWavesTiled];
    const int tile = blockIdx.x, b = blockIdx.y;
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    const int32_t *x = a.tokens + (int64_t)b * a.tok_stride;
    const int64_t T = a.lens[b];
    if (T < 1 || T > a.tok_stride) {   // block-uniform
        if (tile == 0 && threadIdx.x == 0) {
            a.cand_count[b] = 0;
            a.ngram_used[b] = -1;
        }
        return;
    }
    const int32_t *tc = a.tile_counts + (int64_t)b * a.ntiles * kMaxNgram;
    if (threadIdx.x < kMaxNgram) {
        s_tot[threadIdx.x] = 0;
        s_pre[threadIdx.x] = 0;
    }
    __syncthreads();
    if (a.tile_off) {   // uniform: the scan launch wrote n, its count and this tile's offset
        if (threadIdx.x == 0) {
            const int n = a.seq_n[2 * b];
            if (n > 0) {
                s_tot[n - 1] = a.seq_n[2 * b + 1];
                s_pre[n - 1] = a.tile_off[(int64_t)b * a.ntiles + tile];
            }
        }
    } else {
        // totals over all tiles, and over the tiles before this one
        int tot[kMaxNgram], pre[kMaxNgram];
#pragma unroll
        for (int k = 0; k < kMaxNgram; ++k) tot[k] = pre[k] = 0;
        for (int t = threadIdx.x; t < a.ntiles; t += blockDim.x) {
#pragma unroll
            for (int k = 0; k < kMaxNgram; ++k) {
                const int v = tc[(int64_t)t * kMaxNgram + k];
                tot[k] += v;
                if (t < tile) pre[k] += v;
            }
        }
#pragma unroll
        for (int k = 0; k < kMaxNgram; ++k) {
            const int tk = wave_sum_i32(tot[k]), pk = wave_sum_i32(pre[k]);
            if (lane == 0 && (tk | pk)) {
                atomicAdd(&s_tot[k], tk);
                atomicAdd(&s_pre[k], pk);
            }
        }
    }
    __syncthreads();
    int n_used = 0;
    for (int n = a.nmax; n >= a.nmin; --n) {
        if (s_tot[n - 1] > 0) {
            n_used = n;
            break;
        }
    }
    const int64_t t0 = (int64_t)tile * kFindTile;
    if (n_used > 0 && t0 <= T - 2) {   // block-uniform
        const int64_t lo = tile_lo(tile);
        const int64_t hi = (t0 + kFindTile < T - 1) ? t0 + kFindTile : T - 1;
        stage_tokens(x, lo, hi, s_x);
        const Query q = load_query(x, T, a.nmax);
        __syncthreads();
        const int64_t base = t0 + (int64_t)threadIdx.x * kLanePos;
        const uint32_t bits = level_bits(lane_hits(s_x, lo, T, base, q, a.nmax), n_used);
        const int wc = wave_sum_i32(__popc(bits));
        if (lane == 0) s_wc[w] = wc;
        __syncthreads();
        int64_t run = s_pre[n_used - 1];
        for (int i = 0; i < w; ++i) run += s_wc[i];
        emit_bits(bits, base, a.cand_pos + (int64_t)b * a.cap, nullptr, run);
    }
    if (tile == 0 && threadIdx.x == 0) {
        a.cand_count[b] = n_used > 0 ? s_tot[n_used - 1] : 0;
        a.ngram_used[b] = n_used;
    }
}

}  // namespace pld

using namespace pld;

extern "C" size_t pld_find_scratch_bytes(int B, int64_t tok_stride) {
    if (B < 1 || tok_stride < 1 || tok_stride > kMaxTokStride) return 0;
    return find_scratch_bytes(B, tok_stride);
}

extern "C" int pld_find_candidates(const int32_t *tokens, int64_t tok_stride, const int32_t *lens,
                                   int B, int ngram_min, int ngram_max, int32_t *cand_pos,
                                   int64_t cap, int32_t *cand_count, int32_t *ngram_used,
                                   void *scratch, size_t scratch_bytes, void *stream) {
    if (!tokens || !lens || !cand_pos || !cand_count || !ngram_used) return PLD_ERR_INVALID;
    if (B < 1 || B > 65535 || tok_stride < 1 || tok_stride > kMaxTokStride) return PLD_ERR_INVALID;
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
    a.ntiles = (int)((tok_stride + kFindTile - 1) / kFindTile);
    hipStream_t s = (hipStream_t)stream;
    if (tok_stride <= kFindFusedMax) {
        hipLaunchKernelGGL(find_fused_kernel<1>, dim3(B), dim3(kFindWavesFused * kWave), 0, s, a);
    } else if (tok_stride <= kFindFusedPasses * kFindFusedMax) {
        hipLaunchKernelGGL(find_fused_kernel<kFindFusedPasses>, dim3(B),
                           dim3(kFindWavesFused * kWave), 0, s, a);
    } else {
        if (!scratch || scratch_bytes < find_scratch_bytes(B, tok_stride)) return PLD_ERR_WORKSPACE;
        a.tile_counts = (int32_t *)scratch;
        a.tile_off = nullptr;
        a.seq_n = nullptr;
        if (a.ntiles > kFindScanTiles) {
            char *p = (char *)scratch + align_up((size_t)B * a.ntiles * 8 * sizeof(int32_t), 256);
            a.tile_off = (int32_t *)p;
            a.seq_n = (int32_t *)(p + align_up((size_t)B * a.ntiles * sizeof(int32_t), 256));
        }
        dim3 grid(a.ntiles, B);
        hipLaunchKernelGGL(find_count_kernel, grid, dim3(kFindWavesTiled * kWave), 0, s, a);
        if (a.tile_off)
            hipLaunchKernelGGL(find_scan_kernel, dim3(B), dim3(kFindWavesFused * kWave), 0, s, a);
        hipLaunchKernelGGL(find_compact_kernel, grid, dim3(kFindWavesTiled * kWave), 0, s, a);
    }
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}
