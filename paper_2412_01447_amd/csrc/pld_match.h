// pld_match.h -- device pieces of the occurrence search (Eq. 1 of arXiv
// 2412.01447 with longest-first n-gram queries), shared by the find kernels
// and the fused drafting kernel.
#pragma once

#include "pld_device.h"

namespace pld {

// Copies x[lo, hi) of one sequence into s[0, hi-lo) (block-wide).
__device__ __forceinline__ void stage_tokens(const int32_t *x, int64_t lo, int64_t hi, int32_t *s) {
    const int n = (int)(hi - lo);
    constexpr int U = 8;
    for (int i0 = threadIdx.x; i0 < n; i0 += blockDim.x * U) {
        int32_t v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            int i = i0 + u * blockDim.x;
            v[u] = i < n ? x[lo + i] : 0;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            int i = i0 + u * blockDim.x;
            if (i < n) s[i] = v[u];
        }
    }
}

// The query read backwards: q.v[k] = x[T-1-k] for k < nmax (0 beyond T).
struct Query {
    int32_t v[kMaxNgram];
};

// m(p) for the 512 positions of one wave: m[it] belongs to position
// base + it*64 + lane (0 when p is not in [1, T-2]).  `s` holds x[s0 ...].
// p - k >= 0 with p <= T-2 implies T-1-k >= 1, so q.v[k] is a real token.
__device__ __forceinline__ void wave_match(const int32_t *s, int64_t s0, int64_t T, int64_t base,
                                           const Query &q, int nmax, int (&m)[8]) {
    const int lane = lane_id();
#pragma unroll
    for (int it = 0; it < 8; ++it) {
        const int64_t p = base + it * kWave + lane;
        int len = 0;
        if (p >= 1 && p <= T - 2) {
            bool go = true;
#pragma unroll
            for (int k = 0; k < kMaxNgram; ++k) {
                if (k < nmax && go) {
                    const int64_t t = p - k;
                    go = (t >= 0) && (s[t - s0] == q.v[k]);
                    len += go ? 1 : 0;
                }
            }
        }
        m[it] = len;
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

__device__ __forceinline__ int wave_hits(const int (&m)[8], int n) {
    int c = 0;
#pragma unroll
    for (int it = 0; it < 8; ++it) c += __popcll(__ballot(m[it] >= n));
    return c;
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
        const uint64_t mk = __ballot(m[it] >= n);
        if ((mk >> lane) & 1ull) out[run + __popcll(mk & lt)] = (int32_t)(base + it * kWave + lane);
        run += __popcll(mk);
    }
}

}  // namespace pld
