// pld_match.h -- device pieces of the occurrence search (Eq. 1 of arXiv
// 2412.01447 with longest-first n-gram queries), shared by the find kernels
// and the fused drafting kernel.
#pragma once

#include "pld_device.h"

namespace pld {

// Copies x[lo, hi) of one sequence into s[0, hi-lo) (block-wide).  With a
// 16-byte aligned start and a multiple of four tokens, 16-byte loads carry
// four tokens each.  A thread requests up to eight loads before its first
// store; indices past the end are clamped to the last element, for the loads
// and the stores alike (a repeated store of the same value), so there is no
// branch for the compiler to sink the loads into.
__device__ __forceinline__ void stage_tokens(const int32_t *x, int64_t lo, int64_t hi, int32_t *s) {
    const int n = (int)(hi - lo);
    constexpr int U = 8;
    const int32_t *src = x + lo;
    if ((((uintptr_t)src | (uintptr_t)s) & 15) == 0 && (n & 3) == 0) {
        const uint4 *sv = reinterpret_cast<const uint4 *>(src);
        uint4 *dv = reinterpret_cast<uint4 *>(s);
        const int nv = n >> 2;
        for (int i0 = threadIdx.x; i0 < nv; i0 += blockDim.x * U) {
            uint4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) v[u] = sv[min(i0 + u * (int)blockDim.x, nv - 1)];
#pragma unroll
            for (int u = 0; u < U; ++u) dv[min(i0 + u * (int)blockDim.x, nv - 1)] = v[u];
        }
        return;
    }
    for (int i0 = threadIdx.x; i0 < n; i0 += blockDim.x * U) {
        int32_t v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = src[min(i0 + u * (int)blockDim.x, n - 1)];
#pragma unroll
        for (int u = 0; u < U; ++u) s[min(i0 + u * (int)blockDim.x, n - 1)] = v[u];
    }
}

// The query read backwards: q.v[k] = x[T-1-k] for k < nmax (0 beyond T).
struct Query {
    int32_t v[kMaxNgram];
};

// Reads the query from x (T >= 1 tokens, global memory or LDS) with
// unconditional, clamped loads.
__device__ __forceinline__ Query load_query(const int32_t *x, int64_t T, int nmax) {
    Query q;
    int32_t t[kMaxNgram];
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) t[k] = x[T - 1 - k >= 0 ? T - 1 - k : 0];
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) q.v[k] = (k < nmax && T - 1 - k >= 0) ? t[k] : 0;
    return q;
}

// A lane takes 8 consecutive positions base .. base+7 (base a multiple of 8)
// and reads the 16 tokens x[base-8 .. base+7] from LDS with four aligned
// 16-byte loads; every comparison is then a register compare, with no
// branch: one wave covers 512 positions per pass.
constexpr int kLanePos = 8;

__device__ __forceinline__ uint32_t clamp8(int64_t v) {
    return v < 0 ? 0u : (v > 8 ? 8u : (uint32_t)v);
}

// lane_hits: byte k (k < nmax) of the result has bit j set iff position
// p = base + j is an occurrence of the (k+1)-gram query (Eq. 1):
// 1 <= p <= T-2 and x[p-i] == x[T-1-i] for every i <= k.  Levels >= nmax are
// zero.  `s` holds x[s0 ...] with base - s0 a multiple of 4 and at least 8,
// or s0 == 0 (then the window loads below index 0 are clamped and their
// tokens only meet positions p - i < 0, which are masked out).
// p - i >= 0 with p <= T-2 implies T-1-i >= 1, so q.v[i] is a real token.
__device__ __forceinline__ uint64_t lane_hits(const int32_t *s, int64_t s0, int64_t T,
                                              int64_t base, const Query &q, int nmax) {
    // a wave whose first position is past T-2 has nothing to compare (the
    // lanes' bases grow with the lane, so this is the same test for all)
    if (base - (int64_t)kLanePos * lane_id() > T - 2) return 0ull;
    const int i0 = (int)(base - s0) - 8;
    int32_t w[16];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const int idx = i0 + 4 * c;
        const uint4 v = *reinterpret_cast<const uint4 *>(s + (idx < 0 ? 0 : idx));
        w[4 * c] = (int32_t)v.x;
        w[4 * c + 1] = (int32_t)v.y;
        w[4 * c + 2] = (int32_t)v.z;
        w[4 * c + 3] = (int32_t)v.w;
    }
    // positions in [1, T-2]
    uint32_t m = ((0xffu << clamp8(1 - base)) & 0xffu) & ((1u << clamp8(T - 1 - base)) - 1u);
    uint64_t out = 0;
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) {
        if (k >= nmax) break;   // uniform
        uint32_t e = 0;
#pragma unroll
        for (int j = 0; j < kLanePos; ++j) e |= (w[8 + j - k] == q.v[k] ? 1u : 0u) << j;
        m &= e & ((0xffu << clamp8(k - base)) & 0xffu);   // p - k >= 0
        out |= (uint64_t)m << (8 * k);
    }
    return out;
}

__device__ __forceinline__ uint32_t level_bits(uint64_t hits, int n) {
    return (uint32_t)(hits >> (8 * (n - 1))) & 0xffu;
}

// Adds the popcount of every level byte of `hits` to cnt[k], k < nmax.
__device__ __forceinline__ void count_levels(uint64_t hits, int nmax, int (&cnt)[kMaxNgram]) {
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k)
        if (k < nmax) cnt[k] += __popc((uint32_t)(hits >> (8 * k)) & 0xffu);
}

// Writes the positions base + j of the set bits j of `bits` to out[run ...]
// (and out2[run ...] when given) in ascending order across the wave's lanes;
// returns run plus the wave's number of bits.
__device__ __forceinline__ int64_t emit_bits(uint32_t bits, int64_t base, int32_t *out,
                                             int32_t *out2, int64_t run) {
    if (__ballot(bits != 0u) == 0ull) return run;   // nothing in this wave
    int total;
    int64_t o = run + wave_excl_scan(__popc(bits), total);
    while (bits) {
        const int j = __ffs(bits) - 1;
        bits &= bits - 1u;
        out[o] = (int32_t)(base + j);
        if (out2) out2[o] = (int32_t)(base + j);
        ++o;
    }
    return run + total;
}

}  // namespace pld
